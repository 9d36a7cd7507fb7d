// Second layer of the arbitration head for one compacted row, shared by the head's
// epilogue kernel and the chain finish that folds it in (Section 3.3,
// z = w2 . relu(W1 h + b1) + b2): one wave adds the row's k-slice partials of
// W1 h in a fixed order, then b1, the ReLU, w2 and b2, so z is bit-identical in
// both and from run to run.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "launch.h"

namespace cospec {
namespace headz {

template <int DT> __device__ inline float scalar_at(const void *p, int64_t i);
template <> __device__ inline float scalar_at<kBF16>(const void *p, int64_t i) {
    return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t *>(p)[i]) << 16);
}
template <> __device__ inline float scalar_at<kF32>(const void *p, int64_t i) {
    return static_cast<const float *>(p)[i];
}

// Hidden row of list entry m (see HeadArgs::row0).
__device__ inline int64_t hidden_row(const HeadArgs &a, int64_t m) {
    int64_t id = a.list ? static_cast<int64_t>(a.list[m]) : m;
    if (a.row0 && id >= 0) id = a.row0[id / a.slots] + id % a.slots;
    return id;
}

constexpr int kEpiCols = 8;   // columns per lane per pass: every partial a lane needs is
                              // loaded before any is summed (h <= 64 * kEpiCols per pass)

// z of list entry m, in every lane of the calling wave; NaN when its hidden row is
// outside [0, n_rows).
template <int DT>
__device__ inline float head_z(const HeadArgs &a, int64_t m, int lane) {
    float acc = 0.f;
    for (int n0 = 0; n0 < a.h; n0 += 64 * kEpiCols) {
        float u[kEpiCols][kHeadMaxSplit];
#pragma unroll
        for (int i = 0; i < kEpiCols; ++i)
#pragma unroll
            for (int ks = 0; ks < kHeadMaxSplit; ++ks) {
                const int n = n0 + i * 64 + lane;
                u[i][ks] = (ks < a.ksplit && n < a.h)
                               ? a.upart[(static_cast<int64_t>(ks) * a.m_cap + m) * a.h + n] : 0.f;
            }
#pragma unroll
        for (int i = 0; i < kEpiCols; ++i) {
            const int n = n0 + i * 64 + lane;
            if (n < a.h) {
                float v = 0.f;
#pragma unroll
                for (int ks = 0; ks < kHeadMaxSplit; ++ks) v += u[i][ks];
                const float bias = a.b1 ? scalar_at<DT>(a.b1, n) : 0.f;
                acc += fmaxf(v + bias, 0.f) * scalar_at<DT>(a.w2, n);
            }
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
    const int64_t id = hidden_row(a, m);
    return id >= 0 && id < a.n_rows ? acc + a.b2 : NAN;
}

}  // namespace headz
}  // namespace cospec
