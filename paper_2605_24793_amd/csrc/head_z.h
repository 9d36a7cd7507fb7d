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

// Hidden row of decision slot id (see HeadArgs::row0).
__device__ inline int64_t mapped_row(const HeadArgs &a, int64_t id) {
    if (a.row0 && id >= 0) id = a.row0[id / a.slots] + id % a.slots;
    return id;
}

// Hidden row of list entry m.
__device__ inline int64_t hidden_row(const HeadArgs &a, int64_t m) {
    return mapped_row(a, a.list ? static_cast<int64_t>(a.list[m]) : m);
}

// k-slices the persistent GEMM cuts d into for M listed rows: a.ksplit while the
// (tile, k-slice) items fit a.grid workgroups, else as many as fit (at least one).
// The grid-sized form (a.grid = 0) always uses a.ksplit.
__device__ inline int live_ksplit(const HeadArgs &a, int64_t M) {
    const int64_t tiles = ((M + kHeadTileM - 1) / kHeadTileM) * ((a.h + kHeadTileN - 1) / kHeadTileN);
    if (a.grid <= 0 || tiles <= 0 || tiles * a.ksplit <= a.grid) return a.ksplit;
    const int64_t ks = a.grid / tiles;
    return ks < 1 ? 1 : static_cast<int>(ks);
}

// One pass of a lane covers CPL columns (lane, lane + 64, ...) and loads SPL k-slice
// partials of each together, CPL * SPL = 64 loads in flight; narrow heads take fewer
// columns and more slices per pass.  Every load of a pass is unconditional (indexes
// past the end are clamped and their values dropped), b1 and w2 included, so that none
// waits for another.  The partials are read once: nontemporal loads keep them from
// displacing W1 in L2, which the next step's GEMM reads again (measured: the large
// chain batch's GEMM 15.7 -> 13.8 us).
template <int DT, int CPL>
__device__ inline float head_z_cols(const HeadArgs &a, int64_t m, int lane, int ksplit) {
    constexpr int SPL = 64 / CPL;
    const void *b1 = a.b1 ? a.b1 : a.w2;                  // no bias: read w2, use 0
    float acc = 0.f;
    for (int n0 = 0; n0 < a.h; n0 += 64 * CPL) {
        float v[CPL], bias[CPL], w[CPL];
#pragma unroll
        for (int i = 0; i < CPL; ++i) {
            const int nc = min(n0 + i * 64 + lane, a.h - 1);
            bias[i] = scalar_at<DT>(b1, nc);
            w[i] = scalar_at<DT>(a.w2, nc);
            v[i] = 0.f;
        }
        for (int k0 = 0; k0 < ksplit; k0 += SPL) {
            float u[CPL][SPL];
#pragma unroll
            for (int i = 0; i < CPL; ++i)
#pragma unroll
                for (int k = 0; k < SPL; ++k) {
                    const int nc = min(n0 + i * 64 + lane, a.h - 1);
                    const int kc = min(k0 + k, ksplit - 1);
                    u[i][k] = __builtin_nontemporal_load(&a.upart[(static_cast<int64_t>(kc) * a.m_cap + m) * a.h + nc]);
                }
#pragma unroll
            for (int i = 0; i < CPL; ++i)
#pragma unroll
                for (int k = 0; k < SPL; ++k) v[i] += k0 + k < ksplit ? u[i][k] : 0.f;
        }
#pragma unroll
        for (int i = 0; i < CPL; ++i) {
            if (n0 + i * 64 + lane < a.h) {
                const float bi = a.b1 ? bias[i] : 0.f;
                acc = fmaf(fmaxf(v[i] + bi, 0.f), w[i], acc);
            }
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
    return acc;
}

// z of list entry m, in every lane of the calling wave, from the first `ksplit`
// k-slices of upart; NaN when its hidden row is outside [0, n_rows).  Each column's
// k-slices are summed in slice order.
template <int DT>
__device__ inline float head_z(const HeadArgs &a, int64_t m, int lane, int ksplit) {
    const float acc = a.h <= 256 ? head_z_cols<DT, 4>(a, m, lane, ksplit) : head_z_cols<DT, 8>(a, m, lane, ksplit);
    const int64_t id = hidden_row(a, m);
    return id >= 0 && id < a.n_rows ? acc + a.b2 : NAN;
}

}  // namespace headz
}  // namespace cospec
