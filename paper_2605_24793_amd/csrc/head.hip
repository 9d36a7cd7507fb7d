// Arbitration head on the compacted mismatch rows (Section 3.3,
// z_i = g_phi(h_i), read as z = w2 . relu(W1 h + b1) + b2).
//
// U = H_sel W1^T is a dense [M x d] x [d x h] contraction, so it runs on the
// matrix cores: v_mfma_f32_16x16x32_bf16 for bf16 operands (v_mfma_f32_16x16x4_f32
// for fp32), fp32 accumulation.
//
// k_head_gemm: a workgroup owns a 128 x 128 tile of U and one of `ksplit`
// slices of d.  Its 256 threads stage 128-byte k-slices of the 128 gathered
// hidden rows and 128 W1 rows through LDS (double-buffered, rows padded to
// 144 bytes), and each of its four waves accumulates a 64 x 64 sub-tile
// (4 x 4 MFMA tiles).  The slice's partial U goes to the workspace.  M (the
// number of mismatches) is read on the device; workgroups past it exit.
//
// k_head_epilogue: one wave per row adds the k-slices in a fixed order, then
// b1, the ReLU, w2 and b2, so z is bit-identical run to run.
//
// MFMA operand layout used: for the 16x16 shapes, lane l supplies row (l % 16)
// of A and column (l % 16) of B for the k-slice owned by lane group l / 16, and
// receives D[4*(l/16) + j][l % 16] in accumulator element j.  A and B take the
// same k-slice per lane, so the order of k inside an instruction is immaterial.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "launch.h"

namespace cospec {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float floatx4;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kStageBytes = 128;                  // bytes of k per row per stage
constexpr int kLdsRow = kStageBytes + 16;         // padded LDS row
constexpr int kWaveTile = 64;

template <int DT> __device__ inline float scalar_at(const void *p, int64_t i);
template <> __device__ inline float scalar_at<kBF16>(const void *p, int64_t i) {
    return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t *>(p)[i]) << 16);
}
template <> __device__ inline float scalar_at<kF32>(const void *p, int64_t i) {
    return static_cast<const float *>(p)[i];
}

// One 64-byte k-step of a 16x16 tile: one 16-byte operand vector per lane.
template <int DT> __device__ inline floatx4 mma(u32x4 a, u32x4 b, floatx4 c);
template <> __device__ inline floatx4 mma<kBF16>(u32x4 a, u32x4 b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
template <> __device__ inline floatx4 mma<kF32>(u32x4 a, u32x4 b, floatx4 c) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[j]), __uint_as_float(b[j]), c, 0, 0, 0);
    return c;
}

template <int DT>
__global__ __launch_bounds__(256) void k_head_gemm(HeadArgs a) {
    constexpr int EB = DT == kBF16 ? 2 : 4;
    constexpr int BK = kStageBytes / EB;          // elements of k per stage
    constexpr int VE = 16 / EB;                   // elements per 16-byte vector
    const int64_t M = a.count_dev ? static_cast<int64_t>(*a.count_dev) : a.count_host;
    const int64_t m_base = static_cast<int64_t>(blockIdx.x) * kHeadTileM;
    if (m_base >= M) return;
    const int n_base = blockIdx.y * kHeadTileN;
    const int ks = blockIdx.z;
    const int kchunk = ((a.d + a.ksplit - 1) / a.ksplit + BK - 1) / BK * BK;
    const int k0 = ks * kchunk;
    const int k1 = min(a.d, k0 + kchunk);
    const int nst = k1 > k0 ? (k1 - k0 + BK - 1) / BK : 0;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave >> 1, wc = wave & 1;
    const int g = lane >> 4, l16 = lane & 15;

    __shared__ __attribute__((aligned(16))) char sA[2][kHeadTileM * kLdsRow];
    __shared__ __attribute__((aligned(16))) char sB[2][kHeadTileN * kLdsRow];

    // loader: thread t moves 16 bytes of rows (t >> 3) + 32 j, j = 0..3
    const int lrow = tid >> 3, lcol = (tid & 7) * 16;
    const char *ga[4];
    const char *gb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        int64_t m = m_base + lrow + 32 * j;
        if (m >= M) m = M - 1;                     // garbage rows are computed, never stored
        int64_t id = a.list ? static_cast<int64_t>(a.list[m]) : m;
        if (id < 0 || id >= a.n_rows) id = 0;
        ga[j] = static_cast<const char *>(a.hidden) + id * static_cast<int64_t>(a.d) * EB;
        int n = n_base + lrow + 32 * j;
        if (n >= a.h) n = a.h - 1;
        gb[j] = static_cast<const char *>(a.w1) + static_cast<int64_t>(n) * a.d * EB;
    }
    u32x4 ra[4], rb[4];
    auto fetch = [&](int st) {
        const int e = k0 + st * BK + (tid & 7) * VE;     // first element of this thread's vector
        const bool in = e < k1;                          // d is a multiple of VE
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            ra[j] = in ? *reinterpret_cast<const u32x4 *>(ga[j] + static_cast<int64_t>(e) * EB) : u32x4{0, 0, 0, 0};
            rb[j] = in ? *reinterpret_cast<const u32x4 *>(gb[j] + static_cast<int64_t>(e) * EB) : u32x4{0, 0, 0, 0};
        }
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            *reinterpret_cast<u32x4 *>(&sA[buf][(lrow + 32 * j) * kLdsRow + lcol]) = ra[j];
            *reinterpret_cast<u32x4 *>(&sB[buf][(lrow + 32 * j) * kLdsRow + lcol]) = rb[j];
        }
    };

    floatx4 acc[4][4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = floatx4{0.f, 0.f, 0.f, 0.f};

    if (nst > 0) {
        fetch(0);
        stash(0);
    }
    __syncthreads();
    for (int st = 0; st < nst; ++st) {
        const int buf = st & 1;
        if (st + 1 < nst) fetch(st + 1);               // next slice in flight during the MFMAs
#pragma unroll
        for (int kk = 0; kk < kStageBytes; kk += 64) {
            u32x4 av[4], bv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r)
                av[r] = *reinterpret_cast<const u32x4 *>(&sA[buf][(wr * kWaveTile + r * 16 + l16) * kLdsRow + kk + g * 16]);
#pragma unroll
            for (int c = 0; c < 4; ++c)
                bv[c] = *reinterpret_cast<const u32x4 *>(&sB[buf][(wc * kWaveTile + c * 16 + l16) * kLdsRow + kk + g * 16]);
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int c = 0; c < 4; ++c) acc[r][c] = mma<DT>(av[r], bv[c], acc[r][c]);
        }
        if (st + 1 < nst) stash(buf ^ 1);
        __syncthreads();
    }

    // partial U of this k-slice: upart[ks][m][n]
    float *up = a.upart + static_cast<int64_t>(ks) * a.m_cap * a.h;
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t m = m_base + wr * kWaveTile + r * 16 + 4 * g + j;
            if (m < M) {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int n = n_base + wc * kWaveTile + c * 16 + l16;
                    if (n < a.h) up[m * a.h + n] = acc[r][c][j];
                }
            }
        }
}

// z[m] = w2 . relu(sum_ks upart[ks][m] + b1) + b2, one wave per row, fixed order.
template <int DT>
__global__ __launch_bounds__(256) void k_head_epilogue(HeadArgs a) {
    const int64_t M = a.count_dev ? static_cast<int64_t>(*a.count_dev) : a.count_host;
    const int64_t m = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (m >= M) return;
    const int lane = threadIdx.x & 63;
    float acc = 0.f;
    for (int n = lane; n < a.h; n += 64) {
        float u = 0.f;
        for (int ks = 0; ks < a.ksplit; ++ks) u += a.upart[(static_cast<int64_t>(ks) * a.m_cap + m) * a.h + n];
        const float bias = a.b1 ? scalar_at<DT>(a.b1, n) : 0.f;
        acc += fmaxf(u + bias, 0.f) * scalar_at<DT>(a.w2, n);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
    if (lane == 0) a.z[m] = acc + a.b2;
}

__global__ __launch_bounds__(256) void k_arb_finish(ArbFinishArgs a) {
    const int64_t k = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (k >= a.n_sel) return;
    const int64_t r = a.row_index ? static_cast<int64_t>(a.row_index[k]) : k;
    float z = NAN;
    uint8_t acc = 0;
    if (r >= 0 && r < a.n_rows) {
        z = a.z[k];
        const float pi = 1.0f / (1.0f + expf(-z));
        acc = pi > a.lambda;
    }
    if (a.out_z) a.out_z[k] = z;
    if (a.out_accept) a.out_accept[k] = acc;
}

}  // namespace

int32_t head_ksplit(int64_t m_cap, int32_t d, int32_t h, int32_t elem_bytes) {
    const int64_t mt = (m_cap + kHeadTileM - 1) / kHeadTileM;
    const int64_t nt = (h + kHeadTileN - 1) / kHeadTileN;
    if (mt * nt <= 0) return 1;                        // no rows: nothing to split
    const int64_t stages = (static_cast<int64_t>(d) * elem_bytes + kStageBytes - 1) / kStageBytes;
    int64_t ks = (kHeadTargetBlocks + mt * nt - 1) / (mt * nt);
    if (ks > kHeadMaxSplit) ks = kHeadMaxSplit;
    if (ks > stages) ks = stages;
    if (ks < 1) ks = 1;
    return static_cast<int32_t>(ks);
}

hipError_t launch_head(Dtype dt, const HeadArgs &a, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>((a.m_cap + kHeadTileM - 1) / kHeadTileM),
                    static_cast<unsigned>((a.h + kHeadTileN - 1) / kHeadTileN),
                    static_cast<unsigned>(a.ksplit));
    if (grid.x == 0) return hipSuccess;
    const dim3 egrid(static_cast<unsigned>((a.m_cap + 3) / 4));
    if (dt == kBF16) {
        hipLaunchKernelGGL(k_head_gemm<kBF16>, grid, dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_head_epilogue<kBF16>, egrid, dim3(256), 0, s, a);
    } else {
        hipLaunchKernelGGL(k_head_gemm<kF32>, grid, dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_head_epilogue<kF32>, egrid, dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_arb_finish(const ArbFinishArgs &a, hipStream_t s) {
    const unsigned blocks = static_cast<unsigned>((a.n_sel + 255) / 256);
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_arb_finish, dim3(blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace cospec
