// Arbitration head on the compacted mismatch rows (Section 3.3,
// z_i = g_phi(h_i), read as z = w2 . relu(W1 h + b1) + b2).
//
// U = H_sel W1^T is a dense [M x d] x [d x h] contraction, so it runs on the
// matrix cores: v_mfma_f32_16x16x32_bf16 for bf16 operands (v_mfma_f32_16x16x4_f32
// for fp32), fp32 accumulation.  A workgroup owns a 64-row x 64-column tile of
// U; its four waves each own 32 x 32 (2 x 2 MFMA tiles) and run the whole
// d-loop.  The epilogue adds b1, applies the ReLU, multiplies by w2 and sums its
// 64 columns in a fixed order, writing one partial logit per row and column
// tile; the scan kernels add the column tiles in order and b2.  M (the number
// of mismatches) is read on the device, and workgroups past it exit at once.
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

template <int DT> __device__ inline float scalar_at(const void *p, int64_t i);
template <> __device__ inline float scalar_at<kBF16>(const void *p, int64_t i) {
    return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t *>(p)[i]) << 16);
}
template <> __device__ inline float scalar_at<kF32>(const void *p, int64_t i) {
    return static_cast<const float *>(p)[i];
}

// One k-step of the 2x2 wave tile.  bf16: 32 k per step, one 16-byte vector per
// lane and operand.  f32: 16 k per step, one float4 per lane, four MFMAs.
template <int DT> struct Step;
template <> struct Step<kBF16> {
    static constexpr int kK = 32;
    static constexpr int kLaneK = 8;
    __device__ static inline void mma(const u32x4 (&A)[2], const u32x4 (&B)[2], floatx4 (&acc)[2][2]) {
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int c = 0; c < 2; ++c)
                acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    __builtin_bit_cast(bf16x8, A[r]), __builtin_bit_cast(bf16x8, B[c]), acc[r][c], 0, 0, 0);
    }
};
template <> struct Step<kF32> {
    static constexpr int kK = 16;
    static constexpr int kLaneK = 4;
    __device__ static inline void mma(const u32x4 (&A)[2], const u32x4 (&B)[2], floatx4 (&acc)[2][2]) {
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                        __uint_as_float(A[r][j]), __uint_as_float(B[c][j]), acc[r][c], 0, 0, 0);
    }
};

template <int DT>
__global__ __launch_bounds__(256) void k_head(HeadArgs a) {
    using St = Step<DT>;
    constexpr int EB = DT == kBF16 ? 2 : 4;
    const int64_t M = a.count_dev ? static_cast<int64_t>(*a.count_dev) : a.count_host;
    const int64_t m_base = static_cast<int64_t>(blockIdx.x) * kHeadTileM;
    if (m_base >= M) return;
    const int n_base = blockIdx.y * kHeadTileN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave >> 1, wc = wave & 1;
    const int g = lane >> 4, l16 = lane & 15;

    // operand row pointers of this lane (clamped rows/columns compute garbage that is never stored)
    const char *arow[2];
    const char *brow[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        int64_t m = m_base + wr * 32 + r * 16 + l16;
        if (m >= M) m = M - 1;
        int64_t id = a.list ? static_cast<int64_t>(a.list[m]) : m;
        if (id < 0 || id >= a.n_rows) id = 0;
        arow[r] = static_cast<const char *>(a.hidden) + id * static_cast<int64_t>(a.d) * EB;
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        int n = n_base + wc * 32 + c * 16 + l16;
        if (n >= a.h) n = a.h - 1;
        brow[c] = static_cast<const char *>(a.w1) + static_cast<int64_t>(n) * a.d * EB;
    }

    floatx4 acc[2][2];
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int c = 0; c < 2; ++c) acc[r][c] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int lane_k = g * St::kLaneK;
    int kk = 0;
    // whole steps, two at a time so the next step's loads are in flight during the MFMAs
    for (; kk + 2 * St::kK <= a.d; kk += 2 * St::kK) {
        u32x4 A0[2], B0[2], A1[2], B1[2];
        const int64_t o0 = static_cast<int64_t>(kk + lane_k) * EB;
        const int64_t o1 = o0 + static_cast<int64_t>(St::kK) * EB;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            A0[r] = *reinterpret_cast<const u32x4 *>(arow[r] + o0);
            A1[r] = *reinterpret_cast<const u32x4 *>(arow[r] + o1);
        }
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            B0[c] = *reinterpret_cast<const u32x4 *>(brow[c] + o0);
            B1[c] = *reinterpret_cast<const u32x4 *>(brow[c] + o1);
        }
        St::mma(A0, B0, acc);
        St::mma(A1, B1, acc);
    }
    // remaining k (a partial step is zero-filled per lane vector; d is a multiple of the vector)
    for (; kk < a.d; kk += St::kK) {
        u32x4 A[2], Bv[2];
        const bool in = kk + lane_k < a.d;
        const int64_t o = static_cast<int64_t>(kk + lane_k) * EB;
#pragma unroll
        for (int r = 0; r < 2; ++r) A[r] = in ? *reinterpret_cast<const u32x4 *>(arow[r] + o) : u32x4{0, 0, 0, 0};
#pragma unroll
        for (int c = 0; c < 2; ++c) Bv[c] = in ? *reinterpret_cast<const u32x4 *>(brow[c] + o) : u32x4{0, 0, 0, 0};
        St::mma(A, Bv, acc);
    }

    // epilogue: relu(U + b1) * w2, summed over this wave's 32 columns
    float part[2][4];
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j) part[r][j] = 0.f;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        const int n = n_base + wc * 32 + c * 16 + l16;
        float bias = 0.f, w = 0.f;
        if (n < a.h) {
            bias = a.b1 ? scalar_at<DT>(a.b1, n) : 0.f;
            w = scalar_at<DT>(a.w2, n);
        }
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int j = 0; j < 4; ++j) part[r][j] += fmaxf(acc[r][c][j] + bias, 0.f) * w;
    }
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1)
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int j = 0; j < 4; ++j) part[r][j] += __shfl_xor(part[r][j], off);

    __shared__ float s_z[2][kHeadTileM];
    if (l16 == 0) {
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int j = 0; j < 4; ++j) s_z[wc][wr * 32 + r * 16 + 4 * g + j] = part[r][j];
    }
    __syncthreads();
    if (tid < kHeadTileM && m_base + tid < M)
        a.zpart[static_cast<int64_t>(blockIdx.y) * a.m_cap + m_base + tid] = s_z[0][tid] + s_z[1][tid];
}

__global__ __launch_bounds__(256) void k_arb_finish(ArbFinishArgs a) {
    const int64_t k = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (k >= a.n_sel) return;
    const int64_t r = a.row_index ? static_cast<int64_t>(a.row_index[k]) : k;
    float z = NAN;
    uint8_t acc = 0;
    if (r >= 0 && r < a.n_rows) {
        z = a.b2;
        for (int t = 0; t < a.n_htiles; ++t) z += a.zpart[static_cast<int64_t>(t) * a.m_cap + k];
        const float pi = 1.0f / (1.0f + expf(-z));
        acc = pi > a.lambda;
    }
    if (a.out_z) a.out_z[k] = z;
    if (a.out_accept) a.out_accept[k] = acc;
}

}  // namespace

hipError_t launch_head(Dtype dt, const HeadArgs &a, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>((a.m_cap + kHeadTileM - 1) / kHeadTileM),
                    static_cast<unsigned>((a.h + kHeadTileN - 1) / kHeadTileN));
    if (grid.x == 0) return hipSuccess;
    if (dt == kBF16) hipLaunchKernelGGL(k_head<kBF16>, grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_head<kF32>, grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_arb_finish(const ArbFinishArgs &a, hipStream_t s) {
    const unsigned blocks = static_cast<unsigned>((a.n_sel + 255) / 256);
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_arb_finish, dim3(blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace cospec
