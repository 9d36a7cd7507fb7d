// Arbitration head on the compacted mismatch rows (Section 3.3,
// z_i = g_phi(h_i), read as z = w2 . relu(W1 h + b1) + b2).
//
// U = H_sel W1^T is a dense [M x d] x [d x h] contraction, so it runs on the
// matrix cores: v_mfma_f32_16x16x32_bf16 for bf16 operands (v_mfma_f32_16x16x4_f32
// for fp32), fp32 accumulation.
//
// k_head_gemm: a workgroup owns a 128 x 128 tile of U and one of `ksplit`
// slices of d.  Its 512 threads stream 128-byte k-slices of the 128 gathered
// hidden rows and 128 W1 rows into a 4-stage LDS ring with direct loads, and
// each of its eight waves (two per SIMD, so one wave's LDS reads overlap the
// other's MFMAs) accumulates a 64 x 32 sub-tile (4 x 2 MFMA tiles).  The
// slice's partial U goes to the workspace.  M (the number of mismatches) is
// read on the device; workgroups past it exit.
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

#include "head_z.h"
#include "launch.h"

namespace cospec {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float floatx4;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kStageBytes = 128;                  // bytes of k per row per stage
// LDS ring depth: four stages (three in flight while one is used, 128 KiB: one
// workgroup per CU), or two (64 KiB: two workgroups per CU) when the grid has more
// workgroups than there are CUs.
constexpr int kRingDeep = 4;
constexpr int kRingShallow = 2;
constexpr int kWaveTile = 64;                    // rows of a wave's sub-tile
constexpr int kWaveCols = 32;                    // columns of a wave's sub-tile
constexpr int kGemmWaves = 8;                    // 2 x 4 waves per workgroup: two per SIMD

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

typedef __attribute__((address_space(3))) char lds_char;

// Waits until at most N vector-memory operations of this wave are outstanding.
template <int N> __device__ inline void wait_vm() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

// Waits until this wave has at most PER * later of its loads in flight, later <= MAXL.
template <int PER, int MAXL> __device__ inline void wait_later(int later) {
    if constexpr (MAXL > 0) {
        if (later >= MAXL) wait_vm<PER * MAXL>();
        else wait_later<PER, MAXL - 1>(later);
    } else {
        wait_vm<0>();
    }
}

// Workgroup barrier without the memory fence of __syncthreads (which would also wait
// for the stages still in flight); LDS writes of this wave are drained first and the
// compiler may not move memory accesses across it.
__device__ inline void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

using headz::mapped_row;

template <int DT, int kRing>
__global__ __launch_bounds__(64 * kGemmWaves) void k_head_gemm(HeadArgs a) {
    constexpr int EB = DT == kBF16 ? 2 : 4;
    constexpr int BK = kStageBytes / EB;          // elements of k per stage
    constexpr int VE = 16 / EB;                   // elements per 16-byte vector
    // 1-D grid, k-slice fastest: workgroups are dealt to the 8 XCDs round-robin, so with
    // 8 slices each XCD owns one slice of the hidden rows and of W1, which fits its L2
    const int ks = blockIdx.x % a.ksplit;
    const int tile = blockIdx.x / a.ksplit;
    const int mtiles = static_cast<int>((a.m_cap + kHeadTileM - 1) / kHeadTileM);
    const int64_t m_base = static_cast<int64_t>(tile % mtiles) * kHeadTileM;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lrow = lane >> 3, lslot = lane & 7;
    // the list entries of this lane's two loader rows are read together with M (not
    // after it): entries past M are stale and replaced below, so the first operand
    // loads wait for one memory round trip instead of two
    int32_t lid[2] = {0, 0};
    if (a.list) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int64_t m = min(m_base + 8 * (wave * 2 + i) + lrow, a.m_cap - 1);
            lid[i] = a.list[m];
        }
    }
    const int64_t M = a.count_dev ? static_cast<int64_t>(*a.count_dev) : a.count_host;
    if (m_base >= M) return;
    const int n_base = (tile / mtiles) * kHeadTileN;
    const int kchunk = ((a.d + a.ksplit - 1) / a.ksplit + BK - 1) / BK * BK;
    const int k0 = ks * kchunk;
    const int k1 = min(a.d, k0 + kchunk);
    const int nst = k1 > k0 ? (k1 - k0 + BK - 1) / BK : 0;

    const int wr = wave >> 2, wc = wave & 3;
    const int g = lane >> 4, l16 = lane & 15;

    // LDS ring of kRing stages; a stage holds 128 rows of A then 128 rows of B, 128 bytes
    // each, the 16-byte slot s of row r holding k-vector (s ^ (r & 7)) of the stage
    __shared__ __attribute__((aligned(16))) char ring[kRing][2 * kHeadTileM * kStageBytes];

    // async loader: per stage, wave w fills 1 KB blocks w*2+i of A and of B (8 rows each);
    // lane l brings row 8*(w*2+i) + l/8, k-vector (l%8) ^ (row%8)
    const char *ga[2];
    const char *gb[2];
    int lvec[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int row = 8 * (wave * 2 + i) + lrow;
        lvec[i] = lslot ^ (row & 7);
        const int64_t m = m_base + row;
        // rows past M are computed from row 0 and never stored; an invalid id's logit
        // is set to NaN by the epilogue
        int64_t id = m >= M ? 0 : a.list ? mapped_row(a, lid[i]) : mapped_row(a, m);
        if (id < 0 || id >= a.n_rows) id = 0;
        ga[i] = static_cast<const char *>(a.hidden) + id * static_cast<int64_t>(a.d) * EB;
        int n = n_base + row;
        if (n >= a.h) n = a.h - 1;
        gb[i] = static_cast<const char *>(a.w1) + static_cast<int64_t>(n) * a.d * EB;
    }
    auto issue = [&](int st) {
        char *slot = ring[st % kRing];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int e = k0 + st * BK + lvec[i] * VE;          // first element of the vector
            char *la = slot + (wave * 2 + i) * 1024;
            char *lb = slot + kHeadTileM * kStageBytes + (wave * 2 + i) * 1024;
            if (e < k1) {                                       // d is a multiple of VE
                __builtin_amdgcn_global_load_lds(ga[i] + static_cast<int64_t>(e) * EB, (lds_char *)la, 16, 0, 0);
                __builtin_amdgcn_global_load_lds(gb[i] + static_cast<int64_t>(e) * EB, (lds_char *)lb, 16, 0, 0);
            } else {                                            // ragged end of d: zeros
                *reinterpret_cast<u32x4 *>(la + lane * 16) = u32x4{0, 0, 0, 0};
                *reinterpret_cast<u32x4 *>(lb + lane * 16) = u32x4{0, 0, 0, 0};
            }
        }
    };

    floatx4 acc[4][2];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 2; ++c) acc[r][c] = floatx4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
    for (int st = 0; st < kRing - 1; ++st)
        if (st < nst) issue(st);
    for (int st = 0; st < nst; ++st) {
        // this wave's loads of stage st are done once at most the later stages' remain
        wait_later<4, kRing - 2>(min(kRing - 2, nst - 1 - st));   // 4 loads per wave and stage
        lds_barrier();                            // every wave's part of stage st has landed
        if (st + kRing - 1 < nst) issue(st + kRing - 1);   // refills the slot of stage st-1
        const char *sa = ring[st % kRing];
        const char *sb = sa + kHeadTileM * kStageBytes;
        // every fragment of the stage is read before the first product, so the LDS
        // latency is paid once per stage rather than once per k-step
        constexpr int KS = kStageBytes / 64;                // 64-byte k-steps per stage
        u32x4 av[KS][4], bv[KS][2];
#pragma unroll
        for (int q = 0; q < KS; ++q) {
            const int kk = 4 * q;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = wr * kWaveTile + r * 16 + l16;
                av[q][r] = *reinterpret_cast<const u32x4 *>(sa + row * kStageBytes + (((kk + g) ^ (row & 7)) * 16));
            }
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const int row = wc * kWaveCols + c * 16 + l16;
                bv[q][c] = *reinterpret_cast<const u32x4 *>(sb + row * kStageBytes + (((kk + g) ^ (row & 7)) * 16));
            }
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < KS; ++q)
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int c = 0; c < 2; ++c) acc[r][c] = mma<DT>(av[q][r], bv[q][c], acc[r][c]);
    }

    // partial U of this k-slice: upart[ks][m][n].  Nontemporal stores: the partials are
    // read once, by the second layer, and do not stay dirty in this XCD's L2 for the
    // write-back at the kernel's end (measured: 17.4 -> 15.6 us on the large chain batch)
    float *up = a.upart + static_cast<int64_t>(ks) * a.m_cap * a.h;
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t m = m_base + wr * kWaveTile + r * 16 + 4 * g + j;
            if (m < M) {
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    const int n = n_base + wc * kWaveCols + c * 16 + l16;
                    if (n < a.h) __builtin_nontemporal_store(acc[r][c][j], &up[m * a.h + n]);
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
    const float z = headz::head_z<DT>(a, m, threadIdx.x & 63);
    if ((threadIdx.x & 63) == 0) a.z[m] = z;
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

// k-slices of d: one per XCD (each XCD's L2 then holds one slice of the hidden rows
// and of W1), more, in multiples of the XCD count, while the tiles times slices stay
// below one workgroup per CU; never more than there are stages of d.
int32_t head_ksplit(int64_t m_cap, int32_t d, int32_t h, int32_t elem_bytes) {
    const int64_t mt = (m_cap + kHeadTileM - 1) / kHeadTileM;
    const int64_t nt = (h + kHeadTileN - 1) / kHeadTileN;
    if (mt * nt <= 0) return 1;                        // no rows: nothing to split
    const int64_t stages = (static_cast<int64_t>(d) * elem_bytes + kStageBytes - 1) / kStageBytes;
    int64_t ks = kXcds;
    while (ks + kXcds <= kHeadMaxSplit && mt * nt * (ks + kXcds) <= kHeadTargetBlocks) ks += kXcds;
    if (ks > stages) ks = stages;
    if (ks < 1) ks = 1;
    return static_cast<int32_t>(ks);
}

hipError_t launch_head_gemm(Dtype dt, const HeadArgs &a, hipStream_t s) {
    const int64_t tiles = ((a.m_cap + kHeadTileM - 1) / kHeadTileM) * ((a.h + kHeadTileN - 1) / kHeadTileN);
    const dim3 grid(static_cast<unsigned>(tiles * a.ksplit));
    if (grid.x == 0) return hipSuccess;
    const dim3 block(64 * kGemmWaves);
    if (a.two_per_cu) {
        if (dt == kBF16) hipLaunchKernelGGL((k_head_gemm<kBF16, kRingShallow>), grid, block, 0, s, a);
        else hipLaunchKernelGGL((k_head_gemm<kF32, kRingShallow>), grid, block, 0, s, a);
    } else {
        if (dt == kBF16) hipLaunchKernelGGL((k_head_gemm<kBF16, kRingDeep>), grid, block, 0, s, a);
        else hipLaunchKernelGGL((k_head_gemm<kF32, kRingDeep>), grid, block, 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_head(Dtype dt, const HeadArgs &a, hipStream_t s) {
    const dim3 egrid(static_cast<unsigned>((a.m_cap + 3) / 4));
    if (egrid.x == 0) return hipSuccess;
    const hipError_t e = launch_head_gemm(dt, a, s);
    if (e != hipSuccess) return e;
    if (dt == kBF16) hipLaunchKernelGGL(k_head_epilogue<kBF16>, egrid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_head_epilogue<kF32>, egrid, dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_arb_finish(const ArbFinishArgs &a, hipStream_t s) {
    const unsigned blocks = static_cast<unsigned>((a.n_sel + 255) / 256);
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_arb_finish, dim3(blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace cospec
