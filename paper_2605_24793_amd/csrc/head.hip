// Arbitration head on the compacted mismatch rows (Section 3.3,
// z_i = g_phi(h_i), read as z = w2 . relu(W1 h + b1) + b2).
//
// U = H_sel W1^T is a dense [M x d] x [d x h] contraction, so it runs on the
// matrix cores: v_mfma_f32_16x16x32_bf16 for bf16 operands (v_mfma_f32_16x16x4_f32
// for fp32), fp32 accumulation.
//
// gemm_tile: a workgroup computes a 128 x 128 tile of U over one of the slices
// of d.  Its 512 threads stream 128-byte k-slices of the 128 gathered hidden
// rows and 128 W1 rows into a 4-stage LDS ring with direct loads, and each of
// its eight waves (two per SIMD, so one wave's LDS reads overlap the other's
// MFMAs) accumulates a 64 x 32 sub-tile (4 x 2 MFMA tiles).  The slice's
// partial U goes to the workspace.
//
// k_head_gemm (trees): one workgroup per (tile, slice) of the list's capacity;
// M (the number of mismatches) is read on the device, workgroups past it exit.
// k_head_gemm_loop (chains): one workgroup per resident slot; each derives M
// and the list itself (or reads them) and loops over the items of the M rows
// only, the slices cut so that the items fill the grid once.
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

#include <mutex>

#include "head_z.h"
#include "launch.h"
#include "rowstat.h"

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

constexpr int kGemmThreads = 64 * kGemmWaves;
constexpr int kBuildPer = kBuildListMax / kGemmThreads;   // slots per thread in the scan
static_assert(kBuildPer == 8 && kBuildPer * kGemmThreads == kBuildListMax, "build_list: 8 slots per thread");

// Lane exchanges of build_list's combine, all in the VALU: DPP inside rows of 16 lanes,
// the gfx950 permlane swaps across rows.  The combine (larger maximum, then the earlier
// split) is commutative and associative, so pairing lanes by mirrors instead of xor
// masks reduces every group of G = 2, 4, ..., 64 lanes all the same.
constexpr int kDppXor1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int kDppMirror8 = 0x141; // row_half_mirror: lane i <-> 7 - i within 8
constexpr int kDppMirror16 = 0x140;// row_mirror:      lane i <-> 15 - i within 16

struct ArgPick {
    float x;    // the largest maximum so far (-inf: none)
    int s;      // its split (INT_MAX: none)
    int c;      // its argmax
};

__device__ inline ArgPick better(const ArgPick &p, const ArgPick &q) {
    const bool t = (q.x > p.x) | ((q.x == p.x) & (q.s < p.s));
    return ArgPick{t ? q.x : p.x, t ? q.s : p.s, t ? q.c : p.c};
}

template <int CTRL>
__device__ inline int dpp_int(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xf, 0xf, false);
}

template <int CTRL>
__device__ inline ArgPick combine_dpp(const ArgPick &p) {
    const ArgPick q{__int_as_float(dpp_int<CTRL>(__float_as_int(p.x))), dpp_int<CTRL>(p.s), dpp_int<CTRL>(p.c)};
    return better(p, q);
}

// Lane l combined with lane l ^ 16 (ROW32 false) or l ^ 32 (true): each swap returns
// the pair (own, partner) in some order, and the combine is symmetric in it.
template <bool ROW32>
__device__ inline ArgPick combine_swap(const ArgPick &p) {
    auto sw = [](int v) {
        const auto r = ROW32 ? __builtin_amdgcn_permlane32_swap(v, v, false, false)
                             : __builtin_amdgcn_permlane16_swap(v, v, false, false);
        return r;
    };
    const auto x = sw(__float_as_int(p.x)), s = sw(p.s), c = sw(p.c);
    return better(ArgPick{__int_as_float(static_cast<int>(x[0])), static_cast<int>(s[0]), static_cast<int>(c[0])},
                  ArgPick{__int_as_float(static_cast<int>(x[1])), static_cast<int>(s[1]), static_cast<int>(c[1])});
}

// Part 1 of build_list for one batch of NB (slot, split) items per thread: item
// i = base + j * kGemmThreads + tid is split (i mod G) of slot i / G.
template <bool CAND, int NB>
__device__ inline void mark_batch(const HeadArgs &a, int base, int n, int lg, int splits, uint64_t kmag,
                                  uint8_t *s_need) {
    const int tid = threadIdx.x;
    const int G = 1 << lg;
    int tok[NB], r[NB];
    ArgPick p[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int i = base + j * kGemmThreads + tid;
        const int di = (i >> lg) < n ? (i >> lg) : 0;      // past the end: slot 0, dropped
        r[j] = di + static_cast<int>((static_cast<uint64_t>(di) * kmag) >> 32);   // b*(K+1) + i
    }
    // every load of the batch first, unconditionally, so that none waits for another
    if constexpr (CAND) {
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int i = base + j * kGemmThreads + tid;
            tok[j] = a.tokens[(i >> lg) < n ? (i >> lg) : 0];
            p[j] = ArgPick{-INFINITY, INT_MAX, a.cand[r[j]]};
        }
    } else {
        u32x4 q[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int i = base + j * kGemmThreads + tid;
            q[j] = *reinterpret_cast<const u32x4 *>(a.partials + (r[j] * splits + min(i & (G - 1), splits - 1)));
            tok[j] = a.tokens[(i >> lg) < n ? (i >> lg) : 0];
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            // the split's maximum when it holds one (S > 0) and the lane has a split;
            // a single split is taken on S > 0 alone, as merge_row takes it
            const int sub = (base + j * kGemmThreads + tid) & (G - 1);
            const float qx = __uint_as_float(q[j].x), qs = __uint_as_float(q[j].z);
            const bool take = (sub < splits) & (qs > 0.f) & ((qx > -INFINITY) | (splits == 1));
            p[j] = take ? ArgPick{qx, sub, static_cast<int>(q[j].y)} : ArgPick{-INFINITY, INT_MAX, INT_MAX};
        }
        // the loads' unused fourth words stay live until here, so their registers are
        // not reused (which would make the first load wait before the others)
#pragma unroll
        for (int j = 0; j < NB; ++j) asm volatile("" ::"v"(q[j].w));
        if (lg >= 1) {
#pragma unroll
            for (int j = 0; j < NB; ++j) p[j] = combine_dpp<kDppXor1>(p[j]);
        }
        if (lg >= 2) {
#pragma unroll
            for (int j = 0; j < NB; ++j) p[j] = combine_dpp<kDppXor2>(p[j]);
        }
        if (lg >= 3) {
#pragma unroll
            for (int j = 0; j < NB; ++j) p[j] = combine_dpp<kDppMirror8>(p[j]);
        }
        if (lg >= 4) {
#pragma unroll
            for (int j = 0; j < NB; ++j) p[j] = combine_dpp<kDppMirror16>(p[j]);
        }
        if (lg >= 5) {
#pragma unroll
            for (int j = 0; j < NB; ++j) p[j] = combine_swap<false>(p[j]);
        }
        if (lg >= 6) {
#pragma unroll
            for (int j = 0; j < NB; ++j) p[j] = combine_swap<true>(p[j]);
        }
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int i = base + j * kGemmThreads + tid;
        const int di = i >> lg;
        if (di < n && (i & (G - 1)) == 0) s_need[di] = tok[j] >= 0 && tok[j] < a.V && tok[j] != p[j].c;
    }
}

// The head's list for a chain step, derived by the workgroup from the reduction's
// partials (the decision step of Section 3.1 for the rows that need the head): slot
// di = b*K + i is a mismatch when its draft token is valid and differs from the
// candidate of target row b*(K+1) + i, which is the argmax of the row's partials, or
// the candidate already taken (a.cand).  Writes the list (kBuildListMax entries of
// LDS) and returns M, the number of mismatches.
//
// Part 1 marks the mismatches in LDS.  The argmax is the one merge_row takes (the
// first split, in split order, whose maximum is strictly the largest): G lanes
// (G = splits rounded up to a power of two) take one split each and combine their
// (max, split) pairs, larger maximum first and the earlier split on ties.  The
// (slot, split) items are dealt in batches of 4, 8 or 16 per thread (the fewest that
// cover them), every load of a batch issued before the first is used.  Part 2 numbers
// the mismatches in slot order: thread t owns slots [kBuildPer*t, kBuildPer*(t+1)), a
// workgroup-wide exclusive scan gives their positions.
template <bool CAND>
__device__ inline int64_t build_list(const HeadArgs &a, int32_t *list) {
    __shared__ int s_wave[kGemmWaves];
    uint8_t *s_need = reinterpret_cast<uint8_t *>(list);   // part 1's flags: read before part 2 writes
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = static_cast<int>(a.m_cap);
    const int splits = CAND ? 1 : a.plan.splits;
    int lg = 0;
    while ((1 << lg) < splits) ++lg;                  // G = 2^lg <= 64 lanes per slot
    const int items = n << lg;
    // floor(di / K) = (di * kmag) >> 32 with kmag = ceil(2^32 / K), exact for every
    // di < 2^16 and K <= 64 (here di < kBuildListMax)
    const uint64_t kmag = ((uint64_t{1} << 32) + static_cast<uint64_t>(a.K) - 1) / static_cast<uint64_t>(a.K);
    const int per = (items + kGemmThreads - 1) / kGemmThreads;
    if (per <= 4) {
        mark_batch<CAND, 4>(a, 0, n, lg, splits, kmag, s_need);
    } else if (per <= 8) {
        mark_batch<CAND, 8>(a, 0, n, lg, splits, kmag, s_need);
    } else {
        for (int base = 0; base < items; base += 16 * kGemmThreads)      // uniform trip count
            mark_batch<CAND, 16>(a, base, n, lg, splits, kmag, s_need);
    }
    __syncthreads();
    // part 2: exclusive scan of the per-thread counts, within the wave, then over the waves
    const int d0 = tid * kBuildPer;
    uint32_t need = 0;
    if (d0 < n) {
        const uint2 w = *reinterpret_cast<const uint2 *>(s_need + d0);
#pragma unroll
        for (int j = 0; j < kBuildPer; ++j) {
            const uint32_t byte = ((j < 4 ? w.x : w.y) >> (8 * (j & 3))) & 0xffu;
            if (d0 + j < n && byte) need |= 1u << j;
        }
    }
    const int c = __popc(need);
    int incl = c;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(incl, off);
        if (lane >= off) incl += y;
    }
    if (lane == 63) s_wave[wave] = incl;
    __syncthreads();
    int before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < kGemmWaves; ++w) {
        const int t = s_wave[w];
        before += w < wave ? t : 0;
        total += t;
    }
    int pos = before + incl - c;
#pragma unroll
    for (int j = 0; j < kBuildPer; ++j) {
        if (need & (1u << j)) {
            list[pos++] = d0 + j;
        }
    }
    __syncthreads();
    return total;
}

// One 128 x 128 tile of U = X W1^T over k-slice [k0, k1) of d: rows [m_base,
// m_base + 128) of the list (M rows in all), columns [n_base, n_base + 128) of W1.
// lid: the list entries of this lane's two loader rows (m past M: anything).  With
// out_by_slot the stores go by list entry (the decision slot), read from s_list (the
// whole list in LDS) or else from s_rows, where this function puts the tile's entries.
template <int DT, int kRing>
__device__ inline void gemm_tile(const HeadArgs &a, int64_t M, int64_t m_base, int n_base, int ks, int k0, int k1,
                                 const int32_t lid[2], const int32_t *s_list, int32_t *s_rows,
                                 char (*ring)[2 * kHeadTileM * kStageBytes]) {
    constexpr int EB = DT == kBF16 ? 2 : 4;
    constexpr int BK = kStageBytes / EB;          // elements of k per stage
    constexpr int VE = 16 / EB;                   // elements per 16-byte vector
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lrow = lane >> 3, lslot = lane & 7;
    if (a.out_by_slot && !s_list) {   // the tile's slots, for the stores at the end
#pragma unroll
        for (int i = 0; i < 2; ++i)
            if (lslot == 0) s_rows[8 * (wave * 2 + i) + lrow] = lid[i];
        __syncthreads();
    }
    const int nst = k1 > k0 ? (k1 - k0 + BK - 1) / BK : 0;
    const int wr = wave >> 2, wc = wave & 3;
    const int g = lane >> 4, l16 = lane & 15;

    // LDS ring of kRing stages; a stage holds 128 rows of A then 128 rows of B, 128 bytes
    // each, the 16-byte slot s of row r holding k-vector (s ^ (r & 7)) of the stage.
    // Async loader: per stage, wave w fills 1 KB blocks w*2+i of A and of B (8 rows
    // each); lane l brings row 8*(w*2+i) + l/8, k-vector (l%8) ^ (row%8)
    const char *ga[2];
    const char *gb[2];
    int lvec[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int row = 8 * (wave * 2 + i) + lrow;
        lvec[i] = lslot ^ (row & 7);
        // rows past M are computed from row 0 and never stored; an invalid id's logit
        // is set to NaN by the second layer
        int64_t id = m_base + row >= M ? 0 : mapped_row(a, lid[i]);
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

    // partial U of this k-slice: upart[ks][row][n], row the list position m, or with
    // out_by_slot the list entry.  Nontemporal stores: the partials are read once, by the
    // second layer, and do not stay dirty in this XCD's L2 for the write-back at the
    // kernel's end (measured: 17.4 -> 15.6 us on the large chain batch)
    float *up = a.upart + static_cast<int64_t>(ks) * a.m_cap * a.h;
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int trow = wr * kWaveTile + r * 16 + 4 * g + j;
            const int64_t mm = m_base + trow;
            if (mm < M) {
                const int64_t m = !a.out_by_slot ? mm : s_list ? s_list[mm] : s_rows[trow];
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    const int n = n_base + wc * kWaveCols + c * 16 + l16;
                    if (n < a.h) __builtin_nontemporal_store(acc[r][c][j], &up[m * a.h + n]);
                }
            }
        }
}

// Grid-sized GEMM (trees): one workgroup per (tile, k-slice) of the list's capacity;
// workgroups past M leave.  1-D grid, k-slice fastest: workgroups are dealt to the 8
// XCDs round-robin, so with 8 slices each XCD owns one slice of the hidden rows and of
// W1, which fits its L2.
template <int DT, int kRing>
__global__ __launch_bounds__(64 * kGemmWaves) void k_head_gemm(HeadArgs a) {
    constexpr int BK = kStageBytes / (DT == kBF16 ? 2 : 4);
    __shared__ __attribute__((aligned(16))) char ring[kRing][2 * kHeadTileM * kStageBytes];
    __shared__ int32_t s_rows[kHeadTileM];
    const int ks = blockIdx.x % a.ksplit;
    const int tile = blockIdx.x / a.ksplit;
    const int mtiles = static_cast<int>((a.m_cap + kHeadTileM - 1) / kHeadTileM);
    const int64_t m_base = static_cast<int64_t>(tile % mtiles) * kHeadTileM;
    const int wave = threadIdx.x >> 6, lrow = (threadIdx.x & 63) >> 3;
    // the list entries of this lane's two loader rows are read together with M (not
    // after it): entries past M are stale and never used, so the first operand loads
    // wait for one memory round trip instead of two
    int32_t lid[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int64_t m = min(m_base + 8 * (wave * 2 + i) + lrow, a.m_cap - 1);
        lid[i] = a.list ? a.list[m] : static_cast<int32_t>(m);
    }
    const int64_t M = a.count_dev ? static_cast<int64_t>(*a.count_dev) : a.count_host;
    if (m_base >= M) return;
    const int kchunk = ((a.d + a.ksplit - 1) / a.ksplit + BK - 1) / BK * BK;
    const int k0 = ks * kchunk;
    gemm_tile<DT, kRing>(a, M, m_base, (tile / mtiles) * kHeadTileN, ks, k0, min(a.d, k0 + kchunk), lid, nullptr,
                         s_rows, ring);
}

// Persistent GEMM (chains): a.grid workgroups loop over the (tile, k-slice) items of
// the M listed rows only, with the k-slices cut to what fills the grid once
// (headz::live_ksplit, which the second layer repeats).  The list is built in LDS by
// every workgroup (BUILD; workgroup 0 also stores M in a.count_dev, for the second
// layer), or read from a.list (M from a.count_dev).
// LIST: kListRead (a.list), kListArgmax (built, candidates the partials' argmax),
// kListCand (built, candidates from a.cand)
enum { kListRead, kListArgmax, kListCand };

template <int DT, int kRing, int LIST>
__global__ __launch_bounds__(64 * kGemmWaves) void k_head_gemm_loop(HeadArgs a) {
    constexpr bool BUILD = LIST != kListRead;
    constexpr int BK = kStageBytes / (DT == kBF16 ? 2 : 4);
    __shared__ __attribute__((aligned(16))) char ring[kRing][2 * kHeadTileM * kStageBytes];
    __shared__ int32_t s_rows[kHeadTileM];
    __shared__ __attribute__((aligned(16))) int32_t s_list[BUILD ? kBuildListMax : 1];
    const int tid = threadIdx.x, wave = tid >> 6, lrow = (tid & 63) >> 3;
    int64_t M;
    if constexpr (BUILD) {
        M = build_list<LIST == kListCand>(a, s_list);
        if (blockIdx.x == 0 && tid == 0) *a.count_dev = static_cast<int32_t>(M);
    } else {
        M = *a.count_dev;
    }
    const int mt = static_cast<int>((M + kHeadTileM - 1) / kHeadTileM);
    const int nt = (a.h + kHeadTileN - 1) / kHeadTileN;
    const int ksl = headz::live_ksplit(a, M);
    const int kchunk = ((a.d + ksl - 1) / ksl + BK - 1) / BK * BK;
    const int items = mt * nt * ksl;
    for (int w = blockIdx.x; w < items; w += gridDim.x) {
        const int ks = w % ksl, tile = w / ksl;
        const int64_t m_base = static_cast<int64_t>(tile % mt) * kHeadTileM;
        int32_t lid[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int64_t m = min(m_base + 8 * (wave * 2 + i) + lrow, M - 1);
            lid[i] = BUILD ? s_list[m] : a.list[m];
        }
        const int k0 = ks * kchunk;
        gemm_tile<DT, kRing>(a, M, m_base, (tile / mt) * kHeadTileN, ks, k0, min(a.d, k0 + kchunk), lid,
                             BUILD ? s_list : nullptr, s_rows, ring);
        __syncthreads();          // the ring and s_rows are the next item's
    }
}

// z[m] = w2 . relu(sum_ks upart[ks][m] + b1) + b2, one wave per row, fixed order.
template <int DT>
__global__ __launch_bounds__(256) void k_head_epilogue(HeadArgs a) {
    const int64_t M = a.count_dev ? static_cast<int64_t>(*a.count_dev) : a.count_host;
    const int64_t m = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (m >= M) return;
    const float z = headz::head_z<DT>(a, m, threadIdx.x & 63, a.ksplit);
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

int32_t head_gemm_slots(Dtype dt, bool build) {
    constexpr int kMaxDev = 64;
    static std::mutex mu;
    static int32_t cache[kMaxDev][2][2];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) dev = -1;
    const int di = dt == kBF16 ? 1 : 0, bi = build ? 1 : 0;
    if (dev >= 0) {
        std::lock_guard<std::mutex> lock(mu);
        if (cache[dev][di][bi]) return cache[dev][di][bi];
    }
    const void *fn;
    if (build) fn = dt == kBF16 ? reinterpret_cast<const void *>(&k_head_gemm_loop<kBF16, kRingDeep, kListArgmax>)
                                : reinterpret_cast<const void *>(&k_head_gemm_loop<kF32, kRingDeep, kListArgmax>);
    else fn = dt == kBF16 ? reinterpret_cast<const void *>(&k_head_gemm_loop<kBF16, kRingDeep, kListRead>)
                          : reinterpret_cast<const void *>(&k_head_gemm_loop<kF32, kRingDeep, kListRead>);
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kGemmThreads, 0) != hipSuccess || per_cu < 1)
        per_cu = 1;
    if (dev < 0 || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 256;
    const int32_t r = per_cu * cus;
    if (dev >= 0) {
        std::lock_guard<std::mutex> lock(mu);
        cache[dev][di][bi] = r;
    }
    return r;
}

hipError_t launch_head_gemm(Dtype dt, const HeadArgs &a, hipStream_t s) {
    const dim3 block(kGemmThreads);
    if (a.grid > 0) {                                   // persistent (chains)
        if (a.build_list && a.m_cap > kBuildListMax) return hipErrorInvalidValue;
        if (!a.count_dev || !a.out_by_slot || (!a.build_list && !a.list)) return hipErrorInvalidValue;
        const dim3 grid(static_cast<unsigned>(a.grid));
        const int mode = !a.build_list ? kListRead : a.cand ? kListCand : kListArgmax;
        if (dt == kBF16) {
            if (mode == kListArgmax) hipLaunchKernelGGL((k_head_gemm_loop<kBF16, kRingDeep, kListArgmax>), grid, block, 0, s, a);
            else if (mode == kListCand) hipLaunchKernelGGL((k_head_gemm_loop<kBF16, kRingDeep, kListCand>), grid, block, 0, s, a);
            else hipLaunchKernelGGL((k_head_gemm_loop<kBF16, kRingDeep, kListRead>), grid, block, 0, s, a);
        } else {
            if (mode == kListArgmax) hipLaunchKernelGGL((k_head_gemm_loop<kF32, kRingDeep, kListArgmax>), grid, block, 0, s, a);
            else if (mode == kListCand) hipLaunchKernelGGL((k_head_gemm_loop<kF32, kRingDeep, kListCand>), grid, block, 0, s, a);
            else hipLaunchKernelGGL((k_head_gemm_loop<kF32, kRingDeep, kListRead>), grid, block, 0, s, a);
        }
        return hipGetLastError();
    }
    const int64_t tiles = ((a.m_cap + kHeadTileM - 1) / kHeadTileM) * ((a.h + kHeadTileN - 1) / kHeadTileN);
    const dim3 grid(static_cast<unsigned>(tiles * a.ksplit));
    if (grid.x == 0) return hipSuccess;
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
