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
// The MFMA step and its operand layout are in mfma.h.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "head_z.h"
#include "launch.h"
#include "mfma.h"
#include "rowstat.h"
#include "slot_gemm.h"

namespace cospec {
namespace {

typedef __attribute__((address_space(3))) char lds_char;

// Sixteen zero bytes in device memory: the operand loads past the end of d read them.
__device__ __attribute__((aligned(16))) const uint32_t kZeroVec[4] = {0, 0, 0, 0};

// Loads 16 bytes per lane from global memory straight into LDS, lane l's at byte
// lds + 16*l (lds is the wave's base, the same in every lane).  Written as assembly:
// the compiler cannot tell the ring slots apart, and for its own form of this load it
// makes every later LDS read wait until the load has landed, which would stall each
// stage for a full memory round trip.  The GEMM's own vmcnt waits order these loads.
// M0 is declared clobbered; the compiler reserves it and nothing else in this file's
// kernels uses it (their assembly sets M0 only here), so no value of its is lost.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ inline void load_lds16(const void *g, const char *lds) {
    const uint32_t base =
        __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_char *)lds)));
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 :
                 : "s"(base), "v"(g)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

constexpr int kStageBytes = 128;                  // bytes of k per row per stage
// LDS ring depth: four stages (three in flight while one is used, 128 KiB: one
// workgroup per CU), or two (64 KiB: two workgroups per CU) when the grid has more
// workgroups than there are CUs.
constexpr int kRingDeep = 4;
constexpr int kRingShallow = 2;
constexpr int kWaveTile = 64;                    // rows of a wave's sub-tile
constexpr int kWaveCols = 32;                    // columns of a wave's sub-tile
constexpr int kGemmWaves = 8;                    // 2 x 4 waves per workgroup: two per SIMD

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

// Part 1 of build_list, rows of one split (or candidates already taken): NB slots per
// thread, slot base + j * kGemmThreads + tid, every load issued before the first use,
// unconditionally (slots past the end read slot 0 and are dropped).
template <bool CAND, int NB>
__device__ inline void mark_single(const HeadArgs &a, int base, int n, uint64_t kmag, uint8_t *s_need) {
    const int tid = threadIdx.x;
    int tok[NB], r[NB], cand[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int i = base + j * kGemmThreads + tid;
        const int di = i < n ? i : 0;
        r[j] = di + static_cast<int>((static_cast<uint64_t>(di) * kmag) >> 32);   // b*(K+1) + i
    }
    if constexpr (CAND) {
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int i = base + j * kGemmThreads + tid;
            tok[j] = a.tokens[i < n ? i : 0];
            cand[j] = a.cand[r[j]];
        }
    } else {
        u32x4 q[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int i = base + j * kGemmThreads + tid;
            q[j] = *reinterpret_cast<const u32x4 *>(a.partials + r[j]);
            tok[j] = a.tokens[i < n ? i : 0];
        }
        // the single partial's argmax when S > 0, as merge_row takes it
#pragma unroll
        for (int j = 0; j < NB; ++j) cand[j] = __uint_as_float(q[j].z) > 0.f ? static_cast<int>(q[j].y) : INT_MAX;
        // the loads' unused words stay live until here, so their registers are not
        // reused (which would make the first load wait before the others)
#pragma unroll
        for (int j = 0; j < NB; ++j) asm volatile("" ::"v"(q[j].x), "v"(q[j].w));
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int i = base + j * kGemmThreads + tid;
        if (i < n) s_need[i] = tok[j] >= 0 && tok[j] < a.V && tok[j] != cand[j];
    }
}

// Part 1 of build_list, split rows: NS slots per thread, each merged by its thread in
// split order, CH partials of every slot loaded at once; the argmax is the one
// merge_row takes (the first split with S > 0 and the strictly largest maximum).
template <int NS, int CH>
__device__ inline void mark_split(const HeadArgs &a, int base, int n, int splits, uint64_t kmag, uint8_t *s_need) {
    const int tid = threadIdx.x;
    int tok[NS], r[NS], arg[NS];
    float M[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) {
        const int i = base + j * kGemmThreads + tid;
        const int di = i < n ? i : 0;
        r[j] = di + static_cast<int>((static_cast<uint64_t>(di) * kmag) >> 32);
        tok[j] = a.tokens[di];
        M[j] = -INFINITY;
        arg[j] = INT_MAX;
    }
    for (int s0 = 0; s0 < splits; s0 += CH) {       // uniform trip count
        u32x4 q[NS][CH];
#pragma unroll
        for (int j = 0; j < NS; ++j)
#pragma unroll
            for (int k = 0; k < CH; ++k)
                q[j][k] = *reinterpret_cast<const u32x4 *>(a.partials + (r[j] * splits + min(s0 + k, splits - 1)));
#pragma unroll
        for (int j = 0; j < NS; ++j)
#pragma unroll
            for (int k = 0; k < CH; ++k) {
                const float x = __uint_as_float(q[j][k].x);
                const bool take = (s0 + k < splits) & (__uint_as_float(q[j][k].z) > 0.f) & (x > M[j]);
                M[j] = take ? x : M[j];
                arg[j] = take ? static_cast<int>(q[j][k].y) : arg[j];
            }
#pragma unroll
        for (int j = 0; j < NS; ++j)
#pragma unroll
            for (int k = 0; k < CH; ++k) asm volatile("" ::"v"(q[j][k].w));
    }
#pragma unroll
    for (int j = 0; j < NS; ++j) {
        const int i = base + j * kGemmThreads + tid;
        if (i < n) s_need[i] = tok[j] >= 0 && tok[j] < a.V && tok[j] != arg[j];
    }
}

// The head's list for a chain step, derived by the workgroup from the reduction's
// partials (the decision step of Section 3.1 for the rows that need the head): slot
// di = b*K + i is a mismatch when its draft token is valid and differs from the
// candidate of target row b*(K+1) + i, which is the argmax of the row's partials, or
// the candidate already taken (a.cand).  Writes the list (kBuildListMax entries of
// LDS) and returns M, the number of mismatches.
//
// Part 1 marks the mismatches in LDS, one thread per slot (several slots per thread
// when there are more than threads), every load of a batch issued before the first
// is used.  Part 2 numbers the mismatches in slot order: thread t owns slots
// [kBuildPer*t, kBuildPer*(t+1)), a workgroup-wide exclusive scan gives their
// positions.
template <bool CAND>
__device__ inline int64_t build_list(const HeadArgs &a, int32_t *list) {
    __shared__ int s_wave[kGemmWaves];
    uint8_t *s_need = reinterpret_cast<uint8_t *>(list);   // part 1's flags: read before part 2 writes
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = static_cast<int>(a.m_cap);
    const int splits = CAND ? 1 : a.plan.splits;
    // floor(di / K) = (di * kmag) >> 32 with kmag = ceil(2^32 / K), exact for every
    // di < 2^16 and K <= 64 (here di < kBuildListMax)
    const uint64_t kmag = ((uint64_t{1} << 32) + static_cast<uint64_t>(a.K) - 1) / static_cast<uint64_t>(a.K);
    if (splits == 1) {
        if (n <= 4 * kGemmThreads) mark_single<CAND, 4>(a, 0, n, kmag, s_need);
        else mark_single<CAND, 8>(a, 0, n, kmag, s_need);          // n <= kBuildListMax
    } else if (n <= kGemmThreads) {
        mark_split<1, 16>(a, 0, n, splits, kmag, s_need);          // one round trip to 16 splits
    } else {
        for (int base = 0; base < n; base += 2 * kGemmThreads)      // uniform trip count
            mark_split<2, 8>(a, base, n, splits, kmag, s_need);
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
    // Branch-free: a lane past the ragged end of d (d is a multiple of VE) loads the zero
    // vector instead, so a stage's loads are one straight run of instructions.
    auto issue = [&](int st) {
        char *slot = ring[st % kRing];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int e = k0 + st * BK + lvec[i] * VE;          // first element of the vector
            char *la = slot + (wave * 2 + i) * 1024;
            char *lb = slot + kHeadTileM * kStageBytes + (wave * 2 + i) * 1024;
            const bool in = e < k1;
            const char *pa = in ? ga[i] + static_cast<int64_t>(e) * EB : reinterpret_cast<const char *>(kZeroVec);
            const char *pb = in ? gb[i] + static_cast<int64_t>(e) * EB : reinterpret_cast<const char *>(kZeroVec);
            load_lds16(pa, la);
            load_lds16(pb, lb);
        }
    };

    floatx4 acc[4][2];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 2; ++c) acc[r][c] = floatx4{0.f, 0.f, 0.f, 0.f};

    // Fragments of one 64-byte k-step q of stage st: this wave's 4 row tiles of A and 2
    // column tiles of B.
    auto read_frags = [&](int st, int q, u32x4 (&av)[4], u32x4 (&bv)[2]) {
        const char *sa = ring[st % kRing];
        const char *sb = sa + kHeadTileM * kStageBytes;
        const int kk = 4 * q;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = wr * kWaveTile + r * 16 + l16;
            av[r] = *reinterpret_cast<const u32x4 *>(sa + row * kStageBytes + (((kk + g) ^ (row & 7)) * 16));
        }
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int row = wc * kWaveCols + c * 16 + l16;
            bv[c] = *reinterpret_cast<const u32x4 *>(sb + row * kStageBytes + (((kk + g) ^ (row & 7)) * 16));
        }
    };
    auto products = [&](const u32x4 (&av)[4], const u32x4 (&bv)[2]) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int c = 0; c < 2; ++c) acc[r][c] = mma<DT>(av[r], bv[c], acc[r][c]);
    };
    static_assert(kStageBytes == 128, "two 64-byte k-steps per stage");

    // Software pipeline: the fragments of the next k-step are read from LDS while the
    // products of the current one run (the second k-step of a stage during the first's
    // products, the first of the next stage during the second's).  A slot is refilled
    // as soon as every wave has read the stage in it, so all kRing slots are in flight.
    u32x4 a0[4], b0[2], a1[4], b1[2];
#pragma unroll
    for (int st = 0; st < kRing; ++st)
        if (st < nst) issue(st);
    if (nst > 0) {
        wait_later<4, kRing - 1>(min(kRing - 1, nst - 1));     // 4 loads per wave and stage
        lds_barrier();                                          // stage 0 has landed
        read_frags(0, 0, a0, b0);
    }
    int st = 0;
    // steady state, one basic block: every stage after the next is in flight and the
    // refill always happens; the loads, LDS reads and products are interleaved so that
    // a wave's products run while its loads wait to be accepted
    for (; st + kRing < nst; ++st) {
        read_frags(st, 1, a1, b1);
        products(a0, b0);
#pragma unroll
        for (int j = 0; j < 6; ++j) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one product
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        wait_vm<4 * (kRing - 2)>();                             // stage st+1 landed here
        lds_barrier();                                          // ... and everywhere
        issue(st + kRing);
        read_frags(st + 1, 0, a0, b0);
        products(a1, b1);
        // per load: one or two LDS reads, two products
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    }
    for (; st < nst; ++st) {                                    // the last kRing stages
        read_frags(st, 1, a1, b1);
        __builtin_amdgcn_sched_barrier(0);
        products(a0, b0);
        if (st + 1 < nst) {
            // this wave's loads of stage st+1 are done once at most the later stages'
            // remain; the barrier's LDS wait also completes this wave's reads of stage st
            wait_later<4, kRing - 2>(min(kRing - 2, nst - 2 - st));
            lds_barrier();                        // stage st+1 landed, stage st read by all
            read_frags(st + 1, 0, a0, b0);
        }
        __builtin_amdgcn_sched_barrier(0);
        products(a1, b1);
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

// The slot GEMM (slot_gemm.h) on its own, for the second phase of a split chain step
// (whose hidden states arrive after the reduction): the same work and the same
// partials as in the whole step's reduction launch, so both give the same z.
template <int DT>
__global__ __launch_bounds__(kReduceThreads) void k_slot_gemm(HeadArgs a) {
    slotgemm::run<DT>(a, blockIdx.x, reinterpret_cast<const u32x4 *>(kZeroVec));
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

hipError_t launch_slot_gemm(Dtype dt, const HeadArgs &a, hipStream_t s) {
    if (a.m_cap <= 0 || a.m_cap > slotgemm::kMaxSlots || a.ksplit < 1) return hipErrorInvalidValue;
    const int64_t blocks = slotgemm::blocks(a);
    if (blocks > INT32_MAX) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(blocks));
    if (dt == kBF16) hipLaunchKernelGGL(k_slot_gemm<kBF16>, grid, dim3(kReduceThreads), 0, s, a);
    else hipLaunchKernelGGL(k_slot_gemm<kF32>, grid, dim3(kReduceThreads), 0, s, a);
    return hipGetLastError();
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
