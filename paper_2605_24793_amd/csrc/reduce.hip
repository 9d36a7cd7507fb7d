// Vocabulary reductions and the per-sequence decision step.
//
// k_vocab_reduce streams every logit row once (the step's HBM traffic) and
// produces, per (row, split), the partial statistics the softmax quantities
// need: the max, the first index of the max, S = sum 2^(x*log2e - R) and
// T = sum 2^(x*log2e - R) * (x*log2e - R) with R = max*log2e.  From the merged
// (max, S, T) of a whole row:  lse = max + ln2 * log2(S) and the entropy is
// H = ln2 * (log2(S) - T/S) (Shannon entropy of softmax(x) in nats).  The
// running form with a per-lane reference is the one-pass online normaliser of
// Milakov & Gimelshein (2018, "Online normalizer calculation for softmax"),
// extended with the first moment T; the reference is only raised when a chunk
// max exceeds it by more than 2^32, so the rescale is almost never taken.
// One launch covers every target and draft row, one workgroup per (row, split);
// tree draft rows of nodes without a child are skipped.
//
// The decide step (decide_seq) merges the partials of one sequence's target rows
// in fixed split order, takes the target's verification candidates (the greedy
// argmax, ties to the lowest index, or the temperature-1 samples of k_sample), sets
// Delta = 1[draft token == candidate] (Section 3.1), gathers the draft token's target
// logit for log p_T (Section 3.4), and compacts the mismatch decisions into one
// list for the head with a wave ballot and a prefix over the workgroup's waves; it
// runs as k_decide, one workgroup per sequence, after the reduction.  (Run inside the
// reduction instead, by the workgroup that completes a sequence's target rows, it was
// measured slower: its memory round trips, queued behind the streaming loads of every
// other workgroup, took several microseconds each.)
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "launch.h"
#include "rowstat.h"
#include "slot_gemm.h"

// Products and sums are rounded as written in this file: the references (x * log2e
// rounded) must be the same numbers in every kernel that forms them, so no
// multiply-add may be fused unless written as fmaf.
#pragma clang fp contract(off)

namespace cospec {
namespace {

constexpr float kRescaleMargin = 32.0f;   // log2 units of headroom above the reference
constexpr float kFarBelow = -1.0e30f;     // initial reference: any finite logit rescales
constexpr int kUnroll = 8;                // 16-byte loads in flight per lane

// Word 3 of a raw (unswizzled, stride 0) buffer resource: 32-bit data format.
constexpr int kRawBuffer = 0x00020000;
constexpr int kNontemporal = 2;           // cache policy of the loads: streamed once

// The whole 16-byte vectors of one logit row, read through a raw buffer resource: a
// load takes the lane's byte offset in a VGPR and a per-load constant in the scalar
// offset, so it costs no vector address arithmetic.
struct RowReader {
    __amdgpu_buffer_rsrc_t rs;
    __device__ RowReader(const void *row, int bytes)
        : rs(__builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(row), 0, bytes, kRawBuffer)) {}
    __device__ u32x4 load(int voff, int soff) const {
        return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, soff, kNontemporal));
    }
};

typedef __attribute__((address_space(3))) float lds_fw;
constexpr int kSegStage = 1024;           // segments of one split staged in LDS

struct Lane {
    float best;      // largest logit seen
    int chunk;       // first chunk (16-byte vector index) holding `best`, -1 if none
    float nref;      // minus the reference of S and T (log2 units): the exponent of a
                     // logit x is fma(x, log2e, nref)
    float thresh;    // logits above this need a larger reference: (ref + margin) / log2e
    float S, T;
};

__device__ inline void rescale(Lane &st, float new_ref) {
    const float dr = -st.nref - new_ref;          // <= 0, finite
    const float f = __builtin_amdgcn_exp2f(dr);
    st.T = f * fmaf(dr, st.S, st.T);
    st.S = f * st.S;
    st.nref = -new_ref;
    st.thresh = (new_ref + kRescaleMargin) * kLn2;
}

template <int NV>
__device__ inline void consume(const float *x, int chunk, Lane &st) {
    float cm = -INFINITY;
#pragma unroll
    for (int k = 0; k < NV; ++k) cm = fmaxf(cm, x[k]);
    if (cm > st.best) { st.best = cm; st.chunk = chunk; }
    // wave-uniform branch: after the first chunk almost no lane ever takes it.  The
    // test is in the logit domain; the threshold is conservative by its rounding,
    // which only makes a rescale slightly more likely.
    const bool up = cm > st.thresh;
    if (__builtin_expect(__ballot(up) != 0, 0)) {
        if (up) rescale(st, __fmul_rn(cm, kLog2e));
    }
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const float t = fmaf(x[k], kLog2e, st.nref);
        const float e = __builtin_amdgcn_exp2f(t);
        st.S += e;
        st.T = fmaf(e, t, st.T);
    }
}

// Lane exchanges that stay in the VALU (no LDS round trip): DPP patterns inside
// rows of 16 lanes and the gfx950 permlane swaps across rows.
constexpr int kDppXor1 = 0xB1;    // quad_perm [1,0,3,2]: lane i <-> i ^ 1
constexpr int kDppXor2 = 0x4E;    // quad_perm [2,3,0,1]: i <-> i ^ 2
constexpr int kDppXor7 = 0x141;   // row_half_mirror:     i <-> i ^ 7 within 8 lanes
constexpr int kDppXor15 = 0x140;  // row_mirror:          i <-> i ^ 15 within 16 lanes
constexpr int kDppXor8 = 0x128;   // row_ror:8:           i <-> i ^ 8 within 16 lanes

template <int CTRL>
__device__ inline float dpp(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}

// permlane32_swap(x, y): lanes 0..31 of the results hold (x[l], x[l + 32]), lanes
// 32..63 hold (y[l - 32], y[l]); permlane16_swap does the same between the even and
// odd rows of 16 lanes.  Their sum pairs lane l with l ^ 32 (or l ^ 16), taking x in
// the lower and y in the upper half.
__device__ inline float swap32_sum(float x, float y) {
    const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(y), false, false);
    return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

__device__ inline float swap16_sum(float x, float y) {
    const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(y), false, false);
    return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

__device__ inline float wave_max_valu(float x) {
    x = fmaxf(x, dpp<kDppXor1>(x));
    x = fmaxf(x, dpp<kDppXor2>(x));
    x = fmaxf(x, dpp<kDppXor7>(x));
    x = fmaxf(x, dpp<kDppXor15>(x));
    const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
    const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}

// Eight per-lane values m[0..7] -> lane L returns the wave's sum of m[L >> 3].
// Each exchange halves the values a lane carries (lane bits 5, 4, 3), then the
// eight lanes that share bits 3..5 add up (bits 0..2): 7 exchanges + 3 DPP adds.
__device__ inline float transpose_sum8(const float (&m)[8], int lane) {
    float r4[4], r2[2];
#pragma unroll
    for (int j = 0; j < 4; ++j) r4[j] = swap32_sum(m[j], m[j + 4]);     // value j + 4 * bit5
#pragma unroll
    for (int j = 0; j < 2; ++j) r2[j] = swap16_sum(r4[j], r4[j + 2]);   // j + 2 * bit4 + 4 * bit5
    const bool b3 = lane & 8;
    const float send = b3 ? r2[0] : r2[1];
    float r = (b3 ? r2[1] : r2[0]) + dpp<kDppXor8>(send);              // bit3 + 2 * bit4 + 4 * bit5
    r += dpp<kDppXor1>(r);
    r += dpp<kDppXor2>(r);
    r += dpp<kDppXor7>(r);
    return r;
}

// Plain streaming of vectors [v0, v1) of a row: lane `tid` takes v0 + tid, then
// every kReduceThreads-th vector.  Loads roll: while whole batches remain, each
// register slot is refilled with the vector kUnroll steps ahead as soon as it is
// unpacked, so a lane keeps kUnroll loads in flight through the row.
template <int DT>
__device__ inline void stream_plain(const RowReader &rr, int v0, int v1, int tid, Lane &st) {
    using E = Elt<DT>;
    constexpr int NV = E::kPerVec;
    constexpr int T = kReduceThreads;
    constexpr int kStep = kUnroll * T;
    int v = v0 + tid;
    if (v + (kUnroll - 1) * T < v1) {
        u32x4 q[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) q[u] = rr.load(v * 16, u * T * 16);
        for (; v + kStep + (kUnroll - 1) * T < v1; v += kStep) {
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                float x[NV];
                E::unpack(q[u], x);
                q[u] = rr.load(v * 16, (kStep + u * T) * 16);
                consume<NV>(x, v + u * T, st);
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            float x[NV];
            E::unpack(q[u], x);
            consume<NV>(x, v + u * T, st);
        }
        v += kStep;
    }
    // the rest: at most kUnroll - 1 vectors per lane, every load issued before the
    // first is used (one memory round trip, not one per vector)
    u32x4 q[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
        if (v + u * T < v1) q[u] = rr.load(v * 16, u * T * 16);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        if (v + u * T < v1) {
            float x[NV];
            E::unpack(q[u], x);
            consume<NV>(x, v + u * T, st);
        }
    }
}

// Wave-wide rescale to the reference of the wave's largest chunk max; returns the
// factor applied to S.
__device__ inline float rescale_wave(Lane &st, float cm) {
    const float nr = __fmul_rn(wave_max_valu(cm), kLog2e);
    const float dr = -st.nref - nr;
    const float f = __builtin_amdgcn_exp2f(dr);
    st.T = f * fmaf(dr, st.S, st.T);
    st.S = f * st.S;
    st.nref = -nr;
    st.thresh = (nr + kRescaleMargin) * kLn2;
    return f;
}

// The same streaming, for rows that are sampled at temperature 1: it also writes
// the probability mass of every segment of kSegVecs vectors (one wave load, so the
// segments of a row are contiguous and in vocabulary order) as {sum 2^(x*log2e -
// ref), ref}.  Every lane of a wave shares one reference, raised for the whole
// wave when any lane needs it, so a segment's mass is one wave sum.  Requires v0 to
// be a multiple of kSegVecs.
template <int DT>
__device__ inline void stream_segmented(const RowReader &rr, int v0, int v1, int tid, Lane &st, float2 *seg,
                                        lds_fw *sst, int sbase, bool staged) {
    using E = Elt<DT>;
    constexpr int NV = E::kPerVec;
    // a segment's (mass, reference): into the workgroup's LDS stage when the split's
    // segments fit it (LDS writes do not share the vector-memory counter with the
    // rolling loads, so the loads never wait behind a store), else straight to memory
    auto put = [&](int i, float mass) {
        if (staged) {
            sst[2 * (i - sbase)] = mass;
            sst[2 * (i - sbase) + 1] = -st.nref;
        } else {
            seg[i] = make_float2(mass, -st.nref);
        }
    };
    static_assert(kUnroll == 8 && kReduceThreads % kSegVecs == 0, "segment sums assume 8 loads per lane");
    constexpr int kStep = kUnroll * kReduceThreads;
    const int lane = tid & 63;
    int w = v0 + (tid & ~63);                      // this wave's first vector
    // one batch: kUnroll whole segments of this wave; with RELOAD each slot is refilled
    // from the next batch as soon as it is unpacked (loads roll, as in stream_plain)
    auto batch = [&](u32x4 (&q)[kUnroll], auto reload) {
        float m[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            float x[NV];
            E::unpack(q[u], x);
            if constexpr (decltype(reload)::value) q[u] = rr.load((w + lane) * 16, (kStep + u * kReduceThreads) * 16);
            float cm = -INFINITY;
#pragma unroll
            for (int k = 0; k < NV; ++k) cm = fmaxf(cm, x[k]);
            if (cm > st.best) { st.best = cm; st.chunk = w + u * kReduceThreads + lane; }
            if (__builtin_expect(__ballot(cm > st.thresh) != 0, 0)) {
                const float f = rescale_wave(st, cm);
#pragma unroll
                for (int j = 0; j < u; ++j) m[j] *= f;
            }
            const float nref = st.nref;
            float mu = 0.f;
#pragma unroll
            for (int k = 0; k < NV; ++k) {
                const float t = fmaf(x[k], kLog2e, nref);
                const float e = __builtin_amdgcn_exp2f(t);
                mu += e;
                st.T = fmaf(e, t, st.T);
            }
            m[u] = mu;
            st.S += mu;
        }
        const float tot = transpose_sum8(m, lane);
        if ((lane & 7) == 0) put((w + (lane >> 3) * kReduceThreads) / kSegVecs, tot);
    };
    if (w + (kUnroll - 1) * kReduceThreads + 63 < v1) {   // wave-uniform: a whole batch
        u32x4 q[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) q[u] = rr.load((w + lane) * 16, u * kReduceThreads * 16);
        for (; w + kStep + (kUnroll - 1) * kReduceThreads + 63 < v1; w += kStep)
            batch(q, std::true_type{});
        batch(q, std::false_type{});
        w += kStep;
    }
    // the rest: fewer than kUnroll segments of this wave, the last one possibly
    // partial; every load is issued before the first is used
    if (w < v1) {
        u32x4 q[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (w + u * kReduceThreads + lane < v1) q[u] = rr.load((w + lane) * 16, u * kReduceThreads * 16);
        float m[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            m[u] = 0.f;
            if (w + u * kReduceThreads >= v1) continue;            // wave-uniform: no such segment
            const int vi = w + u * kReduceThreads + lane;
            const bool ok = vi < v1;
            float x[NV];
            if (ok) {
                E::unpack(q[u], x);
            } else {
#pragma unroll
                for (int k = 0; k < NV; ++k) x[k] = -INFINITY;
            }
            float cm = -INFINITY;
#pragma unroll
            for (int k = 0; k < NV; ++k) cm = fmaxf(cm, x[k]);
            if (cm > st.best) { st.best = cm; st.chunk = vi; }
            if (__ballot(cm > st.thresh) != 0) {
                const float f = rescale_wave(st, cm);
#pragma unroll
                for (int j = 0; j < u; ++j) m[j] *= f;
            }
            const float nref = st.nref;
            float mu = 0.f;
#pragma unroll
            for (int k = 0; k < NV; ++k) {
                // lanes past the end add exp2(-huge) = 0 and 0 * (finite t) = 0
                const float t = fmaf(ok ? x[k] : kFarBelow, kLog2e, nref);
                const float e = __builtin_amdgcn_exp2f(t);
                mu += e;
                st.T = fmaf(e, t, st.T);
            }
            m[u] = mu;
            st.S += mu;
        }
        const float tot = transpose_sum8(m, lane);
        const int ws = w + (lane >> 3) * kReduceThreads;           // segment of value lane >> 3
        if ((lane & 7) == 0 && ws < v1) put(ws / kSegVecs, tot);
    }
}

static_assert(kReduceThreads >= kMaxSeqRows, "a tree node's children are found by one thread each");

// Reduces 16-byte vectors [v0, v1) of row `row`, plus the row's elements past its last
// whole vector when `with_tail`.  Every thread of the workgroup takes part; thread 0
// returns the piece's partial {max, first index of the max, S, T}.
template <int DT, bool SEG>
__device__ __forceinline__ float4 reduce_piece(const ReduceArgs &a, int row, int v0, int v1, bool with_tail) {
    using E = Elt<DT>;
    constexpr int NV = E::kPerVec;
    const int tid = threadIdx.x;
    const char *rp = row < a.n_tgt_rows ? a.tgt + static_cast<int64_t>(row) * a.ld_bytes
                                        : a.drf + static_cast<int64_t>(row - a.n_tgt_rows) * a.ld_bytes;
    const int nvec = static_cast<int>((static_cast<int64_t>(a.V) * E::kBytes) / 16);
    const int tail = a.V - nvec * NV;
    const u32x4 *rv = reinterpret_cast<const u32x4 *>(rp);

    Lane st{-INFINITY, -1, -kFarBelow, -INFINITY, 0.f, 0.f};   // the first chunk always rescales
    float2 *seg = nullptr;
    if (SEG && row < a.n_tgt_rows) seg = a.seg + static_cast<int64_t>(row) * a.nseg;
    const RowReader rr(rp, nvec * 16);
    __shared__ float s_seg[SEG ? 2 * kSegStage : 1];
    const int sbase = v0 / kSegVecs;
    const int nsg = v1 > v0 ? (v1 - v0 + kSegVecs - 1) / kSegVecs : 0;
    const bool staged = nsg <= kSegStage;
    if (SEG && seg) stream_segmented<DT>(rr, v0, v1, tid, st, seg, (lds_fw *)s_seg, sbase, staged);
    else stream_plain<DT>(rr, v0, v1, tid, st);
    // elements past the last whole vector: the first lane of the piece that ends the
    // row (their own segment, the row's last, when segments are written)
    if (tail > 0 && with_tail && tid == 0) {
        const int64_t e0 = static_cast<int64_t>(nvec) * NV;
        float cm = -INFINITY;
        for (int k = 0; k < tail; ++k) cm = fmaxf(cm, E::at(rp, e0 + k));
        if (cm > st.best) { st.best = cm; st.chunk = nvec; }
        if (cm > st.thresh) rescale(st, __fmul_rn(cm, kLog2e));
        float mu = 0.f;
        for (int k = 0; k < tail; ++k) {
            const float t = fmaf(E::at(rp, e0 + k), kLog2e, st.nref);
            const float e = __builtin_amdgcn_exp2f(t);
            mu += e;
            st.T = fmaf(e, t, st.T);
        }
        st.S += mu;
        if (SEG && seg) seg[a.nseg - 1] = make_float2(mu, -st.nref);
    }

    __shared__ float s_best[kReduceThreads / 64];
    __shared__ int s_idx[kReduceThreads / 64];
    __shared__ float s_S[kReduceThreads / 64], s_T[kReduceThreads / 64];
    __shared__ float s_M;
    const int lane = tid & 63, wave = tid >> 6;

    // the workgroup's max, then its first index: only lanes that hold the max look
    // again at the first chunk where they saw it (one 16-byte load, usually one lane)
    float bv = st.best;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) bv = fmaxf(bv, __shfl_xor(bv, off));
    if (lane == 0) s_best[wave] = bv;
    __syncthreads();
    if (tid == 0) {
        float M = s_best[0];
        for (int w = 1; w < kReduceThreads / 64; ++w) M = fmaxf(M, s_best[w]);
        s_M = M;
    }
    __syncthreads();
    int idx = INT_MAX;
    if (st.chunk >= 0 && st.best == s_M) {
        const int64_t e0 = static_cast<int64_t>(st.chunk) * NV;
        float x[NV];
        if (st.chunk < nvec) {
            E::unpack(__builtin_nontemporal_load(rv + st.chunk), x);
        } else {
#pragma unroll
            for (int k = 0; k < NV; ++k) x[k] = e0 + k < a.V ? E::at(rp, e0 + k) : -INFINITY;
        }
#pragma unroll
        for (int k = NV - 1; k >= 0; --k)
            if (e0 + k < a.V && x[k] == st.best) idx = static_cast<int>(e0 + k);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) idx = min(idx, __shfl_xor(idx, off));
    if (lane == 0) s_idx[wave] = idx;
    __syncthreads();
    if (tid == 0) {
        int I = s_idx[0];
        for (int w = 1; w < kReduceThreads / 64; ++w) I = min(I, s_idx[w]);
        s_idx[0] = I;
    }
    const float M = s_M;
    const float R = __fmul_rn(M, kLog2e);   // the partial's reference: rounded, never contracted
    float S = 0.f, T = 0.f;
    if (st.S > 0.f) {
        const float dr = -st.nref - R;
        const float f = __builtin_amdgcn_exp2f(dr);
        S = f * st.S;
        T = f * fmaf(dr, st.S, st.T);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        S += __shfl_xor(S, off);
        T += __shfl_xor(T, off);
    }
    if (lane == 0) { s_S[wave] = S; s_T[wave] = T; }
    __syncthreads();
    float4 part = make_float4(0.f, 0.f, 0.f, 0.f);
    if (tid == 0) {
        float SS = s_S[0], TT = s_T[0];
        for (int w = 1; w < kReduceThreads / 64; ++w) { SS += s_S[w]; TT += s_T[w]; }
        part = make_float4(M, __int_as_float(s_idx[0]), SS, TT);
    }
    // the staged segment masses, complete since every wave passed the barriers above;
    // nontemporal stores, so that no dirty line waits in L2 for the kernel-end write-back
    // (the large chain batch's temperature-1 step 231.5 -> 226.0 us, the trees' 335.7 ->
    // 323.8 us)
    if (SEG && seg && staged)
        for (int i = tid; i < nsg; i += kReduceThreads) {
            __builtin_nontemporal_store(s_seg[2 * i], &seg[sbase + i].x);
            __builtin_nontemporal_store(s_seg[2 * i + 1], &seg[sbase + i].y);
        }
    return part;
}

// One sequence's (or tree's) decision step, by one workgroup of kDecideThreads:
// merges the partials of its target rows in fixed split order, takes the
// verification candidates (the greedy argmax, ties to the lowest index, or the
// temperature-1 samples k_sample left), sets Delta = 1[draft token == candidate]
// (Section 3.1), gathers the draft token's target logit for log p_T (Section 3.4), and
// compacts the mismatch decisions into the head's list with a wave ballot and a
// prefix over the workgroup's waves (one atomic addition per sequence).
template <int DT>
__device__ __forceinline__ void decide_seq(const DecideArgs &a, int b) {
    using E = Elt<DT>;
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    // per row: max and ln S, so that log p(token) = (x - max) - ln S keeps full
    // precision even when |lse| is large
    __shared__ float s_tmax[kMaxSeqRows], s_tlogs[kMaxSeqRows];
    __shared__ int s_targ[kMaxSeqRows];
    __shared__ int s_wave_cnt[kDecideThreads / 64];
    __shared__ int s_base;
    __shared__ float4 s_parts[kStageParts];

    // this thread's decision slot (D <= kDecideThreads): chain slot t is decision t+1,
    // verified by target row t; tree slot t is node t, verified by its parent's row.
    // Its token and the target logit at it are fetched while the partials merge.
    const int slot = t;
    const int64_t di = static_cast<int64_t>(b) * a.D + slot;
    const bool decides = slot < a.D && !(a.is_tree && slot == 0);
    int p = 0;
    bool valid = false;
    float xt = 0.f;
    if (decides) {
        p = a.is_tree ? a.parent[di] : slot;
        const int tok = a.tokens[di];
        valid = (!a.is_tree || (p >= 0 && p < slot)) && tok >= 0 && tok < a.V;
        if (valid) {
            xt = E::at(a.tgt + (static_cast<int64_t>(b) * a.RT + p) * a.ld_bytes, tok);
        }
    }
    // the sequence's target partials are consecutive slots: staged in LDS when there are
    // several per row (one memory round trip for all of them)
    const int64_t r0 = static_cast<int64_t>(b) * a.RT;
    const RowParts sp = rows_parts(a.plan, r0, r0 + a.RT);
    const float4 *seq_parts = a.partials + sp.first;
    const bool staged = sp.count > a.RT && sp.count <= kStageParts;
    if (staged) {
        stage_partials(seq_parts, sp.count, seq_parts, 0, s_parts, t, kDecideThreads);
        __syncthreads();
    }
    for (int j = t; j < a.RT; j += kDecideThreads) {
        const int64_t r = r0 + j;
        const RowParts rp = row_parts(a.plan, r);
        const int64_t off = rp.first - sp.first;
        const RowStat rs = staged ? merge_row_lds(s_parts + off, rp.count) : merge_row(seq_parts + off, rp.count);
        // the verification candidate: the argmax, or the temperature-1 sample
        // k_sample left in ws_tgt_arg
        const int cand = a.sampled ? a.ws_tgt_arg[r] : rs.arg;
        s_tmax[j] = rs.max;
        s_tlogs[j] = rs.log_s;
        s_targ[j] = cand;
        if (!a.sampled) a.ws_tgt_arg[r] = cand;
        if (a.tgt_cand) a.tgt_cand[r] = cand;
        if (a.tgt_argmax) a.tgt_argmax[r] = rs.arg;
        if (a.tgt_max) a.tgt_max[r] = rs.max;
        if (a.tgt_lse) a.tgt_lse[r] = rs.lse;
        if (a.tgt_ent) a.tgt_ent[r] = rs.ent;
    }
    __syncthreads();

    uint8_t state = kStateMatch;
    float lpt = NAN;
    if (decides) {
        if (valid) {
            state = a.tokens[di] == s_targ[p] ? kStateMatch : kStateMismatch;
            lpt = (xt - s_tmax[p]) - s_tlogs[p];
        } else {
            state = kStateReject;
        }
    }
    const bool need = decides && state == kStateMismatch && a.score_mismatch;
    const uint64_t m = __ballot(need);
    if (lane == 0) s_wave_cnt[wave] = __popcll(m);
    __syncthreads();
    if (t == 0) {
        int tot = 0;
        for (int w = 0; w < kDecideThreads / 64; ++w) { const int c = s_wave_cnt[w]; s_wave_cnt[w] = tot; tot += c; }
        s_base = tot ? atomicAdd(a.ws_count, tot) : 0;
    }
    __syncthreads();
    if (slot < a.D) {
        int pos = -1;
        if (need) {
            pos = s_base + s_wave_cnt[wave] + __popcll(m & ((1ull << lane) - 1ull));
            a.ws_list[pos] = static_cast<int>(di);          // hidden row of the decision
        }
        a.ws_listpos[di] = pos;
        a.ws_state[di] = state;
        if (a.delta) a.delta[di] = state == kStateMatch;
        if (a.logp_tgt) a.logp_tgt[di] = lpt;
        a.ws_logp_tgt[di] = lpt;
    }
}

// Units are (row, split) pairs, split fastest, one workgroup each.  Unit 0 also
// zeroes the decide step's list counter.
template <int DT, bool SEG>
__device__ __forceinline__ void reduce_unit(const ReduceArgs &a, int u) {
    if (u == 0 && threadIdx.x == 0 && a.reset_counter) *a.reset_counter = 0;
    using E = Elt<DT>;
    const int splits = a.plan.splits;
    const int row = u / splits, split = u - row * splits;
    if (row >= a.n_tgt_rows && a.parent) {   // tree: only nodes with a child need their draft row
        const int r = row - a.n_tgt_rows;
        const int b = r / a.N, n = r - b * a.N;
        const int m = n + 1 + threadIdx.x;   // every later node: N <= kMaxSeqRows <= kReduceThreads
        const bool child = m < a.N && a.parent[static_cast<int64_t>(b) * a.N + m] == n;
        if (!__syncthreads_or(child)) return;
    }
    const int nvec = static_cast<int>((static_cast<int64_t>(a.V) * E::kBytes) / 16);
    const int v0 = split * a.vec_per_split;
    const int v1 = min(v0 + a.vec_per_split, nvec);
    // chains: the row's logit at its draft token, read by the piece whose range holds
    // it (the tail past the last whole vector belongs to the last split); the read is
    // issued before the streaming and kept until its end
    bool own = false;
    float xt = 0.f;
    if (a.xtok && threadIdx.x == 0) {
        int tok = -1;
        const char *base;
        if (row < a.n_tgt_rows) {
            const int b = row / (a.K + 1), i = row - b * (a.K + 1);
            if (i < a.K) tok = a.chain_tokens[static_cast<int64_t>(b) * a.K + i];
            base = a.tgt + static_cast<int64_t>(row) * a.ld_bytes;
        } else {
            tok = a.chain_tokens[row - a.n_tgt_rows];
            base = a.drf + static_cast<int64_t>(row - a.n_tgt_rows) * a.ld_bytes;
        }
        if (tok >= 0 && tok < a.V) {
            const int tv = tok / E::kPerVec;
            own = tv < nvec ? (tv >= v0 && tv < v1) : split == splits - 1;
            if (own) xt = E::at(base, tok);
        }
    }
    const float4 part = reduce_piece<DT, SEG>(a, row, v0, v1, split == splits - 1);
    if (threadIdx.x == 0) {
        a.partials[u] = part;
        if (own) a.xtok[row] = xt;
    }
}

template <int DT, bool SEG>
__global__ __launch_bounds__(kReduceThreads) void k_vocab_reduce(ReduceArgs a) {
    reduce_unit<DT, SEG>(a, blockIdx.x);
}

// Sixteen zero bytes in device memory, loaded by the slot GEMM's lanes past the end of d.
__device__ __attribute__((aligned(16))) const u32x4 kZero16 = {0u, 0u, 0u, 0u};

// A small chain step's reduction launch with the head's first layer over every decision
// slot beside it (slot_gemm.h): the first `head_blocks` workgroups are the slot GEMM's,
// dispatched first so that they start at once; the rest are the reduction's units.
// The occupancy bound is k_vocab_reduce's own (eight waves per SIMD for bf16 rows
// without segments, six otherwise): left free, the compiler gives the reduction's code
// more registers here, and the launch fewer resident units.
template <int DT, bool SEG, int HD>
__global__ __launch_bounds__(kReduceThreads) __attribute__((amdgpu_waves_per_eu(DT == kBF16 && !SEG ? 8 : 6)))
void k_vocab_reduce_head(ReduceArgs a, HeadArgs h, int head_blocks) {
    if (static_cast<int>(blockIdx.x) < head_blocks) {
        slotgemm::run<HD>(h, blockIdx.x, &kZero16);
        return;
    }
    reduce_unit<DT, SEG>(a, blockIdx.x - head_blocks);
}

template <int DT>
__global__ __launch_bounds__(kDecideThreads) void k_decide(DecideArgs a) {
    decide_seq<DT>(a, blockIdx.x);
}

}  // namespace

template <int DT>
void launch_reduce_t(const ReduceArgs &a, dim3 grid, hipStream_t s) {
    if (a.seg) hipLaunchKernelGGL((k_vocab_reduce<DT, true>), grid, dim3(kReduceThreads), 0, s, a);
    else hipLaunchKernelGGL((k_vocab_reduce<DT, false>), grid, dim3(kReduceThreads), 0, s, a);
}

// Reduction workgroups resident at once on the current device (greedy variant of the
// dtype: eight per CU for bf16 on MI355X, 2048 in all); the split rule sizes the grid
// by it.  Looked up once per device and dtype.
int32_t reduce_slots(Dtype dt) {
    constexpr int kMaxDev = 64;
    static std::mutex mu;
    static int32_t cache[kMaxDev][2];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) dev = -1;
    const int di = dt == kBF16 ? 1 : 0;
    if (dev >= 0) {
        std::lock_guard<std::mutex> lock(mu);
        if (cache[dev][di]) return cache[dev][di];
    }
    const void *fn = dt == kBF16 ? reinterpret_cast<const void *>(&k_vocab_reduce<kBF16, false>)
                                 : reinterpret_cast<const void *>(&k_vocab_reduce<kF32, false>);
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kReduceThreads, 0) != hipSuccess || per_cu < 1)
        per_cu = 8;
    if (dev < 0 || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 256;
    const int64_t g = static_cast<int64_t>(per_cu) * cus;
    const int32_t r = static_cast<int32_t>(g < kMaxReduceSlots ? g : kMaxReduceSlots);
    if (dev >= 0) {
        std::lock_guard<std::mutex> lock(mu);
        cache[dev][di] = r;
    }
    return r;
}

hipError_t launch_reduce(Dtype dt, const ReduceArgs &a, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(static_cast<int64_t>(a.n_rows) * a.plan.splits));
    if (grid.x == 0) return hipSuccess;
    if (dt == kBF16) launch_reduce_t<kBF16>(a, grid, s);
    else launch_reduce_t<kF32>(a, grid, s);
    return hipGetLastError();
}

template <int DT, bool SEG>
void launch_reduce_head_t(Dtype hdt, const ReduceArgs &a, const HeadArgs &h, int head_blocks, dim3 grid,
                          hipStream_t s) {
    if (hdt == kBF16)
        hipLaunchKernelGGL((k_vocab_reduce_head<DT, SEG, kBF16>), grid, dim3(kReduceThreads), 0, s, a, h, head_blocks);
    else
        hipLaunchKernelGGL((k_vocab_reduce_head<DT, SEG, kF32>), grid, dim3(kReduceThreads), 0, s, a, h, head_blocks);
}

hipError_t launch_reduce_head(Dtype dt, Dtype hdt, const ReduceArgs &a, const HeadArgs &h, hipStream_t s) {
    if (h.m_cap <= 0 || h.m_cap > slotgemm::kMaxSlots || h.ksplit < 1) return hipErrorInvalidValue;
    const int64_t hb = slotgemm::blocks(h);
    const int64_t units = static_cast<int64_t>(a.n_rows) * a.plan.splits;
    if (hb + units > INT32_MAX) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(hb + units));
    const int hbi = static_cast<int>(hb);
    if (dt == kBF16) {
        if (a.seg) launch_reduce_head_t<kBF16, true>(hdt, a, h, hbi, grid, s);
        else launch_reduce_head_t<kBF16, false>(hdt, a, h, hbi, grid, s);
    } else {
        if (a.seg) launch_reduce_head_t<kF32, true>(hdt, a, h, hbi, grid, s);
        else launch_reduce_head_t<kF32, false>(hdt, a, h, hbi, grid, s);
    }
    return hipGetLastError();
}

hipError_t launch_decide(Dtype dt, const DecideArgs &a, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(a.B));
    if (dt == kBF16) hipLaunchKernelGGL(k_decide<kBF16>, grid, dim3(kDecideThreads), 0, s, a);
    else hipLaunchKernelGGL(k_decide<kF32>, grid, dim3(kDecideThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace cospec
