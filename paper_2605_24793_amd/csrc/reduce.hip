// Vocabulary reductions and per-sequence decisions.
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
//
// k_decide merges the partials of one sequence's rows in fixed split order,
// takes the target's greedy verification tokens (argmax, ties to the lowest
// index), sets Delta = 1[draft token == verification token] (Section 3.1),
// gathers the draft token's logits for log p_T and log p_D (Section 3.4), and
// compacts the mismatch decisions into one list for the head with a wave
// ballot and a prefix over the workgroup's waves.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "launch.h"

namespace cospec {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescaleMargin = 32.0f;   // log2 units of headroom above the reference
constexpr float kFarBelow = -1.0e30f;     // initial reference: any finite logit rescales
constexpr int kUnroll = 4;                // 16-byte loads in flight per lane

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <int DT> struct Elt;
template <> struct Elt<kBF16> {
    static constexpr int kPerVec = 8;
    static constexpr int kBytes = 2;
    __device__ static inline void unpack(u32x4 q, float *x) {
        x[0] = __uint_as_float(q.x << 16); x[1] = __uint_as_float(q.x & 0xffff0000u);
        x[2] = __uint_as_float(q.y << 16); x[3] = __uint_as_float(q.y & 0xffff0000u);
        x[4] = __uint_as_float(q.z << 16); x[5] = __uint_as_float(q.z & 0xffff0000u);
        x[6] = __uint_as_float(q.w << 16); x[7] = __uint_as_float(q.w & 0xffff0000u);
    }
    __device__ static inline float at(const char *row, int64_t i) {
        return __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t *>(row)[i]) << 16);
    }
};
template <> struct Elt<kF32> {
    static constexpr int kPerVec = 4;
    static constexpr int kBytes = 4;
    __device__ static inline void unpack(u32x4 q, float *x) {
        x[0] = __uint_as_float(q.x); x[1] = __uint_as_float(q.y);
        x[2] = __uint_as_float(q.z); x[3] = __uint_as_float(q.w);
    }
    __device__ static inline float at(const char *row, int64_t i) {
        return reinterpret_cast<const float *>(row)[i];
    }
};

struct Lane {
    float best;      // largest logit seen
    int chunk;       // first chunk (16-byte vector index) holding `best`, -1 if none
    u32x4 raw;       // that chunk's bits: the exact index is found without a re-read
    float ref;       // reference of S and T, in log2 units
    float S, T;
};

__device__ inline void rescale(Lane &st, float new_ref) {
    const float dr = st.ref - new_ref;            // <= 0, finite
    const float f = __builtin_amdgcn_exp2f(dr);
    st.T = f * fmaf(dr, st.S, st.T);
    st.S = f * st.S;
    st.ref = new_ref;
}

template <int NV>
__device__ inline void consume(const float *x, u32x4 q, int chunk, Lane &st) {
    float cm = -INFINITY;
#pragma unroll
    for (int k = 0; k < NV; ++k) cm = fmaxf(cm, x[k]);
    if (cm > st.best) { st.best = cm; st.chunk = chunk; st.raw = q; }
    const float cms = __fmul_rn(cm, kLog2e);
    const bool up = cms > st.ref + kRescaleMargin;
    // wave-uniform branch: after the first chunk almost no lane ever takes it
    if (__builtin_expect(__ballot(up) != 0, 0)) {
        if (up) rescale(st, cms);
    }
    const float nref = -st.ref;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const float t = fmaf(x[k], kLog2e, nref);
        const float e = __builtin_amdgcn_exp2f(t);
        st.S += e;
        st.T = fmaf(e, t, st.T);
    }
}

__device__ inline bool better(float v, int i, float bv, int bi) {
    return v > bv || (v == bv && i < bi);
}

template <int DT>
__global__ __launch_bounds__(kReduceThreads) void k_vocab_reduce(ReduceArgs a) {
    using E = Elt<DT>;
    constexpr int NV = E::kPerVec;
    const int tid = threadIdx.x;
    const int row = blockIdx.x / a.splits;
    const int split = blockIdx.x - row * a.splits;
    if (blockIdx.x == 0 && tid == 0 && a.reset_counter) *a.reset_counter = 0;

    const char *rp;
    if (row < a.n_tgt_rows) {
        rp = a.tgt + static_cast<int64_t>(row) * a.ld_bytes;
    } else {
        const int r = row - a.n_tgt_rows;
        rp = a.drf + static_cast<int64_t>(r) * a.ld_bytes;
        if (a.parent) {   // tree: only nodes with a child need their draft row
            const int b = r / a.N, n = r - b * a.N;
            const int m = n + 1 + tid;
            const bool child = m < a.N && a.parent[static_cast<int64_t>(b) * a.N + m] == n;
            if (!__syncthreads_or(child)) return;
        }
    }

    const int nvec = static_cast<int>((static_cast<int64_t>(a.V) * E::kBytes) / 16);
    const int tail = a.V - nvec * NV;
    const int v0 = split * a.vec_per_split;
    const int v1 = min(v0 + a.vec_per_split, nvec);
    const u32x4 *rv = reinterpret_cast<const u32x4 *>(rp);

    Lane st{-INFINITY, -1, u32x4{0, 0, 0, 0}, kFarBelow, 0.f, 0.f};
    int v = v0 + tid;
    for (; v + (kUnroll - 1) * kReduceThreads < v1; v += kUnroll * kReduceThreads) {
        u32x4 q[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) q[u] = __builtin_nontemporal_load(rv + v + u * kReduceThreads);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            float x[NV];
            E::unpack(q[u], x);
            consume<NV>(x, q[u], v + u * kReduceThreads, st);
        }
    }
    for (; v < v1; v += kReduceThreads) {
        float x[NV];
        const u32x4 q = __builtin_nontemporal_load(rv + v);
        E::unpack(q, x);
        consume<NV>(x, q, v, st);
    }
    // elements past the last whole vector: the last split's first lane
    if (tail > 0 && split == a.splits - 1 && tid == 0) {
        const int64_t e0 = static_cast<int64_t>(nvec) * NV;
        float cm = -INFINITY;
        for (int k = 0; k < tail; ++k) cm = fmaxf(cm, E::at(rp, e0 + k));
        if (cm > st.best) {
            st.best = cm;
            st.chunk = nvec;
            uint16_t h[8] = {0, 0, 0, 0, 0, 0, 0, 0};      // the partial vector, zero-padded
            for (int k = 0; k < tail * E::kBytes / 2; ++k) h[k] = reinterpret_cast<const uint16_t *>(rp + e0 * E::kBytes)[k];
            st.raw = u32x4{h[0] | (uint32_t(h[1]) << 16), h[2] | (uint32_t(h[3]) << 16),
                           h[4] | (uint32_t(h[5]) << 16), h[6] | (uint32_t(h[7]) << 16)};
        }
        const float cms = __fmul_rn(cm, kLog2e);
        if (cms > st.ref + kRescaleMargin) rescale(st, cms);
        for (int k = 0; k < tail; ++k) {
            const float t = fmaf(E::at(rp, e0 + k), kLog2e, -st.ref);
            const float e = __builtin_amdgcn_exp2f(t);
            st.S += e;
            st.T = fmaf(e, t, st.T);
        }
    }

    // exact first index of the lane's max, from the saved bits of its first chunk
    int idx = INT_MAX;
    if (st.chunk >= 0) {
        float x[NV];
        E::unpack(st.raw, x);
        const int64_t e0 = static_cast<int64_t>(st.chunk) * NV;
#pragma unroll
        for (int k = NV - 1; k >= 0; --k)
            if (e0 + k < a.V && x[k] == st.best) idx = static_cast<int>(e0 + k);
    }

    __shared__ float s_best[kReduceThreads / 64];
    __shared__ int s_idx[kReduceThreads / 64];
    __shared__ float s_S[kReduceThreads / 64], s_T[kReduceThreads / 64];
    __shared__ float s_M;
    const int lane = tid & 63, wave = tid >> 6;

    float bv = st.best;
    int bi = idx;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const float ov = __shfl_xor(bv, off);
        const int oi = __shfl_xor(bi, off);
        if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    if (lane == 0) { s_best[wave] = bv; s_idx[wave] = bi; }
    __syncthreads();
    if (tid == 0) {
        float M = s_best[0];
        int I = s_idx[0];
        for (int w = 1; w < kReduceThreads / 64; ++w)
            if (better(s_best[w], s_idx[w], M, I)) { M = s_best[w]; I = s_idx[w]; }
        s_M = M;
        s_idx[0] = I;
    }
    __syncthreads();
    const float M = s_M;
    const float R = __fmul_rn(M, kLog2e);   // the partial's reference: rounded, never contracted
    float S = 0.f, T = 0.f;
    if (st.S > 0.f) {
        const float dr = st.ref - R;
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
    if (tid == 0) {
        float SS = s_S[0], TT = s_T[0];
        for (int w = 1; w < kReduceThreads / 64; ++w) { SS += s_S[w]; TT += s_T[w]; }
        a.partials[static_cast<int64_t>(row) * a.splits + split] =
            make_float4(M, __int_as_float(s_idx[0]), SS, TT);
    }
}

struct RowStat {
    float max, lse, ent;
    float log_s;     // ln sum exp(x - max): lse - max without the cancellation
    int arg;
};

// Fixed-order merge of one row's split partials.
__device__ inline RowStat merge_row(const float4 *p, int splits) {
    float M = -INFINITY;
    int arg = INT_MAX;
    for (int s = 0; s < splits; ++s) {
        const float4 q = p[s];
        if (q.z > 0.f && q.x > M) { M = q.x; arg = __float_as_int(q.y); }   // earlier split wins ties
    }
    const float R = __fmul_rn(M, kLog2e);
    float S = 0.f, T = 0.f;
    for (int s = 0; s < splits; ++s) {
        const float4 q = p[s];
        if (q.z > 0.f) {
            const float dr = __fmul_rn(q.x, kLog2e) - R;     // the split's reference, as k_vocab_reduce rounded it
            const float f = __builtin_amdgcn_exp2f(dr);
            S += f * q.z;
            T += f * fmaf(dr, q.z, q.w);
        }
    }
    // S = sum 2^(x*log2e - R) = 2^delta * sum e^(x - M) with delta = M*log2e - R the
    // rounding residual of R (exact by one fma); it matters once |M| is in the thousands
    const float delta = fmaf(M, kLog2e, -R);
    const float l2s = __log2f(S);
    RowStat r;
    r.max = M;
    r.arg = arg;
    r.log_s = (l2s - delta) * kLn2;
    r.lse = M + r.log_s;
    r.ent = (l2s - T / S) * kLn2;
    return r;
}

template <int DT>
__global__ __launch_bounds__(kDecideThreads) void k_decide(DecideArgs a) {
    using E = Elt<DT>;
    const int b = blockIdx.x;
    const int t = threadIdx.x;
    // per row: max and ln S, so that log p(token) = (x - max) - ln S keeps full
    // precision even when |lse| is large
    __shared__ float s_tmax[kMaxSeqRows], s_tlogs[kMaxSeqRows];
    __shared__ int s_targ[kMaxSeqRows];
    __shared__ float s_dmax[kMaxSeqRows], s_dlogs[kMaxSeqRows];
    __shared__ int s_child[kMaxSeqRows];
    __shared__ int s_wave_cnt[kDecideThreads / 64];
    __shared__ int s_base;

    // target rows of this sequence
    for (int j = t; j < a.RT; j += kDecideThreads) {
        const int64_t r = static_cast<int64_t>(b) * a.RT + j;
        const RowStat rs = merge_row(a.partials + r * a.splits, a.splits);
        s_tmax[j] = rs.max;
        s_tlogs[j] = rs.log_s;
        s_targ[j] = rs.arg;
        a.ws_tgt_arg[r] = rs.arg;
        if (a.tgt_argmax) a.tgt_argmax[r] = rs.arg;
        if (a.tgt_max) a.tgt_max[r] = rs.max;
        if (a.tgt_lse) a.tgt_lse[r] = rs.lse;
        if (a.tgt_ent) a.tgt_ent[r] = rs.ent;
    }
    // which draft rows were reduced: every chain row; tree nodes with a child
    for (int j = t; j < a.RD; j += kDecideThreads) s_child[j] = a.is_tree ? 0 : 1;
    __syncthreads();
    if (a.is_tree) {
        for (int n = 1 + t; n < a.RD; n += kDecideThreads) {
            const int p = a.parent[static_cast<int64_t>(b) * a.RD + n];
            if (p >= 0 && p < n) s_child[p] = 1;
        }
        __syncthreads();
    }
    for (int j = t; j < a.RD; j += kDecideThreads) {
        const int64_t r = static_cast<int64_t>(b) * a.RD + j;
        RowStat rs{NAN, NAN, NAN, NAN, -1};
        if (s_child[j]) rs = merge_row(a.partials + (static_cast<int64_t>(a.B) * a.RT + r) * a.splits, a.splits);
        s_dmax[j] = rs.max;
        s_dlogs[j] = rs.log_s;
        if (a.drf_argmax) a.drf_argmax[r] = rs.arg;
        if (a.drf_max) a.drf_max[r] = rs.max;
        if (a.drf_lse) a.drf_lse[r] = rs.lse;
        if (a.drf_ent) a.drf_ent[r] = rs.ent;
    }
    __syncthreads();

    // decisions: chain slot t is decision t+1 (verified by row t); tree slot t is node t
    const int lane = t & 63, wave = t >> 6;
    for (int base_slot = 0; base_slot < a.D; base_slot += kDecideThreads) {
        const int slot = base_slot + t;
        const bool active = slot < a.D;
        uint8_t state = kStateMatch;
        float lpt = NAN, lpd = NAN;
        int hrow = 0;
        const int64_t di = static_cast<int64_t>(b) * a.D + slot;
        if (active && !(a.is_tree && slot == 0)) {
            int p;
            bool valid = true;
            if (a.is_tree) {
                p = a.parent[di];
                valid = p >= 0 && p < slot;
                hrow = static_cast<int>(di);
            } else {
                p = slot;
                hrow = static_cast<int>(di);
            }
            const int tok = a.tokens[di];
            valid = valid && tok >= 0 && tok < a.V;
            if (valid) {
                const bool match = tok == s_targ[p];
                const char *trow = a.tgt + (static_cast<int64_t>(b) * a.RT + p) * a.ld_bytes;
                const char *drow = a.drf + (static_cast<int64_t>(b) * a.RD + p) * a.ld_bytes;
                lpt = (E::at(trow, tok) - s_tmax[p]) - s_tlogs[p];
                lpd = (E::at(drow, tok) - s_dmax[p]) - s_dlogs[p];
                state = match ? kStateMatch : kStateMismatch;
            } else {
                state = kStateReject;
            }
        }
        const bool need = active && state == kStateMismatch && a.score_mismatch;
        const uint64_t m = __ballot(need);
        if (lane == 0) s_wave_cnt[wave] = __popcll(m);
        __syncthreads();
        if (t == 0) {
            int tot = 0;
            for (int w = 0; w < kDecideThreads / 64; ++w) { const int c = s_wave_cnt[w]; s_wave_cnt[w] = tot; tot += c; }
            s_base = tot ? atomicAdd(a.ws_count, tot) : 0;
        }
        __syncthreads();
        if (active) {
            int pos = -1;
            if (need) {
                pos = s_base + s_wave_cnt[wave] + __popcll(m & ((1ull << lane) - 1ull));
                a.ws_list[pos] = hrow;
            }
            a.ws_listpos[di] = pos;
            a.ws_state[di] = state;
            if (a.delta) a.delta[di] = state == kStateMatch;
            if (a.logp_tgt) a.logp_tgt[di] = lpt;
            if (a.logp_drf) a.logp_drf[di] = lpd;
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_reduce(Dtype dt, const ReduceArgs &a, hipStream_t s) {
    const int64_t rows = static_cast<int64_t>(a.n_tgt_rows) + a.n_drf_rows;
    const dim3 grid(static_cast<unsigned>(rows * a.splits));
    if (dt == kBF16) hipLaunchKernelGGL(k_vocab_reduce<kBF16>, grid, dim3(kReduceThreads), 0, s, a);
    else hipLaunchKernelGGL(k_vocab_reduce<kF32>, grid, dim3(kReduceThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_decide(Dtype dt, const DecideArgs &a, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(a.B));
    if (dt == kBF16) hipLaunchKernelGGL(k_decide<kBF16>, grid, dim3(kDecideThreads), 0, s, a);
    else hipLaunchKernelGGL(k_decide<kF32>, grid, dim3(kDecideThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace cospec
