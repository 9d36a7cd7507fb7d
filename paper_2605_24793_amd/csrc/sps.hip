// Standard speculative sampling over chain blocks: the distribution-preserving
// baseline the paper runs at temperature 1 (Section 3.1, stochastic decoding; Appendix C.3), on the
// same reductions as the CoSpec step.
//
// k_sps_finish (one wave per sequence, lane i-1 owns draft token i): merges the
//   draft rows, takes log p_D(token), and accepts token i when its uniform is
//   below p_T(token) / p_D(token) = exp(log p_T - log p_D) (so with probability
//   min(1, ratio)); the round stops at the first rejection s (or K+1).
// k_sps_mass: for every sequence, the weight of every segment of kSegVecs
//   16-byte vectors of the distribution its last token is drawn from: the
//   residual max(0, p_T - p_D) of rows s-1 when s <= K, p_T of target row K
//   otherwise.  One wave per four segments, all of its loads issued first.
// k_sps_pick (one wave per sequence): inverts the sequence's last uniform
//   through the segment weights, then through the elements of that segment.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "launch.h"
#include "rowstat.h"

namespace cospec {
namespace {

constexpr int kMassSegsPerWave = 4;
constexpr int kMassSegsPerBlock = 4 * kMassSegsPerWave;
constexpr float kBelowOne = 0x1.fffffep-1f;

// p(x) = exp((x - max) - ln S) of a merged row, in fp32 via exp2.
__device__ inline float prob(float x, const RowStat &rs) {
    return __builtin_amdgcn_exp2f(((x - rs.max) - rs.log_s) * kLog2e);
}

template <int DT>
__global__ __launch_bounds__(256) void k_sps_finish(SpsArgs a) {
    using E = Elt<DT>;
    const int lane = threadIdx.x & 63;
    const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (b >= a.B) return;                                  // whole wave leaves together
    const int K = a.K;
    const int64_t di = static_cast<int64_t>(b) * K + lane;
    bool fail = false;
    if (lane < K) {
        const uint8_t st = a.ws_state[di];
        const bool valid = st != kStateReject;
        const RowParts rp = row_parts(a.plan, a.plan.n_tgt_rows + di);
        const RowStat rs = merge_row(a.partials + rp.first, rp.count);
        const float xd = valid ? E::at(a.drf + di * a.ld_bytes, a.tokens[di]) : 0.f;
        const float lpd = valid ? (xd - rs.max) - rs.log_s : NAN;
        const float ratio = valid ? expf(a.ws_logp_tgt[di] - lpd) : 0.f;
        fail = !(a.uniform[static_cast<int64_t>(b) * (K + 1) + lane] < ratio);   // NaN rejects
        if (a.drf_argmax) a.drf_argmax[di] = rs.arg;
        if (a.drf_max) a.drf_max[di] = rs.max;
        if (a.drf_lse) a.drf_lse[di] = rs.lse;
        if (a.drf_ent) a.drf_ent[di] = rs.ent;
        if (a.logp_drf) a.logp_drf[di] = lpd;
        if (a.accept_prob) a.accept_prob[di] = valid ? fminf(ratio, 1.0f) : NAN;
        if (a.accept) a.accept[di] = !fail;
    }
    const uint64_t rej = __ballot(fail);
    const int s = rej ? __builtin_ctzll(rej) + 1 : K + 1;
    if (lane == 0) a.accept_len[b] = s;
    for (int j = lane; j <= K; j += 64)
        if (j != s - 1) a.out_tokens[static_cast<int64_t>(b) * (K + 1) + j] = j < s - 1 ? a.tokens[static_cast<int64_t>(b) * K + j] : -1;
}

// The rows the last token of sequence b is drawn from: target row s-1 and, when
// s <= K, draft row s-1 (residual), with their merged statistics.
struct LastRows {
    const char *t, *d;    // d null: the bonus token, drawn from p_T
    RowStat ts, ds;
};

// The rows alone (no statistics yet), so that a caller can issue its loads of them
// before the merges' own loads and arithmetic.
__device__ inline LastRows last_row_ptrs(const SpsArgs &a, int b) {
    LastRows r;
    const int s = a.accept_len[b];
    const int64_t trow = static_cast<int64_t>(b) * (a.K + 1) + (s - 1);
    r.t = a.tgt + trow * a.ld_bytes;
    r.d = nullptr;
    if (s <= a.K) r.d = a.drf + (static_cast<int64_t>(b) * a.K + (s - 1)) * a.ld_bytes;
    return r;
}

__device__ inline void last_row_stats(const SpsArgs &a, int b, LastRows &r) {
    const int s = a.accept_len[b];
    const int64_t trow = static_cast<int64_t>(b) * (a.K + 1) + (s - 1);
    const RowParts tp = row_parts(a.plan, trow);
    r.ts = merge_row(a.partials + tp.first, tp.count);
    if (r.d) {
        const RowParts dp = row_parts(a.plan, a.plan.n_tgt_rows + static_cast<int64_t>(b) * a.K + (s - 1));
        r.ds = merge_row(a.partials + dp.first, dp.count);
    }
}

__device__ inline LastRows last_rows(const SpsArgs &a, int b) {
    LastRows r = last_row_ptrs(a, b);
    last_row_stats(a, b, r);
    return r;
}

// Weights of the NV elements of 16-byte vector v of the last rows.
template <int DT>
__device__ inline void vec_weights(const LastRows &r, int v, float *w) {
    using E = Elt<DT>;
    constexpr int NV = E::kPerVec;
    float x[NV];
    E::unpack(*reinterpret_cast<const u32x4 *>(r.t + static_cast<int64_t>(v) * 16), x);
#pragma unroll
    for (int k = 0; k < NV; ++k) w[k] = prob(x[k], r.ts);
    if (r.d) {
        E::unpack(*reinterpret_cast<const u32x4 *>(r.d + static_cast<int64_t>(v) * 16), x);
#pragma unroll
        for (int k = 0; k < NV; ++k) w[k] = fmaxf(w[k] - prob(x[k], r.ds), 0.f);
    }
}

template <int DT>
__device__ inline float elem_weight(const LastRows &r, int64_t i) {
    using E = Elt<DT>;
    float w = prob(E::at(r.t, i), r.ts);
    if (r.d) w = fmaxf(w - prob(E::at(r.d, i), r.ds), 0.f);
    return w;
}

template <int DT>
__global__ __launch_bounds__(256) void k_sps_mass(SpsArgs a) {
    using E = Elt<DT>;
    constexpr int NV = E::kPerVec;
    const int lane = threadIdx.x & 63;
    const int per_seq = (a.nseg + kMassSegsPerBlock - 1) / kMassSegsPerBlock;
    const int b = blockIdx.x / per_seq;
    const int seg0 = (blockIdx.x % per_seq) * kMassSegsPerBlock + (threadIdx.x >> 6) * kMassSegsPerWave;
    if (seg0 >= a.nseg) return;                            // whole wave leaves
    LastRows r = last_row_ptrs(a, b);
    const int nvec = static_cast<int>((static_cast<int64_t>(a.V) * E::kBytes) / 16);
    const int nmain = (nvec + kSegVecs - 1) / kSegVecs;
    // all of this wave's loads first (kMassSegsPerWave segments of both rows), then
    // the weights: the loads overlap instead of one segment's round trip at a time
    u32x4 tq[kMassSegsPerWave], dq[kMassSegsPerWave];
#pragma unroll
    for (int j = 0; j < kMassSegsPerWave; ++j) {
        const int v = (seg0 + j) * kSegVecs + lane;
        tq[j] = u32x4{0, 0, 0, 0};
        dq[j] = u32x4{0, 0, 0, 0};
        if (seg0 + j < nmain && v < nvec) {
            tq[j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(r.t) + v);
            if (r.d) dq[j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(r.d) + v);
        }
    }
    last_row_stats(a, b, r);                               // while the segments are in flight
#pragma unroll
    for (int j = 0; j < kMassSegsPerWave; ++j) {
        const int seg = seg0 + j;
        if (seg >= a.nseg) break;                          // wave-uniform
        float m = 0.f;
        if (seg < nmain) {
            if (seg * kSegVecs + lane < nvec) {
                float x[NV], w[NV];
                E::unpack(tq[j], x);
#pragma unroll
                for (int k = 0; k < NV; ++k) w[k] = prob(x[k], r.ts);
                if (r.d) {
                    E::unpack(dq[j], x);
#pragma unroll
                    for (int k = 0; k < NV; ++k) w[k] = fmaxf(w[k] - prob(x[k], r.ds), 0.f);
                }
#pragma unroll
                for (int k = 0; k < NV; ++k) m += w[k];
            }
        } else {
            const int64_t i = static_cast<int64_t>(nvec) * NV + lane;
            if (i < a.V) m = elem_weight<DT>(r, i);
        }
        m = wave_sum(m);
        if (lane == 0) a.seg_mass[static_cast<int64_t>(b) * a.nseg + seg] = m;
    }
}

__device__ inline float wave_incl_scan(float x, int lane) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const float y = __shfl_up(x, off);
        if (lane >= off) x += y;
    }
    return x;
}

template <int DT>
__global__ __launch_bounds__(256) void k_sps_pick(SpsArgs a) {
    using E = Elt<DT>;
    constexpr int NV = E::kPerVec;
    const int lane = threadIdx.x & 63;
    const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (b >= a.B) return;
    float u = a.uniform[static_cast<int64_t>(b) * (a.K + 1) + a.K];
    u = u >= 0.f ? fminf(u, kBelowOne) : 0.f;
    const float *sm = a.seg_mass + static_cast<int64_t>(b) * a.nseg;

    // 1. the segment: lanes own contiguous runs; only owning lanes may cross
    const int per = (a.nseg + 63) / 64;
    const int s0 = min(lane * per, a.nseg), s1 = min(s0 + per, a.nseg);
    const bool owns = s0 < s1;
    float run = 0.f;
    for (int s = s0; s < s1; ++s) run += sm[s];
    const float incl = wave_incl_scan(run, lane);
    const float up = __shfl_up(incl, 1);
    const float excl = lane ? up : 0.f;
    const float total = __shfl(incl, (a.nseg - 1) / per);
    const float target = u * total;
    const uint64_t hit = __ballot(owns && incl > target);
    const uint64_t has = __ballot(owns && run > 0.f);
    const int L = hit ? __builtin_ctzll(hit) : has ? 63 - __builtin_clzll(has) : 0;
    int segsel = -1;
    float before = 0.f;
    if (lane == L) {
        float cum = excl, cum_last = excl;
        int last = -1;
        for (int s = s0; s < s1; ++s) {
            const float m = sm[s];
            if (m > 0.f) {
                last = s;
                cum_last = cum;
                if (cum + m > target) { segsel = s; before = cum; break; }
            }
            cum += m;
        }
        if (segsel < 0) { segsel = last; before = cum_last; }
    }
    segsel = max(__shfl(segsel, L), 0);
    before = __shfl(before, L);

    // 2. the element
    const LastRows r = last_rows(a, b);
    const int nvec = static_cast<int>((static_cast<int64_t>(a.V) * E::kBytes) / 16);
    const int nmain = (nvec + kSegVecs - 1) / kSegVecs;
    float w[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) w[k] = 0.f;
    int first;
    if (segsel < nmain) {
        const int v = segsel * kSegVecs + lane;
        first = v * NV;
        if (v < nvec) vec_weights<DT>(r, v, w);
    } else {
        first = nvec * NV + lane;
        if (first < a.V) w[0] = elem_weight<DT>(r, first);
    }
    float pre[NV];
    float acc = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) { acc += w[k]; pre[k] = acc; }
    const float lincl = wave_incl_scan(acc, lane);
    const float lup = __shfl_up(lincl, 1);
    const float base = before + (lane ? lup : 0.f);
    int khit = -1, klast = -1;
#pragma unroll
    for (int k = NV - 1; k >= 0; --k) {
        if (w[k] > 0.f && base + pre[k] > target) khit = k;
        if (klast < 0 && w[k] > 0.f) klast = k;
    }
    const uint64_t h2 = __ballot(khit >= 0);
    const uint64_t h3 = __ballot(klast >= 0);
    int idx;
    if (h2) idx = __shfl(first + khit, __builtin_ctzll(h2));
    else if (h3) idx = __shfl(first + klast, 63 - __builtin_clzll(h3));
    else idx = __shfl(first, 0);
    if (lane == 0) a.out_tokens[static_cast<int64_t>(b) * (a.K + 1) + a.accept_len[b] - 1] = idx;
}

}  // namespace

hipError_t launch_sps(Dtype dt, const SpsArgs &a, hipStream_t s) {
    if (a.B == 0) return hipSuccess;
    const dim3 wave_grid(static_cast<unsigned>((a.B + 3) / 4));
    const int per_seq = (a.nseg + kMassSegsPerBlock - 1) / kMassSegsPerBlock;
    const dim3 mass_grid(static_cast<unsigned>(static_cast<int64_t>(a.B) * per_seq));
    if (dt == kBF16) {
        hipLaunchKernelGGL(k_sps_finish<kBF16>, wave_grid, dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_sps_mass<kBF16>, mass_grid, dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_sps_pick<kBF16>, wave_grid, dim3(256), 0, s, a);
    } else {
        hipLaunchKernelGGL(k_sps_finish<kF32>, wave_grid, dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_sps_mass<kF32>, mass_grid, dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_sps_pick<kF32>, wave_grid, dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace cospec
