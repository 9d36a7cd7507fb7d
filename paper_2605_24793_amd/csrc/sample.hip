// Temperature-1 verification candidates (Section 3.1, stochastic decoding; at
// T = 1 the target's candidate is a sample of its next-token distribution,
// Appendix C.3).  The sample is taken by inversion of a caller-supplied uniform
// u: the candidate of a row is the smallest v whose cumulative probability
// p[0] + ... + p[v] (index order, p = softmax(row)) exceeds u.
//
// The reduction kernel leaves, per target row, the probability mass of every
// segment of kSegVecs 16-byte vectors and, last, of the tail elements.  One wave
// per row: each lane sums a contiguous run of segments, a wave scan gives the
// mass before each lane, the lane whose run crosses u * total walks it to the
// segment, and the wave re-reads that one segment (1 KiB) and inverts within it.
// The sums are fp32, so a uniform within about 1e-5 of a boundary of the
// cumulative distribution may select the neighbouring index.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "launch.h"
#include "rowstat.h"

namespace cospec {
namespace {

constexpr float kBelowOne = 0x1.fffffep-1f;   // largest float below 1

__device__ inline float wave_incl_scan(float x, int lane) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const float y = __shfl_up(x, off);
        if (lane >= off) x += y;
    }
    return x;
}

// Mass of a segment relative to the row reference R = fl(max * log2e).
__device__ inline float seg_mass(float2 g, float R) { return g.x * __builtin_amdgcn_exp2f(g.y - R); }

template <int DT>
__global__ __launch_bounds__(256) void k_sample(SampleArgs a) {
    using E = Elt<DT>;
    constexpr int NV = E::kPerVec;
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= a.n_rows) return;                                   // whole wave leaves
    const RowParts parts = row_parts(a.plan, row);
    const RowStat rs = merge_row(a.partials + parts.first, parts.count);
    const float R = __fmul_rn(rs.max, kLog2e);
    float u = a.uniform[row];
    u = u >= 0.f ? fminf(u, kBelowOne) : 0.f;                      // NaN and negatives act as 0

    // 1. the segment where the cumulative mass crosses u * total
    const float2 *sg = a.seg + static_cast<int64_t>(row) * a.nseg;
    const int per = (a.nseg + 63) / 64;
    const int s0 = min(lane * per, a.nseg), s1 = min(s0 + per, a.nseg);
    float run = 0.f;
    for (int s = s0; s < s1; ++s) run += seg_mass(sg[s], R);
    const float incl = wave_incl_scan(run, lane);
    const float up = __shfl_up(incl, 1);
    const float excl = lane ? up : 0.f;
    // lanes past the last segment add only zeros, but the scan rounds their sums
    // in another order: the total is the last owning lane's, and only owning
    // lanes may cross
    const bool owns = s0 < s1;
    const float total = __shfl(incl, (a.nseg - 1) / per);
    const float target = u * total;
    const uint64_t hit = __ballot(owns && incl > target);
    // no lane crosses only when rounding put the target at the very end: take the
    // last lane with mass (the maximal element has mass 1, so there is one)
    const uint64_t has = __ballot(owns && run > 0.f);
    const int L = hit ? __builtin_ctzll(hit) : has ? 63 - __builtin_clzll(has) : 0;
    int segsel = -1;
    float before = 0.f;
    if (lane == L) {
        float cum = excl, cum_last = excl;
        int last = -1;
        for (int s = s0; s < s1; ++s) {
            const float m = seg_mass(sg[s], R);
            if (m > 0.f) {
                last = s;
                cum_last = cum;
                if (cum + m > target) { segsel = s; before = cum; break; }
            }
            cum += m;
        }
        if (segsel < 0) { segsel = last; before = cum_last; }
    }
    segsel = max(__shfl(segsel, L), 0);        // -1 only if no segment had mass at all
    before = __shfl(before, L);

    // 2. invert within that segment
    const char *rp = a.tgt + static_cast<int64_t>(row) * a.ld_bytes;
    const int nvec = static_cast<int>((static_cast<int64_t>(a.V) * E::kBytes) / 16);
    const int nmain = (nvec + kSegVecs - 1) / kSegVecs;
    float e[NV];
    int first;                                                     // vocabulary index of e[0]
#pragma unroll
    for (int k = 0; k < NV; ++k) e[k] = 0.f;
    if (segsel < nmain) {
        const int v = segsel * kSegVecs + lane;
        first = v * NV;
        if (v < nvec) {
            float x[NV];
            E::unpack(*reinterpret_cast<const u32x4 *>(rp + static_cast<int64_t>(v) * 16), x);
#pragma unroll
            for (int k = 0; k < NV; ++k) e[k] = __builtin_amdgcn_exp2f(fmaf(x[k], kLog2e, -R));
        }
    } else {                                                       // the tail segment: one element per lane
        first = nvec * NV + lane;
        if (first < a.V) e[0] = __builtin_amdgcn_exp2f(fmaf(E::at(rp, first), kLog2e, -R));
    }
    float pre[NV];
    float acc = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) { acc += e[k]; pre[k] = acc; }
    const float lincl = wave_incl_scan(acc, lane);
    const float lup = __shfl_up(lincl, 1);
    const float base = before + (lane ? lup : 0.f);
    int khit = -1, klast = -1;
#pragma unroll
    for (int k = NV - 1; k >= 0; --k) {
        if (e[k] > 0.f && base + pre[k] > target) khit = k;
        if (klast < 0 && e[k] > 0.f) klast = k;
    }
    const uint64_t h2 = __ballot(khit >= 0);
    const uint64_t h3 = __ballot(klast >= 0);
    int idx;
    if (h2) {
        idx = __shfl(first + khit, __builtin_ctzll(h2));
    } else if (h3) {                   // rounding left the target past the segment's elements
        idx = __shfl(first + klast, 63 - __builtin_clzll(h3));
    } else {                           // every element underflowed against the row max
        idx = __shfl(first, 0);
    }
    if (lane == 0) a.cand[row] = idx;
}

}  // namespace

hipError_t launch_sample(Dtype dt, const SampleArgs &a, hipStream_t s) {
    if (a.n_rows <= 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>((a.n_rows + 3) / 4));
    if (dt == kBF16) hipLaunchKernelGGL(k_sample<kBF16>, grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_sample<kF32>, grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace cospec
