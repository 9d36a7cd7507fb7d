// Device helpers shared by the reduction, sampling, decide and finish kernels:
// element access for bf16/fp32 rows, wave reductions and the fixed-order merge of
// a row's split partials.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "launch.h"

namespace cospec {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

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

__device__ inline float wave_max(float x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
    return x;
}

__device__ inline float wave_sum(float x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
    return x;
}

struct RowStat {
    float max, lse, ent;
    float log_s;     // ln sum exp(x - max): lse - max without the cancellation
    int arg;
};

// Fixed-order merge of one row's split partials.  Every operation is rounded as
// written (fma only where written, no contraction by the compiler), so that the
// kernels that inline it (decide, finish, sampling) give bit-identical statistics for
// the same partials, whether they read them from global memory or LDS.  The
// partials are read kMergeChunk at a time, every read of a chunk issued before the
// first is used (unconditionally: the index is clamped, the arithmetic skips what is
// past the end); the arithmetic runs over s = 0, 1, ... in order.
constexpr int kMergeChunk = 8;

typedef __attribute__((address_space(3))) const float lds_float;

// ld(s) returns partial s, read from global memory or from LDS through a pointer of
// that address space: a global and an LDS pointer are never merged into one, so
// every access is a global or an LDS instruction, never a flat one.
// The steps of the merge, shared by every form of it so that all of them round alike:
// the maximum and its argmax over one chunk of partials (s0 .. s0 + kMergeChunk - 1,
// those past `splits` skipped; the earlier split wins ties), the sums over one chunk
// against the reference R, and the statistics from the totals.
template <int N>
__device__ inline void merge_max_chunk(const float4 (&q)[N], int s0, int splits, float &M, int &arg) {
#pragma unroll
    for (int i = 0; i < N; ++i)
        if (s0 + i < splits && q[i].z > 0.f && q[i].x > M) { M = q[i].x; arg = __float_as_int(q[i].y); }
}

template <int N>
__device__ inline void merge_sum_chunk(const float4 (&q)[N], int s0, int splits, float R, float &S, float &T) {
#pragma clang fp contract(off)
#pragma unroll
    for (int i = 0; i < N; ++i) {
        if (s0 + i < splits && q[i].z > 0.f) {
            const float dr = __fmul_rn(q[i].x, kLog2e) - R;   // the split's reference, as
                                                              // k_vocab_reduce rounded it
            const float f = __builtin_amdgcn_exp2f(dr);
            S = fmaf(f, q[i].z, S);
            T = fmaf(f, fmaf(dr, q[i].z, q[i].w), T);
        }
    }
}

__device__ inline RowStat merge_final(float M, int arg, float R, float S, float T) {
#pragma clang fp contract(off)
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

template <typename Ld>
__device__ inline RowStat merge_row_t(Ld ld, int splits) {
#pragma clang fp contract(off)
    float M = -INFINITY;
    int arg = INT_MAX;
    float S = 0.f, T = 0.f;
    float R;
    if (splits == 1) {
        // one partial: what the loops below compute for it (its reference is R itself,
        // so dr = 0 and the factor exp2(0) = 1), without them
        const float4 q0 = ld(0);
        if (q0.z > 0.f) { M = q0.x; arg = __float_as_int(q0.y); S = q0.z; T = q0.w; }
        R = __fmul_rn(M, kLog2e);
    } else {
        float4 q[kMergeChunk];
        for (int s0 = 0; s0 < splits; s0 += kMergeChunk) {
#pragma unroll
            for (int i = 0; i < kMergeChunk; ++i) q[i] = ld(min(s0 + i, splits - 1));   // unconditional
            merge_max_chunk(q, s0, splits, M, arg);
        }
        R = __fmul_rn(M, kLog2e);
        for (int s0 = 0; s0 < splits; s0 += kMergeChunk) {
            if (splits > kMergeChunk) {              // else the chunk is still in registers
#pragma unroll
                for (int i = 0; i < kMergeChunk; ++i) q[i] = ld(min(s0 + i, splits - 1));
            }
            merge_sum_chunk(q, s0, splits, R, S, T);
        }
    }
    return merge_final(M, arg, R, S, T);
}

// Two rows of `splits` > 1 partials each, at pa and pb in global memory, merged as
// merge_row merges them (the same steps in split order, so the same bits), the loads
// of both rows' chunk of kWideChunk issued together: one memory round trip when
// splits <= kWideChunk, else two per chunk.
constexpr int kWideChunk = 16;
__device__ inline void merge_rows2(const float4 *pa, const float4 *pb, int splits, RowStat &ra, RowStat &rb) {
#pragma clang fp contract(off)
    constexpr int N = kWideChunk;
    float Ma = -INFINITY, Mb = -INFINITY, Sa = 0.f, Ta = 0.f, Sb = 0.f, Tb = 0.f;
    int aa = INT_MAX, ab = INT_MAX;
    float4 qa[N], qb[N];
    auto load = [&](int s0) {
#pragma unroll
        for (int i = 0; i < N; ++i) {
            const int s = min(s0 + i, splits - 1);   // unconditional
            qa[i] = pa[s];
            qb[i] = pb[s];
        }
        // every word stays live until here, so no load register is reused while the
        // later loads are in flight
#pragma unroll
        for (int i = 0; i < N; ++i)
            asm volatile("" ::"v"(qa[i].x), "v"(qa[i].y), "v"(qa[i].z), "v"(qa[i].w), "v"(qb[i].x), "v"(qb[i].y),
                         "v"(qb[i].z), "v"(qb[i].w));
    };
    for (int s0 = 0; s0 < splits; s0 += N) {
        load(s0);
        merge_max_chunk(qa, s0, splits, Ma, aa);
        merge_max_chunk(qb, s0, splits, Mb, ab);
    }
    const float Ra = __fmul_rn(Ma, kLog2e), Rb = __fmul_rn(Mb, kLog2e);
    for (int s0 = 0; s0 < splits; s0 += N) {
        if (splits > N) load(s0);                  // else the chunk is still in registers
        merge_sum_chunk(qa, s0, splits, Ra, Sa, Ta);
        merge_sum_chunk(qb, s0, splits, Rb, Sb, Tb);
    }
    ra = merge_final(Ma, aa, Ra, Sa, Ta);
    rb = merge_final(Mb, ab, Rb, Sb, Tb);
}

// The candidate merge_row takes (its .arg) from the partials' maxima alone: the first
// split, in split order, with S > 0 and the strictly largest maximum (a single split:
// S > 0 alone, as in merge_row); INT_MAX when none is taken.  One loop, every load
// unconditional (the index clamped) and no branch on the split count, so a caller that
// needs only the argmax issues these loads together with its others.
__device__ inline int merge_arg(const float4 *p, int splits) {
    constexpr int N = 16;                        // one round trip up to 16 splits
    const u32x4 *q = reinterpret_cast<const u32x4 *>(p);
    float M = -INFINITY;
    int arg = INT_MAX;
    for (int s0 = 0; s0 < splits; s0 += N) {
        u32x4 c[N];
#pragma unroll
        for (int i = 0; i < N; ++i) c[i] = q[min(s0 + i, splits - 1)];
#pragma unroll
        for (int i = 0; i < N; ++i) {
            const float x = __uint_as_float(c[i].x);
            const bool take = (s0 + i < splits) & (__uint_as_float(c[i].z) > 0.f) & ((x > M) | (splits == 1));
            M = take ? x : M;
            arg = take ? static_cast<int>(c[i].y) : arg;
        }
    }
    return arg;
}

// A row's partials in global memory.
__device__ inline RowStat merge_row(const float4 *p, int splits) {
    return merge_row_t([p](int s) { return p[s]; }, splits);
}

// A row's partials staged in LDS (p points into a __shared__ array).
__device__ inline RowStat merge_row_lds(const float4 *p, int splits) {
    const lds_float *f = (const lds_float *)p;   // address-space cast to LDS
    return merge_row_t([f](int s) { return make_float4(f[4 * s], f[4 * s + 1], f[4 * s + 2], f[4 * s + 3]); },
                       splits);
}

// A sequence's partials, when a row is split many ways, are first copied into LDS by
// many lanes at once (one memory round trip for all of them); the merges then read
// LDS.  Up to kStageParts partials are staged; beyond that the merges read global
// memory directly.
constexpr int kStageParts = 1024;

// Copies the n1 partials at p1, then the n2 at p2, into stage[0, n1 + n2) with the
// threads [idx, idx + count) of the caller (each copies every count-th, eight loads
// issued before the first write); the caller synchronises before reading them.
__device__ inline void stage_partials(const float4 *p1, int64_t n1, const float4 *p2, int64_t n2, float4 *stage,
                                      int idx, int count) {
    constexpr int kBatch = 8;
    const int64_t n = n1 + n2;
    for (int64_t i0 = idx; i0 < n; i0 += kBatch * static_cast<int64_t>(count)) {
        float4 v[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            int64_t i = i0 + j * static_cast<int64_t>(count);
            i = i < n ? i : n - 1;                       // unconditional: clamped
            v[j] = *(i < n1 ? p1 + i : p2 + (i - n1));
        }
        // unconditional too: an index past the end writes partial n-1's own value to
        // its slot again (a store under a branch would pull its load in after it)
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const int64_t i = i0 + j * static_cast<int64_t>(count);
            stage[i < n ? i : n - 1] = v[j];
        }
    }
}

}  // namespace cospec
