// The arbitrator's hybrid attention (Section 3.3).  The arbitrator reads
// q = [context, SEP, draft 1..K, SEP, candidates 1..K, SEP] (Eq. arb_input) of
// length l = l_c + 2K + 3 under a hybrid mask: context positions attend causally
// within the context; the draft/target region, read as starting at the first SEP
// (position l_c), attends to the whole context and bidirectionally within itself;
// nothing flows from the region back into the context.
//
// k_hybrid_mask writes that mask densely ([B][L][L] bytes, 1 = attend; padding
// rows attend only to themselves) for attention code that takes explicit masks.
//
// k_hybrid_attention computes softmax(q k^T * scale + mask) v for a range of query
// positions of each sequence straight from the rule (no mask in memory), with
// grouped query heads, bf16 inputs and fp32 accumulation on the matrix cores.
// Per round only the region's 2K+3 queries are new: their keys and values are
// the cached context plus the region itself.
//
// Work split: the query rows (position x head) that share one key/value head of
// one sequence go to one workgroup of up to 8 waves, 16 rows per wave, so each
// key and value is read once per group (more rows: more workgroups).  Keys
// stream in blocks of 64 through
// LDS: K row-major (rows padded to D*2+16 bytes) and V transposed (rows of 64 keys
// padded to 136 bytes).  Each wave computes S^T = K Q^T (v_mfma_f32_16x16x32_bf16,
// A = K rows, B = its queries' columns kept in registers), so lane l owns query
// column l % 16 of S^T and keeps that query's running max and sum (online
// softmax).  P^T is packed to bf16 in the same lanes and O^T += V^T P^T leaves
// O^T[d][query] in the same lane too, so rescaling needs no exchange.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>

#include "launch.h"

namespace cospec {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float floatx4;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int kKeyBlock = 64;
constexpr int kMaxWaves = 8;          // per workgroup, 16 query rows each (register budget)
constexpr int kVtPitch = 136;         // bytes per row of V^T in LDS (64 keys + 8 pad)
constexpr float kLog2eA = 1.4426950408889634f;

__device__ inline floatx4 mfma(u32x4 a, u32x4 b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                   c, 0, 0, 0);
}

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

// Two fp32 values -> one word of two bf16 (lo in bits 0-15), round to nearest even
// (v_cvt_pk_bf16_f32).
__device__ inline uint32_t bf16_pair(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, bf16x2{static_cast<__bf16>(lo), static_cast<__bf16>(hi)});
}

// max over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (the rows of 16 lanes), in the VALU
__device__ inline float max_rows(float x) {
    const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
    const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}

__device__ inline float sum_rows(float x) {
    const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(p[0]) + __uint_as_float(p[1]);
    const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}

// The running max of a query is only raised when a block's max exceeds it by more
// than this (log2 units), so that the accumulators are rarely rescaled; weights stay
// below 2^kLazyRescale.
constexpr float kLazyRescale = 8.0f;

__global__ __launch_bounds__(256) void k_hybrid_mask(MaskArgs a) {
    const int64_t row = blockIdx.x;                         // b * L + i
    const int b = static_cast<int>(row / a.L), i = static_cast<int>(row % a.L);
    const int lc = max(a.ctx_len[b], 0);
    const int64_t ln = static_cast<int64_t>(lc) + 2 * a.K + 3;
    uint8_t *out = a.mask + row * a.L;
    for (int j = threadIdx.x; j < a.L; j += blockDim.x) {
        bool m;
        if (i >= ln) m = j == i;
        else if (i < lc) m = j <= i;
        else m = j < ln;
        out[j] = m;
    }
}

template <int D>
__global__ __launch_bounds__(64 * kMaxWaves) void k_hybrid_attention(AttnArgs a) {
    constexpr int KP = D * 2 + 16;                          // bytes per K row in LDS
    constexpr int DS = D / 32;                              // MFMA k-steps over d
    constexpr int DT = D / 16;                              // d tiles of the output
    __shared__ __attribute__((aligned(16))) char s_k[kKeyBlock * KP];
    __shared__ __attribute__((aligned(16))) char s_vt[D * kVtPitch];

    const int grp = a.Hq / a.Hkv;
    const int rows = a.n_q * grp;                           // query rows of one (sequence, kv head)
    const int nthr = blockDim.x, wg_rows = nthr / 4;       // 16 rows per wave
    const int wgs_per = (rows + wg_rows - 1) / wg_rows;
    const int b = blockIdx.x / (a.Hkv * wgs_per);
    const int h = (blockIdx.x / wgs_per) % a.Hkv;
    const int q0 = (blockIdx.x % wgs_per) * wg_rows;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, l16 = lane & 15;

    const int lc = max(a.ctx_len[b], 0);
    const int ln = static_cast<int>(min(static_cast<int64_t>(lc) + 2 * a.K + 3, static_cast<int64_t>(a.L)));
    const int qs = a.q_start[b];
    // the last key any query of this workgroup sees
    const int r_hi = min(q0 + wg_rows, rows) - 1;
    const int p_hi = qs + r_hi / grp;
    const int kend = p_hi >= lc ? ln : min(p_hi + 1, ln);

    // this lane's query column
    const int qi = q0 + wave * 16 + l16;
    const bool qvalid = qi < rows;
    const int r = qvalid ? qi / grp : 0;
    const int hq = h * grp + (qvalid ? qi % grp : 0);
    const int p = qs + r;
    const bool live = qvalid && p >= 0 && p < ln;
    const int vis = p < lc ? p + 1 : ln;                   // keys [0, vis) are visible
    u32x4 qf[DS];
    const char *qrow = static_cast<const char *>(a.q) + ((static_cast<int64_t>(b) * a.n_q + r) * a.Hq + hq) * D * 2;
#pragma unroll
    for (int s = 0; s < DS; ++s)
        qf[s] = live ? *reinterpret_cast<const u32x4 *>(qrow + (32 * s + 8 * g) * 2) : u32x4{0, 0, 0, 0};
    // the query loads complete here, not at their first use inside the key loop (where
    // the wait would also cover every key/value prefetch issued after them)
#pragma unroll
    for (int s = 0; s < DS; ++s) asm volatile("" : "+v"(qf[s]));

    floatx4 o[DT];
#pragma unroll
    for (int t = 0; t < DT; ++t) o[t] = floatx4{0.f, 0.f, 0.f, 0.f};
    // m: running max of the scaled scores (log2 units), common to the four lanes of a
    // query column; l: this lane's share of the running sum (its keys 4g + j)
    float m = -INFINITY, l = 0.f;
    const float sc = a.scale * kLog2eA;
    // blocks that end at or below every lane's visible length need no mask
    int vis_min = vis;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) vis_min = min(vis_min, __shfl_xor(vis_min, off));

    const int64_t kv_row = static_cast<int64_t>(a.Hkv) * D * 2;     // bytes between positions
    const char *kbase = static_cast<const char *>(a.k) + (static_cast<int64_t>(b) * a.L * a.Hkv + h) * D * 2;
    const char *vbase = static_cast<const char *>(a.v) + (static_cast<int64_t>(b) * a.L * a.Hkv + h) * D * 2;

    // Key/value blocks are prefetched into registers one block ahead: the loads of
    // block k0 + 64 are in flight while block k0 is computed from LDS.  The first
    // four waves load (a workgroup has at least four), KPT key chunks and VPT value
    // pairs per thread.  Rows past kend are read as row kend - 1 (no branches around
    // the loads): every query's mask ends at or before kend, so their weights are 0.
    constexpr int CH = D / 8;                               // 16-byte chunks per row
    constexpr int KPT = kKeyBlock * CH / 256;
    constexpr int VPT = (kKeyBlock / 2) * CH / 256;
    const bool loader = tid < 256;
    u32x4 kr[KPT], v0r[VPT], v1r[VPT];
    auto fetch = [&](int kb) {
        const int last = kend - 1;
#pragma unroll
        for (int i = 0; i < KPT; ++i) {
            const int e = tid + i * 256, key = min(kb + e / CH, last), ch = e % CH;
            kr[i] = *reinterpret_cast<const u32x4 *>(kbase + key * kv_row + ch * 16);
        }
#pragma unroll
        for (int i = 0; i < VPT; ++i) {
            const int e = tid + i * 256, k2 = kb + 2 * (e / CH), ch = e % CH;
            v0r[i] = *reinterpret_cast<const u32x4 *>(vbase + min(k2, last) * kv_row + ch * 16);
            v1r[i] = *reinterpret_cast<const u32x4 *>(vbase + min(k2 + 1, last) * kv_row + ch * 16);
        }
    };
    if (kend > 0 && loader) fetch(0);

    for (int k0 = 0; k0 < kend; k0 += kKeyBlock) {
        __syncthreads();                                    // the previous block is consumed
        // K block row-major; V block transposed, pairs of keys as 32-bit words
        if (loader) {
#pragma unroll
            for (int i = 0; i < KPT; ++i) {
                const int e = tid + i * 256, key = e / CH, ch = e % CH;
                *reinterpret_cast<u32x4 *>(s_k + key * KP + ch * 16) = kr[i];
            }
#pragma unroll
            for (int i = 0; i < VPT; ++i) {
                const int e = tid + i * 256, kp = e / CH, ch = e % CH;
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const uint32_t lo = v0r[i][w], hi = v1r[i][w];
                    const int d = ch * 8 + 2 * w;
                    // (lo & 0xffff) | (hi << 16) and (lo >> 16) | (hi & 0xffff0000)
                    *reinterpret_cast<uint32_t *>(s_vt + d * kVtPitch + kp * 4) = __builtin_amdgcn_perm(hi, lo, 0x05040100u);
                    *reinterpret_cast<uint32_t *>(s_vt + (d + 1) * kVtPitch + kp * 4) =
                        __builtin_amdgcn_perm(hi, lo, 0x07060302u);
                }
            }
        }
        __syncthreads();
        if (loader && k0 + kKeyBlock < kend) fetch(k0 + kKeyBlock);

        // S^T[key][query] for the 64 keys: tile c holds keys 16c + 4g + j in element j
        floatx4 st[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            st[c] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < DS; ++s) {
                const u32x4 kf = *reinterpret_cast<const u32x4 *>(s_k + (16 * c + l16) * KP + (32 * s + 8 * g) * 2);
                st[c] = mfma(kf, qf[s], st[c]);
            }
        }
        // online softmax over this block, for the query in this lane's column
        float bm = -INFINITY;
        if (k0 + kKeyBlock <= vis_min) {                     // wave-uniform: no key masked
#pragma unroll
            for (int c = 0; c < 4; ++c)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    st[c][j] *= sc;
                    bm = fmaxf(bm, st[c][j]);
                }
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int key = k0 + 16 * c + 4 * g + j;
                    st[c][j] = key < vis ? st[c][j] * sc : -INFINITY;
                    bm = fmaxf(bm, st[c][j]);
                }
        }
        bm = max_rows(bm);
        const bool raise = bm > m + kLazyRescale;            // always when m is still -inf
        if (__builtin_expect(__ballot(raise) != 0, 0)) {
            const float alpha = raise ? __builtin_amdgcn_exp2f(m - bm) : 1.f;   // 0 from -inf
            if (raise) m = bm;
            l *= alpha;
#pragma unroll
            for (int t = 0; t < DT; ++t) o[t] *= alpha;
        }
        // a lane whose keys so far are all masked keeps m = -inf and adds nothing
        const float mm = m == -INFINITY ? INFINITY : m;
        uint32_t pk[4][2];                                   // P^T as bf16 pairs, tile c
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            float pv[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                pv[j] = __builtin_amdgcn_exp2f(st[c][j] - mm);
                l += pv[j];
            }
            pk[c][0] = bf16_pair(pv[0], pv[1]);
            pk[c][1] = bf16_pair(pv[2], pv[3]);
        }
        // O^T[d][query] += V^T[d][keys] P^T[keys][query]; step u covers tiles 2u, 2u+1
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const u32x4 pb{pk[2 * u][0], pk[2 * u][1], pk[2 * u + 1][0], pk[2 * u + 1][1]};
#pragma unroll
            for (int t = 0; t < DT; ++t) {
                const char *vr = s_vt + (16 * t + l16) * kVtPitch;
                const u32x2 lo = *reinterpret_cast<const u32x2 *>(vr + (32 * u + 4 * g) * 2);
                const u32x2 hi = *reinterpret_cast<const u32x2 *>(vr + (32 * u + 16 + 4 * g) * 2);
                o[t] = mfma(u32x4{lo[0], lo[1], hi[0], hi[1]}, pb, o[t]);
            }
        }
    }

    l = sum_rows(l);
    if (!qvalid) return;
    // O^T tile t, element j: d = 16t + 4g + j of this lane's query
    char *orow = static_cast<char *>(a.out) + ((static_cast<int64_t>(b) * a.n_q + r) * a.Hq + hq) * D * 2;
    const float inv = live && l > 0.f ? 1.f / l : 0.f;
#pragma unroll
    for (int t = 0; t < DT; ++t) {
        const uint32_t w0 = bf16_pair(o[t][0] * inv, o[t][1] * inv);
        const uint32_t w1 = bf16_pair(o[t][2] * inv, o[t][3] * inv);
        *reinterpret_cast<u32x2 *>(orow + (16 * t + 4 * g) * 2) = u32x2{w0, w1};
    }
}

}  // namespace

hipError_t launch_hybrid_mask(const MaskArgs &a, hipStream_t s) {
    const int64_t rows = static_cast<int64_t>(a.B) * a.L;
    if (rows == 0) return hipSuccess;
    hipLaunchKernelGGL(k_hybrid_mask, dim3(static_cast<unsigned>(rows)), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_hybrid_attention(const AttnArgs &a, hipStream_t s) {
    const int64_t rows = static_cast<int64_t>(a.n_q) * (a.Hq / a.Hkv);
    // as many waves as the group's rows need, at most kMaxWaves, spread evenly
    const int64_t per_max = 16 * kMaxWaves;
    const int64_t nwg = (rows + per_max - 1) / per_max;
    const int64_t waves = std::max<int64_t>(4, (((rows + nwg - 1) / nwg) + 15) / 16);   // >= 4: loaders
    const int64_t wgs = static_cast<int64_t>(a.B) * a.Hkv * ((rows + 16 * waves - 1) / (16 * waves));
    if (wgs == 0) return hipSuccess;
    const dim3 block(static_cast<unsigned>(64 * waves));
    if (a.D == 128) hipLaunchKernelGGL(k_hybrid_attention<128>, dim3(static_cast<unsigned>(wgs)), block, 0, s, a);
    else hipLaunchKernelGGL(k_hybrid_attention<64>, dim3(static_cast<unsigned>(wgs)), block, 0, s, a);
    return hipGetLastError();
}

}  // namespace cospec
