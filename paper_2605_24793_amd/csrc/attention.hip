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
// key and value is read once per group (more rows: more workgroups).  Keys and
// values stream through a ring of kStages LDS stages of kKeyBlock rows, filled
// straight from HBM by raw buffer loads into LDS (no register staging): the
// buffers end after the group's last visible row, so the hardware range check
// fills later rows with zeros.  Both tiles are stored row-major with an XOR
// swizzle of their 16- or 32-byte units so that the fragment reads below hit
// distinct LDS banks.  Each wave computes S^T = K Q^T
// (v_mfma_f32_16x16x32_bf16, A = K rows from LDS, B = its queries' columns kept
// in registers), so lane l owns query column l % 16 of S^T and keeps that query's
// running max and sum (online softmax).  P^T is packed to bf16 in the same lanes
// and O^T += V^T P^T takes its A operand (V^T) from the row-major V tile with the
// gfx950 transposing LDS read (ds_read_b64_tr_b16), leaving O^T[d][query] in the
// lane that owns the query, so rescaling needs no exchange.
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

constexpr int kKeyBlock = 32;         // key rows per LDS stage
constexpr int kStages = 4;            // LDS ring: three stages in flight while one is used
// waves that issue the loads (a workgroup has at least 4): two measured 2% faster than
// four at 64 x 2048 context (96.5-98.6 against 99.3-100.0 us on one box), one the same
constexpr int kLoaders = 2;
constexpr int kMaxWaves = 8;          // per workgroup, 16 query rows each (register budget)
constexpr float kLog2eA = 1.4426950408889634f;

// Word 3 of a raw (unswizzled, stride 0) buffer resource: 32-bit data format.
constexpr int kRawBuffer = 0x00020000;

typedef __attribute__((address_space(3))) void lds_void;

constexpr int kNontemporal = 2;       // cache policy of the key/value loads: streamed once

// 16 bytes per lane from a raw buffer into LDS at base + 16 * lane (zeros past the
// buffer's end).  Nontemporal: each key and value is read once per round (measured at
// 64 sequences x 2048 context positions: 109 -> 98 us; a fifth key stage, an earlier
// issue of the value reads or two accumulator chains for S changed nothing more).
__device__ inline void load_lds16(__amdgpu_buffer_rsrc_t r, uint32_t off, const char *lds) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)lds, 16, static_cast<int>(off), 0, 0, kNontemporal);
}

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

// Workgroup barrier that does not wait for the stages still in flight (as the fence
// of __syncthreads would); the compiler may not move memory accesses across it.
__device__ inline void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Transposing LDS read: within each row of 16 lanes, lane j receives element j % 4 of
// the 8-byte chunks addressed by lanes 4k + j / 4, k = 0..3 (in that order).  Issued
// as inline assembly: the compiler does not know which LDS the builtin reads and
// would wait for every load into LDS still in flight before it.  The caller waits for
// the result with lds_wait().
typedef __attribute__((address_space(3))) const char lds_cchar;
__device__ inline u32x2 read_tr(const char *lds) {
    const uint32_t addr = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_cchar *)lds));
    u32x2 r;
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"(addr));
    return r;
}

// Waits for this wave's LDS reads; the values passed through are only used after it.
template <int N> __device__ inline void lds_wait(u32x2 (&x)[N], u32x2 (&y)[N]) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int i = 0; i < N; ++i) asm volatile("" : "+v"(x[i]), "+v"(y[i]));
}

// XOR swizzles of the LDS tiles (rows of RB = 2D bytes).  K: 16-byte units, so that
// 16 consecutive rows read at one column hit distinct banks; V: 32-byte units, so
// that the 8 rows of a transposing read do.
template <int RB> __device__ inline int swz_k(int row) { return RB == 256 ? (row & 15) : ((row >> 1) & 7); }
template <int RB> __device__ inline int swz_v(int row) { return RB == 256 ? (row & 7) : ((row >> 1) & 3); }

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
    constexpr int RB = D * 2;                               // bytes per key/value row
    constexpr int SB = kKeyBlock * RB;                      // bytes of one tile per stage
    constexpr int LPW = SB / 1024 / kLoaders;               // 1 KB load instructions per tile and loader
    constexpr int DS = D / 32;                              // MFMA k-steps over d
    constexpr int DT = D / 16;                              // d tiles of the output
    static_assert(LPW >= 1 && kKeyBlock == 32, "stage shape");
    __shared__ __attribute__((aligned(16))) char s_k[kStages][SB];
    __shared__ __attribute__((aligned(16))) char s_v[kStages][SB];

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
    // the wait would also cover every key/value load issued after them)
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

    // raw buffers over this group's keys and values, ending after row kend - 1;
    // offsets are 32-bit (L * Hkv * D * 2 < 2^32)
    const uint32_t row_b = static_cast<uint32_t>(a.Hkv) * D * 2;   // bytes between positions
    const int64_t head0 = (static_cast<int64_t>(b) * a.L * a.Hkv + h) * D * 2;
    const int nbytes = kend > 0 ? static_cast<int>((kend - 1) * row_b + RB) : 0;
    const __amdgpu_buffer_rsrc_t krs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(static_cast<const char *>(a.k) + head0), 0, nbytes, kRawBuffer);
    const __amdgpu_buffer_rsrc_t vrs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(static_cast<const char *>(a.v) + head0), 0, nbytes, kRawBuffer);

    // loader wave w, instruction q fills bytes (w * LPW + q) KB of a tile: lane l the
    // 16 bytes at 16 l of that KB, i.e. row `lrow`, physical unit `pch` of the tile,
    // which holds logical unit pch ^ swizzle(row)
    const bool loader = wave < kLoaders;
    uint32_t koff[LPW], voff[LPW];
#pragma unroll
    for (int q = 0; q < LPW; ++q) {
        const int o16 = ((wave * LPW + q) * 1024 + lane * 16);
        const int lrow = o16 / RB, pch = (o16 % RB) / 16;
        koff[q] = lrow * row_b + (pch ^ swz_k<RB>(lrow)) * 16;
        voff[q] = lrow * row_b + (((pch >> 1) ^ swz_v<RB>(lrow)) * 2 + (pch & 1)) * 16;
    }
    const int nblk = (kend + kKeyBlock - 1) / kKeyBlock;
    auto issue = [&](int j) {
        const uint32_t off = static_cast<uint32_t>(j * kKeyBlock) * row_b;
        const char *lk = s_k[j % kStages] + wave * LPW * 1024;
        const char *lv = s_v[j % kStages] + wave * LPW * 1024;
#pragma unroll
        for (int q = 0; q < LPW; ++q) {
            load_lds16(krs, koff[q] + off, lk + q * 1024);
            load_lds16(vrs, voff[q] + off, lv + q * 1024);
        }
    };
    if (loader) {
#pragma unroll
        for (int j = 0; j < kStages - 1; ++j)
            if (j < nblk) issue(j);
    }

    for (int j = 0; j < nblk; ++j) {
        // this wave's loads of stage j are done once at most the later stages' remain
        wait_later<2 * LPW, kStages - 2>(min(kStages - 2, nblk - 1 - j));   // 2 LPW loads per stage
        lds_barrier();                                      // stage j landed; stage j-1 consumed
        if (loader && j + kStages - 1 < nblk) issue(j + kStages - 1);
        const char *sk = s_k[j % kStages];
        const char *sv = s_v[j % kStages];
        const int k0 = j * kKeyBlock;

        // S^T[key][query] for the block: tile c holds keys 16c + 4g + jj in element jj
        floatx4 st[2];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int row = 16 * c + l16;
            u32x4 kf[DS];
#pragma unroll
            for (int s = 0; s < DS; ++s)
                kf[s] = *reinterpret_cast<const u32x4 *>(sk + row * RB + ((4 * s + g) ^ swz_k<RB>(row)) * 16);
            st[c] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < DS; ++s) st[c] = mfma(kf[s], qf[s], st[c]);
        }
        // online softmax over this block, for the query in this lane's column
        float bm = -INFINITY;
        if (k0 + kKeyBlock <= vis_min) {                     // wave-uniform: no key masked
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    st[c][jj] *= sc;
                    bm = fmaxf(bm, st[c][jj]);
                }
        } else {
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int key = k0 + 16 * c + 4 * g + jj;
                    st[c][jj] = key < vis ? st[c][jj] * sc : -INFINITY;
                    bm = fmaxf(bm, st[c][jj]);
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
        uint32_t pk[2][2];                                   // P^T as bf16 pairs, tile c
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            float pv[4];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                pv[jj] = __builtin_amdgcn_exp2f(st[c][jj] - mm);
                l += pv[jj];
            }
            pk[c][0] = bf16_pair(pv[0], pv[1]);
            pk[c][1] = bf16_pair(pv[2], pv[3]);
        }
        // O^T[d][query] += V^T[d][keys] P^T[keys][query].  The B operand of lane
        // group g holds keys 4g + 0..3 and 16 + 4g + 0..3; the transposing reads give
        // lane (g, d) the same keys of V column d: lane 4k + c of the group addresses
        // key 4g + k (or 16 + 4g + k), values 16t + 4c .. 16t + 4c + 3.
        const u32x4 pb{pk[0][0], pk[0][1], pk[1][0], pk[1][1]};
        const int vr0 = 4 * g + (l16 >> 2), vr1 = vr0 + 16;
        const int vb = 8 * (l16 & 3);
        u32x2 lo[DT], hi[DT];
#pragma unroll
        for (int t = 0; t < DT; ++t) {
            lo[t] = read_tr(sv + vr0 * RB + (t ^ swz_v<RB>(vr0)) * 32 + vb);
            hi[t] = read_tr(sv + vr1 * RB + (t ^ swz_v<RB>(vr1)) * 32 + vb);
        }
        lds_wait(lo, hi);
#pragma unroll
        for (int t = 0; t < DT; ++t) o[t] = mfma(u32x4{lo[t][0], lo[t][1], hi[t][0], hi[t][1]}, pb, o[t]);
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
