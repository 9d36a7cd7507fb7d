// The arbitration head's first layer over every decision slot of a chain batch
// (Section 3.3: the pre-activations U = H W1^T of z = w2 . relu(W1 h + b1) + b2).
//
// The hidden states do not depend on the vocabulary reduction, only the choice of the
// rows the head must score does.  For small batches it is cheaper to score every slot
// than to wait for that choice: these workgroups run in the reduction's own launch,
// beside its units, and the chain finish takes z of the mismatch slots from their
// partials (headz::head_z by decision slot) and ignores the matches'.  The partials
// have the layout of the mismatch-row GEMM's: upart[ks][slot][n], a.ksplit k-slices.
//
// Work: one wave per 16 x 16 tile of U over one k-slice; a workgroup's four waves take
// four adjacent column tiles of the same sixteen slots and slice, so they read the
// same hidden rows.  The operands go from global memory straight to registers (no
// LDS, and few registers, so the reduction units of the same launch keep their
// occupancy).  A chunk is four 64-byte k-steps; lane group g (lanes 16g .. 16g+15)
// loads the 16-byte piece g of each step, of its hidden row and of its W1 row, at
// four offsets from one address, and product q takes step q.  The k-slices, the steps
// and the lanes' pieces are those of the mismatch-row GEMM (head.hip), so for the same
// slice count the partials of a slot are the same numbers in both.  A chunk cut by
// the end of its slice reads a zero vector for the pieces past it.  Workgroup w takes
// k-slice w % ksplit: with ksplit a multiple of the XCD count (workgroups are dealt to
// the XCDs round-robin) each XCD reads only its own slices of W1 and of the hidden
// rows.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "head_z.h"
#include "launch.h"
#include "mfma.h"

namespace cospec {
namespace slotgemm {

constexpr int kWaves = kReduceThreads / 64;   // waves per workgroup (the reduction's)

// Decision slots this form takes at most (its index arithmetic is 32-bit).
constexpr int64_t kMaxSlots = 1 << 20;

// Workgroups for the a.m_cap decision slots of a.
__host__ __device__ inline int64_t blocks(const HeadArgs &a) {
    const int64_t row_tiles = (a.m_cap + 15) / 16;
    const int64_t col_groups = ((a.h + 15) / 16 + kWaves - 1) / kWaves;
    return row_tiles * col_groups * a.ksplit;
}

// Workgroup w of blocks(a).  zero: sixteen zero bytes in device memory, which a lane
// loads instead of an operand piece past the end of its k-slice (branch-free loads).
template <int DT>
__device__ inline void run(const HeadArgs &a, int64_t w, const u32x4 *zero) {
    constexpr int EB = DT == kBF16 ? 2 : 4;
    constexpr int KE = 64 / EB;                  // elements of a 64-byte k-step
    constexpr int VE = 16 / EB;                  // elements of a lane's 16-byte piece
    // 32-bit index arithmetic (the launchers refuse more than kMaxSlots slots): 64-bit
    // divisions cost registers that the reduction units of the launch would lose
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int l16 = lane & 15, g = lane >> 4;
    const int wi = static_cast<int>(w);
    const int ks = wi % a.ksplit;
    const int t = wi / a.ksplit;
    const int m_cap = static_cast<int>(a.m_cap);
    const int row_tiles = (m_cap + 15) / 16;
    const int s0 = (t % row_tiles) * 16;
    const int n0 = (t / row_tiles * kWaves + wave) * 16;
    if (n0 >= a.h) return;                       // a column tile past h (no barrier follows)
    constexpr int CE = 4 * KE;                   // elements of a chunk
    constexpr int BK = 128 / EB;                 // the slices are whole 128-byte stages
    const int kslice = ((a.d + a.ksplit - 1) / a.ksplit + BK - 1) / BK * BK;
    const int k0 = ks * kslice, k1 = min(a.d, k0 + kslice);

    // this lane's operand rows: slot s0 + l16 (past the last slot: the last slot's row,
    // computed and never stored; an invalid hidden row reads row 0, and the second layer
    // sets its z to NaN) and W1 row n0 + l16 (past h: row h - 1, never stored)
    const int s = min(s0 + l16, m_cap - 1);
    int64_t id = a.row0 ? a.row0[s / a.slots] + s % a.slots : s;   // headz::mapped_row
    if (id < 0 || id >= a.n_rows) id = 0;
    const char *pa = static_cast<const char *>(a.hidden) + id * static_cast<int64_t>(a.d) * EB + g * 16;
    const char *pb = static_cast<const char *>(a.w1) + static_cast<int64_t>(min(n0 + l16, a.h - 1)) * a.d * EB + g * 16;

    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    u32x4 av[4], bv[4];
    int kc = k0;
    for (; kc + CE <= k1; kc += CE) {           // whole chunks: one address per operand
        const char *qa = pa + static_cast<int64_t>(kc) * EB;
        const char *qb = pb + static_cast<int64_t>(kc) * EB;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            av[q] = *reinterpret_cast<const u32x4 *>(qa + 64 * q);
            bv[q] = *reinterpret_cast<const u32x4 *>(qb + 64 * q);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) acc = mma<DT>(av[q], bv[q], acc);
    }
    if (kc < k1) {                               // the chunk cut by the end of the slice
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = kc + q * KE + g * VE;  // first element of the piece; d, k1: multiples of VE
            const bool in = e < k1;
            const int64_t off = static_cast<int64_t>(kc) * EB + 64 * q;
            av[q] = *(in ? reinterpret_cast<const u32x4 *>(pa + off) : zero);
            bv[q] = *(in ? reinterpret_cast<const u32x4 *>(pb + off) : zero);
        }
        // steps wholly past the slice add nothing: the mismatch-row GEMM also runs the
        // zero steps of its last stage, and a product of zeros leaves the sum as it is
#pragma unroll
        for (int q = 0; q < 4; ++q) acc = mma<DT>(av[q], bv[q], acc);
    }

    // nontemporal stores: the partials are read once, by the finish
    float *up = a.upart + static_cast<int64_t>(ks) * m_cap * a.h;
    const int n = n0 + l16;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int sr = s0 + 4 * g + j;
        if (sr < m_cap && n < a.h) __builtin_nontemporal_store(acc[j], &up[static_cast<int64_t>(sr) * a.h + n]);
    }
}

}  // namespace slotgemm
}  // namespace cospec
