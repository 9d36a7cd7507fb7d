// Internal interface between the C ABI (cospec_api.hip) and the kernel files.
// Not installed; the public interface is include/cospec.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cospec {

constexpr int kReduceThreads = 256;   // vocabulary-reduction workgroup
constexpr int kDecideThreads = 256;   // one workgroup per sequence / tree
constexpr int kHeadTileM = 128;       // head GEMM workgroup tile: rows
constexpr int kHeadTileN = 128;       //                            columns of W1
// small heads: k-slices are added (in steps of the XCD count) until the active grid
// reaches this (128 against 64: the serving chain batch, 4 x 2 tiles, 65.1 -> 63.6 us
// per step; 256 gained less and cost the large chain batch 0.5 us)
constexpr int kHeadTargetBlocks = 128;
constexpr int kHeadMaxSplit = 32;
constexpr int kXcds = 8;             // MI355X: 8 XCDs, each with its own L2
constexpr int kMaxSeqRows = 256;      // rows per sequence / nodes per tree held in LDS
constexpr int kSegVecs = 64;          // 16-byte vectors per probability-mass segment (one wave load)
constexpr int kMaxReduceSlots = 4096; // cap on the resident reduction workgroups the split rule assumes

enum Dtype : int32_t { kF32 = 0, kBF16 = 1 };

// Per-decision state byte written by the decide step.
enum : uint8_t { kStateMismatch = 0, kStateMatch = 1, kStateReject = 2 };

// Where the split partials of the logit rows are.  Rows are numbered target rows
// first (0 .. n_tgt_rows-1), then draft rows; every row is cut into `splits` pieces of
// equal length (one workgroup each) and row r's partials are slots r * splits ..
// r * splits + splits - 1, so a sequence's rows' partials are consecutive slots too.
struct PartPlan {
    int32_t splits;
    int64_t n_tgt_rows;
};

struct RowParts {
    int64_t first;
    int32_t count;
};

__host__ __device__ inline RowParts row_parts(const PartPlan &p, int64_t r) {
    return RowParts{r * p.splits, p.splits};
}

// The partials of rows [r0, r1): consecutive slots.
__host__ __device__ inline RowParts rows_parts(const PartPlan &p, int64_t r0, int64_t r1) {
    return RowParts{r0 * p.splits, static_cast<int32_t>((r1 - r0) * p.splits)};
}

struct DecideArgs {
    const char *tgt;
    int64_t ld_bytes;
    int32_t V;
    int32_t B;
    int32_t RT;                // target rows per sequence (K+1 or N)
    int32_t D;                 // decision slots per sequence (K, or N with the root); <= 256
    int32_t is_tree;
    const int32_t *parent;     // tree only
    const int32_t *tokens;     // chain [B][K], tree [B][N]
    const float4 *partials;
    PartPlan plan;
    int32_t score_mismatch;    // compact mismatches for the head
    int32_t sampled;           // ws_tgt_arg already holds the candidates (k_sample)
    int32_t *tgt_argmax; float *tgt_max; float *tgt_lse; float *tgt_ent; int32_t *tgt_cand;
    float *logp_tgt; uint8_t *delta;
    float *ws_logp_tgt;        // [B*D] log p_T(draft token), kept for the finish kernel
    int32_t *ws_tgt_arg;       // [B*RT] verification candidate per target row
    uint8_t *ws_state;         // [B*D]
    int32_t *ws_listpos;       // [B*D] position in the compacted list or -1
    int32_t *ws_list;          // [B*D] compacted hidden-row ids
    int32_t *ws_count;         // compacted length M
};

struct ReduceArgs {
    const char *tgt;           // target rows
    const char *drf;           // draft rows
    int64_t ld_bytes;          // row stride in bytes (multiple of 16)
    int32_t V;
    int32_t n_tgt_rows;        // B * target rows per sequence; rows past it are draft rows
    int32_t n_rows;            // rows of the launch (target rows, then draft rows)
    const int32_t *parent;     // tree: [B][N]; draft rows of leaves are skipped
    int32_t N;                 // tree nodes per tree
    PartPlan plan;
    int32_t vec_per_split;     // 16-byte vectors per split
    float4 *partials;          // {max, argmax bits, S, T} per piece
    int32_t *reset_counter;    // zeroed by workgroup 0 (the decide step's list counter), or null
    float2 *seg;               // [n_tgt_rows][nseg] {mass, reference} of each segment of a
                               // target row, or null; needs vec_per_split % kSegVecs == 0
    int32_t nseg;              // segments per row: ceil(vectors / kSegVecs) + (tail ? 1 : 0)
    // chains, or null: xtok[row] = the row's logit at its draft token (target row
    // b*(K+1)+i and draft row b*K+i: token b*K+i; target row b*(K+1)+K: none), stored
    // by the piece whose range holds it, when the token is in [0, V)
    const int32_t *chain_tokens;
    int32_t K;
    float *xtok;
};

// Temperature-1 candidates: one wave per target row inverts its uniform through
// the segment masses, then through the elements of the segment it lands in.
struct SampleArgs {
    const char *tgt;
    int64_t ld_bytes;
    int32_t V;
    int32_t n_rows;            // target rows
    const float4 *partials;
    PartPlan plan;
    const float2 *seg;
    int32_t nseg;
    const float *uniform;      // [n_rows]
    int32_t *cand;             // [n_rows] out
};


struct HeadArgs {
    const void *hidden;        // [n_rows][d]
    int64_t n_rows;
    const int32_t *list;       // selected rows, or null = identity
    const int64_t *row0;       // packed hidden states: entry e of the list reads row
                               // row0[e / slots] + e % slots, or null (row e)
    int32_t slots;
    int32_t *count_dev;        // M on the device, or null (the persistent GEMM that builds
                               // its list stores M there, for the second layer)
    int64_t count_host;        // M when count_dev is null
    int64_t m_cap;             // capacity of the list (rows of upart and z)
    const void *w1; const void *b1; const void *w2;
    float b2;
    int32_t d, h;
    int32_t ksplit;            // slices of d, one workgroup each (head_ksplit); the
                               // persistent form may use fewer (headz::live_ksplit)
    int32_t grid;              // chains: workgroups of the persistent GEMM (at most one per
                               // resident slot); 0: one workgroup per (tile, k-slice)
    int32_t two_per_cu;        // use the shallow LDS ring: two workgroups fit on a CU
    float *upart;              // [ksplit][m_cap][h] partial pre-activations
    float *z;                  // [m_cap] head logits of the selected rows
    // chains: upart row of a selected row = its decision slot b*K + i (the list entry),
    // not its list position, so that the finish finds it without the list
    int32_t out_by_slot;
    // chains: the list is derived in every workgroup from the reduction's partials
    // instead of read: the decision slots b*K + i (i < K, m_cap = B*K of them) whose
    // valid draft token differs from the candidate of target row b*(K+1) + i, in slot
    // order, M of them
    int32_t build_list;
    const float4 *partials;
    PartPlan plan;
    const int32_t *tokens;     // [B][K] draft tokens
    const int32_t *cand;       // [B][K+1] candidates already taken (temperature-1 samples, or
                               // a split step's first phase), or null: the argmax
    int32_t K, V;
};

// build_list: at most this many decision slots (eight per thread of a GEMM workgroup)
constexpr int kBuildListMax = 4096;

// Finish: draft-row statistics, log p_D, verdicts, first stop, emission.
struct FinishArgs {
    const char *drf;
    int64_t ld_bytes;
    int32_t V;
    int32_t B;
    int32_t RT, RD, D;         // target rows, draft rows, decision slots per sequence
    int32_t is_tree;
    const int32_t *parent;     // tree only
    const int32_t *tokens;     // chain [B][K], tree [B][N]
    const float4 *partials;    // split partials; draft row j is row n_tgt_rows + j of the plan
    PartPlan plan;
    const uint8_t *ws_state;
    const int32_t *ws_listpos;
    const float *z;            // head logits by compacted position
    int32_t head_ran;
    float lambda;
    const float *policy_u;     // [B*D] uniforms of sampled arbitration, or null (threshold)
    const float *ws_logp_tgt;  // [B*D]
    // chain RL statistics (all optional)
    int32_t rl_on;
    const uint8_t *rl_correct; float rl_alpha, rl_beta;
    uint8_t *rl_effective; uint8_t *rl_s_acc; int32_t *rl_first_mismatch; int32_t *rl_first_reject;
    float *rl_rho; float *rl_reward; float *rl_return;
    float *logp_action;
    const int32_t *ws_tgt_arg;
    int32_t *accept_len; int32_t *out_tokens; int32_t *out_path;
    // chains: the decision step is taken in the finish (lane j merges target row j, the
    // row that verifies decision j+1); `sampled`: take the candidates from ws_tgt_arg
    // (temperature-1 samples, or what a split step's first phase stored) instead of the
    // merged argmax; ws_xtok: the logit at each row's token, which the reduction
    // stored (ReduceArgs::xtok)
    const float *ws_xtok;
    int32_t sampled;
    int32_t *tgt_argmax; float *tgt_max; float *tgt_lse; float *tgt_ent; int32_t *tgt_cand;
    uint8_t *delta; float *logp_tgt;
    int32_t *drf_argmax; float *drf_max; float *drf_lse; float *drf_ent; float *logp_drf;
    float *z_tilde; float *policy; uint8_t *accept;
    // chain only: the head's second layer is computed here from its k-slice partials
    // (hd, head dtype head_dt) instead of being read from z
    int32_t fuse_head;
    int32_t head_dt;
    HeadArgs hd;
    // chain only: the first layer ran over every decision slot (hd.ksplit slices, in the
    // reduction's launch), not over the mismatch list of the persistent GEMM
    int32_t head_every_slot;
};

// Speculative sampling baseline (k_sps_finish, k_sps_mass, k_sps_pick).
struct SpsArgs {
    const char *tgt, *drf;
    int64_t ld_bytes;
    int32_t V, B, K;
    const int32_t *tokens;     // [B][K]
    const float *uniform;      // [B][K+1]: K acceptance tests, then the last token's draw
    const float4 *partials;
    PartPlan plan;             // draft row j is row B * (K+1) + j
    const uint8_t *ws_state;   // decide's state (invalid tokens are rejected)
    const float *ws_logp_tgt;
    float *seg_mass;           // [B][nseg] weights of the last token's distribution
    int32_t nseg;
    int32_t *accept_len; int32_t *out_tokens;
    int32_t *drf_argmax; float *drf_max; float *drf_lse; float *drf_ent; float *logp_drf;
    float *accept_prob; uint8_t *accept;
};

// The arbitrator's hybrid mask and attention (attention.hip).
struct MaskArgs {
    const int32_t *ctx_len;    // [B]
    int32_t B, K, L;
    uint8_t *mask;             // [B][L][L]
};

struct AttnArgs {
    const void *q, *k, *v;     // q [B][n_q][Hq][D], k and v [B][L][Hkv][D], bf16
    const int32_t *ctx_len, *q_start;
    int32_t B, n_q, L, Hq, Hkv, D, K;
    float scale;
    void *out;                 // [B][n_q][Hq][D] bf16
};

struct ArbFinishArgs {
    int64_t n_sel, n_rows;
    const int32_t *row_index;
    const float *z;
    float lambda;
    float *out_z; uint8_t *out_accept;
};

hipError_t launch_reduce(Dtype dt, const ReduceArgs &a, hipStream_t s);
// The reduction with the head's first layer over all h.m_cap decision slots in the same
// launch (chains; h.upart by slot, h.ksplit slices; logit dtype dt, head dtype hdt).
hipError_t launch_reduce_head(Dtype dt, Dtype hdt, const ReduceArgs &a, const HeadArgs &h, hipStream_t s);
int32_t reduce_slots(Dtype dt);   // reduction workgroups resident at once on the current device
hipError_t launch_sample(Dtype dt, const SampleArgs &a, hipStream_t s);
hipError_t launch_decide(Dtype dt, const DecideArgs &a, hipStream_t s);
int32_t head_ksplit(int64_t m_cap, int32_t d, int32_t h, int32_t elem_bytes);
hipError_t launch_head(Dtype dt, const HeadArgs &a, hipStream_t s);   // GEMM + epilogue
hipError_t launch_head_gemm(Dtype dt, const HeadArgs &a, hipStream_t s);
// The first layer over all a.m_cap decision slots on its own (slot_gemm.h).
hipError_t launch_slot_gemm(Dtype dt, const HeadArgs &a, hipStream_t s);
// Resident workgroups of the persistent head GEMM on the current device (cached).
int32_t head_gemm_slots(Dtype dt, bool build);   // GEMM only
hipError_t launch_finish(Dtype dt, const FinishArgs &a, hipStream_t s);
hipError_t launch_arb_finish(const ArbFinishArgs &a, hipStream_t s);
hipError_t launch_sps(Dtype dt, const SpsArgs &a, hipStream_t s);   // finish, weights, pick
hipError_t launch_hybrid_mask(const MaskArgs &a, hipStream_t s);
hipError_t launch_hybrid_attention(const AttnArgs &a, hipStream_t s);

}  // namespace cospec
