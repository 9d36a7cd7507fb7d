/*
 * cospec.h -- C ABI of the CoSpec verify-and-arbitrate step for MI355X (gfx950).
 *
 * Method: "Beyond the Target: From Imitation to Collaboration in Speculative
 * Decoding".  In one speculative-decoding round (Section 3.1) the draft model
 * proposes K tokens and the target model scores them in one teacher-forced
 * pass, which gives K+1 next-token rows; with greedy decoding the target's
 * verification token for position i is the argmax of target row i-1 and the
 * mismatch indicator is Delta_i = 1[draft token i == that argmax].  CoSpec
 * (Section 3.3) scores every mismatch with a learned head z_i = g_phi(h_i),
 * accepts the draft token when sigma(z_i) > lambda (Eq. infer_thre; matches are
 * always accepted, Eq. policy-prob), and ends the round at the first rejected
 * mismatch (Eq. cospec_length): it emits the draft tokens before that position
 * and the target token there, or all K draft tokens plus the bonus token.
 *
 * At temperature 1 (Section 3.1, stochastic decoding; Appendix C.3) the target's
 * verification candidate is a sample of softmax(target row) instead of its
 * argmax; the same arbitration rule then applies to the pair.  The library takes
 * that sample by inversion of a caller-supplied uniform (cospec_options).
 *
 * This library computes that step on the GPU from logits, draft tokens,
 * arbitrator hidden states and head weights, and returns accept lengths and the
 * emitted tokens, plus optional per-row and per-decision features.
 *
 * Conventions shared by every entry point
 *  - Array arguments are DEVICE pointers on the current HIP device, owned by the
 *    caller.  The library never allocates, frees or synchronises; all work is
 *    enqueued on `stream` and the call returns before it runs.
 *  - Scratch memory comes from the caller's `workspace` (size from the matching
 *    *_workspace_size function).  Its contents need no initialisation and are
 *    garbage afterwards.  Calls that may overlap in time need distinct workspaces.
 *  - Host structs are read during the call and not retained.  There is no global
 *    mutable state (apart from the static scratch buffer of
 *    cospec_verify_block_static), so the library is reentrant.
 *  - Every argument that lives on the host is checked before anything is
 *    enqueued; an invalid call returns a negative status and enqueues nothing.
 *    Launch failures return COSPEC_ERR_HIP.  No C++ exception crosses the ABI.
 *  - Values that live in device memory (token ids, parent indices, row indices)
 *    cannot be checked on the host.  Out-of-range values never cause an
 *    out-of-bounds access; what they produce is stated per entry point.
 *  - Logits must be finite (a precondition, not checked).
 *  - Row layout: a logit row holds V entries followed by padding up to `ld`
 *    entries; the pointer and ld * element size must be multiples of 16 bytes.
 *  - Head dtype: hidden states, W1, b1 and w2 share head->dtype.
 */
#ifndef COSPEC_H
#define COSPEC_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define COSPEC_ABI_VERSION 5
#define COSPEC_MAX_K 64      /* chain: draft tokens per block              */
#define COSPEC_MAX_N 256     /* tree: nodes per tree, root included        */
#define COSPEC_MAX_SPLITS 64 /* workgroups per logit row (tuning override) */

typedef enum {
    COSPEC_OK = 0,
    COSPEC_ERR_INVALID_ARG = -1,  /* null/misaligned pointer, bad size, NaN lambda ... */
    COSPEC_ERR_UNSUPPORTED = -2,  /* K, N or split count above the documented maximum,
                                     or a logit row (V * element bytes) over 2^31 - 1 B */
    COSPEC_ERR_WORKSPACE = -3,    /* workspace missing, misaligned or too small         */
    COSPEC_ERR_HIP = -4,          /* a HIP call or kernel launch failed                 */
    COSPEC_ERR_SCRATCH_LIMIT = -5 /* cospec_verify_block_static: the sizes need more than
                                     COSPEC_STATIC_SCRATCH_BYTES of scratch             */
} cospec_status;

/* Bytes of the library's static scratch buffer (per GPU), see cospec_verify_block_static. */
#define COSPEC_STATIC_SCRATCH_BYTES (64u << 20)

typedef enum { COSPEC_F32 = 0, COSPEC_BF16 = 1 } cospec_dtype;

/*
 * Arbitration head g_phi (Section 3.3).  The paper gives it no explicit form
 * beyond a small head on the arbitrator's hidden state with one logit out; this
 * library reads it as a two-layer MLP with a ReLU:
 *     z = w2 . max(W1 h + b1, 0) + b2
 * d must be a multiple of 8 (bf16) or 4 (f32); w1 must be 16-byte aligned.
 */
typedef struct {
    int32_t d;            /* hidden size (fan-in)                 */
    int32_t h;            /* inner width                          */
    cospec_dtype dtype;   /* of hidden states, w1, b1 and w2      */
    const void *w1;       /* [h][d] row-major (nn.Linear layout)  */
    const void *b1;       /* [h], or NULL for zeros               */
    const void *w2;       /* [h]                                  */
    float b2;             /* host scalar                          */
} cospec_head;

/*
 * Optional outputs; any member may be NULL.  "Per target row" arrays are
 * [B][K+1] (chain) or [B][N] (tree).  "Per draft row" arrays are [B][K]
 * (chain) or [B][N] (tree; entries of leaf nodes, whose draft rows verify
 * nothing and are not read, are -1 / NaN).  "Per decision" arrays are [B][K]
 * (chain; entry i-1 is decision i) or [B][N] (tree; entry n is the decision on
 * node n; entry 0, the root, reads delta 1, z_tilde +inf, policy 1, accept 1,
 * log-probs NaN).
 */
typedef struct {
    int32_t *tgt_argmax;   /* per target row: first index of the max           */
    float *tgt_max;        /* per target row: max logit                        */
    float *tgt_lse;        /* per target row: log sum exp (log-softmax norm.)  */
    float *tgt_entropy;    /* per target row: Shannon entropy of softmax, nats */
    int32_t *drf_argmax;   /* per draft row, as above                          */
    float *drf_max;
    float *drf_lse;
    float *drf_entropy;
    float *logp_tgt;       /* per decision: log p_T(draft token) (Section 3.4) */
    float *logp_drf;       /* per decision: log p_D(draft token)               */
    uint8_t *delta;        /* per decision: 1 if the draft token matches       */
    float *z_tilde;        /* per decision: head logit, +inf on matches        */
    float *policy;         /* per decision: sigma(z_tilde)                     */
    uint8_t *accept;       /* per decision: a_i (1 on matches)                 */
    int32_t *tgt_candidate; /* per target row: the verification candidate used
                              (the argmax, or the temperature-1 sample)        */
    float *logp_action;    /* per decision: log pi(a_i) of the action taken,
                              log sigma(z) if accepted, log sigma(-z) if not
                              (the rollout-time probability of Section 3.4);
                              0 on matches, NaN where the head did not run or
                              the draft token is invalid                      */
} cospec_features;

/*
 * Per-round statistics of the reinforcement-learning stage (Section 3.4), for
 * chains only.  With decisions i = 1..K, s the round length and Delta, a the
 * mismatch flags and actions:
 *   effective actions  I = {i : Delta_i = 0 and i <= min(s, K)}
 *   first mismatch     i* = min{i : Delta_i = 0}
 *   rho                (s - i*) / ((K+1) - i*)
 *   first rejection    i_rej = min{i : Delta_i = 0 and a_i = 0}, or K+1
 *   S_acc              {i in I : a_i = 1, i < i_rej};  S_rej = {i_rej} if <= K
 *   reward g_i         correct rollout: rho on I; failed rollout
 *                      (Eq. failure_penalty): -alpha |l_i| on S_acc, -beta on
 *                      S_rej, with l_i = log p_T(draft token i)
 *   round return       sum of g over I (the round's share of J)
 * An invalid draft token counts as a rejected mismatch with l_i = NaN.  Every
 * output is optional; `correct` is required when reward or round_return is set.
 */
typedef struct {
    const uint8_t *correct;   /* [B] in: Corr of each sequence's rollout (0 or 1)     */
    float alpha, beta;        /* failure-reward weights (the paper uses 1.0, 0.25)    */
    uint8_t *effective;       /* [B][K] out: 1 if decision i is in I                   */
    uint8_t *in_s_acc;        /* [B][K] out: 1 if decision i is in S_acc               */
    int32_t *first_mismatch;  /* [B] out: i*, or 0 when the round has no mismatch      */
    int32_t *first_reject;    /* [B] out: i_rej (K+1 when no mismatch is rejected)     */
    float *rho;               /* [B] out: rho, NaN when the round has no mismatch      */
    float *reward;            /* [B][K] out: g_i on I, 0 elsewhere                     */
    float *round_return;      /* [B] out: sum of g over I                              */
} cospec_rl;

/*
 * Optional hooks; a NULL options pointer, or zero/NULL members, mean defaults.
 *
 * Order of work inside a verify call: (1) reduce the logit rows, (2) decide
 * (verification tokens, Delta, mismatch list; for chains taken inside the head
 * GEMM, which derives its list, and the finish), (3) the head on the mismatch
 * rows, (4) finish (draft statistics, log p_D, verdicts, first stop, emission).
 * Chain batches of at most 256 decision slots run the head's first layer on
 * every slot inside the reduction's launch instead, and the finish keeps the
 * mismatches' logits (the reduce events then bracket that launch).
 */
typedef struct {
    hipEvent_t reduce_begin;  /* if non-NULL, recorded on `stream` just before ...        */
    hipEvent_t reduce_end;    /* ... and just after the reduction launch                  */
    hipEvent_t reduce2_begin; /* if non-NULL, recorded on `stream` right after reduce_end, */
    hipEvent_t reduce2_end;   /* and this one right after it: an empty interval that
                                 measures what an event pair adds by itself              */
    int32_t splits;           /* workgroups per logit row, 1..COSPEC_MAX_SPLITS; 0 = auto
                                 (one per row for large batches, more for small ones so
                                 that every CU stays busy)                                */
    /*
     * Temperature-1 target candidates.  NULL: the candidate of every target row
     * is its argmax (greedy decoding).  Otherwise a device array with one
     * uniform per target row ([B][K+1] chain, [B][N] tree): the candidate of
     * row r is the smallest v whose cumulative softmax probability
     * p[0] + ... + p[v] exceeds sample_uniform[r] (inversion sampling).  Values
     * below 0 or NaN act as 0, values at or above 1 as the largest float below
     * 1.  Sums are fp32: a uniform within about 1e-5 of a cumulative boundary
     * may select either neighbour.
     */
    const float *sample_uniform;
    /*
     * Sampled arbitration (Section 3.4: rollouts draw mismatch actions from the
     * policy).  NULL: a_i = 1[sigma(z_i) > lambda] (Eq. infer_thre).  Otherwise
     * one uniform per decision ([B][K] chain, [B][N] tree) and a mismatch is
     * accepted when policy_uniform < sigma(z_i) (fp32); lambda is then unused.
     */
    const float *policy_uniform;
    const cospec_rl *rl;      /* chain only: per-round RL statistics, or NULL      */
    /*
     * Packed arbitrator hidden states (for example one row per token of every
     * sequence's input q, Section 3.3).  NULL: `hidden` is [B][K][d] (chain) or
     * [B][N][d] (tree).  Otherwise `hidden` is [hidden_rows][d] and decision
     * slot j of sequence b (chain: decision j+1; tree: node j) reads row
     * hidden_row0[b] + j.  A mismatch whose row falls outside [0, hidden_rows)
     * gets z = NaN and is rejected.
     */
    const int64_t *hidden_row0;
    int64_t hidden_rows;
} cospec_options;

/* COSPEC_ABI_VERSION of the built library. */
int32_t cospec_abi_version(void);

/*
 * Build id of the library: the first 32 hex digits of the SHA-256 of the sources and
 * headers it was compiled from, set by the build ("unknown" if the build set none).
 * Build tooling compares it with the sources on disk to refuse a stale binary.
 */
const char *cospec_build_id(void);

/* Static string naming a status code (never NULL). */
const char *cospec_status_string(int32_t status);

/*
 * Workspace bytes for a step with n_target_rows target rows, n_draft_rows draft rows
 * and n_decisions decision slots over vocabularies of V entries, with the head `head`
 * (NULL: the head does not run, as in cospec_verify_block_sps).  For a chain batch
 * these are B(K+1), BK and BK; for a tree batch BN, BN and BN.  The result equals the
 * matching per-entry query below (0 for negative counts, V < 1 or an invalid head).
 * The workspace must be 256-byte aligned.
 */
size_t cospec_workspace_bytes(int32_t n_target_rows, int32_t n_draft_rows, int32_t n_decisions, int32_t V,
                              const cospec_head *head);

/*
 * Workspace bytes cospec_verify_block needs for these sizes (0 for invalid
 * sizes).  The workspace must be 256-byte aligned.
 */
size_t cospec_verify_block_workspace_size(int32_t B, int32_t K, int32_t V, const cospec_head *head);

/*
 * One chain verify step over B blocks of K draft tokens (Sections 3.1 and 3.3).
 *
 *  target_logits  [B][K+1] rows: row j = target logits after the prefix and
 *                 draft tokens 1..j; row K yields the bonus token.
 *  draft_logits   [B][K] rows: row j = the draft logits token j+1 was drawn from.
 *  logit_dtype, ld  element type of both logit arrays and their row stride in
 *                 elements (ld >= V).
 *  draft_tokens   [B][K] int32, the draft tokens 1..K.
 *  hidden         [B][K][d] arbitrator hidden states; row i-1 feeds decision i.
 *  head, lambda   the head and the acceptance threshold (any non-NaN value;
 *                 lambda >= 1 never accepts a mismatch, lambda < 0 always does).
 *  B >= 0, 0 <= K <= COSPEC_MAX_K, V >= 1.  With K = 0, draft_logits,
 *                 draft_tokens and hidden may be NULL.
 *  accept_len     [B] out: s in [1, K+1] (Eq. cospec_length).
 *  out_tokens     [B][K+1] out: the emitted tokens, then -1.
 *  feats, opts    optional (NULL).
 *
 * A draft token outside [0, V) never matches and is always rejected (its
 * log-probabilities and z are NaN), so it is never emitted.
 */
cospec_status cospec_verify_block(const void *target_logits, const void *draft_logits,
                                  cospec_dtype logit_dtype, int64_t ld,
                                  const int32_t *draft_tokens, const void *hidden,
                                  const cospec_head *head, float lambda, int32_t B, int32_t K,
                                  int32_t V, int32_t *accept_len, int32_t *out_tokens,
                                  const cospec_features *feats, const cospec_options *opts,
                                  void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * cospec_verify_block without a workspace argument, for callers that cannot allocate
 * device memory (code being captured into a HIP graph, tight serving loops, harnesses
 * that forbid allocation): the step's scratch memory is a static buffer of
 * COSPEC_STATIC_SCRATCH_BYTES that the library holds on each GPU it runs on, from
 * when its code object loads until the process ends.  Arguments, results and errors
 * are those of cospec_verify_block, plus:
 *  - COSPEC_ERR_SCRATCH_LIMIT when cospec_verify_block_workspace_size(B, K, V, head)
 *    exceeds COSPEC_STATIC_SCRATCH_BYTES (checked before anything is enqueued);
 *  - COSPEC_ERR_HIP when the buffer's device address cannot be obtained (the first
 *    call on a device looks it up with that device current and keeps it).
 * The call allocates nothing: no hipMalloc, no hipFree, no allocating library routine.
 * Every call on one GPU shares that GPU's buffer, so calls that may overlap in time on
 * one GPU (on different streams, or from different threads) race and must be
 * serialised by the caller; calls in one stream are ordered and safe.  The buffer
 * keeps the last call's contents; the step clears what it needs cleared itself.
 */
cospec_status cospec_verify_block_static(const void *target_logits, const void *draft_logits,
                                         cospec_dtype logit_dtype, int64_t ld,
                                         const int32_t *draft_tokens, const void *hidden,
                                         const cospec_head *head, float lambda, int32_t B, int32_t K,
                                         int32_t V, int32_t *accept_len, int32_t *out_tokens,
                                         const cospec_features *feats, const cospec_options *opts,
                                         hipStream_t stream);

/*
 * The same chain step in two phases, for an arbitrator whose input needs the
 * target's candidates: its input q (Section 3.3) holds the draft tokens next to
 * the target's candidates ytilde_1..K, so its hidden states can only be
 * computed once the target rows are reduced.
 *
 *  phase 1, cospec_verify_block_reduce: the vocabulary reductions, the
 *    candidates, Delta and the mismatch list.  Writes `candidates` ([B][K+1]
 *    int32: the argmax, or the temperature-1 sample, of every target row) and
 *    the features computed there (per target row, delta, logp_tgt).
 *  the caller builds q from the candidates and runs its arbitrator;
 *  phase 2, cospec_verify_block_arbitrate: the head on the mismatch rows, the
 *    verdicts, the first stop, the emission and the remaining features (per
 *    draft row, logp_drf, z_tilde, policy, accept, logp_action, RL statistics).
 *
 * Both phases take the arguments of cospec_verify_block (phase 1 without
 * hidden, lambda and the outputs) with the same values and workspace; the
 * workspace must not be touched between them and phase 2 must be enqueued on a
 * stream ordered after phase 1.  Of the options, phase 1 reads splits (which
 * phase 2 must repeat) and sample_uniform; phase 2 reads policy_uniform, rl and
 * the hidden-row map.  The two phases together
 * give exactly the results of one cospec_verify_block call.
 */
cospec_status cospec_verify_block_reduce(const void *target_logits, const void *draft_logits,
                                         cospec_dtype logit_dtype, int64_t ld,
                                         const int32_t *draft_tokens, const cospec_head *head,
                                         int32_t B, int32_t K, int32_t V, int32_t *candidates,
                                         const cospec_features *feats, const cospec_options *opts,
                                         void *workspace, size_t workspace_bytes, hipStream_t stream);

cospec_status cospec_verify_block_arbitrate(const void *target_logits, const void *draft_logits,
                                            cospec_dtype logit_dtype, int64_t ld,
                                            const int32_t *draft_tokens, const void *hidden,
                                            const cospec_head *head, float lambda, int32_t B, int32_t K,
                                            int32_t V, int32_t *accept_len, int32_t *out_tokens,
                                            const cospec_features *feats, const cospec_options *opts,
                                            void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Standard speculative sampling over B chain blocks: the distribution-
 * preserving baseline the paper compares against at temperature 1 (Section 3.1,
 * stochastic decoding; Appendix C.3), on the same reductions.  Draft token i (drawn by the caller
 * from draft row i-1) is accepted when uniforms[b][i-1] < p_T(token) /
 * p_D(token) (target and draft rows i-1), i.e. with probability min(1, ratio);
 * the round stops at the first rejection s and emits draft tokens 1..s-1, then
 * a sample of max(0, p_T - p_D) (normalised) from rows s-1, or, when all K are
 * accepted, a sample of p_T from target row K; that sample inverts
 * uniforms[b][K] through the distribution's cumulative weights in index order.
 *
 *  uniforms   [B][K+1] float in [0, 1) (device).
 *  accept_len [B] out: s in [1, K+1]; out_tokens [B][K+1] out, -1 after s.
 *  feats      optional: per target row and per draft row statistics, logp_tgt,
 *             logp_drf, accept, and `policy` = min(1, ratio), the acceptance
 *             probability (the other members are not written).
 *  opts       only splits and the four reduction events apply (the second
 *             pair is recorded back to back); any other member is an error.
 * Sums are fp32: a uniform within about 1e-5 (tests: 1e-4) of a boundary may
 * land on the neighbouring outcome.  An invalid draft token is rejected.
 */
size_t cospec_verify_block_sps_workspace_size(int32_t B, int32_t K, int32_t V);

cospec_status cospec_verify_block_sps(const void *target_logits, const void *draft_logits,
                                      cospec_dtype logit_dtype, int64_t ld, const int32_t *draft_tokens,
                                      const float *uniforms, int32_t B, int32_t K, int32_t V,
                                      int32_t *accept_len, int32_t *out_tokens, const cospec_features *feats,
                                      const cospec_options *opts, void *workspace, size_t workspace_bytes,
                                      hipStream_t stream);

/* Workspace bytes cospec_verify_tree needs (0 for invalid sizes). */
size_t cospec_verify_tree_workspace_size(int32_t B, int32_t N, int32_t V, const cospec_head *head);

/*
 * One tree verify step over B token trees of N nodes.  Trees are not in the
 * paper; this applies its chain rule along every root path:
 *  - node 0 is the root (the last verified token) and carries no decision;
 *  - child c of node p is verified against the candidate of target row p
 *    (its argmax, or its temperature-1 sample), its
 *    log-probabilities come from rows p, and its head input is hidden row c;
 *  - a node is reachable when every decision on its root path passes (a match,
 *    or a mismatch whose draft token is accepted); the round accepts the
 *    deepest reachable node n* (ties to the lowest node id) and emits the node
 *    tokens along the path, then the candidate of target row n*.
 * On a path-shaped tree this is exactly the chain rule.
 *
 *  target_logits, draft_logits  [B][N] rows each (row n = distributions after
 *                 node n).  Only draft rows of nodes that have a child are read.
 *  parent         [B][N] int32: parent[0] = -1 and 0 <= parent[n] < n.
 *  node_tokens    [B][N] int32 (entry 0 ignored).
 *  hidden         [B][N][d] (row 0 ignored).
 *  B >= 0, 1 <= N <= COSPEC_MAX_N, V >= 1.
 *  accept_len     [B] out: depth(n*) + 1.
 *  out_tokens     [B][N] out: path tokens then the candidate of target row
 *                 n*, then -1.
 *  out_path       [B][N] out, nullable: node ids 0..n* along the path, then -1.
 *
 * A node whose parent index breaks 0 <= parent[n] < n, or whose token is
 * outside [0, V), fails its decision (it and its subtree are unreachable).
 */
cospec_status cospec_verify_tree(const void *target_logits, const void *draft_logits,
                                 cospec_dtype logit_dtype, int64_t ld, const int32_t *parent,
                                 const int32_t *node_tokens, const void *hidden,
                                 const cospec_head *head, float lambda, int32_t B, int32_t N,
                                 int32_t V, int32_t *accept_len, int32_t *out_tokens,
                                 int32_t *out_path, const cospec_features *feats,
                                 const cospec_options *opts, void *workspace,
                                 size_t workspace_bytes, hipStream_t stream);

/*
 * The arbitrator's hybrid attention (Section 3.3).  The arbitrator reads
 * q = [context, SEP, draft 1..K, SEP, candidates 1..K, SEP] (Eq. arb_input),
 * l = l_c + 2K + 3 positions, under a hybrid mask: context positions attend
 * causally within the context; the draft/target region (read as starting at the
 * first SEP, position l_c) attends to the whole context and bidirectionally
 * within itself; nothing flows from the region back into the context.
 *
 * cospec_hybrid_mask writes that mask: mask[b][i][j] = 1 when position i of
 * sequence b may attend position j, else 0, for a batch padded to L positions;
 * padding positions (i >= l) attend only to themselves.
 *  ctx_len  [B] int32, l_c of each sequence (negative values act as 0).
 *  mask     [B][L][L] uint8 out.
 */
cospec_status cospec_hybrid_mask(const int32_t *ctx_len, int32_t B, int32_t K, int32_t L, uint8_t *mask,
                                 hipStream_t stream);

/*
 * cospec_hybrid_attention: softmax(q k^T * scale + mask) v under the hybrid
 * mask, computed from the rule (no mask array), for n_q consecutive query
 * positions q_start[b] .. q_start[b] + n_q - 1 of each sequence.  Per round the
 * region's 2K+3 positions (q_start = l_c) are the new queries; their keys and
 * values are the cached context plus the region.
 *  q        [B][n_q][Hq][D] bf16;  k, v  [B][L][Hkv][D] bf16, positions 0..L-1.
 *  Hq a multiple of Hkv (query head h reads key/value head h / (Hq / Hkv));
 *  D 64 or 128; pointers 16-byte aligned.
 *  out      [B][n_q][Hq][D] bf16.  A query at a position outside [0, l) gets
 *           zeros; keys at positions >= L do not exist (l is clamped to L).
 * bf16 inputs, fp32 accumulation; the attention weights enter the second
 * product rounded to bf16.
 */
cospec_status cospec_hybrid_attention(const void *q, const void *k, const void *v, const int32_t *ctx_len,
                                      const int32_t *q_start, int32_t B, int32_t n_q, int32_t L, int32_t Hq,
                                      int32_t Hkv, int32_t D, int32_t K, float scale, void *out,
                                      hipStream_t stream);

/* Workspace bytes cospec_arbitrate needs (0 for invalid sizes). */
size_t cospec_arbitrate_workspace_size(int64_t n_sel, const cospec_head *head);

/*
 * The head alone (Section 3.3): for k < n_sel, with r = row_index[k] (or k when
 * row_index is NULL), out_z[k] = g_phi(hidden row r) and out_accept[k] =
 * 1[sigma(out_z[k]) > lambda] (Eq. infer_thre; no match override here).
 *  hidden     [n_rows][d];  row_index [n_sel] int32 or NULL (then n_sel <= n_rows).
 *  out_z      [n_sel] float; out_accept [n_sel] uint8 (either may be NULL).
 * An index outside [0, n_rows) gives z = NaN and accept 0.
 */
cospec_status cospec_arbitrate(const void *hidden, int64_t n_rows, const int32_t *row_index,
                               int64_t n_sel, const cospec_head *head, float lambda, float *out_z,
                               uint8_t *out_accept, void *workspace, size_t workspace_bytes,
                               hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* COSPEC_H */
