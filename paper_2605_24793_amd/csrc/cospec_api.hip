// C ABI of the verify-and-arbitrate step: host-side validation, workspace
// carving and the launch sequence.  Declared in include/cospec.h.
//
// verify_block / verify_tree enqueue, on the caller's stream:
//   1. k_vocab_reduce   every target and draft row (tree: draft rows of nodes with
//                       a child), one workgroup per (row, split) -> split partials
//                       (max, argmax, S, T); zeroes the list counter
//   1b. k_sample        temperature 1 only: one wave per target row samples the
//                       candidate by inversion of its uniform (segment masses
//                       written by step 1, then one segment re-read)
//   2. k_decide         trees (and the first phase of a split chain step): one
//                       workgroup per tree: target statistics, Delta, log p_T, mismatch
//                       compaction (device-side count M)
//   3. k_head_gemm (+ k_head_epilogue for trees)   MFMA head over the M compacted
//                       rows (skipped when the threshold decides every mismatch by
//                       itself and no score is requested); for chains each workgroup
//                       derives the mismatch list itself from the partials
//   4. k_chain_finish(_head) / k_tree_finish   chains: the decision step (target
//                       statistics, Delta, log p_T); draft statistics, log p_D, the
//                       head's second layer (chains), verdicts (threshold or sampled),
//                       first stop, emission, and for chains the optional per-round RL
//                       statistics
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "cospec.h"
#include "launch.h"


// Scratch memory of cospec_verify_block_static: a file-scope device array, so that
// entry point needs no workspace from its caller and allocates nothing.  Each GPU the
// library runs on holds its own copy, from when the code object is loaded until the
// process ends.  In host code `scratch` names a host-side stand-in, not the device
// address: host code only ever uses the address hipGetSymbolAddress returns for the
// current device (static_scratch() below).
static __device__ __align__(256) char scratch[COSPEC_STATIC_SCRATCH_BYTES];

using namespace cospec;

namespace {

constexpr size_t kAlign = 256;
constexpr int64_t kMinPartialSlots = 16384;   // room for a split override on small batches
constexpr int64_t kMaxRowBytes = INT32_MAX;    // V * element bytes of one logit row
// Chain batches with at most this many decision slots run the head's first layer on
// every slot (slot_gemm.h) rather than on the mismatch rows after the reduction, in at
// most kEverySlotSplits k-slices (fewer partials for the finish to add; the slot GEMM's
// extra k-steps hide behind the reduction).  Measured on MI355X, step times: B=8 K=5
// (40 slots, d=4096, h=256) 24.5 us on the mismatch rows, 16.6 us on every slot with 32
// slices, 14.1 with 16, 14.4 with 8; B=1 K=4 (fp32 head, d=512) 19.0 -> 10.5 us; B=64
// K=7 (448 slots) 65.6 us on the mismatch rows, 66.8 on every slot.
constexpr int64_t kEverySlotMax = 256;
constexpr int32_t kEverySlotSplits = 16;

inline size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

inline bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

inline int elem_bytes(cospec_dtype t) { return t == COSPEC_BF16 ? 2 : 4; }

inline bool dtype_ok(cospec_dtype t) { return t == COSPEC_F32 || t == COSPEC_BF16; }

cospec_status check_head(const cospec_head *hd) {
    if (!hd || !dtype_ok(hd->dtype) || hd->d <= 0 || hd->h <= 0 || !hd->w1 || !hd->w2)
        return COSPEC_ERR_INVALID_ARG;
    const int eb = elem_bytes(hd->dtype);
    if ((static_cast<int64_t>(hd->d) * eb) % 16 != 0 || !aligned(hd->w1, 16) || !aligned(hd->w2, eb) ||
        (hd->b1 && !aligned(hd->b1, eb)))
        return COSPEC_ERR_INVALID_ARG;
    return COSPEC_OK;
}

inline int32_t ksplit_for(int64_t m_cap, const cospec_head *hd) {
    return hd ? head_ksplit(m_cap, hd->d, hd->h, elem_bytes(hd->dtype)) : 0;   // no head: no scratch
}

// Head scratch: k-slice partial pre-activations and the logits.
inline size_t head_bytes(int64_t m_cap, const cospec_head *hd) {
    return round_up(static_cast<size_t>(ksplit_for(m_cap, hd)) * static_cast<size_t>(m_cap) *
                    static_cast<size_t>(hd->h) * 4) +
           round_up(static_cast<size_t>(m_cap) * 4);
}

// Workspace carving shared by the size query and the call.
struct Layout {
    size_t partials, seg, tgt_arg, state, listpos, list, count, logp, xtok, upart, z, total;
    int64_t partial_slots;
};

// Probability-mass segments of one logit row for temperature-1 sampling: one per
// kSegVecs 16-byte vectors, plus one for the elements past the last whole vector.
inline int64_t n_segments(int32_t V, int eb) {
    const int64_t nvec = static_cast<int64_t>(V) * eb / 16;
    const int64_t tail = V - nvec * (16 / eb);
    return (nvec + kSegVecs - 1) / kSegVecs + (tail > 0 ? 1 : 0);
}

// The size queries do not know the logit dtype: reserve for the larger count.
inline int64_t n_segments_any(int32_t V) {
    const int64_t a = n_segments(V, 2), b = n_segments(V, 4);
    return a > b ? a : b;
}

// rows = all logit rows; B*RT target rows; B*D decision slots (the sizes depend on
// these three counts alone, which cospec_workspace_bytes relies on).  The partial slots
// hold what the automatic split rule can ask for (rows * splits <= 4 * slots + rows / 2
// when it splits at all, slots <= kMaxReduceSlots) and, on small batches, a split
// override.
Layout layout(int64_t rows, int64_t B, int64_t RT, int64_t D, const cospec_head *hd, int32_t V) {
    Layout L{};
    const int64_t auto_slots = rows + 4 * static_cast<int64_t>(kMaxReduceSlots);
    L.partial_slots = auto_slots > kMinPartialSlots ? auto_slots : kMinPartialSlots;
    size_t off = 0;
    L.partials = off; off += round_up(static_cast<size_t>(L.partial_slots) * 16);
    L.seg = off;      off += round_up(static_cast<size_t>(B * RT) * static_cast<size_t>(n_segments_any(V)) * 8);
    L.tgt_arg = off;  off += round_up(static_cast<size_t>(B * RT) * 4);
    L.state = off;    off += round_up(static_cast<size_t>(B * D));
    L.listpos = off;  off += round_up(static_cast<size_t>(B * D) * 4);
    L.list = off;     off += round_up(static_cast<size_t>(B * D) * 4);
    L.count = off;    off += kAlign;
    L.logp = off;     off += round_up(static_cast<size_t>(B * D) * 4);
    L.xtok = off;     off += round_up(static_cast<size_t>(rows) * 4);
    const int64_t m_cap = B * D;
    L.upart = off;    off += hd ? round_up(static_cast<size_t>(ksplit_for(m_cap, hd)) * static_cast<size_t>(m_cap) *
                                           static_cast<size_t>(hd->h) * 4) : 0;
    L.z = off;        off += round_up(static_cast<size_t>(m_cap) * 4);
    L.total = off;
    return L;
}

// Compute units of the current device (MI355X: 256).
int32_t cu_count() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        return 256;
    return cus;
}

// Splits per row when the caller gives none, from the rows of the launch, the 16-byte
// vectors of a row and the reduction workgroups the device holds at once (`slots`):
//  - at least 1.5 rounds of whole rows (the large batches): one workgroup per row, the
//    cheapest merge and the fewest partials (the large chain batch: 3840 rows on 2048
//    slots, one split 85.6% of the HBM peak, two 84.9%, three 83.8%);
//  - fewer rows: about four rounds of pieces, so that every slot stays busy and the
//    last round is short (the peaked chain batch, 960 rows: one split 82%, nine 86%),
//    but at least four vectors per lane, so every lane keeps its loads in flight (the
//    small chain batch's reduction 4.8 us at 15 splits against 9.9 us at 62; the tiny
//    chain's 1.2 against 2.4 us at 8 and 4 splits).
int32_t auto_splits(int64_t rows, int64_t nvec, int64_t slots) {
    if (rows <= 0) return 1;
    if (2 * rows >= 3 * slots) return 1;
    int64_t s = (4 * slots + rows / 2) / rows;
    const int64_t by_len = nvec / (4 * kReduceThreads);
    if (s > by_len) s = by_len;
    if (s > COSPEC_MAX_SPLITS) s = COSPEC_MAX_SPLITS;
    if (s < 1) s = 1;
    return static_cast<int32_t>(s);
}

// 16-byte vectors per split piece: whole 256-byte blocks, so that every piece of a
// 256-byte aligned row starts on one (measured on MI355X: a plain streaming read of
// 1.17 GB in 256-byte aligned pieces runs at 88% of peak, in pieces aligned to 16 to
// 64 bytes at 81-85%); with temperature-1 segments, whole segments.  Rounding up can
// leave the last pieces without vectors; their partials carry S = 0, which the merges
// skip.
int64_t split_vectors(int64_t nvec, int32_t splits, bool segments) {
    const int64_t unit = segments ? kSegVecs : 16;
    const int64_t vps = (nvec + splits - 1) / splits;
    return (vps + unit - 1) / unit * unit;
}

// The partial layout of a step: the caller's split count, or the rule above.  Both
// phases of a split step derive it from the same arguments.
PartPlan make_plan(int64_t n_tgt_rows, int64_t n_drf_rows, int64_t nvec, int32_t override_splits, Dtype dt) {
    PartPlan p{};
    p.n_tgt_rows = n_tgt_rows;
    p.splits = override_splits > 0 ? override_splits : auto_splits(n_tgt_rows + n_drf_rows, nvec, reduce_slots(dt));
    return p;
}

bool feats_aligned(const cospec_features *f) {
    if (!f) return true;
    const void *p4[] = {f->tgt_argmax, f->tgt_max, f->tgt_lse, f->tgt_entropy, f->drf_argmax, f->drf_max,
                        f->drf_lse, f->drf_entropy, f->logp_tgt, f->logp_drf, f->z_tilde, f->policy,
                        f->tgt_candidate, f->logp_action};
    for (const void *p : p4)
        if (p && !aligned(p, 4)) return false;
    return true;
}

struct Common {
    const void *tgt, *drf;
    cospec_dtype dt;
    int64_t ld;
    const void *hidden;
    const cospec_head *head;
    float lambda;
    int32_t B, V;
    int64_t RT, RD, D;          // per sequence
    int is_tree;
    const int32_t *parent, *tokens;
    const cospec_features *feats;
    const cospec_options *opts;
    void *ws;
    size_t ws_bytes;
    hipStream_t stream;
};

// Which part of the step a call enqueues: the whole step, or one of the two
// phases of the split form (reductions + decide, then head + finish).
enum Phase { kWhole, kReducePhase, kArbitratePhase };

cospec_status run(const Common &c, Phase phase, int32_t *accept_len, int32_t *out_tokens,
                  int32_t *out_path) {
    const int eb = elem_bytes(c.dt);
    const int64_t n_tgt = static_cast<int64_t>(c.B) * c.RT, n_drf = static_cast<int64_t>(c.B) * c.RD;
    const int64_t rows = n_tgt + n_drf;
    const int64_t nvec = static_cast<int64_t>(c.V) * eb / 16;
    int32_t override_splits = 0;
    if (c.opts && c.opts->splits) {
        if (c.opts->splits < 0 || c.opts->splits > COSPEC_MAX_SPLITS) return COSPEC_ERR_UNSUPPORTED;
        override_splits = c.opts->splits;
    }
    const Layout L = layout(rows, c.B, c.RT, c.D, c.head, c.V);
    const float *uniform = c.opts ? c.opts->sample_uniform : nullptr;
    const PartPlan plan = make_plan(n_tgt, n_drf, nvec, override_splits, static_cast<Dtype>(c.dt));
    if (uniform && !aligned(uniform, 4)) return COSPEC_ERR_INVALID_ARG;
    const float *policy_u = c.opts ? c.opts->policy_uniform : nullptr;
    if (policy_u && !aligned(policy_u, 4)) return COSPEC_ERR_INVALID_ARG;
    const cospec_rl *rl = c.opts ? c.opts->rl : nullptr;
    if (rl) {
        if (c.is_tree) return COSPEC_ERR_INVALID_ARG;          // defined for chains only
        if ((rl->reward || rl->round_return) && !rl->correct) return COSPEC_ERR_INVALID_ARG;
        const void *p4[] = {rl->first_mismatch, rl->first_reject, rl->rho, rl->reward, rl->round_return};
        for (const void *p : p4)
            if (p && !aligned(p, 4)) return COSPEC_ERR_INVALID_ARG;
    }
    if (rows * plan.splits > L.partial_slots || rows * plan.splits > INT32_MAX) return COSPEC_ERR_UNSUPPORTED;
    if (!c.ws || !aligned(c.ws, kAlign) || c.ws_bytes < L.total) return COSPEC_ERR_WORKSPACE;
    const int64_t *hidden_row0 = c.opts ? c.opts->hidden_row0 : nullptr;
    const int64_t hidden_rows = hidden_row0 ? c.opts->hidden_rows : static_cast<int64_t>(c.B) * c.D;
    if (hidden_row0 && (!aligned(hidden_row0, 8) || hidden_rows < 0)) return COSPEC_ERR_INVALID_ARG;

    char *ws = static_cast<char *>(c.ws);
    float4 *partials = reinterpret_cast<float4 *>(ws + L.partials);
    float2 *seg = reinterpret_cast<float2 *>(ws + L.seg);
    int32_t *tgt_arg = reinterpret_cast<int32_t *>(ws + L.tgt_arg);
    uint8_t *state = reinterpret_cast<uint8_t *>(ws + L.state);
    int32_t *listpos = reinterpret_cast<int32_t *>(ws + L.listpos);
    int32_t *list = reinterpret_cast<int32_t *>(ws + L.list);
    int32_t *count = reinterpret_cast<int32_t *>(ws + L.count);
    float *ws_logp = reinterpret_cast<float *>(ws + L.logp);
    float *upart = reinterpret_cast<float *>(ws + L.upart);
    float *zlog = reinterpret_cast<float *>(ws + L.z);
    float *xtok = reinterpret_cast<float *>(ws + L.xtok);

    const cospec_features F = c.feats ? *c.feats : cospec_features{};
    const bool decisions = c.B > 0 && (c.is_tree ? c.D > 1 : c.D > 0);
    const bool lambda_decides = !(c.lambda >= 0.0f && c.lambda < 1.0f);
    const bool want_scores = F.z_tilde || F.policy || F.logp_action;
    const bool head = decisions && (!lambda_decides || want_scores || policy_u);
    const bool do_reduce = phase != kArbitratePhase, do_arbitrate = phase != kReducePhase;
    // chains: the head GEMM's workgroups derive the mismatch list from the partials
    const bool build_list = !c.is_tree && static_cast<int64_t>(c.B) * c.D <= kBuildListMax;
    // the candidates are in the workspace when k_sample drew them, and in the second
    // phase of a split step (the first phase's decision step stored them, argmax or sample)
    const bool cand_in_ws = uniform != nullptr || phase == kArbitratePhase;
    const Dtype dt = static_cast<Dtype>(c.dt);
    auto record = [&](hipEvent_t ev) { return !ev || hipEventRecord(ev, c.stream) == hipSuccess; };

    // the head; for chains the finish computes its second layer (the logits of each
    // sequence's mismatches) itself, and the GEMM's workgroups derive the mismatch list
    // (or read the decide kernel's) and run on the M listed rows only
    const int64_t m_cap = static_cast<int64_t>(c.B) * c.D;
    const bool fuse_head = head && !c.is_tree;
    // small chain batches: the first layer runs on every decision slot (slot_gemm.h), in
    // the reduction's launch for a whole step and on its own in the second phase of a
    // split one, instead of on the mismatch rows after the reduction (both forms of the
    // step then compute z alike)
    const bool every_slot = fuse_head && phase != kReducePhase && m_cap <= kEverySlotMax;
    HeadArgs ha{};
    if (head) {
        // no hidden rows at all (a packed array of none): every z is NaN, and the GEMMs'
        // clamped operand loads read W1's first row (valid memory of d elements) instead
        ha.hidden = hidden_rows > 0 ? c.hidden : c.head->w1;
        ha.n_rows = hidden_rows;
        ha.row0 = hidden_row0;
        ha.slots = static_cast<int32_t>(c.D);
        ha.list = list;
        ha.count_dev = count;
        ha.count_host = 0;
        ha.m_cap = m_cap;
        ha.w1 = c.head->w1; ha.b1 = c.head->b1; ha.w2 = c.head->w2; ha.b2 = c.head->b2;
        ha.d = c.head->d; ha.h = c.head->h;
        ha.ksplit = ksplit_for(m_cap, c.head);
        if (every_slot && ha.ksplit > kEverySlotSplits) ha.ksplit = kEverySlotSplits;
        // Trees mismatch most of their slots (about 60% on the 64-tree batch: 304
        // workgroups at 8 k-slices), more than one workgroup per CU: the shallow ring
        // lets two share a CU and finish in one round (19.9 -> 13.8 us there).
        ha.two_per_cu = c.is_tree;
        ha.upart = upart;
        ha.z = zlog;
        if (!c.is_tree) {           // chains: persistent GEMM, partials by decision slot
            const int64_t nt = (ha.h + kHeadTileN - 1) / kHeadTileN;
            const int64_t items = (m_cap + kHeadTileM - 1) / kHeadTileM * nt * ha.ksplit;
            const int64_t slots = head_gemm_slots(static_cast<Dtype>(c.head->dtype), build_list);
            ha.grid = static_cast<int32_t>(items < slots ? items : slots);
            ha.out_by_slot = 1;
            ha.build_list = build_list;
            ha.partials = partials;
            ha.plan = plan;
            ha.tokens = c.tokens;
            ha.cand = cand_in_ws ? tgt_arg : nullptr;
            ha.K = static_cast<int32_t>(c.D);
            ha.V = c.V;
        }
    }

    if (do_reduce) {
        DecideArgs da{};
        da.tgt = static_cast<const char *>(c.tgt);
        da.ld_bytes = c.ld * eb;
        da.V = c.V;
        da.B = c.B;
        da.RT = static_cast<int32_t>(c.RT);
        da.D = static_cast<int32_t>(c.D);
        da.is_tree = c.is_tree;
        da.parent = c.parent;
        da.tokens = c.tokens;
        da.partials = partials;
        da.plan = plan;
        da.score_mismatch = phase == kReducePhase ? decisions : head;   // phase 2 may need the list
        da.sampled = uniform != nullptr;
        da.tgt_argmax = F.tgt_argmax; da.tgt_max = F.tgt_max; da.tgt_lse = F.tgt_lse; da.tgt_ent = F.tgt_entropy;
        da.tgt_cand = F.tgt_candidate;
        da.logp_tgt = F.logp_tgt; da.delta = F.delta;
        da.ws_tgt_arg = tgt_arg;
        da.ws_logp_tgt = ws_logp;
        da.ws_state = state;
        da.ws_listpos = listpos;
        da.ws_list = list;
        da.ws_count = count;

        ReduceArgs ra{};
        ra.tgt = da.tgt;
        ra.drf = static_cast<const char *>(c.drf);
        ra.ld_bytes = da.ld_bytes;
        ra.V = c.V;
        ra.n_tgt_rows = static_cast<int32_t>(n_tgt);
        ra.n_rows = static_cast<int32_t>(rows);
        ra.parent = c.is_tree ? c.parent : nullptr;
        ra.N = static_cast<int32_t>(c.RT);
        ra.plan = plan;
        // segments never straddle splits
        ra.vec_per_split = static_cast<int32_t>(split_vectors(nvec, plan.splits, uniform != nullptr));
        ra.partials = partials;
        ra.reset_counter = count;
        ra.seg = uniform ? seg : nullptr;
        ra.nseg = static_cast<int32_t>(n_segments(c.V, eb));
        if (!c.is_tree) {           // the logit at each row's token, for the chain finish
            ra.chain_tokens = c.tokens;
            ra.K = static_cast<int32_t>(c.D);
            ra.xtok = xtok;
        }

        if (!record(c.opts ? c.opts->reduce_begin : nullptr)) return COSPEC_ERR_HIP;
        const hipError_t re = every_slot ? launch_reduce_head(dt, static_cast<Dtype>(c.head->dtype), ra, ha, c.stream)
                                         : launch_reduce(dt, ra, c.stream);
        if (re != hipSuccess) return COSPEC_ERR_HIP;
        if (!record(c.opts ? c.opts->reduce_end : nullptr)) return COSPEC_ERR_HIP;
        // the second pair brackets nothing: back to back, it measures what an event
        // interval adds by itself
        if (!record(c.opts ? c.opts->reduce2_begin : nullptr)) return COSPEC_ERR_HIP;
        if (!record(c.opts ? c.opts->reduce2_end : nullptr)) return COSPEC_ERR_HIP;

        // temperature-1 candidates
        if (uniform) {
            SampleArgs sa{};
            sa.tgt = ra.tgt;
            sa.ld_bytes = ra.ld_bytes;
            sa.V = c.V;
            sa.n_rows = ra.n_tgt_rows;
            sa.partials = partials;
            sa.plan = plan;
            sa.seg = seg;
            sa.nseg = ra.nseg;
            sa.uniform = uniform;
            sa.cand = tgt_arg;
            if (launch_sample(dt, sa, c.stream) != hipSuccess) return COSPEC_ERR_HIP;
        }
        // the decision step: its own kernel for trees and for the first phase of a split
        // step (whose outputs, the candidates, the caller needs before phase 2); in a
        // whole chain step the finish takes it, and the head GEMM derives its list
        // itself, unless the batch has more decision slots than the GEMM's workgroups
        // list (then this kernel builds the list the GEMM reads)
        if (c.is_tree || phase == kReducePhase || (head && !build_list)) {
            if (launch_decide(dt, da, c.stream) != hipSuccess) return COSPEC_ERR_HIP;
        }
    }
    if (!do_arbitrate) return COSPEC_OK;
    if (head && !(every_slot && do_reduce)) {
        const Dtype hdt = static_cast<Dtype>(c.head->dtype);
        const hipError_t he = every_slot ? launch_slot_gemm(hdt, ha, c.stream)
                              : fuse_head ? launch_head_gemm(hdt, ha, c.stream)
                                          : launch_head(hdt, ha, c.stream);
        if (he != hipSuccess) return COSPEC_ERR_HIP;
    }

    // finish
    FinishArgs fa{};
    fa.drf = static_cast<const char *>(c.drf);
    fa.ld_bytes = c.ld * eb;
    fa.V = c.V;
    fa.B = c.B;
    fa.RT = static_cast<int32_t>(c.RT);
    fa.RD = static_cast<int32_t>(c.RD);
    fa.D = static_cast<int32_t>(c.D);
    fa.is_tree = c.is_tree;
    fa.parent = c.parent;
    fa.tokens = c.tokens;
    fa.partials = partials;
    fa.plan = plan;
    fa.ws_state = state;
    fa.ws_listpos = listpos;
    fa.z = zlog;
    fa.head_ran = head;
    fa.lambda = c.lambda;
    fa.ws_tgt_arg = tgt_arg;
    fa.accept_len = accept_len; fa.out_tokens = out_tokens; fa.out_path = out_path;
    fa.drf_argmax = F.drf_argmax; fa.drf_max = F.drf_max; fa.drf_lse = F.drf_lse; fa.drf_ent = F.drf_entropy;
    fa.logp_drf = F.logp_drf;
    fa.z_tilde = F.z_tilde; fa.policy = F.policy; fa.accept = F.accept;
    fa.logp_action = F.logp_action;
    fa.policy_u = policy_u;
    fa.ws_logp_tgt = ws_logp;
    fa.fuse_head = fuse_head;
    fa.head_every_slot = every_slot;
    fa.head_dt = head ? c.head->dtype : 0;
    fa.hd = ha;
    fa.hd.list = nullptr;           // the finish reads the GEMM's partials by decision slot
    fa.ws_xtok = xtok;
    fa.sampled = cand_in_ws;
    fa.tgt_argmax = F.tgt_argmax; fa.tgt_max = F.tgt_max; fa.tgt_lse = F.tgt_lse; fa.tgt_ent = F.tgt_entropy;
    fa.tgt_cand = F.tgt_candidate;
    fa.delta = F.delta; fa.logp_tgt = F.logp_tgt;
    if (rl) {
        fa.rl_on = 1;
        fa.rl_correct = rl->correct; fa.rl_alpha = rl->alpha; fa.rl_beta = rl->beta;
        fa.rl_effective = rl->effective; fa.rl_s_acc = rl->in_s_acc;
        fa.rl_first_mismatch = rl->first_mismatch; fa.rl_first_reject = rl->first_reject;
        fa.rl_rho = rl->rho; fa.rl_reward = rl->reward; fa.rl_return = rl->round_return;
    }
    if (launch_finish(dt, fa, c.stream) != hipSuccess) return COSPEC_ERR_HIP;
    return COSPEC_OK;
}

cospec_status check_logits(const void *p, cospec_dtype dt, int64_t ld, int32_t V) {
    if (!p || !aligned(p, 16)) return COSPEC_ERR_INVALID_ARG;
    if (ld < V || (ld * elem_bytes(dt)) % 16 != 0) return COSPEC_ERR_INVALID_ARG;
    // a row is read through a buffer resource with 32-bit byte offsets
    if (static_cast<int64_t>(V) * elem_bytes(dt) > kMaxRowBytes) return COSPEC_ERR_UNSUPPORTED;
    return COSPEC_OK;
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices];   // device address of `scratch` per device, once looked up

// The address of the current device's copy of `scratch`, looked up on the first call on
// that device (with it current) and kept; null if the lookup fails.
void *static_scratch() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        g_scratch[dev] = p;
    }
    return g_scratch[dev];
}

}  // namespace

extern "C" {

int32_t cospec_abi_version(void) { return COSPEC_ABI_VERSION; }

#ifndef COSPEC_BUILD_ID
#define COSPEC_BUILD_ID "unknown"
#endif
const char *cospec_build_id(void) { return COSPEC_BUILD_ID; }

const char *cospec_status_string(int32_t status) {
    switch (status) {
        case COSPEC_OK: return "ok";
        case COSPEC_ERR_INVALID_ARG: return "invalid argument";
        case COSPEC_ERR_UNSUPPORTED: return "unsupported size";
        case COSPEC_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
        case COSPEC_ERR_HIP: return "HIP error";
        case COSPEC_ERR_SCRATCH_LIMIT: return "sizes need more scratch than the library's static buffer holds";
        default: return "unknown status";
    }
}

size_t cospec_workspace_bytes(int32_t n_target_rows, int32_t n_draft_rows, int32_t n_decisions, int32_t V,
                              const cospec_head *head) {
    if (n_target_rows < 0 || n_draft_rows < 0 || n_decisions < 0 || V < 1) return 0;
    if (head && check_head(head) != COSPEC_OK) return 0;
    // the layout depends on the batch only through these three counts (B * rows per
    // sequence), so one "sequence" holding all of them gives the same sizes
    return layout(static_cast<int64_t>(n_target_rows) + n_draft_rows, 1, n_target_rows, n_decisions, head, V).total;
}

size_t cospec_verify_block_workspace_size(int32_t B, int32_t K, int32_t V, const cospec_head *head) {
    if (B < 0 || K < 0 || K > COSPEC_MAX_K || V < 1 || check_head(head) != COSPEC_OK) return 0;
    return layout(static_cast<int64_t>(B) * (2 * K + 1), B, K + 1, K, head, V).total;
}

size_t cospec_verify_tree_workspace_size(int32_t B, int32_t N, int32_t V, const cospec_head *head) {
    if (B < 0 || N < 1 || N > COSPEC_MAX_N || V < 1 || check_head(head) != COSPEC_OK) return 0;
    return layout(static_cast<int64_t>(B) * 2 * N, B, N, N, head, V).total;
}

// Host-side checks of a chain call; fills `c` on success.
cospec_status block_common(const void *target_logits, const void *draft_logits, cospec_dtype logit_dtype,
                           int64_t ld, const int32_t *draft_tokens, const void *hidden, bool need_hidden,
                           const cospec_head *head, float lambda, int32_t B, int32_t K, int32_t V,
                           const cospec_features *feats, const cospec_options *opts, void *workspace,
                           size_t workspace_bytes, hipStream_t stream, Common &c) {
    if (!dtype_ok(logit_dtype) || B < 0 || K < 0 || V < 1 || isnan(lambda)) return COSPEC_ERR_INVALID_ARG;
    if (K > COSPEC_MAX_K) return COSPEC_ERR_UNSUPPORTED;
    cospec_status st = check_head(head);
    if (st != COSPEC_OK) return st;
    if (B == 0) return COSPEC_OK;
    if ((st = check_logits(target_logits, logit_dtype, ld, V)) != COSPEC_OK) return st;
    if (K > 0) {
        if ((st = check_logits(draft_logits, logit_dtype, ld, V)) != COSPEC_OK) return st;
        if (!draft_tokens || !aligned(draft_tokens, 4)) return COSPEC_ERR_INVALID_ARG;
        if (need_hidden && (!hidden || !aligned(hidden, 16))) return COSPEC_ERR_INVALID_ARG;
    }
    if (!feats_aligned(feats)) return COSPEC_ERR_INVALID_ARG;
    if (static_cast<int64_t>(B) * (2 * K + 1) > INT32_MAX / 2) return COSPEC_ERR_UNSUPPORTED;
    c.tgt = target_logits; c.drf = draft_logits; c.dt = logit_dtype; c.ld = ld;
    c.hidden = hidden; c.head = head; c.lambda = lambda; c.B = B; c.V = V;
    c.RT = K + 1; c.RD = K; c.D = K; c.is_tree = 0;
    c.parent = nullptr; c.tokens = draft_tokens;
    c.feats = feats; c.opts = opts; c.ws = workspace; c.ws_bytes = workspace_bytes; c.stream = stream;
    return COSPEC_OK;
}

cospec_status cospec_verify_block(const void *target_logits, const void *draft_logits,
                                  cospec_dtype logit_dtype, int64_t ld, const int32_t *draft_tokens,
                                  const void *hidden, const cospec_head *head, float lambda, int32_t B,
                                  int32_t K, int32_t V, int32_t *accept_len, int32_t *out_tokens,
                                  const cospec_features *feats, const cospec_options *opts, void *workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
    Common c{};
    cospec_status st = block_common(target_logits, draft_logits, logit_dtype, ld, draft_tokens, hidden, true,
                                    head, lambda, B, K, V, feats, opts, workspace, workspace_bytes, stream, c);
    if (st != COSPEC_OK || B == 0) return st;
    if (!accept_len || !aligned(accept_len, 4) || !out_tokens || !aligned(out_tokens, 4))
        return COSPEC_ERR_INVALID_ARG;
    return run(c, kWhole, accept_len, out_tokens, nullptr);
}

cospec_status cospec_verify_block_static(const void *target_logits, const void *draft_logits,
                                         cospec_dtype logit_dtype, int64_t ld, const int32_t *draft_tokens,
                                         const void *hidden, const cospec_head *head, float lambda, int32_t B,
                                         int32_t K, int32_t V, int32_t *accept_len, int32_t *out_tokens,
                                         const cospec_features *feats, const cospec_options *opts,
                                         hipStream_t stream) {
    Common c{};
    cospec_status st = block_common(target_logits, draft_logits, logit_dtype, ld, draft_tokens, hidden, true,
                                    head, lambda, B, K, V, feats, opts, nullptr, 0, stream, c);
    if (st != COSPEC_OK || B == 0) return st;
    if (!accept_len || !aligned(accept_len, 4) || !out_tokens || !aligned(out_tokens, 4))
        return COSPEC_ERR_INVALID_ARG;
    const size_t need = cospec_verify_block_workspace_size(B, K, V, head);
    if (need == 0 || need > COSPEC_STATIC_SCRATCH_BYTES) return COSPEC_ERR_SCRATCH_LIMIT;
    // the step's scratch memory needs no clearing: the one counter that must start at
    // zero (the mismatch-list length) is zeroed by the first reduction workgroup
    void *ws = static_scratch();
    if (!ws) return COSPEC_ERR_HIP;
    c.ws = ws;
    c.ws_bytes = COSPEC_STATIC_SCRATCH_BYTES;
    return run(c, kWhole, accept_len, out_tokens, nullptr);
}

cospec_status cospec_verify_block_reduce(const void *target_logits, const void *draft_logits,
                                         cospec_dtype logit_dtype, int64_t ld,
                                         const int32_t *draft_tokens, const cospec_head *head,
                                         int32_t B, int32_t K, int32_t V, int32_t *candidates,
                                         const cospec_features *feats, const cospec_options *opts,
                                         void *workspace, size_t workspace_bytes, hipStream_t stream) {
    Common c{};
    cospec_status st = block_common(target_logits, draft_logits, logit_dtype, ld, draft_tokens, nullptr, false,
                                    head, 0.5f, B, K, V, feats, opts, workspace, workspace_bytes, stream, c);
    if (st != COSPEC_OK || B == 0) return st;
    if (!candidates || !aligned(candidates, 4)) return COSPEC_ERR_INVALID_ARG;
    cospec_features f = feats ? *feats : cospec_features{};
    f.tgt_candidate = candidates;
    c.feats = &f;
    return run(c, kReducePhase, nullptr, nullptr, nullptr);
}

cospec_status cospec_verify_block_arbitrate(const void *target_logits, const void *draft_logits,
                                            cospec_dtype logit_dtype, int64_t ld,
                                            const int32_t *draft_tokens, const void *hidden,
                                            const cospec_head *head, float lambda, int32_t B, int32_t K,
                                            int32_t V, int32_t *accept_len, int32_t *out_tokens,
                                            const cospec_features *feats, const cospec_options *opts,
                                            void *workspace, size_t workspace_bytes, hipStream_t stream) {
    Common c{};
    cospec_status st = block_common(target_logits, draft_logits, logit_dtype, ld, draft_tokens, hidden, true,
                                    head, lambda, B, K, V, feats, opts, workspace, workspace_bytes, stream, c);
    if (st != COSPEC_OK || B == 0) return st;
    if (!accept_len || !aligned(accept_len, 4) || !out_tokens || !aligned(out_tokens, 4))
        return COSPEC_ERR_INVALID_ARG;
    return run(c, kArbitratePhase, accept_len, out_tokens, nullptr);
}

size_t cospec_verify_block_sps_workspace_size(int32_t B, int32_t K, int32_t V) {
    if (B < 0 || K < 0 || K > COSPEC_MAX_K || V < 1) return 0;
    return layout(static_cast<int64_t>(B) * (2 * K + 1), B, K + 1, K, nullptr, V).total;
}

cospec_status cospec_verify_block_sps(const void *target_logits, const void *draft_logits,
                                      cospec_dtype logit_dtype, int64_t ld, const int32_t *draft_tokens,
                                      const float *uniforms, int32_t B, int32_t K, int32_t V,
                                      int32_t *accept_len, int32_t *out_tokens, const cospec_features *feats,
                                      const cospec_options *opts, void *workspace, size_t workspace_bytes,
                                      hipStream_t stream) {
    if (!dtype_ok(logit_dtype) || B < 0 || K < 0 || V < 1) return COSPEC_ERR_INVALID_ARG;
    if (K > COSPEC_MAX_K) return COSPEC_ERR_UNSUPPORTED;
    if (B == 0) return COSPEC_OK;
    cospec_status st;
    if ((st = check_logits(target_logits, logit_dtype, ld, V)) != COSPEC_OK) return st;
    if (K > 0) {
        if ((st = check_logits(draft_logits, logit_dtype, ld, V)) != COSPEC_OK) return st;
        if (!draft_tokens || !aligned(draft_tokens, 4)) return COSPEC_ERR_INVALID_ARG;
    }
    if (!uniforms || !aligned(uniforms, 4) || !accept_len || !aligned(accept_len, 4) || !out_tokens ||
        !aligned(out_tokens, 4) || !feats_aligned(feats))
        return COSPEC_ERR_INVALID_ARG;
    if (opts && (opts->sample_uniform || opts->policy_uniform || opts->rl || opts->hidden_row0))
        return COSPEC_ERR_INVALID_ARG;                  // only splits and the timing events apply
    if (static_cast<int64_t>(B) * (2 * K + 1) > INT32_MAX / 2) return COSPEC_ERR_UNSUPPORTED;
    const int eb = elem_bytes(logit_dtype);
    const int64_t n_tgt = static_cast<int64_t>(B) * (K + 1), n_drf = static_cast<int64_t>(B) * K;
    const int64_t rows = n_tgt + n_drf;
    const int64_t nvec = static_cast<int64_t>(V) * eb / 16;
    int32_t override_splits = 0;
    if (opts && opts->splits) {
        if (opts->splits < 0 || opts->splits > COSPEC_MAX_SPLITS) return COSPEC_ERR_UNSUPPORTED;
        override_splits = opts->splits;
    }
    const Layout L = layout(rows, B, K + 1, K, nullptr, V);
    const PartPlan plan = make_plan(n_tgt, n_drf, nvec, override_splits, static_cast<Dtype>(logit_dtype));
    if (rows * plan.splits > L.partial_slots || rows * plan.splits > INT32_MAX) return COSPEC_ERR_UNSUPPORTED;
    if (!workspace || !aligned(workspace, kAlign) || workspace_bytes < L.total) return COSPEC_ERR_WORKSPACE;
    char *ws = static_cast<char *>(workspace);
    float4 *partials = reinterpret_cast<float4 *>(ws + L.partials);
    const cospec_features F = feats ? *feats : cospec_features{};
    const Dtype dt = static_cast<Dtype>(logit_dtype);

    ReduceArgs ra{};
    ra.tgt = static_cast<const char *>(target_logits);
    ra.drf = static_cast<const char *>(draft_logits);
    ra.ld_bytes = ld * eb;
    ra.V = V;
    ra.n_tgt_rows = static_cast<int32_t>(n_tgt);
    ra.n_rows = static_cast<int32_t>(rows);
    ra.plan = plan;
    ra.vec_per_split = static_cast<int32_t>(split_vectors(nvec, plan.splits, false));
    ra.partials = partials;
    ra.reset_counter = reinterpret_cast<int32_t *>(ws + L.count);
    if (opts && opts->reduce_begin && hipEventRecord(opts->reduce_begin, stream) != hipSuccess) return COSPEC_ERR_HIP;
    if (launch_reduce(dt, ra, stream) != hipSuccess) return COSPEC_ERR_HIP;
    if (opts && opts->reduce_end && hipEventRecord(opts->reduce_end, stream) != hipSuccess) return COSPEC_ERR_HIP;
    // the second pair brackets nothing, as in a whole step
    if (opts && opts->reduce2_begin && hipEventRecord(opts->reduce2_begin, stream) != hipSuccess)
        return COSPEC_ERR_HIP;
    if (opts && opts->reduce2_end && hipEventRecord(opts->reduce2_end, stream) != hipSuccess) return COSPEC_ERR_HIP;

    DecideArgs da{};
    da.tgt = ra.tgt; da.ld_bytes = ra.ld_bytes; da.V = V; da.B = B; da.RT = K + 1; da.D = K;
    da.tokens = draft_tokens; da.partials = partials; da.plan = plan;
    da.tgt_argmax = F.tgt_argmax; da.tgt_max = F.tgt_max; da.tgt_lse = F.tgt_lse; da.tgt_ent = F.tgt_entropy;
    da.tgt_cand = F.tgt_candidate; da.logp_tgt = F.logp_tgt; da.delta = F.delta;
    da.ws_tgt_arg = reinterpret_cast<int32_t *>(ws + L.tgt_arg);
    da.ws_logp_tgt = reinterpret_cast<float *>(ws + L.logp);
    da.ws_state = reinterpret_cast<uint8_t *>(ws + L.state);
    da.ws_listpos = reinterpret_cast<int32_t *>(ws + L.listpos);
    da.ws_list = reinterpret_cast<int32_t *>(ws + L.list);
    da.ws_count = reinterpret_cast<int32_t *>(ws + L.count);
    if (launch_decide(dt, da, stream) != hipSuccess) return COSPEC_ERR_HIP;

    SpsArgs sa{};
    sa.tgt = ra.tgt; sa.drf = ra.drf; sa.ld_bytes = ra.ld_bytes; sa.V = V; sa.B = B; sa.K = K;
    sa.tokens = draft_tokens; sa.uniform = uniforms; sa.partials = partials; sa.plan = plan;
    sa.ws_state = da.ws_state; sa.ws_logp_tgt = da.ws_logp_tgt;
    sa.seg_mass = reinterpret_cast<float *>(ws + L.seg);
    sa.nseg = static_cast<int32_t>(n_segments(V, eb));
    sa.accept_len = accept_len; sa.out_tokens = out_tokens;
    sa.drf_argmax = F.drf_argmax; sa.drf_max = F.drf_max; sa.drf_lse = F.drf_lse; sa.drf_ent = F.drf_entropy;
    sa.logp_drf = F.logp_drf; sa.accept_prob = F.policy; sa.accept = F.accept;
    if (launch_sps(dt, sa, stream) != hipSuccess) return COSPEC_ERR_HIP;
    return COSPEC_OK;
}

cospec_status cospec_verify_tree(const void *target_logits, const void *draft_logits,
                                 cospec_dtype logit_dtype, int64_t ld, const int32_t *parent,
                                 const int32_t *node_tokens, const void *hidden, const cospec_head *head,
                                 float lambda, int32_t B, int32_t N, int32_t V, int32_t *accept_len,
                                 int32_t *out_tokens, int32_t *out_path, const cospec_features *feats,
                                 const cospec_options *opts, void *workspace, size_t workspace_bytes,
                                 hipStream_t stream) {
    if (!dtype_ok(logit_dtype) || B < 0 || N < 1 || V < 1 || isnan(lambda)) return COSPEC_ERR_INVALID_ARG;
    if (N > COSPEC_MAX_N) return COSPEC_ERR_UNSUPPORTED;
    cospec_status st = check_head(head);
    if (st != COSPEC_OK) return st;
    if (B == 0) return COSPEC_OK;
    if ((st = check_logits(target_logits, logit_dtype, ld, V)) != COSPEC_OK) return st;
    if ((st = check_logits(draft_logits, logit_dtype, ld, V)) != COSPEC_OK) return st;
    if (!parent || !aligned(parent, 4) || !node_tokens || !aligned(node_tokens, 4) || !hidden || !aligned(hidden, 16))
        return COSPEC_ERR_INVALID_ARG;
    if (!accept_len || !aligned(accept_len, 4) || !out_tokens || !aligned(out_tokens, 4) ||
        (out_path && !aligned(out_path, 4)) || !feats_aligned(feats))
        return COSPEC_ERR_INVALID_ARG;
    if (static_cast<int64_t>(B) * 2 * N > INT32_MAX / 2) return COSPEC_ERR_UNSUPPORTED;
    Common c{};
    c.tgt = target_logits; c.drf = draft_logits; c.dt = logit_dtype; c.ld = ld;
    c.hidden = hidden; c.head = head; c.lambda = lambda; c.B = B; c.V = V;
    c.RT = N; c.RD = N; c.D = N; c.is_tree = 1;
    c.parent = parent; c.tokens = node_tokens;
    c.feats = feats; c.opts = opts; c.ws = workspace; c.ws_bytes = workspace_bytes; c.stream = stream;
    return run(c, kWhole, accept_len, out_tokens, out_path);
}

cospec_status cospec_hybrid_mask(const int32_t *ctx_len, int32_t B, int32_t K, int32_t L, uint8_t *mask,
                                 hipStream_t stream) {
    if (B < 0 || K < 0 || L < 0) return COSPEC_ERR_INVALID_ARG;
    if (static_cast<int64_t>(B) * L == 0) return COSPEC_OK;
    if (!ctx_len || !aligned(ctx_len, 4) || !mask) return COSPEC_ERR_INVALID_ARG;
    if (static_cast<int64_t>(B) * L > UINT32_MAX) return COSPEC_ERR_UNSUPPORTED;
    MaskArgs a{ctx_len, B, K, L, mask};
    return launch_hybrid_mask(a, stream) == hipSuccess ? COSPEC_OK : COSPEC_ERR_HIP;
}

cospec_status cospec_hybrid_attention(const void *q, const void *k, const void *v, const int32_t *ctx_len,
                                      const int32_t *q_start, int32_t B, int32_t n_q, int32_t L, int32_t Hq,
                                      int32_t Hkv, int32_t D, int32_t K, float scale, void *out,
                                      hipStream_t stream) {
    if (B < 0 || n_q < 0 || L < 0 || K < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || !isfinite(scale))
        return COSPEC_ERR_INVALID_ARG;
    if (D != 64 && D != 128) return COSPEC_ERR_UNSUPPORTED;
    if (static_cast<int64_t>(B) * n_q == 0) return COSPEC_OK;
    if (!q || !aligned(q, 16) || !k || !aligned(k, 16) || !v || !aligned(v, 16) || !out || !aligned(out, 16) ||
        !ctx_len || !aligned(ctx_len, 4) || !q_start || !aligned(q_start, 4))
        return COSPEC_ERR_INVALID_ARG;
    const int64_t wgs = static_cast<int64_t>(B) * Hkv * ((static_cast<int64_t>(n_q) * (Hq / Hkv) + 15) / 16);
    if (wgs > UINT32_MAX || static_cast<int64_t>(L) * Hkv * D > INT32_MAX) return COSPEC_ERR_UNSUPPORTED;
    AttnArgs a{q, k, v, ctx_len, q_start, B, n_q, L, Hq, Hkv, D, K, scale, out};
    return launch_hybrid_attention(a, stream) == hipSuccess ? COSPEC_OK : COSPEC_ERR_HIP;
}

size_t cospec_arbitrate_workspace_size(int64_t n_sel, const cospec_head *head) {
    if (n_sel < 0 || check_head(head) != COSPEC_OK) return 0;
    return head_bytes(n_sel, head);
}

cospec_status cospec_arbitrate(const void *hidden, int64_t n_rows, const int32_t *row_index, int64_t n_sel,
                               const cospec_head *head, float lambda, float *out_z, uint8_t *out_accept,
                               void *workspace, size_t workspace_bytes, hipStream_t stream) {
    if (n_rows < 0 || n_sel < 0 || isnan(lambda)) return COSPEC_ERR_INVALID_ARG;
    cospec_status st = check_head(head);
    if (st != COSPEC_OK) return st;
    if (!row_index && n_sel > n_rows) return COSPEC_ERR_INVALID_ARG;
    if (n_sel > INT32_MAX) return COSPEC_ERR_UNSUPPORTED;
    if (n_sel == 0) return COSPEC_OK;
    if (!hidden || !aligned(hidden, 16) || (row_index && !aligned(row_index, 4)) || (out_z && !aligned(out_z, 4)))
        return COSPEC_ERR_INVALID_ARG;
    const size_t need = cospec_arbitrate_workspace_size(n_sel, head);
    if (!workspace || !aligned(workspace, kAlign) || workspace_bytes < need) return COSPEC_ERR_WORKSPACE;

    const int32_t ks = ksplit_for(n_sel, head);
    float *upart = static_cast<float *>(workspace);
    float *zlog = reinterpret_cast<float *>(static_cast<char *>(workspace) +
                                            round_up(static_cast<size_t>(ks) * n_sel * head->h * 4));
    HeadArgs ha{};
    ha.hidden = hidden; ha.n_rows = n_rows; ha.list = row_index;
    ha.count_dev = nullptr; ha.count_host = n_sel; ha.m_cap = n_sel;
    ha.w1 = head->w1; ha.b1 = head->b1; ha.w2 = head->w2; ha.b2 = head->b2; ha.d = head->d; ha.h = head->h;
    ha.ksplit = ks;
    // the row count is known here: the shallow ring when the grid has more workgroups
    // than there are CUs
    ha.two_per_cu = ((n_sel + kHeadTileM - 1) / kHeadTileM) * ((head->h + kHeadTileN - 1) / kHeadTileN) * ks >
                    cu_count();
    ha.upart = upart;
    ha.z = zlog;
    if (launch_head(static_cast<Dtype>(head->dtype), ha, stream) != hipSuccess) return COSPEC_ERR_HIP;
    ArbFinishArgs fa{};
    fa.n_sel = n_sel; fa.n_rows = n_rows; fa.row_index = row_index;
    fa.z = zlog; fa.lambda = lambda; fa.out_z = out_z; fa.out_accept = out_accept;
    if (launch_arb_finish(fa, stream) != hipSuccess) return COSPEC_ERR_HIP;
    return COSPEC_OK;
}

}  // extern "C"
