// Finish of the verify step: draft-row statistics and log p_D, the per-decision
// verdicts, the first stop and the emitted tokens.
//
// The draft rows are needed only for features (log p_D of the draft token, the
// draft entropy); the decision itself needs the target rows alone, so the draft
// rows' partials are merged here.
//
// Chain (Section 3.3, Eq. cospec_length): one wave per sequence, lane i-1 owns
// decision i, target row i-1 and draft row i-1; it takes the decision step itself
// (the candidate of target row i-1, Delta, log-probabilities).  A matched decision passes (z_tilde = +inf,
// Eq. policy-prob); a mismatch passes when sigma(z) > lambda (Eq. infer_thre),
// or, with sampled arbitration, when its uniform is below sigma(z).
// The first failing decision is the lowest set bit of a wave ballot, s = its
// position (1-based) or K+1; the round emits draft tokens 1..s-1 and the target
// token of row s-1.
//
// Tree (the chain rule along root paths): one workgroup per tree, thread n owns
// node n.  Reachability (every decision on the root path passes) and depth are
// found by pointer jumping in LDS (log2(depth) rounds), the accepted node is the
// deepest reachable one with ties to the lowest id (one key max-reduction), and
// the path is walked back through the parent array.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>

#include "head_z.h"
#include "launch.h"
#include "rowstat.h"

namespace cospec {
namespace {

struct Verdict {
    bool pass;
    float z_tilde, policy;
    float logp_action;   // log pi(a) of the action taken
};

// log sigma(x) without overflow for either sign of x.
__device__ inline float log_sigmoid(float x) { return fminf(x, 0.f) - log1pf(expf(-fabsf(x))); }

// Verdict of one decision slot from its state and its head logit z (read only when
// the head scored the slot): the threshold (Eq. infer_thre), or with sampled
// arbitration (`sampled`) the action u < pi for the slot's uniform u, which the caller
// loaded with its other inputs.
__device__ inline Verdict verdict(uint8_t state, bool scored, float z, float lambda, bool sampled, float u) {
    Verdict v;
    if (state == kStateMatch) {
        v.pass = true; v.z_tilde = INFINITY; v.policy = 1.0f; v.logp_action = 0.0f;
    } else if (state != kStateMismatch) {          // invalid token or parent: always rejected
        v.pass = false; v.z_tilde = NAN; v.policy = NAN; v.logp_action = NAN;
    } else if (!scored) {
        // head skipped: lambda >= 1 or lambda < 0 decides every mismatch by itself
        v.pass = lambda < 0.0f; v.z_tilde = NAN; v.policy = NAN; v.logp_action = NAN;
    } else {
        const float pi = 1.0f / (1.0f + expf(-z));
        v.pass = sampled ? u < pi : pi > lambda;
        v.z_tilde = z; v.policy = pi;
        v.logp_action = log_sigmoid(v.pass ? z : -z);
    }
    return v;
}

__device__ inline void write_drf(const FinishArgs &a, int64_t r, const RowStat &rs) {
    if (a.drf_argmax) a.drf_argmax[r] = rs.arg;
    if (a.drf_max) a.drf_max[r] = rs.max;
    if (a.drf_lse) a.drf_lse[r] = rs.lse;
    if (a.drf_ent) a.drf_ent[r] = rs.ent;
}

// The chain finish of sequence b by one wave, lane i-1 owning decision i, in two
// parts: the decision step and what needs no head logit (the loads, the target- and
// draft-row statistics, Delta, log-probabilities), then the verdicts, the stop, the
// emission and the RL statistics.
struct ChainLane {
    uint8_t st;
    bool scored;      // a mismatch the head scored
    float lpt;        // log p_T of the draft token
    int tok_d, tok_t; // draft token of slot `lane`, target candidate of row `lane`
    int tok_k;        // K = 64 only, in lane 0: the candidate of target row K (no lane of its own)
    float u;          // sampled arbitration: the decision's uniform
};

// Merged statistics of target row tr: its candidate (the argmax, or the candidate
// already taken when `sampled`) and the optional per-row features.
__device__ inline int tgt_row(const FinishArgs &a, int64_t tr, const RowStat &ts) {
    const int cand = a.sampled ? a.ws_tgt_arg[tr] : ts.arg;
    if (a.tgt_cand) a.tgt_cand[tr] = cand;
    if (a.tgt_argmax) a.tgt_argmax[tr] = ts.arg;
    if (a.tgt_max) a.tgt_max[tr] = ts.max;
    if (a.tgt_lse) a.tgt_lse[tr] = ts.lse;
    if (a.tgt_ent) a.tgt_ent[tr] = ts.ent;
    return cand;
}

// The decision step of one chain by one wave (Section 3.1): lane j merges target row
// j in fixed split order (its argmax, ties to the lowest index, is the verification
// candidate of decision j+1, or of the bonus token for j = K; at temperature 1 the
// sample k_sample left, in a split step's second phase the first phase's choice) and
// draft row j; decision j+1 is a match when its draft token
// equals that candidate; log p_T and log p_D of the draft token come from the same
// rows (Section 3.4).  PM, how the partials are read (a template parameter, so that
// each kernel holds one way and no memory wait is placed for another): kPartOne, one
// split per row, each row's partial read with the token; kPartSplit, split rows, the
// lane's target and draft rows merged from registers, their partials loaded together.
enum { kPartOne, kPartSplit };

template <int PM>
__device__ inline ChainLane chain_prefix(const FinishArgs &a, int b, int lane) {
    const int K = a.D;
    const int64_t di = static_cast<int64_t>(b) * K + lane;       // decision lane+1, draft row lane
    const int64_t t0 = static_cast<int64_t>(b) * (K + 1);        // the sequence's first target row
    const int64_t tr = t0 + lane;                                 // target row `lane`
    const PartPlan &plan = a.plan;
    const int64_t d0 = plan.n_tgt_rows + static_cast<int64_t>(b) * K;
    int tok = -1;
    float u = 0.f;
    if (lane < K) {
        tok = a.tokens[di];
        if (a.policy_u) u = a.policy_u[di];
    }
    // the logits at the draft token, which the reduction stored (read whatever the
    // token; used only when it is valid)
    const bool valid = tok >= 0 && tok < a.V;
    float xt = 0.f, xd = 0.f;
    if (lane < K) {
        xt = a.ws_xtok[tr];
        xd = a.ws_xtok[d0 + lane];
    }
    // the merged statistics of target row `lane` (lanes <= K) and draft row `lane`
    // (lanes < K; the others merge a row they drop)
    RowStat ts{}, ds{}, ks{};
    const int64_t trc = lane <= K ? tr : t0, drc = lane < K ? d0 + lane : t0;
    if constexpr (PM == kPartOne) {
        const float4 qt = a.partials[trc], qd = a.partials[drc];
        float4 qk{};
        if (K >= 64 && lane == 0) qk = a.partials[t0 + K];
        ts = merge_row_t([qt](int) { return qt; }, 1);
        ds = merge_row_t([qd](int) { return qd; }, 1);
        if (K >= 64 && lane == 0) ks = merge_row_t([qk](int) { return qk; }, 1);
    } else {
        merge_rows2(a.partials + row_parts(plan, trc).first, a.partials + row_parts(plan, drc).first, plan.splits,
                    ts, ds);
        if (K >= 64 && lane == 0) {
            const RowParts rk = row_parts(plan, t0 + K);
            ks = merge_row(a.partials + rk.first, rk.count);
        }
    }
    ChainLane c{kStateMatch, false, NAN, -1, -1, -1, u};
    if (K >= 64 && lane == 0) c.tok_k = tgt_row(a, t0 + K, ks);
    if (lane <= K) {
        const int cand = tgt_row(a, tr, ts);
        c.tok_t = cand;
        if (lane < K) {
            write_drf(a, di, ds);
            c.tok_d = tok;
            c.st = !valid ? kStateReject : tok == cand ? kStateMatch : kStateMismatch;
            c.lpt = valid ? (xt - ts.max) - ts.log_s : NAN;
            c.scored = a.head_ran && c.st == kStateMismatch;
            if (a.delta) a.delta[di] = c.st == kStateMatch;
            if (a.logp_tgt) a.logp_tgt[di] = c.lpt;
            if (a.logp_drf) a.logp_drf[di] = valid ? (xd - ds.max) - ds.log_s : NAN;
        }
    }
    return c;
}

// z: the head logit of the lane's decision (read only when the head scored it).
__device__ inline void chain_suffix(const FinishArgs &a, int b, int lane, const ChainLane &c, float z) {
    const int K = a.D;
    const int64_t di = static_cast<int64_t>(b) * K + lane;
    bool fail = false;
    const bool mism = lane < K && c.st != kStateMatch;
    const float lpt = c.lpt;
    if (lane < K) {
        const Verdict v = verdict(c.st, c.scored, z, a.lambda, a.policy_u != nullptr, c.u);
        fail = !v.pass;
        if (a.z_tilde) a.z_tilde[di] = v.z_tilde;
        if (a.policy) a.policy[di] = v.policy;
        if (a.accept) a.accept[di] = v.pass;
        if (a.logp_action) a.logp_action[di] = v.logp_action;
    }
    const uint64_t rej = __ballot(fail);
    const int s = rej ? __builtin_ctzll(rej) + 1 : K + 1;
    if (lane == 0) a.accept_len[b] = s;
    // slot j emits draft token j+1 before the stop, the target's token at it (j = K
    // = 64 is lane 0's second slot: no draft token, the bonus row's candidate)
    for (int j = lane; j <= K; j += 64) {
        const int td = j == lane ? c.tok_d : -1;
        const int tt = j == lane ? c.tok_t : c.tok_k;
        a.out_tokens[static_cast<int64_t>(b) * (K + 1) + j] = j < s - 1 ? td : j == s - 1 ? tt : -1;
    }
    if (!a.rl_on) return;
    // Section 3.4: effective actions up to the stop, rho, S_acc / S_rej and the
    // shaped reward; the first rejected mismatch is the stop itself (or K+1)
    const uint64_t mm = __ballot(mism);
    const int i_star = mm ? __builtin_ctzll(mm) + 1 : 0;
    const int i = lane + 1;
    const bool eff = mism && i <= min(s, K);
    const bool acc = eff && !fail && i < s;
    const bool rjt = eff && i == s && s <= K;
    const float rho = mm ? static_cast<float>(s - i_star) / static_cast<float>(K + 1 - i_star) : NAN;
    const bool correct = a.rl_correct && a.rl_correct[b];
    float g = 0.f;
    if (eff) g = correct ? rho : -(acc ? a.rl_alpha * fabsf(lpt) : 0.f) - (rjt ? a.rl_beta : 0.f);
    if (lane < K) {
        if (a.rl_effective) a.rl_effective[di] = eff;
        if (a.rl_s_acc) a.rl_s_acc[di] = acc;
        if (a.rl_reward) a.rl_reward[di] = g;
    }
    const float J = wave_sum(g);
    if (lane == 0) {
        if (a.rl_first_mismatch) a.rl_first_mismatch[b] = i_star;
        if (a.rl_first_reject) a.rl_first_reject[b] = s;
        if (a.rl_rho) a.rl_rho[b] = rho;
        if (a.rl_return) a.rl_return[b] = J;
    }
}

template <int PM>
__global__ __launch_bounds__(256) void k_chain_finish(FinishArgs a) {
    const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (b >= a.B) return;                                  // whole wave leaves together
    const int lane = threadIdx.x & 63;
    const ChainLane c = chain_prefix<PM>(a, b, lane);
    chain_suffix(a, b, lane, c, NAN);                      // the head did not run
}

// One workgroup per sequence: wave 0 takes the decision step while waves 1, 2, ...
// compute the head logits of the slots the head scored (slot t by wave
// 1 + t mod (waves - 1)) from the GEMM's k-slice partials, stored by decision slot;
// then wave 0 finishes the sequence.  A head wave finds out by itself whether its slot
// was scored (its token against the candidate of its target row, merged as wave 0
// merges it), so that its loads wait for no other wave; when the first layer ran on
// every slot, it scores every slot.
constexpr int kFinishWaves = 8;
template <int HD, int PM>
__global__ __launch_bounds__(64 * kFinishWaves) void k_chain_finish_head(FinishArgs a) {
    __shared__ float s_z[64];                              // K <= 64
    const int b = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int waves = blockDim.x >> 6;                     // >= 2
    const int K = a.D;
    ChainLane c{};
    if (wave == 0) {
        c = chain_prefix<PM>(a, b, lane);
    } else if (a.head_every_slot) {
        // the first layer ran on every slot: z of every slot, waiting for nothing (wave 0
        // uses the mismatches' only)
        for (int t = wave - 1; t < K; t += waves - 1) {    // wave-uniform
            const float z = headz::head_z<HD>(a.hd, static_cast<int64_t>(b) * K + t, lane, a.hd.ksplit);
            if (lane == 0) s_z[t] = z;
        }
    } else {
        const int64_t M = *a.hd.count_dev;                 // rows the GEMM ran on
        for (int t = wave - 1; t < K; t += waves - 1) {    // wave-uniform
            const int64_t di = static_cast<int64_t>(b) * K + t;
            const int64_t tr = static_cast<int64_t>(b) * (K + 1) + t;
            // both candidate sources are read (the workspace always holds ws_tgt_arg) and
            // one is chosen: no branch for the loads to wait at
            const int tok = a.tokens[di];
            const int taken = a.ws_tgt_arg[tr];
            const RowParts rp = row_parts(a.plan, tr);
            const int am = merge_arg(a.partials + rp.first, rp.count);
            const int cand = a.sampled ? taken : am;
            if (a.head_ran && tok >= 0 && tok < a.V && tok != cand) {
                const int ksl = headz::live_ksplit(a.hd, M);
                const float z = headz::head_z<HD>(a.hd, di, lane, ksl);
                if (lane == 0) s_z[t] = z;
            }
        }
    }
    __syncthreads();
    if (wave == 0) chain_suffix(a, b, lane, c, lane < K && c.scored ? s_z[lane] : NAN);
}

template <int DT>
__global__ __launch_bounds__(kMaxSeqRows) void k_tree_finish(FinishArgs a) {
    using E = Elt<DT>;
    const int b = blockIdx.x;
    const int n = threadIdx.x;
    const int N = a.D;
    const int64_t base = static_cast<int64_t>(b) * N;
    __shared__ int s_anc[2][kMaxSeqRows];
    __shared__ int s_dep[2][kMaxSeqRows];
    __shared__ int s_ok[2][kMaxSeqRows];
    __shared__ int s_par[kMaxSeqRows];
    __shared__ int s_path[kMaxSeqRows];
    __shared__ int s_child[kMaxSeqRows];
    __shared__ float s_dmax[kMaxSeqRows], s_dlogs[kMaxSeqRows];
    __shared__ int s_key[kMaxSeqRows / 64];
    __shared__ int s_tok[kMaxSeqRows], s_cand[kMaxSeqRows];

    // Two memory round trips: first every input that depends on the node alone (its
    // state, parent, token, list position, target candidate and uniform), then what
    // those locate (the draft logit of its token in the parent's row, its head logit)
    // together with the partials of its own draft row, merged for every node (leaves'
    // draft rows were not reduced: their stale partials are dropped below).  Later
    // steps read all of it from LDS.
    int par = -1, tok = -1, pos = -1;
    uint8_t st = kStateMatch;
    float u = 0.f;
    if (n < N) {
        st = a.ws_state[base + n];
        tok = a.tokens[base + n];
        if (a.head_ran) pos = a.ws_listpos[base + n];
        if (a.policy_u) u = a.policy_u[base + n];
        s_cand[n] = a.ws_tgt_arg[base + n];
        if (n > 0) {
            par = a.parent[base + n];
            if (!(par >= 0 && par < n)) par = -1;
        }
        s_par[n] = par;
        s_tok[n] = tok;
        s_child[n] = 0;
    }
    float xd = 0.f, z = NAN;
    RowStat rs{NAN, NAN, NAN, NAN, -1};
    if (n < N) {
        if (n > 0 && st != kStateReject && par >= 0) xd = E::at(a.drf + (base + par) * a.ld_bytes, tok);
        if (pos >= 0) z = a.z[pos];
        const RowParts rp = row_parts(a.plan, a.plan.n_tgt_rows + base + n);
        rs = merge_row(a.partials + rp.first, rp.count);
    }
    __syncthreads();
    if (n < N && par >= 0) s_child[par] = 1;
    __syncthreads();
    // draft rows were reduced for nodes with a child only
    if (n < N) {
        if (!s_child[n]) rs = RowStat{NAN, NAN, NAN, NAN, -1};
        write_drf(a, base + n, rs);
        s_dmax[n] = rs.max;
        s_dlogs[n] = rs.log_s;
    }
    __syncthreads();

    int anc = -1, dep = 0, ok = 1;
    if (n < N) {
        const bool scored = pos >= 0;
        const Verdict v = verdict(st, scored, z, a.lambda, a.policy_u != nullptr, u);
        if (n > 0) {
            anc = par;
            dep = 1;
            ok = par >= 0 && v.pass;
            if (a.logp_drf)
                a.logp_drf[base + n] = (st != kStateReject && par >= 0) ? (xd - s_dmax[par]) - s_dlogs[par] : NAN;
        } else if (a.logp_drf) {
            a.logp_drf[base] = NAN;
        }
        if (a.z_tilde) a.z_tilde[base + n] = v.z_tilde;
        if (a.policy) a.policy[base + n] = v.policy;
        if (a.accept) a.accept[base + n] = n == 0 ? 1 : v.pass;
        if (a.logp_action) a.logp_action[base + n] = n == 0 ? 0.0f : v.logp_action;
    }
    // pointer jumping: anc = ancestor 2^k steps up (or -1), dep = distance to it,
    // ok = every decision from this node up to (not including) anc passes
    int cur = 0;
    if (n < N) { s_anc[0][n] = anc; s_dep[0][n] = dep; s_ok[0][n] = ok; }
    __syncthreads();
    while (__syncthreads_or(n < N && s_anc[cur][n] >= 0)) {
        if (n < N) {
            const int x = s_anc[cur][n];
            if (x >= 0) {
                s_anc[cur ^ 1][n] = s_anc[cur][x];
                s_dep[cur ^ 1][n] = s_dep[cur][n] + s_dep[cur][x];
                s_ok[cur ^ 1][n] = s_ok[cur][n] & s_ok[cur][x];
            } else {
                s_anc[cur ^ 1][n] = -1;
                s_dep[cur ^ 1][n] = s_dep[cur][n];
                s_ok[cur ^ 1][n] = s_ok[cur][n];
            }
        }
        cur ^= 1;
        __syncthreads();
    }
    // a node with a broken parent link (anc -1 before the root) is never reachable:
    // its ok is 0 and so is every descendant's
    int key = -1;
    if (n < N && s_ok[cur][n]) key = (s_dep[cur][n] << 9) | (511 - n);
    for (int off = 32; off >= 1; off >>= 1) key = max(key, __shfl_xor(key, off));
    if ((n & 63) == 0) s_key[n >> 6] = key;
    __syncthreads();
    if (n == 0) {
        int k = s_key[0];
        for (int w = 1; w < kMaxSeqRows / 64; ++w) k = max(k, s_key[w]);
        const int best = 511 - (k & 511);
        const int depth = k >> 9;
        int x = best;
        for (int d = depth; d >= 0; --d) { s_path[d] = x; x = d > 0 ? s_par[x] : x; }
        s_key[0] = best;
        s_key[1] = depth;
        a.accept_len[b] = depth + 1;
    }
    __syncthreads();
    const int best = s_key[0], depth = s_key[1];
    if (n < N) {
        int t = -1;
        if (n < depth) t = s_tok[s_path[n + 1]];
        else if (n == depth) t = s_cand[best];
        a.out_tokens[base + n] = t;
        if (a.out_path) a.out_path[base + n] = n <= depth ? s_path[n] : -1;
    }
}

}  // namespace

hipError_t launch_finish(Dtype dt, const FinishArgs &a, hipStream_t s) {
    if (a.B == 0) return hipSuccess;
    if (a.is_tree) {
        if (dt == kBF16) hipLaunchKernelGGL(k_tree_finish<kBF16>, dim3(a.B), dim3(kMaxSeqRows), 0, s, a);
        else hipLaunchKernelGGL(k_tree_finish<kF32>, dim3(a.B), dim3(kMaxSeqRows), 0, s, a);
    } else {
        const bool one = a.plan.splits == 1;
        if (a.fuse_head) {
            const dim3 block(64 * std::min(a.D + 1, kFinishWaves));   // D >= 1 when the head ran
            const bool bf = a.head_dt == kBF16;
            if (one) {
                if (bf) hipLaunchKernelGGL((k_chain_finish_head<kBF16, kPartOne>), dim3(a.B), block, 0, s, a);
                else hipLaunchKernelGGL((k_chain_finish_head<kF32, kPartOne>), dim3(a.B), block, 0, s, a);
            } else {
                if (bf) hipLaunchKernelGGL((k_chain_finish_head<kBF16, kPartSplit>), dim3(a.B), block, 0, s, a);
                else hipLaunchKernelGGL((k_chain_finish_head<kF32, kPartSplit>), dim3(a.B), block, 0, s, a);
            }
        } else {
            const unsigned blocks = static_cast<unsigned>((a.B + 3) / 4);
            if (one) hipLaunchKernelGGL(k_chain_finish<kPartOne>, dim3(blocks), dim3(256), 0, s, a);
            else hipLaunchKernelGGL(k_chain_finish<kPartSplit>, dim3(blocks), dim3(256), 0, s, a);
        }
    }
    return hipGetLastError();
}

}  // namespace cospec
