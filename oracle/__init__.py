"""CPU oracle for the CoSpec verify-and-arbitrate step.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import this package.  It is never a fallback
for the GPU path and shares no code with it: the two vocabulary/weight loops are
plain C in double precision (cospec_oracle.c, built with gcc), the rest is plain
Python/numpy written from the paper's definitions ("Beyond the Target: From
Imitation to Collaboration in Speculative Decoding", Section 3).

Arrays are numpy: logits and hidden states are float32 arrays or uint16 arrays
holding raw bf16 bit patterns (the dtype says which).

Readings of the paper used here (each also listed with the design notes):
  * ties in an argmax go to the lowest index;
  * entropy is the Shannon entropy in nats of softmax(logits) over the whole
    vocabulary; log-probabilities are reported (logp = x[token] - lse);
  * the head g_phi is a two-layer MLP  z = w2 . relu(W1 h + b1) + b2;
  * the threshold is strict (a = 1[pi > lambda], decided in fp64); decisions with
    |sigma(z) - lambda| <= 1e-3 are flagged ambiguous;
  * every mismatch decision is scored, not only those before the stop;
  * at temperature 1 the target's verification candidate of a row is a sample
    of softmax(row), taken by inversion of a caller-supplied uniform u: the
    smallest v whose cumulative probability (index order) exceeds u;
  * trees: node 0 is the root; child c of p is verified by target row p and
    scored on hidden row c; the accepted node is the deepest node whose whole
    root path passes (match or accepted), ties to the lowest node id.
Parity for the tree tie-break and for the head form is pinned only by these
stated rules (no printed value in the paper covers them).
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

__all__ = [
    "F32", "BF16", "AMBIGUITY_BAND", "build", "row_stats", "element", "head_logits",
    "policy_accept", "chain_length", "chain_tokens", "tree_select", "verify_block",
    "verify_tree", "arbitrate", "chain_outcomes", "tree_outcomes", "RowStats", "sample_rows",
    "cdf_at", "candidates", "policy_sample", "action_logprob", "rl_round", "RL_ALPHA", "RL_BETA",
    "residual_sample", "sps_block", "SPS_BAND", "arbitrator_length", "hybrid_mask",
    "hybrid_attention",
]

F32, BF16 = 0, 1
AMBIGUITY_BAND = 1e-3
RL_ALPHA, RL_BETA = 1.0, 0.25       # failure-reward weights the paper trains with (Appendix C.2)
SPS_BAND = 1e-4                     # speculative-sampling tests closer than this to their uniform

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cospec_oracle.c")
# COSPEC_ORACLE_SANITIZE=1 builds and loads a copy instrumented with AddressSanitizer and
# UndefinedBehaviorSanitizer (host code only; the process must preload libasan), so that
# the pins can be run with every array access of the C loops checked.
_SANITIZE = os.environ.get("COSPEC_ORACLE_SANITIZE") == "1"
_SO = os.path.join(_HERE, "libcospec_oracle_san.so" if _SANITIZE else "libcospec_oracle.so")
_lib = None


def build(sanitize: bool = _SANITIZE) -> str:
    """Compile the C half of the oracle with gcc (IEEE semantics, no fast-math); with
    `sanitize`, instrumented for out-of-bounds accesses and undefined behaviour, any
    finding fatal."""
    so = os.path.join(_HERE, "libcospec_oracle_san.so" if sanitize else "libcospec_oracle.so")
    tmp = so + ".tmp"
    extra = (["-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
              "-fno-sanitize-recover=all"] if sanitize else [])
    subprocess.run(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fno-fast-math"] + extra +
                   ["-o", tmp, _SRC, "-lm"], check=True)
    os.replace(tmp, so)
    return so


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(_SRC):
            build()
        lib = ctypes.CDLL(_SO)
        P = ctypes.c_void_p
        I64 = ctypes.c_int64
        lib.oracle_row_stats.restype = I64
        lib.oracle_row_stats.argtypes = [P, ctypes.c_int, I64, I64, I64, P, P, P, P]
        lib.oracle_sample_rows.restype = I64
        lib.oracle_sample_rows.argtypes = [P, ctypes.c_int, I64, I64, I64, P, P, P, P, P]
        lib.oracle_cdf_at.restype = I64
        lib.oracle_cdf_at.argtypes = [P, ctypes.c_int, I64, I64, I64, P, P, P, P]
        lib.oracle_residual_sample.restype = I64
        lib.oracle_residual_sample.argtypes = [P, P, ctypes.c_int, I64, I64, I64, P, P, P, P, P, P]
        lib.oracle_head.restype = None
        lib.oracle_head.argtypes = [P, ctypes.c_int, I64, P, I64, P, P, P, ctypes.c_double, I64,
                                    I64, P]
        _lib = lib
    return _lib


def _code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError(f"oracle arrays are float32 or uint16 (bf16 bits), got {a.dtype}")


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def element(a: np.ndarray) -> np.ndarray:
    """Exact float64 values of an fp32 or bf16-bit array."""
    if a.dtype == np.float32:
        return a.astype(np.float64)
    return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


@dataclass
class RowStats:
    max: np.ndarray      # float64
    arg: np.ndarray      # int64
    lse: np.ndarray      # float64
    ent: np.ndarray      # float64


def row_stats(rows: np.ndarray) -> RowStats:
    """max, first argmax, log-sum-exp and entropy (nats) of every row of a [..., V]
    array (Section 3.1 greedy verification token; see cospec_oracle.c)."""
    rows = np.ascontiguousarray(rows)
    shape = rows.shape[:-1]
    V = rows.shape[-1]
    n = int(np.prod(shape)) if shape else 1
    mx = np.empty(n, np.float64)
    arg = np.empty(n, np.int64)
    lse = np.empty(n, np.float64)
    ent = np.empty(n, np.float64)
    if n:
        rc = _load().oracle_row_stats(_ptr(rows), _code(rows), V, n, V, _ptr(mx), _ptr(arg),
                                      _ptr(lse), _ptr(ent))
        if rc != 0:
            raise ValueError(f"non-finite logit in row {-rc - 1}")
    return RowStats(mx.reshape(shape), arg.reshape(shape), lse.reshape(shape), ent.reshape(shape))


def sample_rows(rows: np.ndarray, u):
    """Temperature-1 samples of every row of a [..., V] array by inversion (see
    oracle_sample_rows): the smallest v with P(v) > u, P the cumulative softmax in
    index order.  Returns (index, P(index-1), P(index)) with the rows' shape."""
    rows = np.ascontiguousarray(rows)
    shape = rows.shape[:-1]
    V = rows.shape[-1]
    n = int(np.prod(shape)) if shape else 1
    uu = np.ascontiguousarray(np.asarray(u, dtype=np.float64).reshape(n))
    idx = np.empty(n, np.int64)
    lo = np.empty(n, np.float64)
    hi = np.empty(n, np.float64)
    work = np.empty(max(V, 1), np.float64)
    if n:
        rc = _load().oracle_sample_rows(_ptr(rows), _code(rows), V, n, V, _ptr(uu), _ptr(work),
                                        _ptr(idx), _ptr(lo), _ptr(hi))
        if rc != 0:
            raise ValueError(f"non-finite logit in row {-rc - 1}")
    return idx.reshape(shape), lo.reshape(shape), hi.reshape(shape)


def cdf_at(rows: np.ndarray, idx):
    """(P(idx-1), P(idx)) of every row for given candidate indices: the interval of
    uniforms that inversion sampling maps to idx."""
    rows = np.ascontiguousarray(rows)
    shape = rows.shape[:-1]
    V = rows.shape[-1]
    n = int(np.prod(shape)) if shape else 1
    ii = np.ascontiguousarray(np.asarray(idx, dtype=np.int64).reshape(n))
    lo = np.empty(n, np.float64)
    hi = np.empty(n, np.float64)
    work = np.empty(max(V, 1), np.float64)
    if n:
        rc = _load().oracle_cdf_at(_ptr(rows), _code(rows), V, n, V, _ptr(ii), _ptr(work),
                                   _ptr(lo), _ptr(hi))
        if rc == -(n + 1):
            raise IndexError("candidate index out of range")
        if rc != 0:
            raise ValueError(f"non-finite logit in row {-rc - 1}")
    return lo.reshape(shape), hi.reshape(shape)


def residual_sample(target_rows, draft_rows, u=None, query=None):
    """Speculative sampling's resampling step for rows [n, V] (see
    oracle_residual_sample): a sample of max(0, p_T - p_D) / Z by inversion of u,
    or of p_T when draft_rows is None; with `query` the given candidates are
    placed instead.  Returns (index, P(index-1), P(index)), P normalised by Z."""
    t = np.ascontiguousarray(target_rows)
    n, V = t.shape
    d = None if draft_rows is None else np.ascontiguousarray(draft_rows)
    if d is not None and (d.shape != t.shape or _code(d) != _code(t)):
        raise TypeError("target and draft rows must share shape and dtype")
    uu = np.ascontiguousarray(np.zeros(n) if u is None else np.asarray(u, np.float64).reshape(n))
    qq = None if query is None else np.ascontiguousarray(np.asarray(query, np.int64).reshape(n))
    idx = np.empty(n, np.int64) if query is None else qq.copy()
    lo = np.empty(n, np.float64)
    hi = np.empty(n, np.float64)
    work = np.empty(2 * max(V, 1), np.float64)
    if n:
        rc = _load().oracle_residual_sample(_ptr(t), None if d is None else _ptr(d), _code(t), V, n, V,
                                            _ptr(uu), None if qq is None else _ptr(qq), _ptr(work),
                                            _ptr(idx), _ptr(lo), _ptr(hi))
        if rc == -(n + 1):
            raise IndexError("candidate index out of range")
        if rc != 0:
            raise ValueError(f"non-finite logit in row {-rc - 1}")
    return idx, lo, hi


def sps_block(target, draft, draft_tokens, u) -> dict:
    """Standard speculative sampling over a chain block, the distribution-preserving
    baseline the paper runs at T = 1 (Section 3.1, stochastic decoding; Appendix C.3).

    target [B, K+1, V], draft [B, K, V], draft_tokens [B, K] (drawn from the draft),
    u [B, K+1] uniforms.  Draft token i (rows i-1) is accepted when u[b, i-1] <
    min(1, p_T(token) / p_D(token)); the round stops at the first rejection s and
    emits draft tokens 1..s-1, then a sample of max(0, p_T - p_D) from rows s-1 by
    inversion of u[b, K], or, with every token accepted (s = K+1), a sample of p_T
    from target row K.  The test is taken in fp64; tests within SPS_BAND of their
    uniform are flagged ambiguous, and `stops` lists every round length the
    ambiguous tests allow.
    """
    B, K1, V = target.shape
    K = K1 - 1
    toks = np.asarray(draft_tokens, dtype=np.int64)
    uu = np.asarray(u, dtype=np.float64)
    if toks.size and (toks.min() < 0 or toks.max() >= V):
        raise ValueError("draft token out of range")
    ts = row_stats(target)
    ds = row_stats(draft)
    logp_t = _gather(target[:, :K, :], toks) - ts.lse[:, :K]
    logp_d = _gather(draft, toks) - ds.lse
    ratio = np.exp(logp_t - logp_d)
    accept = uu[:, :K] < ratio
    ambiguous = np.abs(uu[:, :K] - ratio) <= SPS_BAND
    accept_len = np.empty(B, np.int64)
    tokens = np.full((B, K + 1), -1, np.int64)
    stops = []
    for b in range(B):
        s = K + 1
        for i in range(1, K + 1):
            if not accept[b, i - 1]:
                s = i
                break
        accept_len[b] = s
        tokens[b, : s - 1] = toks[b, : s - 1]
        tokens[b, s - 1] = final_token(target[b], draft[b], s, uu[b, K])
        possible, certain = set(), False
        for i in range(1, K + 1):                  # the stop can be any ambiguous test before
            if ambiguous[b, i - 1]:                # the first certain rejection
                possible.add(i)
            elif not accept[b, i - 1]:
                possible.add(i)
                certain = True
                break
        if not certain:
            possible.add(K + 1)
        stops.append(possible)
    return dict(tgt_lse=ts.lse, drf_lse=ds.lse, logp_tgt=logp_t, logp_drf=logp_d, ratio=ratio,
                accept=accept, ambiguous=ambiguous, accept_len=accept_len, tokens=tokens, stops=stops)


def final_token(target_seq, draft_seq, s: int, u_last: float, query=None):
    """The token a speculative-sampling round of length s emits last (see sps_block):
    from the residual of rows s-1 when s <= K, from target row K when s = K+1.
    With `query`, returns (P(query-1), P(query)) of that distribution instead."""
    K = draft_seq.shape[0]
    t = target_seq[s - 1: s]
    d = draft_seq[s - 1: s] if s <= K else None
    if query is None:
        return int(residual_sample(t, d, [u_last])[0][0])
    _, lo, hi = residual_sample(t, d, query=[query])
    return float(lo[0]), float(hi[0])


def candidates(target, stats: "RowStats", sample_u=None, override=None):
    """The target's verification candidate of every target row: the argmax at
    T = 0 (Section 3.1), a temperature-1 sample by inversion of the uniform
    `sample_u` at T = 1 (Section 3.1, stochastic decoding; Appendix C.3).  `override` replaces the
    computed candidates (a test passes another implementation's candidates
    after checking each against cdf_at)."""
    if override is not None:
        return np.asarray(override, dtype=np.int64).reshape(stats.arg.shape)
    if sample_u is None:
        return stats.arg
    return sample_rows(target, sample_u)[0]


def head_logits(hidden: np.ndarray, rows, w1: np.ndarray, b1: Optional[np.ndarray],
                w2: np.ndarray, b2: float) -> np.ndarray:
    """z = w2 . relu(W1 h + b1) + b2 (Section 3.3, z_i = g_phi(h)) for hidden rows `rows`
    of a [n, d] array, in float64."""
    hidden = np.ascontiguousarray(hidden)
    w1 = np.ascontiguousarray(w1)
    w2 = np.ascontiguousarray(w2)
    code = _code(hidden)
    if _code(w1) != code or _code(w2) != code or (b1 is not None and _code(b1) != code):
        raise TypeError("hidden states and head weights must share one dtype")
    hdim, d = w1.shape
    assert hidden.shape[-1] == d and w2.shape == (hdim,)
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    n_hidden = int(np.prod(hidden.shape[:-1]))
    if rows.size and (rows.min() < 0 or rows.max() >= n_hidden):
        raise IndexError("hidden row index out of range")
    b1c = None if b1 is None else np.ascontiguousarray(b1)
    out = np.empty(rows.size, np.float64)
    if rows.size:
        _load().oracle_head(_ptr(hidden), code, d, _ptr(rows), rows.size, _ptr(w1),
                            None if b1c is None else _ptr(b1c), _ptr(w2), float(b2), d, hdim,
                            _ptr(out))
    return out


def policy_accept(z: np.ndarray, lam: float):
    """pi = sigma(z) (Eq. policy-prob) and a = 1[pi > lambda] (Eq. infer_thre), both in
    fp64 with lambda as given.  Decisions with |pi - lambda| <= 1e-3 are flagged
    ambiguous: an implementation that rounds differently may take them either way."""
    z = np.asarray(z, dtype=np.float64)
    lam = float(lam)
    with np.errstate(over="ignore"):
        pi = 1.0 / (1.0 + np.exp(-z))
    accept = pi > lam
    ambiguous = np.abs(pi - lam) <= AMBIGUITY_BAND
    return accept, pi, ambiguous


def policy_sample(z: np.ndarray, u):
    """Sampled arbitration (Section 3.4: at training time mismatch actions are drawn
    from pi_theta): a = 1[u < pi] for a caller-supplied uniform u, with pi = sigma(z),
    in fp64; decisions with |pi - u| <= 1e-3 are flagged ambiguous."""
    z = np.asarray(z, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    with np.errstate(over="ignore"):
        pi = 1.0 / (1.0 + np.exp(-z))
    accept = u < pi
    ambiguous = np.abs(pi - u) <= AMBIGUITY_BAND
    return accept, pi, ambiguous


def action_logprob(z: np.ndarray, accept) -> np.ndarray:
    """log pi_theta(a | q) of the action taken on a mismatch decision (the rollout-time
    probability in the PPO ratio of Section 3.4): log sigma(z) when a = 1 and
    log(1 - sigma(z)) = log sigma(-z) when a = 0, in fp64."""
    z = np.asarray(z, dtype=np.float64)
    x = np.where(np.asarray(accept, bool), z, -z)
    # log sigma(x) = -log(1 + e^-x), written without overflow for either sign of x
    return np.where(x >= 0, -np.log1p(np.exp(-np.abs(x))), x - np.log1p(np.exp(-np.abs(x))))


def rl_round(delta, accept, logp_tgt, correct: bool, alpha: float = RL_ALPHA,
             beta: float = RL_BETA) -> dict:
    """Per-round statistics of the reinforcement-learning stage (Section 3.4) for one
    chain round with decisions i = 1..K (index i-1 of each array).

      s      the round length (Eq. cospec_length);
      I_r    effective actions {i : Delta_i = 0 and i <= min(s, K)};
      i*     the first mismatch min{i : Delta_i = 0} (0 here when there is none);
      rho    (s - i*) / ((K+1) - i*), NaN without a mismatch;
      i_rej  the first rejected mismatch, K+1 when none is rejected;
      S_acc  {i in I_r : a_i = 1, i < i_rej};  S_rej = {i_rej} if i_rej <= K;
      g      correct rollout: rho on every effective decision; failed rollout
             (Eq. failure_penalty): -alpha |l_i| on S_acc, -beta on S_rej.
             g is reported as 0 outside I_r, where the paper defines no term;
      J      the round's share of the rollout return, the sum of g over I_r.
    """
    K = len(delta)
    s = chain_length(delta, accept)
    mism = [i for i in range(1, K + 1) if not delta[i - 1]]
    i_star = mism[0] if mism else 0
    rho = (s - i_star) / ((K + 1) - i_star) if mism else math.nan
    rejected = [i for i in mism if not accept[i - 1]]
    i_rej = rejected[0] if rejected else K + 1
    eff = [False] * K
    s_acc = [False] * K
    s_rej = [False] * K
    g = [0.0] * K
    for i in mism:
        if i <= min(s, K):
            eff[i - 1] = True
            s_acc[i - 1] = bool(accept[i - 1]) and i < i_rej
            s_rej[i - 1] = i == i_rej and i_rej <= K
            if correct:
                g[i - 1] = rho
            else:
                g[i - 1] = (-alpha * abs(float(logp_tgt[i - 1])) * s_acc[i - 1]
                            - beta * s_rej[i - 1])
    J = float(sum(g[i] for i in range(K) if eff[i]))
    return dict(s=s, i_star=i_star, rho=rho, i_rej=i_rej, effective=np.array(eff),
                s_acc=np.array(s_acc), s_rej=np.array(s_rej), g=np.array(g), J=J)


def chain_length(delta, accept) -> int:
    """Eq. cospec_length: s = min{i : Delta_i = 0 and a_i = 0} (1-based), else K+1."""
    K = len(delta)
    rejected = [i for i in range(1, K + 1) if not delta[i - 1] and not accept[i - 1]]
    return min(rejected) if rejected else K + 1


def chain_tokens(s: int, draft_tokens, target_argmax) -> list:
    """Tokens a round of length s emits (Section 3.3): draft tokens 1..s-1, then the
    target's token at position s (the bonus token when s = K+1).  target_argmax[j]
    is the argmax of target row j, i.e. ytilde_{j+1}.  Padded with -1 to K+1."""
    K = len(draft_tokens)
    out = [int(t) for t in draft_tokens[: s - 1]] + [int(target_argmax[s - 1])]
    return out + [-1] * (K + 1 - len(out))


def tree_select(parent, passed):
    """Accepted node of a token tree (tree reading of Eq. cospec_length): a node is
    reachable when every node on its root path (root excluded) passes; the
    accepted node is the deepest reachable node, ties to the lowest id.
    Returns (node, depth of every node, path from the root to the node)."""
    N = len(parent)
    ok = [False] * N
    depth = [0] * N
    ok[0] = True
    for n in range(1, N):
        p = int(parent[n])
        ok[n] = ok[p] and bool(passed[n])
        depth[n] = depth[p] + 1
    best = 0
    for n in range(1, N):
        if ok[n] and depth[n] > depth[best]:
            best = n
    path = [best]
    while path[-1] != 0:
        path.append(int(parent[path[-1]]))
    return best, depth, path[::-1]


def _tree_emit(best, path, node_tokens, target_argmax, N):
    toks = [int(node_tokens[n]) for n in path[1:]] + [int(target_argmax[best])]
    return toks + [-1] * (N - len(toks)), list(path) + [-1] * (N - len(path))


def _gather(rows: np.ndarray, tokens: np.ndarray) -> np.ndarray:
    """rows[..., tokens[...]] as exact float64 (one logit per decision)."""
    g = np.take_along_axis(rows, tokens[..., None].astype(np.int64), axis=-1)[..., 0]
    return element(g)


def _head_arrays(head):
    w1, b1, w2, b2 = head
    return w1, b1, w2, float(b2)


def verify_block(target, draft, draft_tokens, hidden, head, lam: float, sample_u=None,
                 cand_override=None, policy_u=None, correct=None, alpha: float = RL_ALPHA,
                 beta: float = RL_BETA) -> dict:
    """Oracle of one chain verify step.

    target [B, K+1, V], draft [B, K, V] (float32 or bf16 bits), draft_tokens int
    [B, K], hidden [B, K, d], head = (W1 [h, d], b1 [h] or None, w2 [h], b2).
    Decision i (1..K) compares draft token i with the target's candidate from row
    i-1 (Section 3.1, Delta_i): its argmax, or with sample_u [B, K+1] its
    temperature-1 sample (see candidates()).  Mismatches are scored with the head
    (Section 3.3) and the round stops at the first rejected mismatch
    (Eq. cospec_length), emitting the candidate of row s-1 last.  With policy_u
    [B, K] mismatch actions are sampled (policy_sample) instead of thresholded.
    With correct [B] (the rollouts' Corr flags) the per-round RL statistics of
    rl_round are added, from the nominal actions.
    """
    B, K1, V = target.shape
    K = K1 - 1
    assert draft.shape == (B, K, V) and draft_tokens.shape == (B, K)
    toks = np.asarray(draft_tokens, dtype=np.int64)
    if toks.size and (toks.min() < 0 or toks.max() >= V):
        raise ValueError("draft token out of range")
    ts = row_stats(target)
    ds = row_stats(draft)
    cand = candidates(target, ts, sample_u, cand_override)
    ytil = cand[:, :K]                                     # ytilde_i = candidate of row i-1
    delta = (toks == ytil)
    logp_tgt = _gather(target[:, :K, :], toks) - ts.lse[:, :K]
    logp_drf = _gather(draft, toks) - ds.lse
    w1, b1, w2, b2 = _head_arrays(head)
    mism = np.argwhere(~delta)                             # (b, i-1) pairs
    z = np.full((B, K), np.nan)
    if len(mism):
        rows = mism[:, 0] * K + mism[:, 1]
        z[mism[:, 0], mism[:, 1]] = head_logits(hidden.reshape(B * K, -1), rows, w1, b1, w2, b2)
    if policy_u is None:
        acc_m, pi_m, amb_m = policy_accept(np.where(delta, 0.0, z), lam)
    else:
        acc_m, pi_m, amb_m = policy_sample(np.where(delta, 0.0, z), policy_u)
    accept = np.where(delta, True, acc_m)
    pi = np.where(delta, 1.0, pi_m)
    ambiguous = np.where(delta, False, amb_m)
    z_tilde = np.where(delta, np.inf, z)
    logp_action = np.where(delta, 0.0, action_logprob(np.where(delta, 0.0, z), accept))
    accept_len = np.empty(B, np.int64)
    tokens = np.empty((B, K + 1), np.int64)
    outcomes = []
    rl = []
    for b in range(B):
        s = chain_length(delta[b], accept[b])
        accept_len[b] = s
        tokens[b] = chain_tokens(s, toks[b], cand[b])
        outcomes.append(chain_outcomes(delta[b], accept[b], ambiguous[b], toks[b], cand[b]))
        if correct is not None:
            rl.append(rl_round(delta[b], accept[b], logp_tgt[b], bool(correct[b]), alpha, beta))
    return dict(logp_action=logp_action, rl=rl if correct is not None else None,
                tgt_max=ts.max, tgt_arg=ts.arg, tgt_lse=ts.lse, tgt_ent=ts.ent, tgt_cand=cand,
                drf_max=ds.max, drf_arg=ds.arg, drf_lse=ds.lse, drf_ent=ds.ent,
                delta=delta, logp_tgt=logp_tgt, logp_drf=logp_drf, z=z, z_tilde=z_tilde,
                pi=pi, accept=accept, ambiguous=ambiguous, accept_len=accept_len,
                tokens=tokens, outcomes=outcomes)


def chain_outcomes(delta, accept, ambiguous, draft_tokens, target_argmax, cap: int = 16):
    """Every (s, tokens) the round can produce when each ambiguous mismatch decision
    may go either way; None when more than `cap` such decisions could matter."""
    K = len(delta)
    certain_stop = [i for i in range(K) if not delta[i] and not ambiguous[i] and not accept[i]]
    limit = certain_stop[0] if certain_stop else K
    free = [i for i in range(limit) if not delta[i] and ambiguous[i]]
    if len(free) > cap:
        return None
    outs = set()
    for mask in range(1 << len(free)):
        a = [bool(x) for x in accept]
        for j, i in enumerate(free):
            a[i] = bool((mask >> j) & 1)
        s = chain_length(delta, a)
        outs.add((s, tuple(chain_tokens(s, draft_tokens, target_argmax))))
    return outs


def _internal(parent) -> np.ndarray:
    N = len(parent)
    has_child = np.zeros(N, bool)
    for n in range(1, N):
        has_child[int(parent[n])] = True
    return has_child


def verify_tree(target, draft, parent, node_tokens, hidden, head, lam: float, sample_u=None,
                cand_override=None, policy_u=None) -> dict:
    """Oracle of one tree verify step (tree reading of Section 3.1/3.3).

    target, draft [B, N, V]; parent int [B, N] (parent[0] = -1, parent[n] < n);
    node_tokens int [B, N]; hidden [B, N, d].  Only draft rows of nodes with a
    child are reduced (leaf draft rows verify nothing); their statistics are NaN /
    -1 for leaves.  Node 0 carries no decision.  With sample_u [B, N] the
    candidate of each target row is its temperature-1 sample (see candidates()).
    """
    B, N, V = target.shape
    par = np.asarray(parent, dtype=np.int64)
    toks = np.asarray(node_tokens, dtype=np.int64)
    for b in range(B):
        if par[b, 0] != -1 or any(not (0 <= par[b, n] < n) for n in range(1, N)):
            raise ValueError("parent array must satisfy parent[0] = -1, 0 <= parent[n] < n")
    if N > 1 and (toks[:, 1:].min() < 0 or toks[:, 1:].max() >= V):
        raise ValueError("node token out of range")
    ts = row_stats(target)
    cand = candidates(target, ts, sample_u, cand_override)
    internal = np.stack([_internal(par[b]) for b in range(B)])
    drf_max = np.full((B, N), np.nan)
    drf_arg = np.full((B, N), -1, np.int64)
    drf_lse = np.full((B, N), np.nan)
    drf_ent = np.full((B, N), np.nan)
    ib, inn = np.nonzero(internal)
    if len(ib):
        ds = row_stats(draft[ib, inn])
        drf_max[ib, inn], drf_arg[ib, inn], drf_lse[ib, inn], drf_ent[ib, inn] = (
            ds.max, ds.arg, ds.lse, ds.ent)
    delta = np.ones((B, N), bool)
    logp_tgt = np.full((B, N), np.nan)
    logp_drf = np.full((B, N), np.nan)
    for b in range(B):
        for n in range(1, N):
            p = par[b, n]
            t = toks[b, n]
            delta[b, n] = t == cand[b, p]
            logp_tgt[b, n] = element(target[b, p, t:t + 1])[0] - ts.lse[b, p]
            logp_drf[b, n] = element(draft[b, p, t:t + 1])[0] - drf_lse[b, p]
    w1, b1, w2, b2 = _head_arrays(head)
    z = np.full((B, N), np.nan)
    mb, mn = np.nonzero(~delta)
    if len(mb):
        z[mb, mn] = head_logits(hidden.reshape(B * N, -1), mb * N + mn, w1, b1, w2, b2)
    if policy_u is None:
        acc_m, pi_m, amb_m = policy_accept(np.where(delta, 0.0, z), lam)
    else:
        acc_m, pi_m, amb_m = policy_sample(np.where(delta, 0.0, z), policy_u)
    accept = np.where(delta, True, acc_m)
    pi = np.where(delta, 1.0, pi_m)
    ambiguous = np.where(delta, False, amb_m)
    z_tilde = np.where(delta, np.inf, z)
    logp_action = np.where(delta, 0.0, action_logprob(np.where(delta, 0.0, z), accept))
    accept_len = np.empty(B, np.int64)
    tokens = np.empty((B, N), np.int64)
    path = np.empty((B, N), np.int64)
    outcomes = []
    for b in range(B):
        passed = delta[b] | accept[b]
        best, depth, pth = tree_select(par[b], passed)
        accept_len[b] = depth[best] + 1
        tokens[b], path[b] = _tree_emit(best, pth, toks[b], cand[b], N)
        outcomes.append(tree_outcomes(par[b], delta[b], accept[b], ambiguous[b], toks[b],
                                      cand[b]))
    return dict(logp_action=logp_action, tgt_max=ts.max, tgt_arg=ts.arg, tgt_lse=ts.lse,
                tgt_ent=ts.ent, tgt_cand=cand, drf_max=drf_max, drf_arg=drf_arg, drf_lse=drf_lse, drf_ent=drf_ent,
                internal=internal, delta=delta, logp_tgt=logp_tgt, logp_drf=logp_drf, z=z,
                z_tilde=z_tilde, pi=pi, accept=accept, ambiguous=ambiguous,
                accept_len=accept_len, tokens=tokens, path=path, outcomes=outcomes)


def tree_outcomes(parent, delta, accept, ambiguous, node_tokens, target_argmax, cap: int = 16):
    """Every (accept_len, tokens, path) a tree round can produce when each ambiguous
    mismatch decision may go either way; None when more than `cap` could matter."""
    N = len(parent)
    # a node's decision can matter only if no certain failure lies on its root path
    blocked = [False] * N
    for n in range(1, N):
        p = int(parent[n])
        certain_fail = (not delta[n]) and (not ambiguous[n]) and (not accept[n])
        blocked[n] = blocked[p] or certain_fail
    free = [n for n in range(1, N) if not delta[n] and ambiguous[n] and not blocked[int(parent[n])]]
    if len(free) > cap:
        return None
    outs = set()
    for mask in range(1 << len(free)):
        a = [bool(x) for x in accept]
        for j, n in enumerate(free):
            a[n] = bool((mask >> j) & 1)
        passed = [bool(delta[n]) or a[n] for n in range(N)]
        best, depth, pth = tree_select(parent, passed)
        toks, pth_pad = _tree_emit(best, pth, node_tokens, target_argmax, N)
        outs.add((depth[best] + 1, tuple(toks), tuple(pth_pad)))
    return outs


def arbitrate(hidden, rows, head, lam: float) -> dict:
    """Head alone over selected hidden rows (rows=None: all rows): z, pi, a and the
    ambiguity flag (Section 3.3, Eq. policy-prob and Eq. infer_thre without the
    match override, which needs Delta)."""
    hidden2 = hidden.reshape(-1, hidden.shape[-1])
    if rows is None:
        rows = np.arange(hidden2.shape[0])
    w1, b1, w2, b2 = _head_arrays(head)
    z = head_logits(hidden2, rows, w1, b1, w2, b2)
    a, pi, amb = policy_accept(z, lam)
    return dict(z=z, pi=pi, accept=a, ambiguous=amb)


# ---------------------------------------------------------------- the arbitrator's hybrid attention

def arbitrator_length(ctx_len: int, K: int) -> int:
    """Length of the arbitrator input q = [context, SEP, draft 1..K, SEP, candidates
    1..K, SEP] (Eq. arb_input): l_c + 2K + 3."""
    return int(ctx_len) + 2 * K + 3


def hybrid_mask(ctx_len, K: int, L: int) -> np.ndarray:
    """Attention mask of the arbitrator (Section 3.3) for a batch padded to length L:
    mask[b, i, j] = 1 when query position i of sequence b may attend key position j.
    Positions before l_c (the context) attend causally within the context; the
    draft/target region, read here as starting at the first [SEP] (position l_c)
    and ending at l = l_c + 2K + 3, attends to every position of the context and of
    the region; nothing flows from the region back into the context.  Padding
    positions i >= l attend only to themselves (no row is empty)."""
    ctx = np.asarray(ctx_len, dtype=np.int64)
    B = ctx.shape[0]
    out = np.zeros((B, L, L), np.uint8)
    for b in range(B):
        lc = int(ctx[b])
        ln = arbitrator_length(lc, K)
        for i in range(L):
            for j in range(L):
                if i >= ln:
                    out[b, i, j] = i == j
                elif i < lc:
                    out[b, i, j] = j <= i
                else:
                    out[b, i, j] = j < ln
    return out


def hybrid_attention(q, k, v, ctx_len, q_start, K: int, scale: float) -> np.ndarray:
    """softmax(q k^T * scale + mask) v for the queries of each sequence, in fp64.

    q [B, n_q, Hq, D]: queries at positions q_start[b] .. q_start[b] + n_q - 1;
    k, v [B, L, Hkv, D]: keys and values of positions 0..L-1; Hq is a multiple of
    Hkv and query head h reads key/value head h // (Hq / Hkv) (grouped queries).
    The mask is hybrid_mask's rule for that sequence; queries at padding positions
    (>= l) give zeros.  Arrays are float32 or uint16 bf16 bits."""
    qf, kf, vf = element(np.asarray(q)), element(np.asarray(k)), element(np.asarray(v))
    B, nq, Hq, D = qf.shape
    L, Hkv = kf.shape[1], kf.shape[2]
    grp = Hq // Hkv
    out = np.zeros((B, nq, Hq, D))
    for b in range(B):
        lc = int(ctx_len[b])
        ln = arbitrator_length(lc, K)
        if ln > L:
            raise ValueError(f"sequence {b}: input length {ln} exceeds the {L} cached positions")
        for r in range(nq):
            p = int(q_start[b]) + r
            if p >= ln:
                continue
            vis = np.arange(p + 1) if p < lc else np.arange(ln)
            for h in range(Hq):
                kh = h // grp
                s = (kf[b, vis, kh, :] @ qf[b, r, h, :]) * scale
                w = np.exp(s - s.max())
                out[b, r, h, :] = (w / w.sum()) @ vf[b, vis, kh, :]
    return out
