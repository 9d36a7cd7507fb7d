"""Comparison of a verify step's GPU outputs with the oracle's.

TEST INFRASTRUCTURE ONLY (used by tests/, the package smoke check and the
benchmark's parity re-check).  The rules:
  * integers (argmax, Delta, accept flags outside the ambiguity band, accept
    lengths, tokens, paths) must be bit-exact;
  * where a decision lies within 1e-3 of the threshold, the GPU's
    (accept_len, tokens[, path]) must be one member of the oracle's outcome set;
  * floating-point features must agree within `contract` = 2e-3 * max(1, |ref|)
    (the stated fp32-accumulation tolerance) and, as a tighter engineering
    check that fp32 arithmetic easily meets, within the per-feature bounds in
    TIGHT.
"""
from __future__ import annotations

import numpy as np

CONTRACT_RTOL = 2e-3
# fp32 cumulative sums over up to ~300 segment masses and 512 elements: a few ulp
# each, so 5e-5 in probability covers the worst accumulation with margin
CDF_TOL = 5e-5
# (rtol, atol) per feature for the tighter check
TIGHT = dict(max=(0.0, 0.0), lse=(1e-5, 1e-5), ent=(1e-5, 1e-4), logp=(1e-5, 1e-4),
             z=(1e-4, 1e-4), pi=(0.0, 2e-5))


class ParityError(AssertionError):
    pass


def _np(x):
    if hasattr(x, "detach"):
        x = x.detach().cpu().numpy()
    return np.asarray(x)


def _close(name, got, ref, kind, stats, mask=None):
    got = _np(got).astype(np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if mask is not None:
        got, ref = got[mask], ref[mask]
    if got.size == 0:
        return
    err = np.abs(got - ref)
    scale = np.maximum(1.0, np.abs(ref))
    bad_contract = ~(err <= CONTRACT_RTOL * scale)
    rtol, atol = TIGHT[kind]
    bad_tight = ~(err <= atol + rtol * np.abs(ref))
    stats[name] = float(np.max(err / scale))
    if bad_contract.any() or bad_tight.any():
        i = int(np.flatnonzero(bad_contract | bad_tight)[0])
        raise ParityError(f"{name}: {int((bad_contract | bad_tight).sum())} of {got.size} outside "
                          f"tolerance; first at flat index {i}: gpu {got.flat[i]!r} oracle {ref.flat[i]!r}")


def _exact(name, got, ref, mask=None):
    got = _np(got).astype(np.int64)
    ref = np.asarray(ref).astype(np.int64)
    if mask is not None:
        got, ref = got[mask], ref[mask]
    if not np.array_equal(got, ref):
        i = int(np.flatnonzero(got != ref)[0])
        raise ParityError(f"{name}: {int((got != ref).sum())} of {got.size} differ; first at flat "
                          f"index {i}: gpu {got.flat[i]} oracle {ref.flat[i]}")


def _decisions(gpu, ref, dmask, stats):
    """Per-decision features; dmask selects real decision slots."""
    delta = ref["delta"]
    _exact("delta", gpu["delta"], delta, dmask)
    _close("logp_tgt", gpu["logp_tgt"], ref["logp_tgt"], "logp", stats, dmask)
    _close("logp_drf", gpu["logp_drf"], ref["logp_drf"], "logp", stats, dmask)
    zt = _np(gpu["z_tilde"])
    match = dmask & delta
    mism = dmask & ~delta
    if not np.all(np.isposinf(zt[match])):
        raise ParityError("z_tilde must be +inf on matched decisions")
    _close("z", zt, ref["z"], "z", stats, mism)
    _close("policy", gpu["policy"], ref["pi"], "pi", stats, dmask)
    acc = _np(gpu["accept"]).astype(bool)
    firm = dmask & ~ref["ambiguous"]
    _exact("accept", acc, ref["accept"], firm)
    stats["ambiguous_decisions"] = int((dmask & ref["ambiguous"]).sum())
    if "logp_action" in gpu and "logp_action" in ref:
        la = _np(gpu["logp_action"])
        if not np.all(la[match] == 0.0):
            raise ParityError("logp_action must be 0 on matched decisions")
        scored = mism & firm & np.isfinite(ref["logp_action"]) & np.isfinite(_np(gpu["z_tilde"]))
        _close("logp_action", la, ref["logp_action"], "logp", stats, scored)


def _outcomes(got_len, got_tok, got_path, ref, stats):
    n_amb_seq = 0
    for b, outs in enumerate(ref["outcomes"]):
        key_len = int(got_len[b])
        key_tok = tuple(int(x) for x in got_tok[b])
        nominal = (int(ref["accept_len"][b]), tuple(int(x) for x in ref["tokens"][b]))
        if got_path is not None:
            key = (key_len, key_tok, tuple(int(x) for x in got_path[b]))
            nominal = nominal + (tuple(int(x) for x in ref["path"][b]),)
        else:
            key = (key_len, key_tok)
        if outs is None:
            raise ParityError(f"sequence {b}: too many ambiguous decisions to enumerate")
        if len(outs) > 1:
            n_amb_seq += 1
        if key not in outs:
            raise ParityError(f"sequence {b}: gpu outcome {key} not among the oracle's {sorted(outs)[:4]} "
                              f"(nominal {nominal})")
    stats["sequences_with_ambiguity"] = n_amb_seq


def check_candidates(got, rows, u, stats: dict = None):
    """Temperature-1 candidates chosen on the GPU against the oracle's inversion of
    the same uniforms.  rows [..., V] (the logits the GPU read), u [...].  Returns
    the GPU's candidates (each one checked) for the oracle's downstream steps."""
    from . import sample_rows, cdf_at
    got = _np(got).astype(np.int64)
    u = np.asarray(u, dtype=np.float64)
    ref, _, _ = sample_rows(rows, u)
    diff = got != ref
    if diff.any():
        lo, hi = cdf_at(rows[diff], got[diff])
        ud = u[diff]
        ok = (lo - CDF_TOL <= ud) & (ud < hi + CDF_TOL)
        if not ok.all():
            i = int(np.flatnonzero(~ok)[0])
            raise ParityError(f"temperature-1 candidate {got[diff][i]} (oracle {ref[diff][i]}) does not "
                              f"invert u={ud[i]!r}: its interval is [{lo[i]!r}, {hi[i]!r})")
    if stats is not None:
        stats["candidates_at_boundary"] = int(diff.sum())
    return got


def check_block(gpu: dict, ref: dict) -> dict:
    """GPU result of cospec_verify_block (features included) against oracle.verify_block."""
    stats = {}
    _exact("tgt_argmax", gpu["tgt_argmax"], ref["tgt_arg"])
    _exact("tgt_candidate", gpu["tgt_candidate"], ref["tgt_cand"])
    _exact("drf_argmax", gpu["drf_argmax"], ref["drf_arg"])
    _close("tgt_max", gpu["tgt_max"], ref["tgt_max"], "max", stats)
    _close("drf_max", gpu["drf_max"], ref["drf_max"], "max", stats)
    _close("tgt_lse", gpu["tgt_lse"], ref["tgt_lse"], "lse", stats)
    _close("drf_lse", gpu["drf_lse"], ref["drf_lse"], "lse", stats)
    _close("tgt_entropy", gpu["tgt_entropy"], ref["tgt_ent"], "ent", stats)
    _close("drf_entropy", gpu["drf_entropy"], ref["drf_ent"], "ent", stats)
    dmask = np.ones(ref["delta"].shape, bool)
    _decisions(gpu, ref, dmask, stats)
    _outcomes(_np(gpu["accept_len"]), _np(gpu["tokens"]), None, ref, stats)
    return stats


def check_tree(gpu: dict, ref: dict) -> dict:
    """GPU result of cospec_verify_tree (features included) against oracle.verify_tree."""
    stats = {}
    _exact("tgt_argmax", gpu["tgt_argmax"], ref["tgt_arg"])
    _exact("tgt_candidate", gpu["tgt_candidate"], ref["tgt_cand"])
    _close("tgt_max", gpu["tgt_max"], ref["tgt_max"], "max", stats)
    _close("tgt_lse", gpu["tgt_lse"], ref["tgt_lse"], "lse", stats)
    _close("tgt_entropy", gpu["tgt_entropy"], ref["tgt_ent"], "ent", stats)
    internal = ref["internal"]
    _exact("drf_argmax", gpu["drf_argmax"], ref["drf_arg"])          # -1 on leaves on both sides
    _close("drf_lse", gpu["drf_lse"], ref["drf_lse"], "lse", stats, internal)
    _close("drf_entropy", gpu["drf_entropy"], ref["drf_ent"], "ent", stats, internal)
    if not np.all(np.isnan(_np(gpu["drf_lse"])[~internal])):
        raise ParityError("draft statistics of leaf nodes must be NaN")
    dmask = np.ones(ref["delta"].shape, bool)
    dmask[:, 0] = False
    _decisions(gpu, ref, dmask, stats)
    _outcomes(_np(gpu["accept_len"]), _np(gpu["tokens"]), _np(gpu["path"]), ref, stats)
    return stats


def check_outputs_only(gpu: dict, ref: dict, tree: bool = False) -> dict:
    """Accept lengths and tokens alone (for calls made without features)."""
    stats = {}
    _outcomes(_np(gpu["accept_len"]), _np(gpu["tokens"]), _np(gpu["path"]) if tree else None,
              ref, stats)
    return stats


def check_rl(gpu: dict, ref: dict, correct, alpha: float, beta: float) -> dict:
    """Per-round RL statistics of a chain step (the rl_* outputs) against
    oracle.rl_round, evaluated on the GPU's own actions (which check_block has
    already matched to the oracle's outside the ambiguity band) and the oracle's
    log p_T."""
    from . import rl_round
    stats = {}
    acc = _np(gpu["accept"]).astype(bool)
    B, K = acc.shape
    eff, sacc, g = np.zeros((B, K), bool), np.zeros((B, K), bool), np.zeros((B, K))
    istar, irej, rho, J = (np.zeros(B, np.int64), np.zeros(B, np.int64), np.zeros(B), np.zeros(B))
    for b in range(B):
        r = rl_round(ref["delta"][b], acc[b], ref["logp_tgt"][b], bool(correct[b]), alpha, beta)
        eff[b], sacc[b], g[b] = r["effective"], r["s_acc"], r["g"]
        istar[b], irej[b], rho[b], J[b] = r["i_star"], r["i_rej"], r["rho"], r["J"]
    _exact("rl_effective", gpu["rl_effective"], eff)
    _exact("rl_in_s_acc", gpu["rl_in_s_acc"], sacc)
    _exact("rl_first_mismatch", gpu["rl_first_mismatch"], istar)
    _exact("rl_first_reject", gpu["rl_first_reject"], irej)
    has = istar > 0
    if not np.all(np.isnan(_np(gpu["rl_rho"])[~has])):
        raise ParityError("rho must be NaN for rounds without a mismatch")
    _close("rl_rho", gpu["rl_rho"], rho, "logp", stats, has)
    _close("rl_reward", gpu["rl_reward"], g, "logp", stats)
    _close("rl_return", gpu["rl_round_return"], J, "logp", stats)
    return stats


def check_sps(gpu: dict, ref: dict, target, draft, u) -> dict:
    """GPU result of cospec_verify_block_sps against oracle.sps_block: acceptance
    tests outside SPS_BAND bit-exact, the round length one the ambiguous tests allow,
    the draft prefix exact, and the last token inside its interval of the
    distribution it is drawn from (residual or target row), up to CDF_TOL plus the
    fp32 cancellation of p_T - p_D relative to the residual's total weight."""
    from . import final_token, element, SPS_BAND  # noqa: F401
    stats = {}
    acc = _np(gpu["accept"]).astype(bool)
    firm = ~ref["ambiguous"]
    _exact("sps accept", acc, ref["accept"], firm)
    s = _np(gpu["accept_len"]).astype(np.int64)
    tok = _np(gpu["tokens"]).astype(np.int64)
    B, K1 = tok.shape
    K = K1 - 1
    u = np.asarray(u, np.float64)
    worst = 0.0
    for b in range(B):
        if int(s[b]) not in ref["stops"][b]:
            raise ParityError(f"sequence {b}: round length {s[b]} not among {sorted(ref['stops'][b])}")
        toks_in = np.asarray(ref["tokens"][b])
        if s[b] == ref["accept_len"][b] and not np.array_equal(tok[b, : s[b] - 1], toks_in[: s[b] - 1]):
            raise ParityError(f"sequence {b}: draft prefix differs")
        if (tok[b, s[b]:] != -1).any():
            raise ParityError(f"sequence {b}: tokens after the round are not -1")
        lo, hi = final_token(target[b], draft[b], int(s[b]), u[b, K], query=int(tok[b, s[b] - 1]))
        if s[b] <= K:
            pt = np.exp(element(target[b, s[b] - 1]) - ref["tgt_lse"][b, s[b] - 1])
            pd = np.exp(element(draft[b, s[b] - 1]) - ref["drf_lse"][b, s[b] - 1])
            z = np.maximum(pt - pd, 0.0).sum()
        else:
            z = 1.0
        tol = CDF_TOL + 3e-6 / z
        if not (lo - tol <= u[b, K] < hi + tol):
            raise ParityError(f"sequence {b}: last token {tok[b, s[b] - 1]} does not invert u={u[b, K]!r}: "
                              f"interval [{lo!r}, {hi!r}), tolerance {tol:.1e}")
        worst = max(worst, max(lo - u[b, K], u[b, K] - hi, 0.0))
    stats["last_token_interval_excess"] = worst
    _close("tgt_lse", gpu["tgt_lse"], ref["tgt_lse"], "lse", stats)
    _close("drf_lse", gpu["drf_lse"], ref["drf_lse"], "lse", stats)
    _close("logp_tgt", gpu["logp_tgt"], ref["logp_tgt"], "logp", stats)
    _close("logp_drf", gpu["logp_drf"], ref["logp_drf"], "logp", stats)
    _close("accept_prob", gpu["policy"], np.minimum(ref["ratio"], 1.0), "pi", stats)
    stats["ambiguous_decisions"] = int(ref["ambiguous"].sum())
    return stats
