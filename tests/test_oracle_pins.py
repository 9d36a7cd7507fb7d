"""Pins of the CPU oracle against what the paper and mathematics fix.

Nothing here compares the oracle with itself: every expected value is a closed
form, a hand-worked fixture (tests/golden/), a brute-force enumeration, an
independent formulation of the same definition, or a numpy/scipy routine that
the oracle does not call.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

from paper_2605_24793_amd import workloads

# The mutation tests re-run these pins against a copy of the oracle with a planted
# mistake; they name that copy's directory here.  Normal runs use oracle/.
_UNDER_TEST = os.environ.get("COSPEC_ORACLE_UNDER_TEST")
if _UNDER_TEST:
    import importlib.util
    _spec = importlib.util.spec_from_file_location(
        "oracle_under_test", os.path.join(_UNDER_TEST, "__init__.py"),
        submodule_search_locations=[_UNDER_TEST])
    oracle = importlib.util.module_from_spec(_spec)
    _spec.loader.exec_module(oracle)
else:
    import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _rows_from_fixture(r):
    if "two_level" in r:
        t = r["two_level"]
        x = np.full(t["V"], t["c"], np.float32)
        x[t["k"]] = t["c"] + t["L"]
        return x
    if r["dtype"] == "bf16":
        return np.array(r["bits"], np.uint16)
    return np.array(r["values"], np.float32)


# ---------------------------------------------------------------- row statistics

@pytest.mark.parametrize("r", _load("row_stats.json")["rows"], ids=lambda r: r["name"])
def test_row_stats_golden(r):
    env = {k: getattr(math, k) for k in ("log", "exp")}
    if "two_level" in r:
        env.update(r["two_level"])
    assert eval(r["lse_expr"], env) == pytest.approx(r["lse"], rel=1e-15)
    st = oracle.row_stats(_rows_from_fixture(r)[None])
    assert st.arg[0] == r["argmax"]
    assert st.max[0] == r["max"]
    assert st.lse[0] == pytest.approx(r["lse"], rel=1e-12, abs=1e-12)
    assert st.ent[0] == pytest.approx(r["entropy"], rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("V,c", [(1, 0.0), (7, -3.25), (32000, 1.5), (151936, -20.0)])
def test_constant_row_closed_form(V, c):
    st = oracle.row_stats(np.full((1, V), c, np.float32))
    assert st.arg[0] == 0
    assert st.lse[0] == pytest.approx(c + math.log(V), rel=1e-12, abs=1e-12)
    assert st.ent[0] == pytest.approx(math.log(V), rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("V,c,L,k", [(2, 0.0, 1.0, 1), (1000, 3.0, -2.0, 5), (128256, -1.0, 12.0, 128255),
                                     (151936, 4.0, 30.0, 0)])
def test_two_level_row_closed_form(V, c, L, k):
    x = np.full(V, c, np.float32)
    x[k] = c + L
    st = oracle.row_stats(x[None])
    if L > 0:
        assert st.arg[0] == k
    else:
        assert st.arg[0] == (0 if k != 0 else 1)
    # p = e^L / (e^L + V - 1) at index k, q = 1 - p spread over the other V - 1,
    # written without cancellation so the closed form itself stays exact to ~1e-15
    lse = c + math.log(math.exp(L) + V - 1)
    log_p = -math.log1p((V - 1) * math.exp(-L))
    log_q1 = -math.log1p(math.exp(L) / (V - 1)) - math.log(V - 1)   # log(q / (V - 1))
    p, q = math.exp(log_p), (V - 1) * math.exp(log_q1)
    ent = -p * log_p - q * log_q1
    assert st.lse[0] == pytest.approx(lse, rel=1e-12, abs=1e-12)
    # a plain sequential fp64 sum of V terms onto the dominant one carries an absolute
    # error of about sqrt(V) * 2^-53; with a +30 peak the entropy itself is ~4e-7
    assert st.ent[0] == pytest.approx(ent, rel=1e-9, abs=1e-10)


def test_argmax_ties_lowest_index():
    rng = np.random.default_rng(5)
    for V in (2, 9, 4096, 151936):
        x = rng.normal(size=V).astype(np.float32)
        pos = np.sort(rng.choice(V, size=min(V, 5), replace=False))
        x[pos] = 100.0
        st = oracle.row_stats(x[None])
        assert st.arg[0] == pos[0]
        assert int(np.argmax(x)) == pos[0]          # numpy documents first occurrence


def test_row_stats_against_scipy_float64():
    rng = np.random.default_rng(11)
    for V, scale in ((17, 1.0), (4099, 4.0), (32000, 3.0)):
        x = (rng.normal(size=(6, V)) * scale).astype(np.float32)
        st = oracle.row_stats(x)
        x64 = x.astype(np.float64)
        lse = scipy.special.logsumexp(x64, axis=-1)
        p = scipy.special.softmax(x64, axis=-1)
        ent = scipy.special.entr(p).sum(axis=-1)
        np.testing.assert_allclose(st.lse, lse, rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(st.ent, ent, rtol=1e-10, atol=1e-12)
        np.testing.assert_array_equal(st.arg, np.argmax(x, axis=-1))
        np.testing.assert_array_equal(st.max, x.max(axis=-1))


def test_bf16_widening_matches_torch():
    g = torch.Generator().manual_seed(3)
    t = (torch.randn(3, 1000, generator=g) * 8).to(torch.bfloat16)
    bits = workloads.bf16_bits(t)
    np.testing.assert_array_equal(oracle.element(bits), t.double().numpy())
    st = oracle.row_stats(bits)
    np.testing.assert_allclose(st.lse, torch.logsumexp(t.double(), -1).numpy(), rtol=1e-13)
    np.testing.assert_array_equal(st.arg, torch.argmax(t.float(), -1).numpy())


def test_shift_invariance():
    rng = np.random.default_rng(2)
    # multiples of 2^-10 below 64 in magnitude: adding 8 is exact in fp32
    x = (np.round(rng.normal(size=(3, 5000)) * 4 * 1024) / 1024).astype(np.float32)
    a = oracle.row_stats(x)
    b = oracle.row_stats((x + np.float32(8.0)).astype(np.float32))
    np.testing.assert_allclose(b.lse, a.lse + 8.0, rtol=1e-13)
    np.testing.assert_allclose(b.ent, a.ent, rtol=1e-10, atol=1e-12)
    np.testing.assert_array_equal(b.arg, a.arg)


def test_nonfinite_rejected():
    x = np.zeros((2, 8), np.float32)
    x[1, 3] = np.inf
    with pytest.raises(ValueError, match="row 1"):
        oracle.row_stats(x)


# ---------------------------------------------------------------- temperature-1 sampling

@pytest.mark.parametrize("V,c", [(1, 0.0), (7, 2.0), (1000, -5.5)])
def test_sample_constant_row_closed_form(V, c):
    # p = 1/V everywhere: inversion maps u to floor(u V), with P(k-1) = k/V, P(k) = (k+1)/V
    k = np.arange(V)
    u = (k + 0.5) / V
    idx, lo, hi = oracle.sample_rows(np.full((V, V), c, np.float32), u)
    np.testing.assert_array_equal(idx, k)
    np.testing.assert_allclose(lo, k / V, rtol=0, atol=1e-13)
    np.testing.assert_allclose(hi, (k + 1) / V, rtol=0, atol=1e-13)


def test_sample_grid_counts_match_softmax():
    # inversion of the quasi-uniform grid u_k = (k + 1/2)/N hits index v exactly
    # #{k : P(v-1) <= u_k < P(v)} times, which is within 1 of N p_v
    rng = np.random.default_rng(41)
    V, N = 40, 20000
    x = (rng.normal(size=V) * 3).astype(np.float32)
    p = scipy.special.softmax(x.astype(np.float64))
    idx, _, _ = oracle.sample_rows(np.tile(x, (N, 1)), (np.arange(N) + 0.5) / N)
    counts = np.bincount(idx, minlength=V)
    assert np.abs(counts - N * p).max() <= 1.0 + 1e-9
    assert (np.diff(idx) >= 0).all()                 # monotone in u


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sample_against_cumsum_searchsorted(dtype):
    rng = np.random.default_rng(43)
    rows, V = 64, 3001
    x = torch.from_numpy((rng.normal(size=(rows, V)) * 4).astype(np.float32))
    if dtype == "bf16":
        arr = workloads.bf16_bits(x.to(torch.bfloat16))
    else:
        arr = x.numpy()
    u = rng.random(rows).astype(np.float32).astype(np.float64)
    idx, lo, hi = oracle.sample_rows(arr, u)
    cdf = np.cumsum(scipy.special.softmax(oracle.element(arr), axis=-1), axis=-1)
    want = np.array([np.searchsorted(cdf[r], u[r], side="right") for r in range(rows)])
    np.testing.assert_array_equal(idx, want)
    r = np.arange(rows)
    np.testing.assert_allclose(hi, cdf[r, idx], rtol=0, atol=1e-12)
    np.testing.assert_allclose(lo, np.where(idx > 0, cdf[r, np.maximum(idx - 1, 0)], 0.0), rtol=0,
                               atol=1e-12)
    assert ((lo <= u) & (u < hi)).all()
    lo2, hi2 = oracle.cdf_at(arr, want)
    np.testing.assert_allclose(lo2, lo, rtol=0, atol=1e-12)
    np.testing.assert_allclose(hi2, hi, rtol=0, atol=1e-12)


def test_sample_peaked_and_edge_uniforms():
    V = 1000
    x = np.zeros((4, V), np.float32)
    x[:, 321] = 60.0                                  # every other index carries < 1e-23 of the mass
    idx, _, _ = oracle.sample_rows(x, [1e-9, 0.25, 0.5, 1 - 1e-9])
    assert (idx == 321).all()
    y = np.zeros((2, 5), np.float32)
    idx, lo, _ = oracle.sample_rows(y, [0.0, np.nextafter(1.0, 0.0)])
    assert idx[0] == 0 and lo[0] == 0.0
    assert idx[1] == 4
    with pytest.raises(IndexError):
        oracle.cdf_at(y, [0, 5])


# ---------------------------------------------------------------- head

def test_head_identity_block_closed_form():
    rng = np.random.default_rng(7)
    d, h = 48, 16
    w1 = np.zeros((h, d), np.float32)
    w1[np.arange(h), np.arange(h)] = 1.0          # W1 = [I, 0]
    w2 = np.ones(h, np.float32)
    hid = rng.normal(size=(5, d)).astype(np.float32)
    z = oracle.head_logits(hid, np.arange(5), w1, None, w2, 0.25)
    expect = np.maximum(hid[:, :h].astype(np.float64), 0).sum(axis=1) + 0.25
    np.testing.assert_allclose(z, expect, rtol=1e-15)


def test_head_bias_paths():
    rng = np.random.default_rng(8)
    d, h = 32, 8
    w1 = rng.normal(size=(h, d)).astype(np.float32)
    w2 = rng.normal(size=h).astype(np.float32)
    hid = rng.normal(size=(3, d)).astype(np.float32)
    # b1 so negative that every unit is off: z = b2 exactly
    b1 = np.full(h, -1e6, np.float32)
    np.testing.assert_array_equal(oracle.head_logits(hid, [0, 1, 2], w1, b1, w2, -0.5), -0.5)
    # b1 so positive that every unit is on: z = w2.(W1 h + b1) + b2 (linear)
    b1 = np.full(h, 1e4, np.float32)
    lin = (hid.astype(np.float64) @ w1.astype(np.float64).T + 1e4) @ w2.astype(np.float64) + 0.5
    np.testing.assert_allclose(oracle.head_logits(hid, [0, 1, 2], w1, b1, w2, 0.5), lin, rtol=1e-12)


def test_head_against_numpy_matmul_bf16():
    g = torch.Generator().manual_seed(9)
    d, h = 256, 64
    hid = torch.randn(10, d, generator=g).to(torch.bfloat16)
    w1 = (torch.randn(h, d, generator=g) / 16).to(torch.bfloat16)
    b1 = (torch.randn(h, generator=g) * 0.3).to(torch.bfloat16)
    w2 = (torch.randn(h, generator=g) / 8).to(torch.bfloat16)
    rows = np.array([9, 0, 3, 3])
    z = oracle.head_logits(workloads.bf16_bits(hid), rows, workloads.bf16_bits(w1),
                           workloads.bf16_bits(b1), workloads.bf16_bits(w2), 0.125)
    H, W1, B1, W2 = (t.double().numpy() for t in (hid, w1, b1, w2))
    expect = np.maximum(H[rows] @ W1.T + B1, 0.0) @ W2 + 0.125
    np.testing.assert_allclose(z, expect, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- policy threshold

def test_policy_sigmoid_and_strict_threshold():
    z = np.array([0.0, -3.0, 2.0, 40.0, -120.0])
    a, pi, amb = oracle.policy_accept(z, 0.5)
    np.testing.assert_allclose(pi, scipy.special.expit(z), rtol=1e-15)
    assert pi[0] == 0.5 and not a[0] and amb[0]       # sigma(0) = 0.5 is not > 0.5
    assert list(a[1:]) == [False, True, True, False]
    a, _, _ = oracle.policy_accept(np.array([0.0]), 0.4999)
    assert a[0]


@pytest.mark.parametrize("lam", [1.0, 1.5, 1e9])
def test_policy_lambda_ge_one_never_accepts(lam):
    a, _, _ = oracle.policy_accept(np.array([-50.0, 0.0, 17.0, 100.0, 1e30]), lam)
    assert not a.any()


@pytest.mark.parametrize("lam", [-1e-7, -0.5, -1e9])
def test_policy_lambda_negative_always_accepts(lam):
    a, _, _ = oracle.policy_accept(np.array([-200.0, -17.0, 0.0, 50.0]), lam)
    assert a.all()


# ---------------------------------------------------------------- chain scan

def _sequential(delta, accept):
    for i in range(len(delta)):
        if not delta[i] and not accept[i]:
            return i + 1
    return len(delta) + 1


def _longest_passing_prefix(delta, accept):
    L = 0
    while L < len(delta) and (delta[L] or accept[L]):
        L += 1
    return L + 1


@pytest.mark.parametrize("K", [1, 2, 3, 5, 7])
def test_chain_length_brute_force(K):
    for delta in itertools.product([0, 1], repeat=K):
        strict = oracle.chain_length(delta, [0] * K)
        for acc in itertools.product([0, 1], repeat=K):
            s = oracle.chain_length(delta, acc)
            assert s == _sequential(delta, acc) == _longest_passing_prefix(delta, acc)
            assert 1 <= s <= K + 1
            assert s >= strict
            for j in range(K):                  # accepting one more never shortens the round
                if not acc[j]:
                    up = list(acc)
                    up[j] = 1
                    assert oracle.chain_length(delta, up) >= s


@pytest.mark.parametrize("c", _load("chain_rounds.json")["cases"], ids=lambda c: c["name"])
def test_chain_golden(c):
    delta = [int(a == b) for a, b in zip(c["draft"], c["target_tokens"])]
    assert delta == c["delta"]
    s = oracle.chain_length(delta, c["accept"])
    assert s == c["s"]
    assert oracle.chain_tokens(s, c["draft"], c["target_tokens"]) == c["tokens"]
    assert oracle.chain_length(delta, [0] * c["K"]) == c["strict_s"]


# ---------------------------------------------------------------- tree scan

def _tree_brute(parent, passed):
    N = len(parent)
    best, best_depth = 0, 0
    for n in range(N):
        path = [n]
        while path[-1] != 0:
            path.append(parent[path[-1]])
        if all(passed[m] for m in path[:-1]):
            if len(path) - 1 > best_depth:
                best, best_depth = n, len(path) - 1
    return best, best_depth


@pytest.mark.parametrize("seed", range(12))
def test_tree_select_brute_force(seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(1, 10))
    parent = [-1] + [int(rng.integers(0, n)) for n in range(1, N)]
    for bits in itertools.product([0, 1], repeat=N - 1):
        passed = [1] + list(bits)
        node, depth, path = oracle.tree_select(parent, passed)
        bnode, bdepth = _tree_brute(parent, passed)
        assert node == bnode and depth[node] == bdepth
        assert path[0] == 0 and path[-1] == node and len(path) == bdepth + 1
        assert all(parent[path[k + 1]] == path[k] for k in range(len(path) - 1))


def test_tree_golden():
    g = _load("tree_rounds.json")
    for c in g["cases"]:
        node, depth, path = oracle.tree_select(g["parent"], c["passed"])
        assert node == c["node"] and depth[node] + 1 == c["accept_len"] and path == c["path"]
        toks = [g["node_tokens"][n] for n in path[1:]] + [g["target_argmax"][node]]
        assert toks == c["tokens"]


def test_path_tree_equals_chain_scan():
    for K in range(1, 7):
        parent = [-1] + list(range(K))
        for delta in itertools.product([0, 1], repeat=K):
            for acc in itertools.product([0, 1], repeat=K):
                passed = [1] + [d or a for d, a in zip(delta, acc)]
                node, depth, _ = oracle.tree_select(parent, passed)
                assert depth[node] + 1 == oracle.chain_length(delta, acc)


# ---------------------------------------------------------------- whole verify step

def _np_chain(wl):
    conv = (lambda t: workloads.bf16_bits(t)) if wl.target.dtype == torch.bfloat16 else (
        lambda t: t.contiguous().numpy())
    head = (conv(wl.head.w1), None if wl.head.b1 is None else conv(wl.head.b1), conv(wl.head.w2),
            wl.head.b2)
    return conv(wl.target), conv(wl.draft), wl.draft_tokens.numpy(), conv(wl.hidden), head


def _small_chain(dtype="bf16", B=6, K=5, V=3001, noise=1.0, seed=21, bias=True, **kw):
    return workloads.make_chain(B=B, K=K, V=V, d=64, h=32, dtype=dtype, noise=noise, seed=seed,
                                bias=bias, **kw)


def _greedy_spd(target64, draft_tokens):
    """Textbook greedy speculative decoding, one position at a time."""
    K = len(draft_tokens)
    out = []
    for i in range(K):
        t = int(np.argmax(target64[i]))
        if t != int(draft_tokens[i]):
            out.append(t)
            return len(out), out
        out.append(int(draft_tokens[i]))
    out.append(int(np.argmax(target64[K])))
    return K + 1, out


@pytest.mark.parametrize("lam", [1.0, 2.5])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_always_defer_is_greedy_spd(lam, dtype):
    wl = _small_chain(dtype=dtype, B=10, noise=0.7, peaked=0.3)
    t, d, toks, hid, head = _np_chain(wl)
    r = oracle.verify_block(t, d, toks, hid, head, lam)
    t64 = oracle.element(t)
    for b in range(wl.B):
        s, out = _greedy_spd(t64[b], toks[b])
        assert r["accept_len"][b] == s
        assert list(r["tokens"][b][:s]) == out and all(x == -1 for x in r["tokens"][b][s:])
        strict = [i + 1 for i in range(wl.K) if not r["delta"][b, i]]
        assert s == (strict[0] if strict else wl.K + 1)     # Eq. strict-spd-len


@pytest.mark.parametrize("lam", [-1e-6, -3.0])
def test_always_accept_emits_block_plus_bonus(lam):
    wl = _small_chain(B=5)
    t, d, toks, hid, head = _np_chain(wl)
    r = oracle.verify_block(t, d, toks, hid, head, lam)
    t64 = oracle.element(t)
    for b in range(wl.B):
        assert r["accept_len"][b] == wl.K + 1
        assert list(r["tokens"][b]) == list(toks[b]) + [int(np.argmax(t64[b, wl.K]))]


def test_block_features_against_scipy():
    wl = _small_chain(B=4, K=6, V=2049, peaked=0.25)
    t, d, toks, hid, head = _np_chain(wl)
    r = oracle.verify_block(t, d, toks, hid, head, 0.5)
    t64, d64 = oracle.element(t), oracle.element(d)
    K = wl.K
    lt = scipy.special.log_softmax(t64, axis=-1)
    ld = scipy.special.log_softmax(d64, axis=-1)
    for b in range(wl.B):
        for i in range(1, K + 1):
            y = toks[b, i - 1]
            # l_i = log p_T(yhat_i | prefix, yhat_<i): target row i-1 (Section 3.4)
            assert r["logp_tgt"][b, i - 1] == pytest.approx(lt[b, i - 1, y], abs=1e-12)
            assert r["logp_drf"][b, i - 1] == pytest.approx(ld[b, i - 1, y], abs=1e-12)
            assert r["delta"][b, i - 1] == (y == np.argmax(t64[b, i - 1]))
    np.testing.assert_allclose(r["tgt_ent"], scipy.special.entr(np.exp(lt)).sum(-1), rtol=1e-9)
    np.testing.assert_allclose(r["drf_ent"], scipy.special.entr(np.exp(ld)).sum(-1), rtol=1e-9)
    # z only on mismatches, +inf (forced accept) on matches (Eq. policy-prob)
    assert np.isinf(r["z_tilde"][r["delta"]]).all() and r["accept"][r["delta"]].all()
    mism = ~r["delta"]
    W1, W2 = (oracle.element(x).astype(np.float64) for x in (head[0], head[2]))
    B1 = oracle.element(head[1])
    Hh = oracle.element(hid)
    zz = np.maximum(Hh @ W1.T + B1, 0) @ W2 + head[3]
    np.testing.assert_allclose(r["z"][mism], zz[mism], rtol=1e-12, atol=1e-14)


def test_chain_outcome_set_enumerates_ambiguous_decisions():
    delta = [1, 0, 0, 1]
    accept = [1, 1, 0, 1]
    amb = [False, True, False, False]
    outs = oracle.chain_outcomes(delta, accept, amb, [7, 8, 9, 10], [7, 1, 2, 10, 5])
    assert outs == {(3, (7, 8, 2, -1, -1)), (2, (7, 1, -1, -1, -1))}
    # an ambiguous decision after a certain rejection cannot matter
    outs = oracle.chain_outcomes([0, 0], [0, 1], [False, True], [3, 4], [5, 6, 7])
    assert outs == {(1, (5, -1, -1))}


def test_chain_outcome_sets_hand_worked():
    draft, cand = [1, 2, 3, 4, 5], [10, 11, 12, 13, 14, 15]
    # decision 4 is a certain rejection, so only the ambiguous decision 1 before it can
    # matter: accepted, the round runs to the stop at 4; rejected, it stops at 1.  The
    # ambiguous decision 5 lies after the certain stop and cannot matter.
    outs = oracle.chain_outcomes([0, 0, 1, 0, 0], [1, 1, 1, 0, 1], [True, False, False, False, True],
                                 draft, cand)
    assert outs == {(4, (1, 2, 3, 13, -1, -1)), (1, (10, -1, -1, -1, -1, -1))}
    # two ambiguous decisions and no certain rejection: (1, 3) both accepted gives the whole
    # block and the bonus token; 3 rejected stops at 3; 1 rejected stops at 1 whatever 3 does
    outs = oracle.chain_outcomes([0, 1, 0], [0, 1, 1], [True, False, True], [1, 2, 3], [7, 8, 9, 6])
    assert outs == {(4, (1, 2, 3, 6)), (3, (1, 2, 9, -1)), (1, (7, -1, -1, -1))}
    # no ambiguous decision: the one nominal outcome, a certain rejection included
    outs = oracle.chain_outcomes([0, 0], [1, 0], [False, False], [1, 2], [7, 8, 9])
    assert outs == {(2, (1, 8, -1))}


# A 7-node tree for the hand-worked outcome sets below:
#     0 -> 1 -> 3 -> 6,   1 -> 4,   0 -> 2 -> 5
_T_PARENT = [-1, 0, 0, 1, 1, 2, 3]
_T_TOKENS = [-1, 11, 12, 13, 14, 15, 16]
_T_CAND = [21, 22, 23, 24, 25, 26, 27]         # the candidate of target row n


def _tree_outcome(accept_len, tokens, path, N=7):
    return (accept_len, tuple(tokens + [-1] * (N - len(tokens))), tuple(path + [-1] * (N - len(path))))


def test_tree_outcomes_ambiguous_node_under_a_certain_failure():
    # node 1 is a certain rejection; the ambiguous node 3 lies below it and cannot
    # matter.  Reachable: 0, 2, 5 -> the deepest is node 5
    delta = [1, 0, 1, 0, 1, 1, 1]
    accept = [1, 0, 1, 1, 1, 1, 1]
    amb = [False, False, False, True, False, False, False]
    outs = oracle.tree_outcomes(_T_PARENT, delta, accept, amb, _T_TOKENS, _T_CAND)
    assert outs == {_tree_outcome(3, [12, 15, 26], [0, 2, 5])}


def test_tree_outcomes_ambiguous_node_on_a_live_path():
    # node 3 is ambiguous with every ancestor passing: accepted, the round reaches node 6
    # (depth 3); rejected, the deepest reachable nodes are 4 and 5 (depth 2) and the
    # lower id, 4, wins
    delta = [1, 1, 1, 0, 1, 1, 1]
    accept = [1, 1, 1, 1, 1, 1, 1]
    amb = [False, False, False, True, False, False, False]
    outs = oracle.tree_outcomes(_T_PARENT, delta, accept, amb, _T_TOKENS, _T_CAND)
    assert outs == {_tree_outcome(4, [11, 13, 16, 27], [0, 1, 3, 6]),
                    _tree_outcome(3, [11, 14, 25], [0, 1, 4])}


def test_tree_outcomes_ambiguous_siblings_tie_to_the_lower_id():
    # node 3 is a certain rejection (its child 6 is unreachable); the ambiguous nodes 4 and
    # 5 share depth 2.  Node 4 accepted: it wins the tie whatever 5 does.  Only 5
    # accepted: node 5.  Neither: depth 1, nodes 1 and 2 tie and node 1 wins.
    delta = [1, 1, 1, 0, 0, 0, 1]
    accept = [1, 1, 1, 0, 1, 0, 1]
    amb = [False, False, False, False, True, True, False]
    outs = oracle.tree_outcomes(_T_PARENT, delta, accept, amb, _T_TOKENS, _T_CAND)
    assert outs == {_tree_outcome(3, [11, 14, 25], [0, 1, 4]),
                    _tree_outcome(3, [12, 15, 26], [0, 2, 5]),
                    _tree_outcome(2, [11, 22], [0, 1])}


def test_tree_outcomes_count_only_decisions_that_can_matter():
    # node 1 is a certain rejection with a matched child 2 under it, and the 17 ambiguous
    # nodes 3..19 hang below node 2; node 20 is a matched child of the root.  None of the
    # 17 can matter, so the set is the single nominal outcome and the cap of 16 free
    # decisions is not reached.
    N = 21
    parent = [-1, 0, 1] + [2] * 17 + [0]
    delta = [1, 0, 1] + [0] * 17 + [1]
    accept = [1, 0, 1] + [1] * 17 + [1]
    amb = [False, False, False] + [True] * 17 + [False]
    toks = [-1] + list(range(100, 100 + N - 1))
    cand = list(range(200, 200 + N))
    outs = oracle.tree_outcomes(parent, delta, accept, amb, toks, cand)
    assert outs == {(2, tuple([119, 220] + [-1] * (N - 2)), tuple([0, 20] + [-1] * (N - 2)))}
    # the same 17 on a live path exceed the cap: the set is not enumerated
    delta2 = [1, 1] + delta[2:]
    assert oracle.tree_outcomes(parent, delta2, accept, amb, toks, cand) is None


def test_path_tree_verify_equals_chain_verify():
    wl = _small_chain(B=4, K=5, V=1500, noise=0.6)
    t, d, toks, hid, head = _np_chain(wl)
    rc = oracle.verify_block(t, d, toks, hid, head, 0.5)
    B, K = wl.B, wl.K
    N = K + 1
    dpad = np.concatenate([d, d[:, :1]], axis=1)          # leaf draft row: never read
    parent = np.tile(np.array([-1] + list(range(K))), (B, 1))
    node_tokens = np.concatenate([np.full((B, 1), -1), toks], axis=1)
    hpad = np.concatenate([hid[:, :1], hid], axis=1)       # hidden row n <-> decision n
    rt = oracle.verify_tree(t, dpad, parent, node_tokens, hpad, head, 0.5)
    np.testing.assert_array_equal(rt["accept_len"], rc["accept_len"])
    np.testing.assert_array_equal(rt["tokens"][:, :K + 1], rc["tokens"])
    np.testing.assert_array_equal(rt["delta"][:, 1:], rc["delta"])
    np.testing.assert_allclose(rt["z"][:, 1:], rc["z"], rtol=0, atol=0, equal_nan=True)
    np.testing.assert_array_equal(rt["drf_arg"][:, :K], rc["drf_arg"])
    assert (rt["drf_arg"][:, K] == -1).all()


def test_tree_config_structure():
    tr = workloads.make_config(5, B=2)
    assert tr.N == 60
    par = tr.parent.numpy()
    for b in range(tr.B):
        assert par[b, 0] == -1 and all(0 <= par[b, n] < n for n in range(1, 60))
        _, depth, _ = oracle.tree_select(par[b], [1] * 60)
        assert max(depth) == 6


def _sampled_spd(target64, draft_tokens, u):
    """Exact-match speculative decoding whose target candidates are temperature-1
    samples (inversion of u through numpy's cumulative softmax), position by position."""
    K = len(draft_tokens)
    cand = [int(np.searchsorted(np.cumsum(scipy.special.softmax(target64[i])), u[i], side="right"))
            for i in range(K + 1)]
    out = []
    for i in range(K):
        if cand[i] != int(draft_tokens[i]):
            return len(out) + 1, out + [cand[i]], cand
        out.append(int(draft_tokens[i]))
    return K + 1, out + [cand[K]], cand


def test_sampled_candidates_always_defer_is_sampled_spd():
    wl = _small_chain(B=12, K=5, V=400, noise=0.5)
    t, d, toks, hid, head = _np_chain(wl)
    rng = np.random.default_rng(47)
    u = rng.random((wl.B, wl.K + 1)).astype(np.float32).astype(np.float64)
    r = oracle.verify_block(t, d, toks, hid, head, 1.0, sample_u=u)
    t64 = oracle.element(t)
    differs = 0
    for b in range(wl.B):
        s, out, cand = _sampled_spd(t64[b], toks[b], u[b])
        assert list(r["tgt_cand"][b]) == cand
        assert r["accept_len"][b] == s
        assert list(r["tokens"][b][:s]) == out
        differs += int(cand != list(np.argmax(t64[b], axis=-1)))
    assert differs > 0                      # the samples are not the argmax everywhere


def test_sampled_candidates_on_peaked_rows_equal_greedy():
    wl = _small_chain(B=6, K=4, V=500, noise=0.8)
    t, d, toks, hid, head = _np_chain(wl)
    t = t.copy()
    t64 = oracle.element(t)
    am = np.argmax(t64, axis=-1)
    # lift each row's argmax by 64: every other entry keeps less than 1e-25 of the mass
    bits = workloads.bf16_bits(torch.from_numpy(t64 + 64.0 * (np.arange(t.shape[-1]) == am[..., None]))
                               .to(torch.bfloat16))
    u = np.random.default_rng(3).uniform(1e-6, 1 - 1e-6, size=(wl.B, wl.K + 1))
    r1 = oracle.verify_block(bits, d, toks, hid, head, 0.5, sample_u=u)
    r0 = oracle.verify_block(bits, d, toks, hid, head, 0.5)
    np.testing.assert_array_equal(r1["tgt_cand"], r0["tgt_arg"])
    np.testing.assert_array_equal(r1["tokens"], r0["tokens"])


# ---------------------------------------------------------------- sampled arbitration and RL statistics

@pytest.mark.parametrize("r", _load("rl_rounds.json")["rounds"], ids=lambda r: r["name"])
def test_rl_round_golden(r):
    for correct, gk, jk in ((True, "g_correct", "J_correct"), (False, "g_failed", "J_failed")):
        out = oracle.rl_round(r["delta"], r["accept"], r["logp"], correct, r["alpha"], r["beta"])
        assert out["s"] == r["s"] and out["i_star"] == r["i_star"] and out["i_rej"] == r["i_rej"]
        if r["rho"] is None:
            assert math.isnan(out["rho"])
        else:
            assert out["rho"] == pytest.approx(r["rho"], abs=1e-15)
        np.testing.assert_array_equal(out["effective"], np.array(r["effective"], bool))
        np.testing.assert_array_equal(out["s_acc"], np.array(r["s_acc"], bool))
        np.testing.assert_array_equal(out["s_rej"], np.array(r["s_rej"], bool))
        np.testing.assert_allclose(out["g"], r[gk], rtol=0, atol=1e-15)
        assert out["J"] == pytest.approx(r[jk], abs=1e-15)


@pytest.mark.parametrize("K", [1, 2, 4, 6])
def test_rl_round_invariants_brute_force(K):
    logp = -np.linspace(0.1, 3.0, K)
    for delta in itertools.product([0, 1], repeat=K):
        for acc in itertools.product([0, 1], repeat=K):
            a = [1 if d else x for d, x in zip(delta, acc)]         # matches are forced accepts
            ok = oracle.rl_round(delta, a, logp, True)
            bad = oracle.rl_round(delta, a, logp, False)
            s = oracle.chain_length(delta, a)
            mism = [i + 1 for i in range(K) if not delta[i]]
            eff = ok["effective"]
            assert ok["s"] == s == ok["i_rej"] or (ok["i_rej"] == K + 1 and s == K + 1)
            assert all(not delta[i] for i in range(K) if eff[i])      # I_r holds mismatches only
            assert all(i + 1 <= min(s, K) for i in range(K) if eff[i])
            assert not (bad["s_acc"] & bad["s_rej"]).any()
            assert ((bad["s_acc"] | bad["s_rej"]) <= eff).all()
            assert bad["s_rej"].sum() <= 1 and (bad["s_rej"].sum() == 0) == (s == K + 1)
            assert all(g <= 0 for g in bad["g"])
            if mism:
                assert 0.0 <= ok["rho"] <= 1.0
                assert (ok["rho"] == 1.0) == (s == K + 1)
                assert ok["J"] == pytest.approx(eff.sum() * ok["rho"], abs=1e-12)
                if not any(a[i - 1] for i in mism):                    # always defer: rho = 0
                    assert ok["rho"] == 0.0 and ok["J"] == 0.0
                    assert bad["J"] == -oracle.RL_BETA
            else:
                assert math.isnan(ok["rho"]) and not eff.any() and ok["J"] == 0.0 == bad["J"]


def test_policy_sample_strict_and_grid():
    a, pi, amb = oracle.policy_sample(np.zeros(3), [0.5, 0.4999, 0.50001])
    assert list(a) == [False, True, False] and amb.all()          # u < pi, pi(0) = 1/2 exactly
    a, _, _ = oracle.policy_sample(np.array([80.0, -80.0]), [1 - 1e-7, 1e-7])
    assert list(a) == [True, False]
    z = 0.37
    n = 20000
    a, pi, _ = oracle.policy_sample(np.full(n, z), (np.arange(n) + 0.5) / n)
    assert abs(a.mean() - scipy.special.expit(z)) <= 1.0 / n + 1e-7


def test_action_logprob_closed_form():
    z = np.array([-40.0, -3.0, 0.0, 0.5, 7.0, 40.0])
    np.testing.assert_allclose(oracle.action_logprob(z, np.ones(6, bool)), scipy.special.log_expit(z),
                               rtol=1e-13, atol=1e-300)
    np.testing.assert_allclose(oracle.action_logprob(z, np.zeros(6, bool)), scipy.special.log_expit(-z),
                               rtol=1e-13, atol=1e-300)
    assert oracle.action_logprob(np.array([0.0]), [True])[0] == pytest.approx(math.log(0.5), abs=1e-16)


def test_verify_block_sampled_policy_and_rl():
    wl = _small_chain(B=10, K=6, V=700, noise=1.2)
    t, d, toks, hid, head = _np_chain(wl)
    u = np.random.default_rng(5).random((wl.B, wl.K))
    corr = np.arange(wl.B) % 2
    r = oracle.verify_block(t, d, toks, hid, head, 0.5, policy_u=u, correct=corr)
    for b in range(wl.B):
        for i in range(wl.K):
            if not r["delta"][b, i]:
                assert r["accept"][b, i] == (np.float32(u[b, i]) < np.float32(1) / (np.float32(1) + np.exp(
                    -np.float32(r["z"][b, i]))))
        st = r["rl"][b]
        assert st["s"] == r["accept_len"][b]
        ref = oracle.rl_round(r["delta"][b], r["accept"][b], r["logp_tgt"][b], bool(corr[b]))
        np.testing.assert_array_equal(st["g"], ref["g"])
    # sampled actions differ from the lambda = 0.5 threshold somewhere
    r2 = oracle.verify_block(t, d, toks, hid, head, 0.5)
    assert (r["accept"] != r2["accept"]).any()


# ---------------------------------------------------------------- speculative sampling baseline

def _logits_of(p):
    return np.log(np.asarray(p, np.float64)).astype(np.float32)


def test_sps_preserves_the_target_distribution():
    # the defining property of speculative sampling: with the draft token drawn from
    # p_D, the first emitted token is distributed as p_T.  Weight each draft token
    # by p_D and sweep both uniforms over an n x n grid.
    rng = np.random.default_rng(17)
    V, n = 6, 64
    t_logit = (rng.normal(size=V) * 1.5).astype(np.float32)
    d_logit = (rng.normal(size=V) * 1.5).astype(np.float32)
    pT = scipy.special.softmax(t_logit.astype(np.float64))
    pD = scipy.special.softmax(d_logit.astype(np.float64))
    g = (np.arange(n) + 0.5) / n
    ua, ur = np.meshgrid(g, g, indexing="ij")
    m = n * n
    dist = np.zeros(V)
    for y in range(V):
        target = np.tile(t_logit, (m, 2, 1))
        draft = np.tile(d_logit, (m, 1, 1))
        toks = np.full((m, 1), y)
        u = np.stack([ua.ravel(), ur.ravel()], axis=1)
        r = oracle.sps_block(target, draft, toks, u)
        first = r["tokens"][:, 0]
        dist += pD[y] * np.bincount(first, minlength=V) / m
    assert np.abs(dist - pT).max() <= 2.0 / n


def test_sps_equal_models_accept_everything():
    rng = np.random.default_rng(3)
    B, K, V = 5, 4, 50
    x = (rng.normal(size=(B, K + 1, V)) * 2).astype(np.float32)
    toks = rng.integers(0, V, size=(B, K))
    u = rng.random((B, K + 1)) * 0.999
    r = oracle.sps_block(x, x[:, :K].copy(), toks, u)
    assert (r["accept_len"] == K + 1).all()
    np.testing.assert_allclose(r["ratio"], 1.0, rtol=1e-12)
    cdf = np.cumsum(scipy.special.softmax(x[:, K].astype(np.float64), axis=-1), axis=-1)
    for b in range(B):                      # the bonus token: inversion of p_T from row K
        assert r["tokens"][b, K] == np.searchsorted(cdf[b], u[b, K], side="right")
        assert list(r["tokens"][b, :K]) == list(toks[b])


def test_sps_residual_closed_form():
    pT = [0.5, 0.3, 0.2]
    pD = [0.2, 0.5, 0.3]
    target = np.stack([_logits_of(pT), _logits_of(pT)])[None]     # K = 1
    draft = _logits_of(pD)[None, None]
    # token 1: ratio 0.3 / 0.5 = 0.6.  u = 0.7 rejects it; the residual max(0, pT - pD)
    # = (0.3, 0, 0) puts everything on token 0, whatever the second uniform
    for u2 in (0.0, 0.5, 0.999):
        r = oracle.sps_block(target, draft, np.array([[1]]), np.array([[0.7, u2]]))
        assert r["accept_len"][0] == 1 and r["tokens"][0, 0] == 0
        assert r["ratio"][0, 0] == pytest.approx(0.6, rel=1e-6)
    r = oracle.sps_block(target, draft, np.array([[1]]), np.array([[0.5, 0.9]]))
    assert r["accept_len"][0] == 2 and r["tokens"][0, 0] == 1      # accepted: bonus from p_T
    assert r["tokens"][0, 1] == 2                                  # 0.9 > 0.5 + 0.3
    # token 0: ratio 0.5 / 0.2 > 1, accepted for every u < 1
    r = oracle.sps_block(target, draft, np.array([[0]]), np.array([[0.999, 0.1]]))
    assert r["accept_len"][0] == 2


def test_sps_residual_interval_closed_form():
    # p_T = (0.4, 0.1, 0.3, 0.2), p_D = (0.1, 0.4, 0.1, 0.4): the residual max(0, p_T - p_D)
    # = (0.3, 0, 0.2, 0) has Z = 0.5, so its normalised cumulative weights are
    # 0.6, 0.6, 1, 1 and token v takes the uniforms in [P(v-1), P(v))
    pT, pD = [0.4, 0.1, 0.3, 0.2], [0.1, 0.4, 0.1, 0.4]
    t, d = _logits_of(pT)[None], _logits_of(pD)[None]
    want = {0: (0.0, 0.6), 1: (0.6, 0.6), 2: (0.6, 1.0), 3: (1.0, 1.0)}
    for q, (lo, hi) in want.items():
        idx, l, h = oracle.residual_sample(t, d, query=[q])
        assert idx[0] == q
        assert l[0] == pytest.approx(lo, abs=1e-6) and h[0] == pytest.approx(hi, abs=1e-6)
    for u, v in ((0.0, 0), (0.59, 0), (0.61, 2), (0.999, 2)):
        assert oracle.residual_sample(t, d, [u])[0][0] == v
    # without a draft row: the cumulative weights of p_T itself
    want = {0: (0.0, 0.4), 1: (0.4, 0.5), 2: (0.5, 0.8), 3: (0.8, 1.0)}
    for q, (lo, hi) in want.items():
        _, l, h = oracle.residual_sample(t, None, query=[q])
        assert l[0] == pytest.approx(lo, abs=1e-6) and h[0] == pytest.approx(hi, abs=1e-6)
    # final_token's interval: a round that stops at s <= K resamples the residual of rows
    # s-1; a full round (s = K+1) draws from target row K.  K = 2 here, with row 1 of the
    # draft equal to row 1 of the target except for the residual above
    target = np.stack([_logits_of([0.25] * 4), _logits_of(pT), _logits_of([0.7, 0.1, 0.1, 0.1])])
    draft = np.stack([_logits_of([0.25] * 4), _logits_of(pD)])
    assert oracle.final_token(target, draft, 2, 0.0, query=2) == pytest.approx((0.6, 1.0), abs=1e-6)
    assert oracle.final_token(target, draft, 3, 0.0, query=1) == pytest.approx((0.7, 0.8), abs=1e-6)
    assert oracle.final_token(target, draft, 3, 0.75) == 1
    assert oracle.final_token(target, draft, 2, 0.75) == 2
    with pytest.raises(IndexError):
        oracle.residual_sample(t, d, query=[4])


def test_sps_ambiguous_stops():
    pT = [0.5, 0.3, 0.2]
    pD = [0.2, 0.5, 0.3]
    target = np.tile(_logits_of(pT), (1, 3, 1))
    draft = np.tile(_logits_of(pD), (1, 2, 1))
    r = oracle.sps_block(target, draft, np.array([[1, 0]]), np.array([[0.6, 0.2, 0.4]]))
    assert r["ambiguous"][0, 0] == (abs(0.6 - r["ratio"][0, 0]) <= oracle.SPS_BAND)
    assert r["stops"][0] == ({1, 3} if r["ambiguous"][0, 0] else {r["accept_len"][0]})


# ---------------------------------------------------------------- arbitrator hybrid attention

def test_hybrid_mask_golden():
    g = _load("hybrid_mask.json")
    m = oracle.hybrid_mask([g["ctx_len"]], g["K"], g["L"])[0]
    want = np.array([[int(c) for c in row] for row in g["rows"]], np.uint8)
    np.testing.assert_array_equal(m, want)


@pytest.mark.parametrize("lc,K,L", [(0, 1, 5), (5, 3, 16), (9, 7, 40)])
def test_hybrid_mask_structure(lc, K, L):
    m = oracle.hybrid_mask([lc], K, L)[0].astype(bool)
    ln = lc + 2 * K + 3
    assert ln == oracle.arbitrator_length(lc, K)
    np.testing.assert_array_equal(m[:lc, :lc], np.tril(np.ones((lc, lc), bool)))   # causal context
    assert not m[:lc, lc:].any()                       # no flow from the region into the context
    assert m[lc:ln, :ln].all()                         # the region sees everything up to l
    assert not m[:ln, ln:].any()                       # nobody sees padding
    assert (m.sum(1) >= 1).all()                       # no empty row


def _attn_inputs(B=2, nq=5, Hq=4, Hkv=2, D=16, L=12, seed=0):
    rng = np.random.default_rng(seed)
    q = rng.normal(size=(B, nq, Hq, D)).astype(np.float32)
    k = rng.normal(size=(B, L, Hkv, D)).astype(np.float32)
    v = rng.normal(size=(B, L, Hkv, D)).astype(np.float32)
    return q, k, v


def test_hybrid_attention_against_torch_sdpa():
    # torch's scaled_dot_product_attention in float64 with a boolean mask built here
    # from the rule (not from oracle.hybrid_mask) as an independent formulation
    B, nq, Hq, Hkv, D, L, K = 3, 9, 4, 2, 16, 14, 2
    q, k, v = _attn_inputs(B, nq, Hq, Hkv, D, L, seed=4)
    ctx = [2, 5, 7]
    qs = [0, 3, 5]
    out = oracle.hybrid_attention(q, k, v, ctx, qs, K, 0.25)
    for b in range(B):
        ln = ctx[b] + 2 * K + 3
        pos = np.arange(nq) + qs[b]
        keys = np.arange(L)
        allow = np.where((pos < ctx[b])[:, None], keys[None, :] <= pos[:, None], keys[None, :] < ln)
        for h in range(Hq):
            qq = torch.from_numpy(q[b, :, h].astype(np.float64))[None]
            kk = torch.from_numpy(k[b, :, h // 2].astype(np.float64))[None]
            vv = torch.from_numpy(v[b, :, h // 2].astype(np.float64))[None]
            ref = torch.nn.functional.scaled_dot_product_attention(
                qq, kk, vv, attn_mask=torch.from_numpy(allow)[None], scale=0.25)[0].numpy()
            valid = pos < ln
            np.testing.assert_allclose(out[b, valid, h], ref[valid], rtol=1e-12, atol=1e-12)
            assert (out[b, ~valid, h] == 0).all()


def test_hybrid_attention_closed_forms():
    q, k, v = _attn_inputs(B=1, nq=4, Hq=2, Hkv=1, D=8, L=10, seed=1)
    # the first context position sees only key 0: the output is v_0 exactly
    out = oracle.hybrid_attention(q, k, v, [5], [0], 1, 0.3)
    np.testing.assert_allclose(out[0, 0, 0], v[0, 0, 0], rtol=0, atol=1e-15)
    # all-equal keys: uniform weights, the mean of the visible values
    k[:] = k[:, :1]
    out = oracle.hybrid_attention(q, k, v, [4], [3], 1, 0.3)      # positions 3..6, l = 4 + 5 = 9
    v64 = v.astype(np.float64)
    np.testing.assert_allclose(out[0, 0, 1], v64[0, :4, 0].mean(0), rtol=1e-12)    # context row 3
    np.testing.assert_allclose(out[0, 1, 0], v64[0, :9, 0].mean(0), rtol=1e-12)    # region row, 9 keys
    with pytest.raises(ValueError):
        oracle.hybrid_attention(q, k, v, [6], [0], 1, 0.3)        # l = 11 > L = 10 keys
