"""GPU parity: libcospec.so (through the C ABI) against the CPU oracle.

Integers (argmax, Delta, accept flags outside the 1e-3 band, accept lengths,
tokens, paths) must be bit-exact; floating-point features within the stated
2e-3 * max(1, |ref|) and the tighter bounds of oracle/parity.py.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from oracle import parity
import paper_2605_24793_amd as cs
from paper_2605_24793_amd import workloads
from paper_2605_24793_amd.workloads import bf16_bits

import oracle_pool

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _conv(t):
    return bf16_bits(t) if t.dtype == torch.bfloat16 else t.contiguous().numpy()


def _head_np(h):
    return (_conv(h.w1), None if h.b1 is None else _conv(h.b1), _conv(h.w2), h.b2)


def _head_dev(h):
    return workloads.Head(h.w1.to(DEV), None if h.b1 is None else h.b1.to(DEV), h.w2.to(DEV), h.b2)


def _padded(t, pad):
    """Device copy of a [B, R, V] tensor whose rows are at least `pad` elements longer
    than V, rounded up to the 16-byte row alignment the library requires (the
    padding holds NaN, which must never be read)."""
    B, R, V = t.shape
    per = 16 // t.element_size()
    ld = (V + pad + per - 1) // per * per
    if ld == V:
        return t.to(DEV)
    big = torch.full((B, R, ld), float("nan"), dtype=t.dtype, device=DEV)
    big[:, :, :V] = t.to(DEV)
    return big[:, :, :V]


def _gpu_block(wl, lam, splits=0, pad=0, features=True, u=None):
    out = cs.verify_block(_padded(wl.target, pad), _padded(wl.draft, pad), wl.draft_tokens.to(DEV),
                          wl.hidden.to(DEV), _head_dev(wl.head), lam, features=features,
                          splits=splits,
                          sample_u=None if u is None else u.to(DEV))
    torch.cuda.synchronize()
    return {k: v.cpu() for k, v in out.items()}


def _ref_block(wl, lam, u=None, cand=None):
    return oracle.verify_block(_conv(wl.target), _conv(wl.draft), wl.draft_tokens.numpy(),
                               _conv(wl.hidden), _head_np(wl.head), lam,
                               sample_u=None if u is None else u.double().numpy(), cand_override=cand)


def _gpu_tree(tr, lam, splits=0, pad=0, u=None):
    out = cs.verify_tree(_padded(tr.target, pad), _padded(tr.draft, pad), tr.parent.to(DEV),
                         tr.node_tokens.to(DEV), tr.hidden.to(DEV), _head_dev(tr.head), lam,
                         splits=splits, sample_u=None if u is None else u.to(DEV))
    torch.cuda.synchronize()
    return {k: v.cpu() for k, v in out.items()}


def _ref_tree(tr, lam, u=None, cand=None):
    return oracle.verify_tree(_conv(tr.target), _conv(tr.draft), tr.parent.numpy(),
                              tr.node_tokens.numpy(), _conv(tr.hidden), _head_np(tr.head), lam,
                              sample_u=None if u is None else u.double().numpy(), cand_override=cand)


def _report(name, stats, gpu):
    s = gpu["accept_len"].float().mean().item() if gpu["accept_len"].numel() else float("nan")
    print(f"[{name}] mean accept_len {s:.3f} max rel err "
          + " ".join(f"{k}={v:.1e}" for k, v in stats.items() if isinstance(v, float))
          + f" ambiguous={stats.get('ambiguous_decisions', 0)}", flush=True)


# ------------------------------------------------------------------ named workloads

@pytest.mark.parametrize("cfg", [1, 2])
def test_config_full(cfg):
    wl = workloads.make_config(cfg)
    for lam in wl.lambdas:
        gpu = _gpu_block(wl, lam)
        stats = parity.check_block(gpu, _ref_block(wl, lam))
        _report(f"config {cfg} lambda {lam}", stats, gpu)


def test_config3_full_lambda_sweep():
    """The peaked serving batch (B=64, K=7, V=151936) at every threshold it names, in the
    launch sequence bench.py times, every sequence against the oracle."""
    wl = workloads.make_config(3)
    for lam in wl.lambdas:
        gpu = _gpu_block(wl, lam)
        stats = parity.check_block(gpu, oracle_pool.verify_block(wl, lam))
        _report(f"config 3 lambda {lam} (all {wl.B} sequences)", stats, gpu)


def test_config4_full_size():
    """The large chain batch (B=256, K=7, V=151936, head 5120->512->1) in the launch
    sequence bench.py times; all 256 sequences against the oracle."""
    wl = workloads.make_config(4)
    lam = wl.lambdas[0]
    gpu = _gpu_block(wl, lam)
    stats = parity.check_block(gpu, oracle_pool.verify_block(wl, lam))
    _report(f"config 4 (all {wl.B} sequences)", stats, gpu)
    _chain_properties(wl, gpu)


def test_config5_full_size():
    """The tree batch (64 trees of 60 nodes, V=151936) in the launch sequence bench.py
    --config 5 times; all 64 trees against the oracle."""
    tr = workloads.make_config(5)
    lam = tr.lambdas[0]
    gpu = _gpu_tree(tr, lam)
    stats = parity.check_tree(gpu, oracle_pool.verify_tree(tr, lam))
    _report(f"config 5 (all {tr.B} trees)", stats, gpu)
    _tree_properties(tr, gpu)


def _sample(B, n, seed):
    rng = np.random.default_rng(seed)
    return sorted(rng.choice(B, size=min(n, B), replace=False).tolist())


def _chain_properties(wl, gpu):
    """Properties every sequence must satisfy whatever the values (Section 3.3)."""
    K = wl.K
    s = gpu["accept_len"].numpy()
    tok = gpu["tokens"].numpy()
    dt = wl.draft_tokens.numpy()
    targ = gpu["tgt_argmax"].numpy()
    delta = gpu["delta"].numpy().astype(bool)
    acc = gpu["accept"].numpy().astype(bool)
    assert ((s >= 1) & (s <= K + 1)).all()
    for b in range(wl.B):
        assert list(tok[b, : s[b] - 1]) == list(dt[b, : s[b] - 1])
        assert tok[b, s[b] - 1] == targ[b, s[b] - 1]
        assert (tok[b, s[b]:] == -1).all()
        assert (delta[b] == (dt[b] == targ[b, :K])).all()
        assert acc[b, : s[b] - 1].all() and (s[b] == K + 1 or not acc[b, s[b] - 1])
        strict = np.flatnonzero(~delta[b])
        assert s[b] >= (strict[0] + 1 if strict.size else K + 1)


def _tree_properties(tr, gpu):
    par = tr.parent.numpy()
    s = gpu["accept_len"].numpy()
    path = gpu["path"].numpy()
    acc = gpu["accept"].numpy().astype(bool)
    for b in range(tr.B):
        p = path[b, : s[b]]
        assert p[0] == 0 and all(par[b, p[k + 1]] == p[k] for k in range(s[b] - 1))
        assert acc[b, p].all()
        assert (path[b, s[b]:] == -1).all()


# ------------------------------------------------------------------ fuzz and edges

FUZZ = [
    # (B, K, V, dtype, pad, splits, lam, tscale, noise)
    (1, 1, 1, "bf16", 0, 0, 0.5, 4.0, 1.0),
    (3, 2, 7, "f32", 4, 0, 0.5, 4.0, 1.0),
    (2, 3, 9, "bf16", 0, 0, 0.3, 4.0, 1.0),
    (4, 5, 4095, "bf16", 8, 3, 0.5, 4.0, 0.5),
    (5, 6, 4097, "f32", 0, 7, 0.7, 3.0, 1.5),
    (7, 8, 32001, "bf16", 24, 0, 0.45, 4.0, 1.0),
    (2, 25, 50001, "bf16", 0, 0, 0.6, 4.0, 0.6),
    (3, 64, 2053, "bf16", 0, 2, 0.5, 4.0, 0.3),
    (300, 3, 513, "bf16", 0, 0, 0.5, 4.0, 1.0),
    (9, 7, 20000, "f32", 0, 64, 0.2, 2.0, 2.0),
    # merges across a chunk boundary (9 splits), and rows split so many ways that a
    # sequence's partials do not fit the LDS stage (41 x 30 > 1024): merged from memory
    (4, 5, 30011, "f32", 0, 9, 0.5, 4.0, 1.0),
    (2, 40, 60001, "bf16", 0, 30, 0.5, 4.0, 0.8),
    # vocabularies far past the workloads' (2 MiB and 4 MiB rows, ragged tails)
    (2, 3, 1048583, "bf16", 0, 0, 0.5, 4.0, 1.0),
    (1, 2, 1048577, "f32", 3, 0, 0.5, 4.0, 1.0),
    # more decision slots (600 x 8) than the head GEMM's workgroups list themselves:
    # the decide kernel builds the list
    (600, 8, 257, "bf16", 0, 0, 0.5, 4.0, 1.0),
    # either side of the 256-slot limit of the head's first layer on every slot
    (32, 8, 4099, "bf16", 0, 0, 0.5, 4.0, 1.0),
    (37, 7, 4099, "f32", 0, 0, 0.5, 4.0, 1.0),
]


@pytest.mark.parametrize("B,K,V,dtype,pad,splits,lam,tscale,noise", FUZZ)
def test_fuzz_chain(B, K, V, dtype, pad, splits, lam, tscale, noise):
    wl = workloads.make_chain(B=B, K=K, V=V, d=96 if dtype == "bf16" else 100, h=40, dtype=dtype,
                              tscale=tscale, noise=noise, seed=B * 1000 + K * 10 + V % 97,
                              bias=True, peaked=0.2)
    gpu = _gpu_block(wl, lam, splits=splits, pad=pad)
    stats = parity.check_block(gpu, _ref_block(wl, lam))
    _report(f"fuzz B={B} K={K} V={V} {dtype} pad={pad} splits={splits}", stats, gpu)


def _adversarial_rows(B, R, V, seed):
    """Rows built to stress the argmax tie-break and the normaliser: all-equal rows,
    a tied maximum placed on split/vector boundaries, huge and tiny magnitudes."""
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(B, R, V, generator=g) * 4
    flat = x.view(-1, V)
    for r in range(flat.shape[0]):
        kind = r % 6
        if kind == 0:
            flat[r] = 1.5                                       # constant row
        elif kind == 1:
            pos = torch.tensor([0, 8, 2048, V // 2, V - 1]).clamp(max=V - 1)
            flat[r, pos] = 40.0                                 # ties on vector edges
        elif kind == 2:
            flat[r] = flat[r] * 2500.0                          # logits to about +-1e4
        elif kind == 3:
            flat[r] = -1e4 + flat[r] * 1e-3                     # far-negative narrow row
        elif kind == 4:
            flat[r, -1] = 1e4                                   # max in the last element
        else:
            flat[r, torch.randperm(V, generator=g)[:3]] = flat[r].max() + 1.0
    return x


@pytest.mark.parametrize("dtype,V,splits", [("bf16", 16384, 0), ("bf16", 16391, 5), ("f32", 9000, 3),
                                            ("bf16", 151936, 0)])
def test_adversarial_rows(dtype, V, splits):
    B, K = 4, 5
    wl = workloads.make_chain(B=B, K=K, V=V, d=64, h=32, dtype=dtype, seed=77, bias=True)
    dt = wl.target.dtype
    wl.target = _adversarial_rows(B, K + 1, V, 1).to(dt)
    wl.draft = (wl.target[:, :K].float() + torch.randn(B, K, V, generator=torch.Generator().manual_seed(2))).to(dt)
    wl.draft[:, 0] = wl.target[:, 0]                     # some exact copies: ties everywhere
    wl.draft_tokens = torch.argmax(wl.draft.float(), -1).to(torch.int32)
    gpu = _gpu_block(wl, 0.5, splits=splits)
    stats = parity.check_block(gpu, _ref_block(wl, 0.5))
    _report(f"adversarial {dtype} V={V}", stats, gpu)


@pytest.mark.parametrize("shape,N", [("random", 9), ("random", 60), ("star", 33), ("path", 12),
                                     ("random", 256)])
def test_fuzz_tree(shape, N):
    tr = workloads.make_random_tree(B=5, N=N, V=3001, d=64, h=48, shape=shape, seed=N, bias=True,
                                    noise=0.5)
    for lam in (0.3, 0.5):
        ref = _ref_tree(tr, lam)
        # rows split 5 ways too: a tree's partials staged in LDS (N x 5 <= 1024) or,
        # for 256 nodes, merged from memory
        for splits in (0, 5):
            gpu = _gpu_tree(tr, lam, pad=8, splits=splits)
            stats = parity.check_tree(gpu, ref)
            _report(f"tree {shape} N={N} lambda {lam} splits {splits}", stats, gpu)


def test_path_tree_equals_chain_on_gpu():
    wl = workloads.make_chain(B=6, K=7, V=2999, d=64, h=32, seed=5, bias=True, noise=0.6)
    K = wl.K
    chain = _gpu_block(wl, 0.5)
    tr = workloads.TreeBatch("path", wl.target, torch.cat([wl.draft, wl.draft[:, :1]], 1),
                             torch.tensor([-1] + list(range(K)), dtype=torch.int32).repeat(wl.B, 1),
                             torch.cat([torch.full((wl.B, 1), -1, dtype=torch.int32), wl.draft_tokens], 1),
                             torch.cat([wl.hidden[:, :1], wl.hidden], 1), wl.head, (0.5,))
    tree = _gpu_tree(tr, 0.5)
    assert torch.equal(tree["accept_len"], chain["accept_len"])
    assert torch.equal(tree["tokens"], chain["tokens"])
    assert torch.equal(tree["z_tilde"][:, 1:], chain["z_tilde"])


@pytest.mark.parametrize("lam", [1.0, 3.0])
def test_always_defer_is_greedy_on_gpu(lam):
    wl = workloads.make_config(3, B=16)
    gpu = _gpu_block(wl, lam, features=False)
    ref = _ref_block(wl, lam)
    t64 = oracle.element(_conv(wl.target))
    for b in range(wl.B):
        s, toks = wl.K + 1, []
        for i in range(wl.K):
            y = int(np.argmax(t64[b, i]))
            if y != int(wl.draft_tokens[b, i]):
                s, toks = i + 1, toks + [y]
                break
            toks.append(y)
        else:
            toks.append(int(np.argmax(t64[b, wl.K])))
        assert gpu["accept_len"][b].item() == s == ref["accept_len"][b]
        assert gpu["tokens"][b, :s].tolist() == toks


@pytest.mark.parametrize("lam", [-1e-6, -2.0])
def test_always_accept_on_gpu(lam):
    wl = workloads.make_config(2, B=4)
    gpu = _gpu_block(wl, lam, features=False)
    assert (gpu["accept_len"] == wl.K + 1).all()
    assert torch.equal(gpu["tokens"][:, : wl.K], wl.draft_tokens)


def _replays_match_eager(p, perturb):
    """Capture p.launch() in a HIP graph; every replay, with its outputs poisoned first
    and another eager step (perturb) run in between, must give the eager results."""
    p.launch()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in p.result().items()}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        p.launch()                                       # warm-up off the default stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        p.launch()
    for i in range(4):
        for v in p.result().values():
            v.fill_(7)
        perturb()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, v in p.result().items():
            a, b = ref[k], v
            same = torch.equal(a.view(torch.uint8), b.view(torch.uint8)) if a.dtype == torch.float32 else torch.equal(a, b)
            assert same, f"replay {i}: {k}"


def test_step_replays_from_a_hip_graph():
    # the step enqueues kernels only (no allocation, copy or memset node): a captured
    # step replays bit for bit, chains and trees, also with split rows
    wl = workloads.make_chain(B=32, K=7, V=30001, d=256, h=128, seed=21, bias=True, noise=1.0)
    other = workloads.make_chain(B=32, K=7, V=30001, d=256, h=128, seed=22, bias=True, noise=1.5)
    dev = lambda w: (_padded(w.target, 0), _padded(w.draft, 0), w.draft_tokens.to(DEV), w.hidden.to(DEV))
    q = cs.prepare_block(*dev(other), _head_dev(other.head), 0.5)
    for splits in (0, 3):
        p = cs.prepare_block(*dev(wl), _head_dev(wl.head), 0.5, splits=splits)
        _replays_match_eager(p, q.launch)
    tr = workloads.make_random_tree(B=6, N=40, V=3001, d=64, h=32, seed=23, bias=True)
    pt = cs.prepare_tree(_padded(tr.target, 0), _padded(tr.draft, 0), tr.parent.to(DEV), tr.node_tokens.to(DEV),
                         tr.hidden.to(DEV), _head_dev(tr.head), 0.5)
    _replays_match_eager(pt, q.launch)


@pytest.mark.parametrize("logit_dtype,head_dtype", [("bf16", "f32"), ("f32", "bf16")])
def test_mixed_logit_and_head_dtypes(logit_dtype, head_dtype):
    wl = workloads.make_chain(B=9, K=6, V=5003, d=128, h=96, dtype=logit_dtype, seed=31, bias=True)
    wl.head = workloads.make_head(31, 128, 96, head_dtype, bias=True)
    wl.hidden = wl.hidden.to(wl.head.w1.dtype)
    gpu = _gpu_block(wl, 0.5)
    stats = parity.check_block(gpu, _ref_block(wl, 0.5))
    _report(f"mixed logits {logit_dtype} head {head_dtype}", stats, gpu)
    tr = workloads.make_random_tree(B=3, N=20, V=3001, d=128, h=96, dtype=logit_dtype, seed=32)
    tr.head = workloads.make_head(32, 128, 96, head_dtype, bias=True)
    tr.hidden = tr.hidden.to(tr.head.w1.dtype)
    gpu = _gpu_tree(tr, 0.5)
    parity.check_tree(gpu, _ref_tree(tr, 0.5))


def test_splits_and_repeat_are_deterministic():
    wl = workloads.make_chain(B=6, K=5, V=40000, d=128, h=64, seed=8, bias=True)
    runs = [_gpu_block(wl, 0.5, splits=s) for s in (1, 1, 4, 17)]
    for k in ("accept_len", "tokens", "tgt_argmax", "drf_argmax", "delta", "accept"):
        for r in runs[1:]:
            assert torch.equal(runs[0][k], r[k]), k
    for k in ("tgt_lse", "tgt_entropy", "z_tilde"):
        assert torch.equal(runs[0][k], runs[1][k]), k          # same split: bitwise
        for r in runs[2:]:
            torch.testing.assert_close(runs[0][k], r[k], rtol=1e-5, atol=1e-5)


def test_empty_and_degenerate_sizes():
    wl = workloads.make_chain(B=2, K=3, V=100, d=32, h=16, seed=3)
    hd = _head_dev(wl.head)
    # B = 0: nothing to do
    e = torch.empty(0, 4, 100, dtype=torch.bfloat16, device=DEV)
    out = cs.verify_block(e, e[:, :3], torch.empty(0, 3, dtype=torch.int32, device=DEV),
                          torch.empty(0, 3, 32, dtype=torch.bfloat16, device=DEV), hd, 0.5)
    assert out["accept_len"].numel() == 0
    # K = 0: the round emits the target's token from row 0
    t = _padded(wl.target[:, :1].contiguous(), 0)         # rows padded to 16-byte multiples
    out = cs.verify_block(t, t[:, :0], torch.empty(2, 0, dtype=torch.int32, device=DEV),
                          torch.empty(2, 0, 32, dtype=torch.bfloat16, device=DEV), hd, 0.5)
    torch.cuda.synchronize()
    assert out["accept_len"].tolist() == [1, 1]
    assert out["tokens"][:, 0].cpu().tolist() == torch.argmax(wl.target[:, 0].float(), -1).tolist()
    # N = 1: the root alone
    tr = workloads.make_random_tree(B=2, N=1, V=100, d=32, h=16, seed=4)
    gpu = _gpu_tree(tr, 0.5)
    assert gpu["accept_len"].tolist() == [1, 1]
    assert gpu["path"][:, 0].tolist() == [0, 0]


def test_invalid_device_values_are_safe():
    wl = workloads.make_chain(B=3, K=4, V=1000, d=32, h=16, seed=6, bias=True)
    wl.draft_tokens[0, 1] = 1000          # out of range: never matches, always rejected
    wl.draft_tokens[1, 0] = -5
    gpu = _gpu_block(wl, -1.0)            # even when every valid mismatch is accepted
    assert gpu["accept_len"][0].item() <= 2 and gpu["accept_len"][1].item() == 1
    assert (gpu["tokens"] < 1000).all()
    assert gpu["accept"][0, 1].item() == 0 and torch.isnan(gpu["logp_tgt"][0, 1])
    tr = workloads.make_random_tree(B=2, N=8, V=500, d=32, h=16, seed=7)
    tr.parent[0, 5] = 7                   # breaks parent[n] < n: node 5 unreachable
    tr.parent[1, 3] = -2
    gpu = _gpu_tree(tr, -1.0)
    assert 5 not in gpu["path"][0].tolist() and 3 not in gpu["path"][1].tolist()


def test_arbitrate_matches_oracle():
    for dtype, d, h in (("bf16", 4096, 256), ("f32", 512, 128), ("bf16", 136, 72)):
        hd = workloads.make_head(11, d, h, dtype, bias=True)
        g = torch.Generator().manual_seed(d)
        hid = torch.randn(300, d, generator=g).to(hd.w1.dtype)
        idx = torch.tensor([5, 0, 299, 17, 17, 123, 300, -1] + list(range(40, 140)), dtype=torch.int32)
        out = cs.arbitrate(hid.to(DEV), _head_dev(hd), 0.5, row_index=idx.to(DEV))
        torch.cuda.synchronize()
        z = out["z"].cpu().double().numpy()
        valid = (idx >= 0) & (idx < 300)
        ref = oracle.arbitrate(_conv(hid), idx[valid].numpy(), _head_np(hd), 0.5)
        np.testing.assert_allclose(z[valid.numpy()], ref["z"], rtol=1e-4, atol=1e-4)
        assert np.isnan(z[~valid.numpy()]).all()
        a = out["accept"].cpu().numpy().astype(bool)[valid.numpy()]
        firm = ~ref["ambiguous"]
        assert np.array_equal(a[firm], ref["accept"][firm])


# ------------------------------------------------------------------ temperature 1

def _uniforms(shape, seed):
    return torch.rand(shape, generator=torch.Generator().manual_seed(seed), dtype=torch.float32)


def _t1_block(wl, lam, seed, **kw):
    """GPU chain step with temperature-1 candidates against the oracle: the candidates
    are checked against inversion of the same uniforms, then the oracle runs the rest
    of the step on them."""
    u = _uniforms((wl.B, wl.K + 1), seed)
    gpu = _gpu_block(wl, lam, u=u, **kw)
    stats = {}
    cand = parity.check_candidates(gpu["tgt_candidate"], _conv(wl.target), u.double().numpy(), stats)
    stats.update(parity.check_block(gpu, _ref_block(wl, lam, u, cand)))
    return gpu, stats


def _t1_tree(tr, lam, seed, **kw):
    u = _uniforms((tr.B, tr.N), seed)
    gpu = _gpu_tree(tr, lam, u=u, **kw)
    stats = {}
    cand = parity.check_candidates(gpu["tgt_candidate"], _conv(tr.target), u.double().numpy(), stats)
    stats.update(parity.check_tree(gpu, _ref_tree(tr, lam, u, cand)))
    return gpu, stats


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_t1_configs_full(cfg):
    wl = workloads.make_config(cfg)
    gpu, stats = _t1_block(wl, wl.lambdas[0], 100 + cfg)
    _report(f"T=1 config {cfg}", stats, gpu)
    assert (gpu["tgt_candidate"] != gpu["tgt_argmax"]).any()


def test_t1_config4_full_size():
    wl = workloads.make_config(4)
    u = _uniforms((wl.B, wl.K + 1), 104)
    gpu = _gpu_block(wl, wl.lambdas[0], u=u)
    stats = {}
    cand = oracle_pool.check_candidates(parity, gpu["tgt_candidate"], wl, u, stats)
    stats.update(parity.check_block(gpu, oracle_pool.verify_block(wl, wl.lambdas[0], u=u, cand=cand)))
    _report(f"T=1 config 4 (all {wl.B} sequences)", stats, gpu)


def test_t1_config5_full_size():
    tr = workloads.make_config(5)
    u = _uniforms((tr.B, tr.N), 105)
    gpu = _gpu_tree(tr, tr.lambdas[0], u=u)
    stats = {}
    cand = oracle_pool.check_candidates(parity, gpu["tgt_candidate"], tr, u, stats)
    stats.update(parity.check_tree(gpu, oracle_pool.verify_tree(tr, tr.lambdas[0], u=u, cand=cand)))
    _report(f"T=1 config 5 (all {tr.B} trees)", stats, gpu)


T1_FUZZ = [
    # (B, K, V, dtype, pad, splits): tails, rows shorter than one vector, split rounding
    (2, 3, 1, "bf16", 0, 0), (3, 2, 7, "f32", 4, 0), (2, 4, 9, "bf16", 0, 3),
    (4, 5, 4095, "bf16", 8, 3), (5, 6, 4097, "f32", 0, 7), (3, 7, 32001, "bf16", 24, 0),
    (2, 9, 50001, "f32", 0, 64), (40, 3, 513, "bf16", 0, 0), (2, 3, 151936, "bf16", 0, 13),
    # one split per row over 2 MiB and 4 MiB rows: the segment masses are written
    # without staging
    (2, 3, 1048583, "bf16", 0, 1), (1, 2, 1048577, "f32", 3, 1),
]


@pytest.mark.parametrize("B,K,V,dtype,pad,splits", T1_FUZZ)
def test_t1_fuzz_chain(B, K, V, dtype, pad, splits):
    wl = workloads.make_chain(B=B, K=K, V=V, d=64, h=32, dtype=dtype, seed=7 * B + V % 89, bias=True,
                              noise=0.7, peaked=0.2)
    gpu, stats = _t1_block(wl, 0.5, V + splits, splits=splits, pad=pad)
    _report(f"T=1 fuzz B={B} K={K} V={V} {dtype} pad={pad} splits={splits}", stats, gpu)


@pytest.mark.parametrize("shape,N", [("random", 60), ("star", 17), ("path", 9)])
def test_t1_fuzz_tree(shape, N):
    tr = workloads.make_random_tree(B=4, N=N, V=3001, d=64, h=48, shape=shape, seed=N + 1, bias=True,
                                    noise=0.5)
    gpu, stats = _t1_tree(tr, 0.4, N, pad=8)
    _report(f"T=1 tree {shape} N={N}", stats, gpu)


def test_t1_adversarial_rows_and_edge_uniforms():
    B, K, V = 4, 5, 16391
    wl = workloads.make_chain(B=B, K=K, V=V, d=64, h=32, dtype="bf16", seed=78, bias=True)
    wl.target = _adversarial_rows(B, K + 1, V, 3).to(torch.bfloat16)
    wl.draft_tokens = torch.argmax(wl.draft.float(), -1).to(torch.int32)
    u = _uniforms((B, K + 1), 9)
    u[0, :] = torch.tensor([0.0, -1.0, float("nan"), 1.0, 2.0, 0.9999999])
    gpu = _gpu_block(wl, 0.5, splits=5, u=u)
    uc = u.double().numpy()
    uc = np.where(np.isnan(uc) | (uc < 0), 0.0, np.minimum(uc, float(np.nextafter(np.float32(1), np.float32(0)))))
    stats = {}
    cand = parity.check_candidates(gpu["tgt_candidate"], _conv(wl.target), uc, stats)
    stats.update(parity.check_block(gpu, _ref_block(wl, 0.5, torch.from_numpy(uc), cand)))
    _report("T=1 adversarial rows", stats, gpu)
    assert gpu["tgt_candidate"][0, 0] == 0 and gpu["tgt_candidate"][0, 1] == 0


@pytest.mark.parametrize("V,dtype", [(100, "bf16"), (16391, "bf16"), (4097, "f32"), (151936, "bf16")])
def test_t1_uniforms_next_to_one(V, dtype):
    # u just below 1 puts the target in the last segments, where the wave scan's
    # lanes past the last segment round their (zero-padded) sums differently
    wl = workloads.make_chain(B=6, K=3, V=V, d=64, h=32, dtype=dtype, seed=V % 101, bias=True,
                              peaked=0.3)
    u = torch.full((wl.B, wl.K + 1), 0.99999994, dtype=torch.float32)
    u[:, 1] = 0.9999
    u[:, 2] = 0.99999
    gpu = _gpu_block(wl, 0.5, u=u)
    stats = {}
    cand = parity.check_candidates(gpu["tgt_candidate"], _conv(wl.target), u.double().numpy(), stats)
    stats.update(parity.check_block(gpu, _ref_block(wl, 0.5, u, cand)))
    _report(f"T=1 u next to 1, V={V} {dtype}", stats, gpu)


def test_t1_grid_counts_follow_softmax():
    # every target row is the same logit row; inverting the grid u_k = (k + 1/2)/n
    # must hit index v within a rounding step of n * p_v times
    V, B, K = 1000, 512, 7
    row = torch.randn(V, generator=torch.Generator().manual_seed(12)) * 2
    wl = workloads.make_chain(B=B, K=K, V=V, d=64, h=32, dtype="f32", seed=1)
    wl.target = row.expand(B, K + 1, V).contiguous()
    n = B * (K + 1)
    u = ((torch.arange(n, dtype=torch.float64) + 0.5) / n).float().reshape(B, K + 1)
    gpu = _gpu_block(wl, 0.5, u=u)
    counts = np.bincount(gpu["tgt_candidate"].numpy().ravel(), minlength=V)
    p = torch.softmax(row.double(), 0).numpy()
    assert np.abs(counts - n * p).max() <= 2.0


def test_t1_greedy_path_unchanged_and_deterministic():
    wl = workloads.make_config(3, B=8)
    g0 = _gpu_block(wl, 0.5)
    assert torch.equal(g0["tgt_candidate"], g0["tgt_argmax"])
    u = _uniforms((wl.B, wl.K + 1), 33)
    a = _gpu_block(wl, 0.5, u=u)
    b = _gpu_block(wl, 0.5, u=u)
    for k in a:
        assert torch.equal(a[k], b[k]) or (a[k].dtype.is_floating_point and
                                           torch.equal(torch.nan_to_num(a[k]), torch.nan_to_num(b[k]))), k


# ------------------------------------------------------------------ sampled arbitration and RL statistics

def _policy_block(wl, lam, pu, correct=None, alpha=1.0, beta=0.25, **kw):
    out = cs.verify_block(_padded(wl.target, 0), _padded(wl.draft, 0), wl.draft_tokens.to(DEV),
                          wl.hidden.to(DEV), _head_dev(wl.head), lam, policy_u=pu.to(DEV),
                          correct=None if correct is None else correct.to(DEV), alpha=alpha, beta=beta,
                          **kw)
    torch.cuda.synchronize()
    return {k: v.cpu() for k, v in out.items()}


@pytest.mark.parametrize("cfg", [2, 3])
def test_sampled_arbitration_and_rl_statistics(cfg):
    wl = workloads.make_config(cfg)
    pu = _uniforms((wl.B, wl.K), 200 + cfg)
    correct = (torch.arange(wl.B) % 3 != 0).to(torch.uint8)
    gpu = _policy_block(wl, 0.5, pu, correct)
    ref = oracle.verify_block(_conv(wl.target), _conv(wl.draft), wl.draft_tokens.numpy(),
                              _conv(wl.hidden), _head_np(wl.head), 0.5, policy_u=pu.double().numpy())
    stats = parity.check_block(gpu, ref)
    stats.update(parity.check_rl(gpu, ref, correct.numpy(), 1.0, 0.25))
    _report(f"sampled arbitration + RL, config {cfg}", stats, gpu)
    thr = _gpu_block(wl, 0.5)
    assert not torch.equal(thr["accept"], gpu["accept"])          # the uniforms, not lambda, decide


@pytest.mark.parametrize("lam", [0.5, 1.0, -1.0])
def test_rl_statistics_under_threshold_policy(lam):
    wl = workloads.make_chain(B=40, K=9, V=5003, d=64, h=32, seed=31, bias=True, noise=0.9)
    correct = (torch.arange(wl.B) % 2).to(torch.uint8)
    out = cs.verify_block(_padded(wl.target, 1), _padded(wl.draft, 1), wl.draft_tokens.to(DEV),
                          wl.hidden.to(DEV), _head_dev(wl.head), lam, correct=correct.to(DEV),
                          alpha=2.0, beta=0.5)
    torch.cuda.synchronize()
    gpu = {k: v.cpu() for k, v in out.items()}
    ref = _ref_block(wl, lam)
    stats = parity.check_block(gpu, ref)
    stats.update(parity.check_rl(gpu, ref, correct.numpy(), 2.0, 0.5))
    _report(f"RL statistics, lambda {lam}", stats, gpu)
    if lam >= 1.0:                       # always defer: rho = 0 on every round with a mismatch
        has = gpu["rl_first_mismatch"] > 0
        assert (gpu["rl_rho"][has] == 0).all()


def test_rl_statistics_with_invalid_tokens_and_k_zero():
    wl = workloads.make_chain(B=6, K=5, V=1000, d=64, h=32, seed=3, bias=True)
    wl.draft_tokens[1, 2] = -7
    wl.draft_tokens[4, 0] = 5000
    correct = torch.tensor([0, 0, 1, 0, 0, 1], dtype=torch.uint8)
    out = cs.verify_block(wl.target.to(DEV), wl.draft.to(DEV), wl.draft_tokens.to(DEV),
                          wl.hidden.to(DEV), _head_dev(wl.head), 0.3, correct=correct.to(DEV))
    torch.cuda.synchronize()
    gpu = {k: v.cpu() for k, v in out.items()}
    # an invalid token is a rejected mismatch: the stop, in S_rej, reward -beta
    assert gpu["accept_len"][1] <= 3 and gpu["accept_len"][4] == 1
    assert gpu["rl_first_reject"][4] == 1 and gpu["rl_reward"][4, 0] == pytest.approx(-0.25)
    w0 = workloads.make_chain(B=3, K=0, V=256, d=64, h=32, seed=4, dtype="f32")
    out = cs.verify_block(w0.target.to(DEV), w0.draft.to(DEV), w0.draft_tokens.to(DEV), w0.hidden.to(DEV),
                          _head_dev(w0.head), 0.5, correct=torch.ones(3, dtype=torch.uint8, device=DEV))
    torch.cuda.synchronize()
    assert (out["rl_first_mismatch"].cpu() == 0).all() and (out["rl_first_reject"].cpu() == 1).all()
    assert torch.isnan(out["rl_rho"].cpu()).all() and (out["rl_round_return"].cpu() == 0).all()


def test_sampled_arbitration_on_trees():
    tr = workloads.make_random_tree(B=5, N=60, V=3001, d=64, h=48, shape="random", seed=8, bias=True,
                                    noise=0.5)
    pu = _uniforms((tr.B, tr.N), 300)
    out = cs.verify_tree(_padded(tr.target, 1), _padded(tr.draft, 1), tr.parent.to(DEV),
                         tr.node_tokens.to(DEV), tr.hidden.to(DEV), _head_dev(tr.head), 0.5,
                         policy_u=pu.to(DEV))
    torch.cuda.synchronize()
    gpu = {k: v.cpu() for k, v in out.items()}
    ref = oracle.verify_tree(_conv(tr.target), _conv(tr.draft), tr.parent.numpy(), tr.node_tokens.numpy(),
                             _conv(tr.hidden), _head_np(tr.head), 0.5, policy_u=pu.double().numpy())
    stats = parity.check_tree(gpu, ref)
    _report("sampled arbitration, random trees", stats, gpu)


# ------------------------------------------------------------------ split phases and packed hidden states

def _same(a, b, keys):
    for k in keys:
        x, y = a[k].cpu(), b[k].cpu()
        if x.dtype.is_floating_point:
            assert torch.equal(torch.nan_to_num(x, nan=-7.0), torch.nan_to_num(y, nan=-7.0)), k
        else:
            assert torch.equal(x, y), k


# 24 x 7 decision slots: the head's first layer runs on every slot (beside the
# reduction, and on its own in phase 2); 80 x 7 = 560: on the mismatch rows only
@pytest.mark.parametrize("t1,B", [(False, 24), (True, 24), (False, 80)])
def test_split_phases_equal_the_whole_step(t1, B):
    wl = workloads.make_config(3, B=B)
    u = _uniforms((wl.B, wl.K + 1), 61) if t1 else None
    pu = _uniforms((wl.B, wl.K), 62)
    corr = (torch.arange(wl.B) % 2).to(torch.uint8)
    tgt, drf, tok = wl.target.to(DEV), wl.draft.to(DEV), wl.draft_tokens.to(DEV)
    head = _head_dev(wl.head)
    whole = cs.verify_block(tgt, drf, tok, wl.hidden.to(DEV), head, 0.5, sample_u=None if u is None else u.to(DEV),
                            policy_u=pu.to(DEV), correct=corr.to(DEV))
    sb = cs.SplitBlock(tgt, drf, tok, head, sample_u=None if u is None else u.to(DEV))
    torch.cuda.synchronize()
    cand = sb.candidates.cpu()
    assert torch.equal(cand, whole["tgt_candidate"].cpu())     # what the arbitrator's input needs
    split = sb.arbitrate(wl.hidden.to(DEV), 0.5, policy_u=pu.to(DEV), correct=corr.to(DEV))
    torch.cuda.synchronize()
    _same(whole, split, [k for k in whole if k in split])


def test_packed_hidden_rows():
    wl = workloads.make_config(3, B=16)
    B, K, d = wl.B, wl.K, wl.head.d
    # each sequence's arbitrator input q = [context, SEP, draft 1..K, SEP, candidates, SEP]
    # packed back to back; decision i reads the row of draft token i
    g = torch.Generator().manual_seed(4)
    ctx = torch.randint(3, 40, (B,), generator=g)
    qlen = ctx + 2 * K + 3
    start = torch.cumsum(qlen, 0) - qlen
    packed = torch.randn(int(qlen.sum()), d, generator=g).to(wl.hidden.dtype)
    row0 = start + ctx + 1
    for b in range(B):
        packed[row0[b]:row0[b] + K] = wl.hidden[b]
    ref = _gpu_block(wl, 0.5)
    sb = cs.SplitBlock(wl.target.to(DEV), wl.draft.to(DEV), wl.draft_tokens.to(DEV), _head_dev(wl.head))
    out = sb.arbitrate(packed.to(DEV), 0.5, hidden_row0=row0.to(DEV))
    torch.cuda.synchronize()
    _same(ref, out, ["accept_len", "tokens", "z_tilde", "accept", "policy"])
    # a row outside the packed array: z = NaN and the mismatch is rejected
    bad = row0.clone()
    bad[3] = packed.shape[0] - 2                     # decisions 3.. of sequence 3 fall off the end
    out = sb.arbitrate(packed.to(DEV), 0.5, hidden_row0=bad.to(DEV))
    torch.cuda.synchronize()
    zt, acc, delta = out["z_tilde"].cpu()[3], out["accept"].cpu()[3], out["delta"].cpu()[3]
    for i in range(2, K):
        if not delta[i]:
            assert torch.isnan(zt[i]) and acc[i] == 0


@pytest.mark.parametrize("B", [16, 90])
def test_packed_hidden_rows_whole_step(B):
    # the whole step with packed hidden states (16 x 7 slots: first layer on every slot;
    # 90 x 7 = 630: on the mismatch rows) equals the step on [B, K, d] bit for bit
    wl = workloads.make_config(3, B=B)
    K, d = wl.K, wl.head.d
    g = torch.Generator().manual_seed(5)
    gap = torch.randint(0, 9, (B,), generator=g)
    start = torch.cumsum(gap + K, 0) - K
    packed = torch.randn(int(start[-1]) + K + 3, d, generator=g).to(wl.hidden.dtype)
    for b in range(B):
        packed[start[b]:start[b] + K] = wl.hidden[b]
    ref = _gpu_block(wl, 0.5)
    tgt, drf, tok = wl.target.to(DEV), wl.draft.to(DEV), wl.draft_tokens.to(DEV)
    out = cs.verify_block(tgt, drf, tok, packed.to(DEV), _head_dev(wl.head), 0.5, hidden_row0=start.to(DEV))
    torch.cuda.synchronize()
    _same(ref, out, ["accept_len", "tokens", "z_tilde", "accept", "policy", "delta"])
    # rows past the packed array's end: their mismatches get z = NaN and are rejected
    bad = start.clone()
    bad[B // 2] = packed.shape[0] - 2
    out = cs.verify_block(tgt, drf, tok, packed.to(DEV), _head_dev(wl.head), 0.5, hidden_row0=bad.to(DEV))
    torch.cuda.synchronize()
    zt, acc, delta = out["z_tilde"].cpu(), out["accept"].cpu(), out["delta"].cpu()
    for i in range(2, K):
        if not delta[B // 2, i]:
            assert torch.isnan(zt[B // 2, i]) and acc[B // 2, i] == 0
    others = torch.arange(B) != B // 2
    for k in ("z_tilde", "accept"):
        x, y = ref[k].cpu()[others], out[k].cpu()[others]
        assert torch.equal(torch.nan_to_num(x, nan=-7.0), torch.nan_to_num(y, nan=-7.0)), k
    # a packed array of no rows (hidden_rows = 0 with a valid pointer): every mismatch has
    # z = NaN and is rejected, so each round stops at its first mismatch
    p = cs.prepare_block(tgt, drf, tok, packed.to(DEV), _head_dev(wl.head), 0.5, hidden_row0=start.to(DEV))
    p.hidden_rows = 0
    p.launch()
    torch.cuda.synchronize()
    out = p.result()
    delta, zt, acc = out["delta"].cpu().bool(), out["z_tilde"].cpu(), out["accept"].cpu().bool()
    assert torch.equal(acc, delta) and torch.isnan(zt[~delta]).all() and torch.isinf(zt[delta]).all()
    first = torch.where((~delta).any(1), (~delta).int().argmax(1) + 1, torch.full((B,), K + 1))
    assert torch.equal(out["accept_len"].cpu(), first.int())


# ------------------------------------------------------------------ speculative sampling baseline

def _sps(wl, seed, splits=0, pad=0):
    u = _uniforms((wl.B, wl.K + 1), seed)
    gpu = cs.sps_block(_padded(wl.target, pad), _padded(wl.draft, pad), wl.draft_tokens.to(DEV), u.to(DEV),
                       splits=splits)
    torch.cuda.synchronize()
    gpu = {k: v.cpu() for k, v in gpu.items()}
    t, d = _conv(wl.target), _conv(wl.draft)
    ref = oracle.sps_block(t, d, wl.draft_tokens.numpy(), u.double().numpy())
    return gpu, parity.check_sps(gpu, ref, t, d, u.double().numpy())


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_sps_configs(cfg):
    wl = workloads.make_config(cfg)
    gpu, stats = _sps(wl, 400 + cfg)
    _report(f"SpS config {cfg}", stats, gpu)


def test_sps_config4_full_size():
    # the launch configuration bench.py --sps times (256 sequences, automatic splits),
    # every sequence checked, a chunk of sequences per oracle task
    wl = workloads.make_config(4)
    u = _uniforms((wl.B, wl.K + 1), 404)
    gpu = cs.sps_block(wl.target.to(DEV), wl.draft.to(DEV), wl.draft_tokens.to(DEV), u.to(DEV))
    torch.cuda.synchronize()
    gpu = {k: v.cpu() for k, v in gpu.items()}

    def one(seqs):
        sub = wl.take(seqs)
        gsub = {k: v[seqs] for k, v in gpu.items()}
        t, d, us = _conv(sub.target), _conv(sub.draft), u[seqs].double().numpy()
        return parity.check_sps(gsub, oracle.sps_block(t, d, sub.draft_tokens.numpy(), us), t, d, us)
    chunks = [list(range(s, min(wl.B, s + 8))) for s in range(0, wl.B, 8)]
    with ThreadPoolExecutor(max_workers=oracle_pool.threads()) as pool:
        parts = list(pool.map(one, chunks))
    stats = {k: max(p.get(k, 0.0) for p in parts) for k in parts[0] if isinstance(parts[0][k], float)}
    _report(f"SpS config 4 (all {wl.B} sequences)", stats, gpu)


@pytest.mark.parametrize("B,K,V,dtype,pad,splits", [(3, 1, 7, "f32", 1, 0), (4, 4, 9, "bf16", 0, 2),
                                                     (5, 6, 4097, "bf16", 8, 3), (3, 5, 32001, "f32", 3, 0),
                                                     (2, 0, 3000, "bf16", 0, 0), (6, 9, 151936, "bf16", 0, 5)])
def test_sps_fuzz(B, K, V, dtype, pad, splits):
    wl = workloads.make_chain(B=B, K=K, V=V, d=64, h=32, dtype=dtype, seed=V % 53 + K, noise=0.6,
                              peaked=0.2)
    gpu, stats = _sps(wl, V + K, splits=splits, pad=pad)
    _report(f"SpS fuzz B={B} K={K} V={V} {dtype}", stats, gpu)


def test_sps_preserves_the_target_distribution_on_gpu():
    # draft token y drawn from p_D (weighted), both uniforms on an n x n grid: the first
    # emitted token must follow p_T
    V, n = 8, 64
    g = torch.Generator().manual_seed(19)
    t_logit = torch.randn(V, generator=g) * 1.5
    d_logit = torch.randn(V, generator=g) * 1.5
    pT = torch.softmax(t_logit.double(), 0).numpy()
    pD = torch.softmax(d_logit.double(), 0).numpy()
    grid = (torch.arange(n, dtype=torch.float64) + 0.5) / n
    ua, ur = torch.meshgrid(grid, grid, indexing="ij")
    m = n * n
    u = torch.stack([ua.reshape(-1), ur.reshape(-1)], 1).float().to(DEV)
    target = t_logit.expand(m, 2, V).contiguous().to(DEV)
    draft = d_logit.expand(m, 1, V).contiguous().to(DEV)
    dist = np.zeros(V)
    for y in range(V):
        toks = torch.full((m, 1), y, dtype=torch.int32, device=DEV)
        out = cs.sps_block(target, draft, toks, u, features=False)
        torch.cuda.synchronize()
        first = out["tokens"][:, 0].cpu().numpy()
        dist += pD[y] * np.bincount(first, minlength=V) / m
    assert np.abs(dist - pT).max() <= 2.5 / n


# ------------------------------------------------------------------ arbitrator hybrid attention

def test_hybrid_mask_matches_oracle():
    ctx = torch.tensor([0, 5, 20, -3], dtype=torch.int32)
    for K, L in ((2, 40), (7, 64), (1, 5)):
        got = cs.hybrid_mask(ctx.to(DEV), K, L).cpu().numpy()
        np.testing.assert_array_equal(got, oracle.hybrid_mask(np.maximum(ctx.numpy(), 0), K, L))


def _attn_case(B, nq, Hq, Hkv, D, L, ctx, qs, K, seed):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(B, nq, Hq, D, generator=g).to(torch.bfloat16)
    k = torch.randn(B, L, Hkv, D, generator=g).to(torch.bfloat16)
    v = torch.randn(B, L, Hkv, D, generator=g).to(torch.bfloat16)
    ctx_t, qs_t = torch.tensor(ctx, dtype=torch.int32), torch.tensor(qs, dtype=torch.int32)
    scale = 1.0 / np.sqrt(D)
    out = cs.hybrid_attention(q.to(DEV), k.to(DEV), v.to(DEV), ctx_t.to(DEV), qs_t.to(DEV), K, scale)
    torch.cuda.synchronize()
    ref = oracle.hybrid_attention(bf16_bits(q), bf16_bits(k), bf16_bits(v), ctx, qs, K, scale)
    got = out.float().cpu().numpy()
    # P enters the second product as bf16 (relative 2^-9) and the output is stored as bf16:
    # |error| <= about 2 * 2^-9 * max|v| per element; 6e-3 * max|v| leaves margin
    tol = 6e-3 * float(v.float().abs().max())
    err = np.abs(got - ref).max()
    print(f"[hybrid attention B={B} n_q={nq} Hq={Hq} Hkv={Hkv} D={D} L={L}] max err {err:.2e} (tol {tol:.2e})",
          flush=True)
    assert err <= tol


def test_hybrid_attention_bench_shape_sampled():
    # the shape bench.py --attention times: 64 sequences x 2048 context tokens, K = 7
    # (17 region queries each), 32 query / 8 key-value heads, D = 128; the oracle checks
    # four sampled sequences
    B, ctx_len, K, Hq, Hkv, D = 64, 2048, 7, 32, 8, 128
    nq = 2 * K + 3
    L = (ctx_len + nq + 15) // 16 * 16
    g = torch.Generator().manual_seed(12)
    q = torch.randn(B, nq, Hq, D, generator=g).to(torch.bfloat16)
    k = torch.randn(B, L, Hkv, D, generator=g).to(torch.bfloat16)
    v = torch.randn(B, L, Hkv, D, generator=g).to(torch.bfloat16)
    ctx = torch.full((B,), ctx_len, dtype=torch.int32)
    scale = 1.0 / np.sqrt(D)
    out = cs.hybrid_attention(q.to(DEV), k.to(DEV), v.to(DEV), ctx.to(DEV), ctx.to(DEV), K, scale)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    for b in _sample(B, 4, 13):
        ref = oracle.hybrid_attention(bf16_bits(q[b:b + 1]), bf16_bits(k[b:b + 1]), bf16_bits(v[b:b + 1]),
                                      [ctx_len], [ctx_len], K, scale)
        tol = 6e-3 * float(v[b].float().abs().max())
        err = np.abs(got[b:b + 1] - ref).max()
        print(f"[hybrid attention bench shape, sequence {b}] max err {err:.2e} (tol {tol:.2e})", flush=True)
        assert err <= tol


@pytest.mark.parametrize("D", [128, 64])
def test_hybrid_attention_region_queries(D):
    K = 7
    ctx = [37, 100, 0]
    L = 100 + 2 * K + 3 + 5
    _attn_case(3, 2 * K + 3, 8, 2, D, L, ctx, ctx, K, seed=D)


def test_hybrid_attention_whole_input_prefill():
    # every position of q at once: causal context rows, region rows, padding rows
    K = 3
    ctx = [10, 70]
    L = 70 + 2 * K + 3 + 4
    _attn_case(2, L, 4, 4, 128, L, ctx, [0, 0], K, seed=3)


def test_hybrid_attention_long_context_gqa():
    K = 7
    ctx = [1000, 2041]
    L = 2041 + 2 * K + 3
    _attn_case(2, 2 * K + 3, 64, 8, 128, L, ctx, ctx, K, seed=9)


# ------------------------------------------------------------------ option combinations

@pytest.mark.parametrize("splits,pad,dtype", [(0, 0, "bf16"), (5, 24, "bf16"), (3, 4, "f32")])
def test_t1_with_sampled_arbitration_and_rl(splits, pad, dtype):
    wl = workloads.make_chain(B=12, K=6, V=20011, d=64, h=32, dtype=dtype, seed=91 + splits, bias=True,
                              noise=0.6, peaked=0.2)
    u = _uniforms((wl.B, wl.K + 1), 500 + splits)
    pu = _uniforms((wl.B, wl.K), 600 + splits)
    corr = (torch.arange(wl.B) % 3 == 0).to(torch.uint8)
    out = cs.verify_block(_padded(wl.target, pad), _padded(wl.draft, pad), wl.draft_tokens.to(DEV),
                          wl.hidden.to(DEV), _head_dev(wl.head), 0.5, splits=splits, sample_u=u.to(DEV),
                          policy_u=pu.to(DEV), correct=corr.to(DEV), alpha=1.5, beta=0.3)
    torch.cuda.synchronize()
    gpu = {k: v.cpu() for k, v in out.items()}
    stats = {}
    cand = parity.check_candidates(gpu["tgt_candidate"], _conv(wl.target), u.double().numpy(), stats)
    ref = oracle.verify_block(_conv(wl.target), _conv(wl.draft), wl.draft_tokens.numpy(), _conv(wl.hidden),
                              _head_np(wl.head), 0.5, sample_u=u.double().numpy(), cand_override=cand,
                              policy_u=pu.double().numpy())
    stats.update(parity.check_block(gpu, ref))
    stats.update(parity.check_rl(gpu, ref, corr.numpy(), 1.5, 0.3))
    _report(f"T=1 + sampled arbitration + RL, splits={splits} pad={pad} {dtype}", stats, gpu)


@pytest.mark.parametrize("shape,N,splits", [("random", 60, 0), ("random", 37, 6), ("star", 20, 2)])
def test_t1_trees_with_sampled_arbitration(shape, N, splits):
    tr = workloads.make_random_tree(B=4, N=N, V=4099, d=64, h=48, shape=shape, seed=N + 7, bias=True,
                                    noise=0.5)
    u = _uniforms((tr.B, tr.N), 700 + N)
    pu = _uniforms((tr.B, tr.N), 800 + N)
    out = cs.verify_tree(_padded(tr.target, 4), _padded(tr.draft, 4), tr.parent.to(DEV), tr.node_tokens.to(DEV),
                         tr.hidden.to(DEV), _head_dev(tr.head), 0.5, splits=splits, sample_u=u.to(DEV),
                         policy_u=pu.to(DEV))
    torch.cuda.synchronize()
    gpu = {k: v.cpu() for k, v in out.items()}
    stats = {}
    cand = parity.check_candidates(gpu["tgt_candidate"], _conv(tr.target), u.double().numpy(), stats)
    ref = oracle.verify_tree(_conv(tr.target), _conv(tr.draft), tr.parent.numpy(), tr.node_tokens.numpy(),
                             _conv(tr.hidden), _head_np(tr.head), 0.5, sample_u=u.double().numpy(),
                             cand_override=cand, policy_u=pu.double().numpy())
    stats.update(parity.check_tree(gpu, ref))
    _report(f"T=1 + sampled arbitration, tree {shape} N={N} splits={splits}", stats, gpu)


def test_split_phases_with_everything():
    wl = workloads.make_config(3, B=10)
    B, K = wl.B, wl.K
    u = _uniforms((B, K + 1), 71)
    pu = _uniforms((B, K), 72)
    corr = torch.ones(B, dtype=torch.uint8)
    head = _head_dev(wl.head)
    tgt, drf, tok = wl.target.to(DEV), wl.draft.to(DEV), wl.draft_tokens.to(DEV)
    whole = cs.verify_block(tgt, drf, tok, wl.hidden.to(DEV), head, 0.5, splits=7, sample_u=u.to(DEV),
                            policy_u=pu.to(DEV), correct=corr.to(DEV))
    # packed hidden rows: q = [context, SEP, draft, SEP, candidates, SEP] per sequence
    ctx = torch.randint(1, 30, (B,), generator=torch.Generator().manual_seed(3))
    qlen = ctx + 2 * K + 3
    start = torch.cumsum(qlen, 0) - qlen
    packed = torch.randn(int(qlen.sum()), wl.head.d, generator=torch.Generator().manual_seed(4)).to(wl.hidden.dtype)
    row0 = start + ctx + 1
    for b in range(B):
        packed[row0[b]:row0[b] + K] = wl.hidden[b]
    sb = cs.SplitBlock(tgt, drf, tok, head, splits=7, sample_u=u.to(DEV))
    split = sb.arbitrate(packed.to(DEV), 0.5, policy_u=pu.to(DEV), correct=corr.to(DEV),
                         hidden_row0=row0.to(DEV))
    torch.cuda.synchronize()
    _same(whole, split, [k for k in whole if k in split])
    # a second arbitration on the same phase 1 (another threshold) equals a whole step at it
    again = sb.arbitrate(packed.to(DEV), 0.3, hidden_row0=row0.to(DEV))
    whole2 = cs.verify_block(tgt, drf, tok, wl.hidden.to(DEV), head, 0.3, splits=7, sample_u=u.to(DEV))
    torch.cuda.synchronize()
    _same(whole2, again, ["accept_len", "tokens", "z_tilde", "accept"])


def test_sps_long_blocks():
    wl = workloads.make_chain(B=5, K=64, V=2053, d=64, h=32, dtype="bf16", seed=17, noise=0.2)
    gpu, stats = _sps(wl, 77)
    _report("SpS K=64", stats, gpu)
    assert gpu["accept_len"].max() > 8                # low noise: long accepted runs


def test_hybrid_attention_long_prefill_several_workgroups():
    # 300 positions x 1 head per group: three workgroups share each group's keys
    K = 2
    ctx = [250, 120]
    L = 250 + 2 * K + 3 + 9
    _attn_case(2, L, 2, 2, 64, L, ctx, [0, 0], K, seed=21)
