"""The C ABI without a GPU: libcospec.so loads, exports every function that
include/cospec.h declares, and rejects invalid host-side arguments before it
enqueues anything (these calls never reach a kernel launch)."""
import ctypes
import math
import os
import re

import pytest

import paper_2605_24793_amd as cs
from paper_2605_24793_amd import binding

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "cospec.h")
OK, INVALID, UNSUPPORTED, WORKSPACE = 0, -1, -2, -3
FAKE = 0x10000          # an aligned address; validation never dereferences device pointers


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cospec_\w+)\s*\(", text)))


def test_header_symbols_exported():
    names = _declared()
    assert {"cospec_verify_block", "cospec_verify_tree", "cospec_arbitrate"} <= set(names)
    L = cs.lib()
    for n in names:
        assert hasattr(L, n), f"{n} declared in cospec.h but not exported"


def test_abi_version_and_status_strings():
    L = cs.lib()
    ver = int(re.search(r"#define COSPEC_ABI_VERSION (\d+)", open(HEADER).read()).group(1))
    assert L.cospec_abi_version() == ver
    for code, word in ((OK, "ok"), (INVALID, "invalid"), (UNSUPPORTED, "unsupported"),
                       (WORKSPACE, "workspace"), (-4, "HIP"), (7, "unknown")):
        assert word in binding.status_string(code)


def _head(d=512, h=128, dtype=1, w1=FAKE, w2=FAKE, b1=None):
    return binding._Head(d, h, dtype, w1, b1, w2, 0.0)


def test_workspace_sizes():
    L = cs.lib()
    hd = _head()
    sz = L.cospec_verify_block_workspace_size(64, 7, 151936, ctypes.byref(hd))
    assert sz > 0 and sz % 256 == 0
    assert L.cospec_verify_block_workspace_size(256, 7, 151936, ctypes.byref(hd)) >= sz
    assert L.cospec_verify_block_workspace_size(64, 65, 151936, ctypes.byref(hd)) == 0
    assert L.cospec_verify_block_workspace_size(-1, 7, 100, ctypes.byref(hd)) == 0
    assert L.cospec_verify_block_workspace_size(1, 7, 0, ctypes.byref(hd)) == 0
    assert L.cospec_verify_tree_workspace_size(64, 60, 151936, ctypes.byref(hd)) > 0
    assert L.cospec_verify_tree_workspace_size(64, 257, 151936, ctypes.byref(hd)) == 0
    assert L.cospec_verify_tree_workspace_size(64, 0, 151936, ctypes.byref(hd)) == 0
    assert L.cospec_arbitrate_workspace_size(1000, ctypes.byref(hd)) > 0
    # no decision rows at all (empty batch, K = 0, a lone root, no selection)
    assert L.cospec_verify_block_workspace_size(0, 7, 151936, ctypes.byref(hd)) > 0
    assert L.cospec_verify_block_workspace_size(5, 0, 151936, ctypes.byref(hd)) > 0
    assert L.cospec_verify_tree_workspace_size(0, 60, 151936, ctypes.byref(hd)) > 0
    assert L.cospec_verify_tree_workspace_size(3, 1, 151936, ctypes.byref(hd)) > 0
    assert L.cospec_arbitrate_workspace_size(0, ctypes.byref(hd)) >= 0
    bad = _head(d=12)                                      # 24 bytes: not a 16-byte multiple
    assert L.cospec_verify_block_workspace_size(1, 4, 100, ctypes.byref(bad)) == 0


@pytest.mark.parametrize("B,K,V", [(64, 7, 151936), (256, 7, 151936), (1, 4, 32000), (8, 5, 128256),
                                   (0, 7, 100), (5, 0, 1000), (300, 64, 9)])
def test_generic_workspace_query_matches_the_per_entry_queries(B, K, V):
    L = cs.lib()
    hd = _head(d=5120, h=512)
    block = L.cospec_verify_block_workspace_size(B, K, V, ctypes.byref(hd))
    assert L.cospec_workspace_bytes(B * (K + 1), B * K, B * K, V, ctypes.byref(hd)) == block
    N = K + 1
    tree = L.cospec_verify_tree_workspace_size(B, N, V, ctypes.byref(hd))
    assert L.cospec_workspace_bytes(B * N, B * N, B * N, V, ctypes.byref(hd)) == tree
    sps = L.cospec_verify_block_sps_workspace_size(B, K, V)
    assert L.cospec_workspace_bytes(B * (K + 1), B * K, B * K, V, None) == sps


def test_generic_workspace_query_rejects_invalid_sizes():
    L = cs.lib()
    hd = _head()
    assert L.cospec_workspace_bytes(-1, 0, 0, 100, ctypes.byref(hd)) == 0
    assert L.cospec_workspace_bytes(8, -1, 0, 100, ctypes.byref(hd)) == 0
    assert L.cospec_workspace_bytes(8, 7, -1, 100, ctypes.byref(hd)) == 0
    assert L.cospec_workspace_bytes(8, 7, 7, 0, ctypes.byref(hd)) == 0
    bad = _head(d=12)
    assert L.cospec_workspace_bytes(8, 7, 7, 100, ctypes.byref(bad)) == 0


def test_build_id_matches_the_sources():
    from paper_2605_24793_amd import _build
    L = cs.lib()
    assert L.cospec_build_id().decode() == _build.source_hash()
    assert re.fullmatch(r"[0-9a-f]{32}", _build.source_hash())


def _block(L, **kw):
    a = dict(tgt=FAKE, drf=FAKE, dt=1, ld=151936, toks=FAKE, hid=FAKE, head=_head(), lam=0.5,
             B=4, K=7, V=151936, alen=FAKE, otok=FAKE, feats=None, opts=None, ws=FAKE, wsb=1 << 30)
    a.update(kw)
    return L.cospec_verify_block(a["tgt"], a["drf"], a["dt"], a["ld"], a["toks"], a["hid"],
                                 ctypes.byref(a["head"]), a["lam"], a["B"], a["K"], a["V"],
                                 a["alen"], a["otok"], a["feats"], a["opts"], a["ws"], a["wsb"],
                                 None)


@pytest.mark.parametrize("kw,code", [
    (dict(tgt=None), INVALID),
    (dict(tgt=FAKE + 8), INVALID),                 # logits not 16-byte aligned
    (dict(drf=None), INVALID),
    (dict(toks=None), INVALID),
    (dict(hid=None), INVALID),
    (dict(alen=None), INVALID),
    (dict(otok=None), INVALID),
    (dict(ld=151935), INVALID),                    # ld < V
    (dict(ld=151940, V=151937), INVALID),          # ld * 2 bytes not a 16-byte multiple
    (dict(dt=5), INVALID),
    (dict(B=-1), INVALID),
    (dict(K=-1), INVALID),
    (dict(K=65), UNSUPPORTED),
    (dict(V=0), INVALID),
    (dict(dt=0, V=1 << 29, ld=1 << 29), UNSUPPORTED),   # an fp32 row of 2^31 bytes
    (dict(lam=math.nan), INVALID),
    (dict(head=_head(d=0)), INVALID),
    (dict(head=_head(h=0)), INVALID),
    (dict(head=_head(w1=None)), INVALID),
    (dict(head=_head(w1=FAKE + 4)), INVALID),
    (dict(head=_head(dtype=3)), INVALID),
    (dict(ws=None), WORKSPACE),
    (dict(ws=FAKE + 64), WORKSPACE),               # not 256-byte aligned
    (dict(wsb=1024), WORKSPACE),
    (dict(B=0), OK),                               # empty batch: nothing to enqueue
])
def test_verify_block_rejects_before_launch(kw, code):
    assert _block(cs.lib(), **kw) == code


def test_verify_block_split_override_limits():
    L = cs.lib()
    assert _block(L, opts=ctypes.byref(binding._Options(splits=65))) == UNSUPPORTED
    assert _block(L, opts=ctypes.byref(binding._Options(splits=-2))) == UNSUPPORTED
    # 4 x 15 rows x 64 splits fits the partial buffer; the workspace is checked after
    assert _block(L, wsb=16, opts=ctypes.byref(binding._Options(splits=64))) == WORKSPACE


def test_verify_block_sample_uniform_alignment():
    L = cs.lib()
    assert _block(L, opts=ctypes.byref(binding._Options(sample_uniform=FAKE + 2))) == INVALID
    f = binding._Features(tgt_candidate=FAKE + 1)
    assert _block(L, feats=ctypes.byref(f)) == INVALID


def test_rl_and_policy_uniform_arguments():
    L = cs.lib()
    assert _block(L, opts=ctypes.byref(binding._Options(policy_uniform=FAKE + 1))) == INVALID
    rl = binding._RL(reward=FAKE)                                   # reward needs correct flags
    assert _block(L, opts=ctypes.byref(binding._Options(rl=ctypes.pointer(rl)))) == INVALID
    rl = binding._RL(correct=FAKE, rho=FAKE + 2)                    # misaligned output
    assert _block(L, opts=ctypes.byref(binding._Options(rl=ctypes.pointer(rl)))) == INVALID
    rl = binding._RL(correct=FAKE, reward=FAKE, alpha=1.0, beta=0.25)
    assert _block(L, B=0, opts=ctypes.byref(binding._Options(rl=ctypes.pointer(rl)))) == OK
    assert _tree(L, opts=ctypes.byref(binding._Options(rl=ctypes.pointer(rl)))) == INVALID


def test_split_phase_arguments():
    L = cs.lib()
    hd = _head()

    def reduce(cand=FAKE, opts=None, toks=FAKE, B=4):
        return L.cospec_verify_block_reduce(FAKE, FAKE, 1, 151936, toks, ctypes.byref(hd), B, 7, 151936,
                                            cand, None, opts, FAKE, 1 << 30, None)
    assert reduce(cand=None) == INVALID                        # candidates are required
    assert reduce(cand=FAKE + 2) == INVALID
    assert reduce(toks=None) == INVALID
    assert reduce(B=0, cand=None) == OK
    # phase 2 checks like cospec_verify_block; a packed hidden map must be 8-byte aligned
    a = L.cospec_verify_block_arbitrate
    args = [FAKE, FAKE, 1, 151936, FAKE, FAKE, ctypes.byref(hd), 0.5, 4, 7, 151936, FAKE, FAKE, None]
    assert a(*args, ctypes.byref(binding._Options(hidden_row0=FAKE + 4, hidden_rows=10)), FAKE, 1 << 30,
             None) == INVALID
    assert a(*args[:11], None, FAKE, None, None, FAKE, 1 << 30, None) == INVALID   # accept_len missing


def test_sps_arguments():
    L = cs.lib()
    assert L.cospec_verify_block_sps_workspace_size(64, 7, 151936) > 0
    assert L.cospec_verify_block_sps_workspace_size(64, 65, 151936) == 0

    def call(u=FAKE, opts=None, B=4, K=7, wsb=1 << 30):
        return L.cospec_verify_block_sps(FAKE, FAKE, 1, 151936, FAKE, u, B, K, 151936, FAKE, FAKE, None,
                                         opts, FAKE, wsb, None)
    assert call(u=None) == INVALID
    assert call(u=FAKE + 2) == INVALID
    assert call(K=65) == UNSUPPORTED
    assert call(wsb=100) == WORKSPACE
    assert call(B=0, u=None) == OK
    for bad in (binding._Options(policy_uniform=FAKE), binding._Options(sample_uniform=FAKE)):
        assert call(opts=ctypes.byref(bad)) == INVALID


def test_hybrid_attention_arguments():
    L = cs.lib()
    assert L.cospec_hybrid_mask(None, 2, 1, 8, FAKE, None) == INVALID
    assert L.cospec_hybrid_mask(FAKE, 0, 1, 8, None, None) == OK
    assert L.cospec_hybrid_mask(FAKE, -1, 1, 8, FAKE, None) == INVALID

    def attn(Hq=8, Hkv=2, D=128, q=FAKE, scale=0.1, n_q=17):
        return L.cospec_hybrid_attention(q, FAKE, FAKE, FAKE, FAKE, 2, n_q, 100, Hq, Hkv, D, 7, scale, FAKE,
                                         None)
    assert attn(Hq=6, Hkv=4) == INVALID            # Hq not a multiple of Hkv
    assert attn(D=96) == UNSUPPORTED
    assert attn(q=FAKE + 8) == INVALID
    assert attn(scale=math.inf) == INVALID
    assert attn(n_q=0) == OK


def _tree(L, **kw):
    a = dict(tgt=FAKE, drf=FAKE, dt=1, ld=151936, par=FAKE, toks=FAKE, hid=FAKE, head=_head(),
             lam=0.5, B=4, N=60, V=151936, alen=FAKE, otok=FAKE, path=None, ws=FAKE, wsb=1 << 30,
             opts=None)
    a.update(kw)
    return L.cospec_verify_tree(a["tgt"], a["drf"], a["dt"], a["ld"], a["par"], a["toks"], a["hid"],
                                ctypes.byref(a["head"]), a["lam"], a["B"], a["N"], a["V"],
                                a["alen"], a["otok"], a["path"], None, a["opts"], a["ws"], a["wsb"],
                                None)


@pytest.mark.parametrize("kw,code", [
    (dict(par=None), INVALID), (dict(toks=None), INVALID), (dict(drf=None), INVALID),
    (dict(N=0), INVALID), (dict(N=257), UNSUPPORTED), (dict(path=FAKE + 2), INVALID),
    (dict(wsb=100), WORKSPACE), (dict(B=0), OK),
])
def test_verify_tree_rejects_before_launch(kw, code):
    assert _tree(cs.lib(), **kw) == code


def test_arbitrate_rejects_before_launch():
    L = cs.lib()
    hd = _head()

    def call(hid=FAKE, n_rows=10, idx=None, n_sel=10, lam=0.5, ws=FAKE, wsb=1 << 20):
        return L.cospec_arbitrate(hid, n_rows, idx, n_sel, ctypes.byref(hd), lam, FAKE, FAKE, ws,
                                  wsb, None)
    assert call(n_sel=11) == INVALID                       # more rows than exist, no index
    assert call(hid=None) == INVALID
    assert call(lam=math.nan) == INVALID
    assert call(ws=None) == WORKSPACE
    assert call(wsb=8) == WORKSPACE
    assert call(n_sel=0) == OK


def test_static_scratch_entry_point_rejects_before_any_launch():
    L = cs.lib()
    hd = _head(d=5120, h=512)
    args = [FAKE, FAKE, 1, 151936, FAKE, FAKE, ctypes.byref(hd), 0.5]

    def call(B, K, V, **kw):
        a = list(args)
        a[3] = V
        return L.cospec_verify_block_static(*a, B, K, V, FAKE, FAKE, None, kw.get("opts"), None)
    assert L.cospec_verify_block_workspace_size(4096, 64, 151936, ctypes.byref(hd)) > (64 << 20)
    assert call(4096, 64, 151936) == -5                   # needs more than the static buffer
    assert call(4, 65, 151936) == UNSUPPORTED             # K above the maximum
    assert call(-1, 7, 151936) == INVALID
    assert call(0, 7, 151936) == OK                       # empty batch: nothing to do
    assert "static buffer" in binding.status_string(-5)


def test_bench_names_the_launch_the_library_takes():
    # bench.py labels the timed launch of chain batches of at most EVERY_SLOT_MAX decision
    # slots as the reduction with the head's first layer; the library's limit must agree
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    src = open(os.path.join(root, "paper_2605_24793_amd", "csrc", "cospec_api.hip")).read()
    lib_max = int(re.search(r"constexpr int64_t kEverySlotMax = (\d+);", src).group(1))
    bench_src = open(os.path.join(root, "bench.py")).read()
    bench_max = int(re.search(r"^EVERY_SLOT_MAX = (\d+)$", bench_src, flags=re.M).group(1))
    assert lib_max == bench_max
