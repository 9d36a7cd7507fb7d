"""cospec_verify_block_static (the chain step on the library's static scratch buffer)
against cospec_verify_block with a caller workspace, through the C ABI.

The two run the same kernels, so every output must be the same bits.  Two calls in a
row, the second on a smaller batch, check that the buffer's leftover contents from the
first call change nothing; an oversized batch must be refused before any launch.
"""
import ctypes

import pytest
import torch

import paper_2605_24793_amd as cs
from paper_2605_24793_amd import binding, workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _dev_head(h):
    return workloads.Head(h.w1.to(DEV), None if h.b1 is None else h.b1.to(DEV), h.w2.to(DEV), h.b2)


def _both(wl, lam, **kw):
    args = (wl.target.to(DEV), wl.draft.to(DEV), wl.draft_tokens.to(DEV), wl.hidden.to(DEV),
            _dev_head(wl.head), lam)
    ref = cs.verify_block(*args, **kw)
    got = cs.verify_block_static(*args, **kw)
    torch.cuda.synchronize()
    return {k: v.cpu() for k, v in ref.items()}, {k: v.cpu() for k, v in got.items()}


def _identical(ref, got):
    assert set(ref) == set(got)
    for k in ref:
        a, b = ref[k], got[k]
        if a.dtype == torch.float32:
            a, b = a.view(torch.int32), b.view(torch.int32)      # bits, NaN included
        assert torch.equal(a, b), k


def test_static_scratch_matches_the_workspace_entry_point():
    big = workloads.make_chain(B=96, K=7, V=151936, d=4096, h=256, seed=31, noise=0.9, bias=True)
    ref, got = _both(big, 0.5)
    _identical(ref, got)
    assert (ref["delta"] == 0).any()                             # the head ran on mismatches
    # second call, smaller batch, other dtype and sizes: leftovers of the first must not matter
    small = workloads.make_chain(B=5, K=4, V=32004, d=512, h=128, dtype="f32", seed=32, noise=1.5)
    ref, got = _both(small, 0.3)
    _identical(ref, got)
    # temperature-1 candidates and a split override through the same buffer
    u = torch.rand((big.B, big.K + 1), generator=torch.Generator().manual_seed(33)).to(DEV)
    ref, got = _both(big, 0.7, sample_u=u, splits=3)
    _identical(ref, got)


def test_static_scratch_refuses_oversized_batches():
    L = cs.lib()
    head = _dev_head(workloads.make_chain(B=1, K=1, V=16, d=5120, h=512, seed=1).head)
    hs = binding._head_struct(head)
    B, K, V = 4096, 64, 151936
    assert L.cospec_verify_block_workspace_size(B, K, V, ctypes.byref(hs)) > (64 << 20)
    x = torch.empty(16, dtype=torch.bfloat16, device=DEV)
    i = torch.empty(16, dtype=torch.int32, device=DEV)
    code = L.cospec_verify_block_static(x.data_ptr(), x.data_ptr(), 1, V, i.data_ptr(), x.data_ptr(),
                                        ctypes.byref(hs), 0.5, B, K, V, i.data_ptr(), i.data_ptr(), None, None,
                                        None)
    assert code == -5 and "static buffer" in binding.status_string(code)
