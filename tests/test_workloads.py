"""The seeded input generator: determinism, batch independence and the recipe."""
import numpy as np
import torch

from paper_2605_24793_amd import workloads


def test_deterministic_and_batch_independent():
    a = workloads.make_config(4, B=3)
    b = workloads.make_config(4, B=2)
    assert torch.equal(a.target[:2].view(torch.int16), b.target.view(torch.int16))
    assert torch.equal(a.draft[:2].view(torch.int16), b.draft.view(torch.int16))
    assert torch.equal(a.draft_tokens[:2], b.draft_tokens)
    assert torch.equal(a.hidden[:2].view(torch.int16), b.hidden.view(torch.int16))
    assert torch.equal(a.head.w1.view(torch.int16), b.head.w1.view(torch.int16))
    c = workloads.make_config(4, B=2)
    assert torch.equal(c.target.view(torch.int16), b.target.view(torch.int16))


def test_shapes_and_dtypes():
    c1 = workloads.make_config(1)
    assert c1.target.shape == (1, 5, 32000) and c1.draft.shape == (1, 4, 32000)
    assert c1.target.dtype == torch.float32 and c1.hidden.dtype == torch.float32
    assert c1.head.w1.shape == (128, 512) and c1.head.w2.shape == (128,) and c1.head.b1 is None
    c3 = workloads.make_config(3, B=2)
    assert c3.target.shape == (2, 8, 151936) and c3.target.dtype == torch.bfloat16
    assert c3.hidden.shape == (2, 7, 4096) and c3.head.w1.shape == (256, 4096)
    assert tuple(c3.lambdas) == (0.3, 0.5, 0.7)


def test_draft_tokens_are_greedy_draft_choices():
    c = workloads.make_config(2, B=3)
    assert torch.equal(c.draft_tokens.long(), torch.argmax(c.draft.float(), -1))


def test_peaked_fraction_and_noise_levels():
    c = workloads.make_config(3, B=32)
    n_peaked = sum(len(p) for p in c.meta["peaks"])
    assert 0.12 < n_peaked / (32 * 8) < 0.28
    # the draft inherits the peak: draft row = peaked target row + noise (sigma 0.8)
    for b, peaks in enumerate(c.meta["peaks"]):
        for r, v in peaks:
            if r < c.K:
                assert abs(float(c.draft[b, r, v]) - float(c.target[b, r, v])) < 6.0
    c4 = workloads.make_config(4, B=8)
    assert all(0.3 <= s <= 2.0 for s in c4.meta["sigma"])


def test_tree_recipe():
    t = workloads.make_config(5, B=2)
    assert t.target.shape == (2, 60, 151936) and t.hidden.shape == (2, 60, 4096)
    par = t.parent.numpy()
    tok = t.node_tokens.numpy()
    for b in range(2):
        assert par[b, 0] == -1 and tok[b, 0] == -1
        assert all(0 <= par[b, n] < n for n in range(1, 60))
        # depth-1 nodes are the root's top-4 draft tokens, in rank order
        kids = [n for n in range(1, 60) if par[b, n] == 0]
        assert len(kids) == 4
        row = t.draft[b, 0].float()
        top4 = torch.topk(row, 4).values
        assert np.allclose(sorted(row[tok[b, kids]].tolist(), reverse=True), top4.tolist())
        assert row[tok[b, kids[0]]] == row.max()


def test_random_tree_shapes():
    for shape in ("random", "path", "star"):
        t = workloads.make_random_tree(B=2, N=9, V=300, d=32, h=16, shape=shape, seed=1)
        par = t.parent.numpy()
        assert all(0 <= par[b, n] < n for b in range(2) for n in range(1, 9))
        # siblings carry distinct tokens
        for b in range(2):
            for p in range(9):
                kids = [t.node_tokens[b, n].item() for n in range(1, 9) if par[b, n] == p]
                assert len(kids) == len(set(kids))
