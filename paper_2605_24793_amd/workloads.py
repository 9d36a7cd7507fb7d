"""Seeded synthetic inputs for the CoSpec verify-and-arbitrate step.

This module draws random numbers and lays them out as the verify step's inputs:
target logits, draft logits, draft tokens (or a token tree), arbitrator hidden
states and the arbitration head's weights.  It computes nothing that the verify
step computes (no softmax statistics, no mismatch flags, no head, no scan), so
it can feed both the GPU path and the CPU oracle without either depending on
the other.

What it does model is the draft model's own proposal (Section 3.1, Eq. 1): at
greedy decoding (Appendix C.3) a chain's draft token is the first index of the
maximum of its stored draft row, and a token tree is grown from the top-k tokens
of each node's stored draft row.  Those choices are inputs of the verify step
and are made here with torch library routines on the stored (already rounded)
rows.

Every sequence (chain or tree) draws from its own generator keyed by
(seed, sequence index), so sequence b is the same whatever the batch size:
a bounded sample of a workload is its first few sequences.

The five named workloads follow the shapes of the paper's model pairs
(Section 4.1: V = 128256 for the LLaMA-3 pair, V = 151936 for Qwen3); the
paper's benchmark suites themselves are not used anywhere.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Optional, Sequence

import torch

__all__ = [
    "Head", "ChainBatch", "TreeBatch", "CONFIGS", "make_config", "make_chain",
    "make_tree", "make_random_tree", "make_head", "bf16_bits",
]

_MASK63 = (1 << 63) - 1


def _gen(seed: int, *stream: int) -> torch.Generator:
    """A CPU generator whose seed is a fixed mix of `seed` and the stream ids."""
    h = (seed * 0x9E3779B97F4A7C15 + 0x632BE59BD9B4E019) & _MASK63
    for s in stream:
        h = ((h ^ (s + 0x9E3779B9)) * 0xBF58476D1CE4E5B9 + 0x94D049BB133111EB) & _MASK63
    g = torch.Generator()
    g.manual_seed(h)
    return g


def _dt(name: str) -> torch.dtype:
    if name == "bf16":
        return torch.bfloat16
    if name == "f32":
        return torch.float32
    raise ValueError(f"unknown dtype {name!r}")


def bf16_bits(t: torch.Tensor):
    """uint16 numpy view of a bfloat16 tensor's stored bits (no copy when contiguous)."""
    assert t.dtype == torch.bfloat16
    return t.contiguous().view(torch.int16).numpy().view("uint16")


@dataclass
class Head:
    """Arbitration head g_phi as a 2-layer MLP: z = w2 . relu(W1 h + b1) + b2."""
    w1: torch.Tensor                 # [h, d]  (row-major, nn.Linear layout)
    b1: Optional[torch.Tensor]       # [h] or None (= zeros)
    w2: torch.Tensor                 # [h]
    b2: float

    @property
    def d(self) -> int:
        return int(self.w1.shape[1])

    @property
    def h(self) -> int:
        return int(self.w1.shape[0])


@dataclass
class ChainBatch:
    """One verify step over B chain blocks of K draft tokens.

    target[b, j] are the target's next-token logits after prefix + draft tokens
    1..j (j = 0..K; row K gives the bonus token); draft[b, j] are the draft's
    logits from which draft token j+1 was chosen (j = 0..K-1); hidden[b, i-1] is
    the arbitrator hidden state for decision i.
    """
    name: str
    target: torch.Tensor             # [B, K+1, V]
    draft: torch.Tensor              # [B, K, V]
    draft_tokens: torch.Tensor       # int32 [B, K]
    hidden: torch.Tensor             # [B, K, d]
    head: Head
    lambdas: Sequence[float]
    meta: dict = field(default_factory=dict)

    @property
    def B(self) -> int:
        return int(self.target.shape[0])

    @property
    def K(self) -> int:
        return int(self.draft.shape[1])

    @property
    def V(self) -> int:
        return int(self.target.shape[2])

    @property
    def rows(self) -> int:
        """Verified rows of the step: B * (K + 1)."""
        return self.B * (self.K + 1)

    def take(self, seqs) -> "ChainBatch":
        """The same step restricted to the listed sequences."""
        idx = torch.as_tensor(list(seqs), dtype=torch.long)
        return ChainBatch(self.name, self.target[idx].contiguous(), self.draft[idx].contiguous(),
                          self.draft_tokens[idx].contiguous(), self.hidden[idx].contiguous(),
                          self.head, self.lambdas, dict(self.meta))


@dataclass
class TreeBatch:
    """One verify step over B token trees of N nodes.

    Node 0 is the root (the last verified token).  target[b, n] / draft[b, n]
    are the distributions after node n; a child c of p is verified by target row
    p.  parent[b, 0] = -1 and 0 <= parent[b, n] < n.  node_tokens[b, 0] = -1.
    hidden[b, n] is the hidden state for the decision at node n (row 0 unused).
    """
    name: str
    target: torch.Tensor             # [B, N, V]
    draft: torch.Tensor              # [B, N, V]
    parent: torch.Tensor             # int32 [B, N]
    node_tokens: torch.Tensor        # int32 [B, N]
    hidden: torch.Tensor             # [B, N, d]
    head: Head
    lambdas: Sequence[float]
    meta: dict = field(default_factory=dict)

    @property
    def B(self) -> int:
        return int(self.target.shape[0])

    @property
    def N(self) -> int:
        return int(self.target.shape[1])

    @property
    def V(self) -> int:
        return int(self.target.shape[2])

    @property
    def rows(self) -> int:
        return self.B * self.N

    def take(self, seqs) -> "TreeBatch":
        idx = torch.as_tensor(list(seqs), dtype=torch.long)
        return TreeBatch(self.name, self.target[idx].contiguous(), self.draft[idx].contiguous(),
                         self.parent[idx].contiguous(), self.node_tokens[idx].contiguous(),
                         self.hidden[idx].contiguous(), self.head, self.lambdas, dict(self.meta))


# The five named workloads.  Readings where the description leaves a value open:
# target scale 4 for the large chain and the tree, b1 absent and b2 = 0 for the
# head, fp32 hidden states and weights for the tiny fp32 case, seeds 0..4.
CONFIGS = {
    1: dict(kind="chain", name="tiny-chain B=1 K=4 V=32000 f32", B=1, K=4, V=32000, dtype="f32",
            tscale=3.0, noise=1.5, d=512, h=128, lambdas=(0.5,), seed=0),
    2: dict(kind="chain", name="chain B=8 K=5 V=128256 bf16", B=8, K=5, V=128256, dtype="bf16",
            tscale=4.0, noise=1.0, d=4096, h=256, lambdas=(0.5,), seed=1),
    3: dict(kind="chain", name="serving chain B=64 K=7 V=151936 bf16", B=64, K=7, V=151936,
            dtype="bf16", tscale=4.0, noise=0.8, peaked=0.2, peak=12.0, d=4096, h=256,
            lambdas=(0.3, 0.5, 0.7), seed=2),
    4: dict(kind="chain", name="large chain B=256 K=7 V=151936 bf16", B=256, K=7, V=151936,
            dtype="bf16", tscale=4.0, noise=(0.3, 2.0), d=5120, h=512, lambdas=(0.5,), seed=3),
    5: dict(kind="tree", name="tree B=64 N=60 depth=6 V=151936 bf16", B=64, branch=4, keep=11,
            depth=6, V=151936, dtype="bf16", tscale=4.0, noise=1.0, d=4096, h=256,
            lambdas=(0.5,), seed=4),
}


def make_head(seed: int, d: int, h: int, dtype: str = "bf16", bias: bool = False) -> Head:
    """Head weights ~ N(0, 1/fan_in); with `bias`, b1 ~ N(0, 0.25) and b2 ~ N(0, 0.25)."""
    g = _gen(seed, 2)
    w1 = torch.randn(h, d, generator=g) / math.sqrt(d)
    w2 = torch.randn(h, generator=g) / math.sqrt(h)
    b1 = None
    b2 = 0.0
    if bias:
        b1 = (torch.randn(h, generator=g) * 0.5).to(_dt(dtype))
        b2 = float(torch.randn(1, generator=g).item() * 0.5)
    return Head(w1.to(_dt(dtype)), b1, w2.to(_dt(dtype)), b2)


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _chain_seq(seed, b, K, V, d, dtype, tscale, noise, peaked, peak):
    g = _gen(seed, 1, b)
    if isinstance(noise, tuple):                       # per-sequence noise level
        lo, hi = noise
        sigma = lo + (hi - lo) * float(torch.rand(1, generator=g).item())
    else:
        sigma = float(noise)
    t = torch.randn(K + 1, V, generator=g).mul_(tscale)
    z = torch.randn(K, V, generator=g)
    peaks = []
    if peaked:
        mask = torch.rand(K + 1, generator=g) < peaked
        pidx = torch.randint(0, V, (K + 1,), generator=g)
        for r in range(K + 1):
            if bool(mask[r]):
                t[r, int(pidx[r])] += peak
                peaks.append((r, int(pidx[r])))
    dr = z.mul_(sigma).add_(t[:K])
    hid = torch.randn(K, d, generator=g)
    t = t.to(_dt(dtype))
    dr = dr.to(_dt(dtype))
    # greedy draft proposal on the stored row: first index of the maximum
    tok = torch.argmax(dr.float(), dim=-1).to(torch.int32)
    return t, dr, tok, hid.to(_dt(dtype)), sigma, peaks


def make_chain(B: int, K: int, V: int, d: int, h: int, dtype: str = "bf16", tscale: float = 4.0,
               noise=1.0, peaked: float = 0.0, peak: float = 12.0, seed: int = 0,
               lambdas=(0.5,), bias: bool = False, name: Optional[str] = None,
               threads: Optional[int] = None) -> ChainBatch:
    """B chain blocks: target ~ N(0,1)*tscale (+peak on a `peaked` fraction of target
    rows, added before the draft noise), draft = target + N(0,1)*sigma, draft tokens =
    greedy choices of the draft rows, hidden ~ N(0,1)."""
    with ThreadPoolExecutor(threads or _threads()) as ex:
        seqs = list(ex.map(lambda b: _chain_seq(seed, b, K, V, d, dtype, tscale, noise, peaked,
                                                peak), range(B)))
    target = torch.stack([s[0] for s in seqs])
    draft = torch.stack([s[1] for s in seqs])
    tokens = torch.stack([s[2] for s in seqs])
    hidden = torch.stack([s[3] for s in seqs])
    head = make_head(seed, d, h, dtype, bias)
    meta = dict(sigma=[s[4] for s in seqs], peaks=[s[5] for s in seqs], seed=seed, dtype=dtype)
    return ChainBatch(name or f"chain B={B} K={K} V={V} {dtype}", target, draft, tokens, hidden,
                      head, tuple(lambdas), meta)


def _ranked_tokens(row: torch.Tensor, k: int) -> list:
    """The k largest entries of a row, ordered by value (desc) then index (asc)."""
    k = min(k, row.numel())
    thr = torch.topk(row, k).values[-1]
    cand = torch.nonzero(row >= thr).flatten()
    vals = row[cand]
    order = sorted(range(cand.numel()), key=lambda i: (-float(vals[i]), int(cand[i])))
    return [int(cand[i]) for i in order[:k]]


def _tree_seq(seed, b, V, d, dtype, tscale, noise, branch, keep, depth):
    g = _gen(seed, 1, b)
    n_nodes = 1 + branch + (depth - 1) * keep
    t = torch.randn(n_nodes, V, generator=g).mul_(tscale)
    dr = torch.randn(n_nodes, V, generator=g).mul_(noise).add_(t)
    hid = torch.randn(n_nodes, d, generator=g)
    t = t.to(_dt(dtype))
    dr = dr.to(_dt(dtype))
    drf = dr.float()
    parent = [-1]
    tokens = [-1]
    cum = [0.0]
    level = [0]
    for lev in range(1, depth + 1):
        cands = []
        for p in level:
            lp = torch.log_softmax(drf[p], dim=-1)
            for rank, tok in enumerate(_ranked_tokens(drf[p], branch)):
                cands.append((cum[p] + float(lp[tok]), p, rank, tok))
        if lev > 1:
            cands = sorted(cands, key=lambda c: (-c[0], c[1], c[2]))[:keep]
        cands = sorted(cands, key=lambda c: (c[1], c[2]))
        level = []
        for score, p, rank, tok in cands:
            level.append(len(parent))
            parent.append(p)
            tokens.append(tok)
            cum.append(score)
    assert len(parent) == n_nodes
    return (t, dr, torch.tensor(parent, dtype=torch.int32), torch.tensor(tokens, dtype=torch.int32),
            hid.to(_dt(dtype)))


def make_tree(B: int, V: int, d: int, h: int, dtype: str = "bf16", tscale: float = 4.0,
              noise: float = 1.0, branch: int = 4, keep: int = 11, depth: int = 6, seed: int = 0,
              lambdas=(0.5,), bias: bool = False, name: Optional[str] = None,
              threads: Optional[int] = None) -> TreeBatch:
    """B token trees grown from the draft rows: depth 1 holds the root's top-`branch`
    tokens; each deeper level keeps the `keep` candidates (every node of the level
    above offering its top-`branch` tokens) with the highest cumulative draft
    log-probability, ties to the lower parent id then the lower rank; node ids are
    given in (parent id, rank) order.  With 4 / 11 / 6 every tree has 60 nodes."""
    with ThreadPoolExecutor(threads or _threads()) as ex:
        seqs = list(ex.map(lambda b: _tree_seq(seed, b, V, d, dtype, tscale, noise, branch, keep,
                                               depth), range(B)))
    head = make_head(seed, d, h, dtype, bias)
    return TreeBatch(name or f"tree B={B} V={V} {dtype}",
                     torch.stack([s[0] for s in seqs]), torch.stack([s[1] for s in seqs]),
                     torch.stack([s[2] for s in seqs]), torch.stack([s[3] for s in seqs]),
                     torch.stack([s[4] for s in seqs]), head, tuple(lambdas),
                     dict(seed=seed, dtype=dtype))


def make_random_tree(B: int, N: int, V: int, d: int, h: int, dtype: str = "bf16",
                     tscale: float = 4.0, noise: float = 1.0, seed: int = 0, lambdas=(0.5,),
                     bias: bool = False, shape: str = "random") -> TreeBatch:
    """Trees of N nodes with parent[n] drawn uniformly from [0, n) (shape='random'),
    parent[n] = n-1 (shape='path') or parent[n] = 0 (shape='star').  A node's token
    is its parent's r-th ranked draft token, r = number of earlier siblings."""
    trees_t, trees_d, trees_p, trees_k, trees_h = [], [], [], [], []
    for b in range(B):
        g = _gen(seed, 3, b)
        t = torch.randn(N, V, generator=g).mul_(tscale)
        dr = torch.randn(N, V, generator=g).mul_(noise).add_(t)
        hid = torch.randn(N, d, generator=g)
        if shape == "path":
            par = [-1] + list(range(N - 1))
        elif shape == "star":
            par = [-1] + [0] * (N - 1)
        else:
            par = [-1] + [int(torch.randint(0, n, (1,), generator=g)) for n in range(1, N)]
        t = t.to(_dt(dtype))
        dr = dr.to(_dt(dtype))
        drf = dr.float()
        nkids = [0] * N
        toks = [-1]
        ranked = {}
        for n in range(1, N):
            p = par[n]
            if p not in ranked:
                ranked[p] = _ranked_tokens(drf[p], sum(1 for q in par[1:] if q == p))
            toks.append(ranked[p][nkids[p]])
            nkids[p] += 1
        trees_t.append(t)
        trees_d.append(dr)
        trees_p.append(torch.tensor(par, dtype=torch.int32))
        trees_k.append(torch.tensor(toks, dtype=torch.int32))
        trees_h.append(hid.to(_dt(dtype)))
    head = make_head(seed, d, h, dtype, bias)
    return TreeBatch(f"{shape} tree B={B} N={N} V={V} {dtype}", torch.stack(trees_t),
                     torch.stack(trees_d), torch.stack(trees_p), torch.stack(trees_k),
                     torch.stack(trees_h), head, tuple(lambdas), dict(seed=seed, dtype=dtype))


def make_config(i: int, B: Optional[int] = None, threads: Optional[int] = None):
    """Named workload i (1..5).  `B` keeps only the first B sequences (same data)."""
    c = dict(CONFIGS[i])
    kind = c.pop("kind")
    name = c.pop("name")
    if B is not None:
        c["B"] = B
        name = f"{name} [first {B} sequences]"
    if kind == "chain":
        return make_chain(name=name, threads=threads, **c)
    return make_tree(name=name, threads=threads, **c)
