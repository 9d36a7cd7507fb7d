"""The oracle over a whole batch, a few sequences per task on a thread pool.

Sequences (and trees) are independent, so running the oracle on chunks of them and
concatenating the results gives exactly what one call over the batch gives; the
oracle's C loops release the interpreter lock, so the chunks run in parallel.  This
lets the parity tests compare every sequence of the full-size workloads.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

import oracle
from paper_2605_24793_amd.workloads import bf16_bits

CHUNK = 8


def conv(t):
    """Oracle array of a CPU tensor: fp32 values, or the raw bits of bf16."""
    return bf16_bits(t) if t.dtype == torch.bfloat16 else t.contiguous().numpy()


def head_np(h):
    return (conv(h.w1), None if h.b1 is None else conv(h.b1), conv(h.w2), h.b2)


def threads() -> int:
    """The CPUs this process may use, at most 16."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _merge(parts):
    out = {}
    for k, v in parts[0].items():
        if v is None:
            out[k] = None
        elif isinstance(v, np.ndarray):
            out[k] = np.concatenate([p[k] for p in parts], axis=0)
        elif isinstance(v, list):
            out[k] = [x for p in parts for x in p[k]]
        else:
            raise TypeError(f"cannot merge oracle result field {k!r} of type {type(v)}")
    return out


def _run(batch, fn):
    chunks = [list(range(s, min(batch.B, s + CHUNK))) for s in range(0, batch.B, CHUNK)]
    with ThreadPoolExecutor(max_workers=threads()) as pool:
        return _merge(list(pool.map(fn, chunks)))


def _rows(a, seqs):
    return None if a is None else np.asarray(a)[seqs]


def verify_block(wl, lam, u=None, cand=None, policy_u=None, correct=None):
    """oracle.verify_block over every sequence of a chain workload.  u, cand, policy_u
    and correct are per-sequence arrays (torch or numpy) or None."""
    u = None if u is None else (u.double().numpy() if hasattr(u, "double") else np.asarray(u, np.float64))
    pu = None if policy_u is None else (policy_u.double().numpy() if hasattr(policy_u, "double")
                                        else np.asarray(policy_u, np.float64))
    cor = None if correct is None else np.asarray(correct)
    hd = head_np(wl.head)

    def one(seqs):
        sub = wl.take(seqs)
        return oracle.verify_block(conv(sub.target), conv(sub.draft), sub.draft_tokens.numpy(),
                                   conv(sub.hidden), hd, lam, sample_u=_rows(u, seqs),
                                   cand_override=_rows(cand, seqs), policy_u=_rows(pu, seqs),
                                   correct=_rows(cor, seqs))
    return _run(wl, one)


def verify_tree(tr, lam, u=None, cand=None, policy_u=None):
    """oracle.verify_tree over every tree of a tree workload."""
    u = None if u is None else (u.double().numpy() if hasattr(u, "double") else np.asarray(u, np.float64))
    pu = None if policy_u is None else (policy_u.double().numpy() if hasattr(policy_u, "double")
                                        else np.asarray(policy_u, np.float64))
    hd = head_np(tr.head)

    def one(seqs):
        sub = tr.take(seqs)
        return oracle.verify_tree(conv(sub.target), conv(sub.draft), sub.parent.numpy(),
                                  sub.node_tokens.numpy(), conv(sub.hidden), hd, lam,
                                  sample_u=_rows(u, seqs), cand_override=_rows(cand, seqs),
                                  policy_u=_rows(pu, seqs))
    return _run(tr, one)


def check_candidates(parity, gpu_cand, batch, u, stats=None):
    """parity.check_candidates over every target row, a chunk of sequences per task."""
    uu = u.double().numpy() if hasattr(u, "double") else np.asarray(u, np.float64)
    gc = gpu_cand.numpy() if hasattr(gpu_cand, "numpy") else np.asarray(gpu_cand)
    chunks = [list(range(s, min(batch.B, s + CHUNK))) for s in range(0, batch.B, CHUNK)]
    parts = []

    def one(seqs):
        st = {}
        c = parity.check_candidates(gc[seqs], conv(batch.take(seqs).target), uu[seqs], st)
        return c, st
    with ThreadPoolExecutor(max_workers=threads()) as pool:
        parts = list(pool.map(one, chunks))
    if stats is not None:
        for _, st in parts:
            for k, v in st.items():
                if isinstance(v, (int, np.integer)):
                    stats[k] = stats.get(k, 0) + int(v)
                elif isinstance(v, float):
                    stats[k] = max(stats.get(k, 0.0), v)
    return np.concatenate([c for c, _ in parts], axis=0)
