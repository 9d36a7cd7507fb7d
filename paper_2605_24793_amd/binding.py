"""Thin ctypes binding of libcospec.so (include/cospec.h).

Marshalling only: torch tensors supply device memory and the current stream,
this module turns them into pointers and sizes and calls the C ABI.  Every step
of the computation runs in the library's HIP kernels.  There is no fallback: if
the library cannot be loaded or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

from . import _build

__all__ = ["lib", "verify_block", "verify_block_static", "verify_tree", "arbitrate", "CospecError", "Prepared",
           "prepare_block", "prepare_tree", "prepare_sps", "SplitBlock", "sps_block", "hybrid_mask",
           "hybrid_attention", "status_string", "MAX_K",
           "MAX_N", "MAX_SPLITS"]

MAX_K, MAX_N, MAX_SPLITS = 64, 256, 64
_F32, _BF16 = 0, 1
_lib = None


class CospecError(RuntimeError):
    pass


class _Head(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("h", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("w1", ctypes.c_void_p), ("b1", ctypes.c_void_p), ("w2", ctypes.c_void_p),
                ("b2", ctypes.c_float)]


_FEATURE_FIELDS = ["tgt_argmax", "tgt_max", "tgt_lse", "tgt_entropy", "drf_argmax", "drf_max",
                   "drf_lse", "drf_entropy", "logp_tgt", "logp_drf", "delta", "z_tilde", "policy",
                   "accept", "tgt_candidate", "logp_action"]


class _Features(ctypes.Structure):
    _fields_ = [(f, ctypes.c_void_p) for f in _FEATURE_FIELDS]


class _RL(ctypes.Structure):
    _fields_ = [("correct", ctypes.c_void_p), ("alpha", ctypes.c_float), ("beta", ctypes.c_float),
                ("effective", ctypes.c_void_p), ("in_s_acc", ctypes.c_void_p),
                ("first_mismatch", ctypes.c_void_p), ("first_reject", ctypes.c_void_p),
                ("rho", ctypes.c_void_p), ("reward", ctypes.c_void_p),
                ("round_return", ctypes.c_void_p)]


class _Options(ctypes.Structure):
    _fields_ = [("reduce_begin", ctypes.c_void_p), ("reduce_end", ctypes.c_void_p),
                ("reduce2_begin", ctypes.c_void_p), ("reduce2_end", ctypes.c_void_p),
                ("splits", ctypes.c_int32),
                ("sample_uniform", ctypes.c_void_p), ("policy_uniform", ctypes.c_void_p),
                ("rl", ctypes.POINTER(_RL)), ("hidden_row0", ctypes.c_void_p),
                ("hidden_rows", ctypes.c_int64)]


def _event_handle(ev) -> int:
    """Raw hipEvent_t of a torch event (torch creates it at its first record)."""
    if ev.cuda_event == 0:
        ev.record()
    return ev.cuda_event


def lib():
    """The loaded library, built first if no build exists.  A build whose id (the hash
    of the sources it was compiled from) differs from the sources on disk is refused:
    the kernels it holds are not the ones in csrc/."""
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        HP = ctypes.POINTER(_Head)
        L.cospec_build_id.restype = ctypes.c_char_p
        L.cospec_build_id.argtypes = []
        built, want = L.cospec_build_id().decode(), _build.source_hash()
        if built != want:
            raise CospecError(f"{_build.LIB} is stale: built from sources {built}, the sources on disk are "
                              f"{want}; rebuild it (python -m paper_2605_24793_amd._build)")
        L.cospec_abi_version.restype = I32
        L.cospec_abi_version.argtypes = []
        L.cospec_workspace_bytes.restype = SZ
        L.cospec_workspace_bytes.argtypes = [I32, I32, I32, I32, HP]
        L.cospec_status_string.restype = ctypes.c_char_p
        L.cospec_status_string.argtypes = [I32]
        L.cospec_verify_block_workspace_size.restype = SZ
        L.cospec_verify_block_workspace_size.argtypes = [I32, I32, I32, HP]
        L.cospec_verify_tree_workspace_size.restype = SZ
        L.cospec_verify_tree_workspace_size.argtypes = [I32, I32, I32, HP]
        L.cospec_arbitrate_workspace_size.restype = SZ
        L.cospec_arbitrate_workspace_size.argtypes = [I64, HP]
        L.cospec_verify_block.restype = I32
        L.cospec_verify_block.argtypes = [P, P, I32, I64, P, P, HP, ctypes.c_float, I32, I32, I32,
                                          P, P, ctypes.POINTER(_Features),
                                          ctypes.POINTER(_Options), P, SZ, P]
        L.cospec_verify_tree.restype = I32
        L.cospec_verify_tree.argtypes = [P, P, I32, I64, P, P, P, HP, ctypes.c_float, I32, I32,
                                         I32, P, P, P, ctypes.POINTER(_Features),
                                         ctypes.POINTER(_Options), P, SZ, P]
        L.cospec_verify_block_static.restype = I32
        L.cospec_verify_block_static.argtypes = [P, P, I32, I64, P, P, HP, ctypes.c_float, I32, I32, I32,
                                                 P, P, ctypes.POINTER(_Features), ctypes.POINTER(_Options), P]
        L.cospec_verify_block_reduce.restype = I32
        L.cospec_verify_block_reduce.argtypes = [P, P, I32, I64, P, HP, I32, I32, I32, P,
                                                 ctypes.POINTER(_Features), ctypes.POINTER(_Options),
                                                 P, SZ, P]
        L.cospec_verify_block_arbitrate.restype = I32
        L.cospec_verify_block_arbitrate.argtypes = L.cospec_verify_block.argtypes
        L.cospec_verify_block_sps_workspace_size.restype = SZ
        L.cospec_verify_block_sps_workspace_size.argtypes = [I32, I32, I32]
        L.cospec_verify_block_sps.restype = I32
        L.cospec_verify_block_sps.argtypes = [P, P, I32, I64, P, P, I32, I32, I32, P, P,
                                              ctypes.POINTER(_Features), ctypes.POINTER(_Options), P,
                                              SZ, P]
        L.cospec_hybrid_mask.restype = I32
        L.cospec_hybrid_mask.argtypes = [P, I32, I32, I32, P, P]
        L.cospec_hybrid_attention.restype = I32
        L.cospec_hybrid_attention.argtypes = [P, P, P, P, P, I32, I32, I32, I32, I32, I32, I32,
                                              ctypes.c_float, P, P]
        L.cospec_arbitrate.restype = I32
        L.cospec_arbitrate.argtypes = [P, I64, P, I64, HP, ctypes.c_float, P, P, P, SZ, P]
        _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().cospec_status_string(code).decode()


def _check(code: int, what: str):
    if code != 0:
        raise CospecError(f"{what}: {status_string(code)} ({code})")


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return _BF16
    if t.dtype == torch.float32:
        return _F32
    raise TypeError(f"logits, hidden states and head weights are bf16 or f32, got {t.dtype}")


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _head_struct(head) -> _Head:
    w1, b1, w2, b2 = head.w1, head.b1, head.w2, head.b2
    for t in (w1, w2) + ((b1,) if b1 is not None else ()):
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError("head weights must be contiguous device tensors")
    return _Head(int(w1.shape[1]), int(w1.shape[0]), _dtype_code(w1), _ptr(w1), _ptr(b1),
                 _ptr(w2), float(b2))


def _row_stride(t: torch.Tensor) -> int:
    """Row stride in elements of a [B, R, V] logit tensor whose rows may be padded."""
    if t.dim() != 3 or (t.shape[2] > 1 and t.stride(2) != 1):
        raise ValueError("logits must be [B, R, V] with unit element stride")
    if t.shape[0] > 1 and t.shape[1] > 0 and t.stride(0) != t.shape[1] * t.stride(1):
        raise ValueError("logit rows must be uniformly spaced: stride(0) == R * stride(1)")
    return int(t.stride(1))


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


class Prepared:
    """Pre-marshalled arguments of one verify call: outputs, features, workspace and
    are allocated once, so
    `launch()` enqueues the step with no allocation."""

    def __init__(self, fn, args_before_feats, outputs, feats, feats_struct, workspace, splits,
                 uniform=None, policy_u=None, rl=None):
        self._fn = fn
        self._args = args_before_feats
        self.outputs = outputs
        self.features = feats
        self._feats = feats_struct
        self.workspace = workspace
        self.splits = int(splits)
        self.uniform = uniform
        self.policy_u = policy_u
        self.rl = rl                    # (struct, output tensors, correct tensor) or None
        self.hidden_row0 = None         # packed hidden rows: int64 [B] device tensor, and
        self.hidden_rows = 0            # the rows of the packed array
        self._keep = []

    def _options(self, timing):
        if (timing is None and not self.splits and self.uniform is None
                and self.policy_u is None and self.rl is None and self.hidden_row0 is None):
            return None
        ev = [None] * 4 if timing is None else [None if e is None else _event_handle(e) for e in timing]
        rl = None if self.rl is None else ctypes.pointer(self.rl[0])
        return _Options(ev[0], ev[1], ev[2], ev[3], self.splits, _ptr(self.uniform),
                        _ptr(self.policy_u), rl, _ptr(self.hidden_row0), int(self.hidden_rows))

    def launch(self, timing=None):
        """Enqueue the step on torch's current stream.  `timing` = four torch events
        recorded around the target-row and the draft-row reduction launches."""
        opts = self._options(timing)
        code = self._fn(*self._args, ctypes.byref(self._feats) if self._feats is not None else None,
                        ctypes.byref(opts) if opts is not None else None,
                        _ptr(self.workspace), self.workspace.numel(), _stream())
        _check(code, self._fn.__name__)

    def result(self) -> dict:
        out = dict(self.outputs)
        out.update(self.features or {})
        if self.rl is not None:
            out.update({"rl_" + k: v for k, v in self.rl[1].items()})
        return out


def _features(alloc: bool, dev, B, RT, RD, D):
    if not alloc:
        return None, None
    i32, f32, u8 = torch.int32, torch.float32, torch.uint8
    shapes = dict(tgt_argmax=((B, RT), i32), tgt_max=((B, RT), f32), tgt_lse=((B, RT), f32),
                  tgt_entropy=((B, RT), f32), drf_argmax=((B, RD), i32), drf_max=((B, RD), f32),
                  drf_lse=((B, RD), f32), drf_entropy=((B, RD), f32), logp_tgt=((B, D), f32),
                  logp_drf=((B, D), f32), delta=((B, D), u8), z_tilde=((B, D), f32),
                  policy=((B, D), f32), accept=((B, D), u8), tgt_candidate=((B, RT), i32),
                  logp_action=((B, D), f32))
    feats = {k: torch.empty(s, dtype=t, device=dev) for k, (s, t) in shapes.items()}
    st = _Features(*[_ptr(feats[f]) for f in _FEATURE_FIELDS])
    return feats, st


def _uniforms(u: Optional[torch.Tensor], B: int, RT: int):
    if u is None:
        return None
    if tuple(u.shape) != (B, RT) or u.dtype != torch.float32 or not u.is_contiguous() or not u.is_cuda:
        raise ValueError("sample_u must be a contiguous float32 device tensor [B, target rows]")
    return u


def _policy_uniforms(u: Optional[torch.Tensor], B: int, D: int):
    if u is None:
        return None
    if tuple(u.shape) != (B, D) or u.dtype != torch.float32 or not u.is_contiguous() or not u.is_cuda:
        raise ValueError("policy_u must be a contiguous float32 device tensor [B, decisions]")
    return u


def _rl(correct: Optional[torch.Tensor], alpha: float, beta: float, B: int, K: int, dev):
    if correct is None:
        return None
    if tuple(correct.shape) != (B,) or correct.dtype != torch.uint8 or not correct.is_cuda:
        raise ValueError("correct must be a uint8 device tensor [B]")
    correct = correct.contiguous()
    outs = dict(effective=torch.empty((B, K), dtype=torch.uint8, device=dev),
                in_s_acc=torch.empty((B, K), dtype=torch.uint8, device=dev),
                first_mismatch=torch.empty(B, dtype=torch.int32, device=dev),
                first_reject=torch.empty(B, dtype=torch.int32, device=dev),
                rho=torch.empty(B, dtype=torch.float32, device=dev),
                reward=torch.empty((B, K), dtype=torch.float32, device=dev),
                round_return=torch.empty(B, dtype=torch.float32, device=dev))
    st = _RL(_ptr(correct), float(alpha), float(beta), *[_ptr(outs[k]) for k in (
        "effective", "in_s_acc", "first_mismatch", "first_reject", "rho", "reward", "round_return")])
    return st, outs, correct


def prepare_block(target, draft, draft_tokens, hidden, head, lam: float, features: bool = True,
                  splits: int = 0,
                  sample_u: Optional[torch.Tensor] = None,
                  policy_u: Optional[torch.Tensor] = None,
                  correct: Optional[torch.Tensor] = None, alpha: float = 1.0,
                  beta: float = 0.25, hidden_row0: Optional[torch.Tensor] = None) -> Prepared:
    """sample_u: one uniform per target row [B, K+1] for temperature-1 candidates
    (cospec_options.sample_uniform); None for the greedy argmax.  policy_u: one
    uniform per decision [B, K] for sampled arbitration.  correct: uint8 [B]
    rollout correctness; turns on the per-round RL statistics (returned with an
    "rl_" prefix) with failure-reward weights alpha and beta.  hidden_row0: int64 [B]
    device tensor; hidden is then a packed [rows, d] array and decision i of sequence
    b reads row hidden_row0[b] + i - 1 (cospec_options.hidden_row0)."""
    B, R, V = target.shape
    K = R - 1
    ld = _row_stride(target)
    if K > 0 and _row_stride(draft) != ld:
        raise ValueError("target and draft rows must share one stride")
    if hidden_row0 is not None:
        if tuple(hidden_row0.shape) != (B,) or hidden_row0.dtype != torch.int64 or not hidden_row0.is_cuda:
            raise ValueError("hidden_row0 must be an int64 device tensor [B]")
        if hidden.dim() != 2 or not hidden.is_contiguous():
            raise ValueError("with hidden_row0, hidden must be a contiguous [rows, d] array")
        hidden_row0 = hidden_row0.contiguous()
    packed_ok = hidden_row0 is not None or (hidden.shape[:2] == (B, K) and hidden.is_contiguous())
    if K > 0 and (tuple(draft.shape) != (B, K, V) or tuple(draft_tokens.shape) != (B, K)
                  or draft_tokens.dtype != torch.int32 or not draft_tokens.is_contiguous()
                  or not packed_ok):
        raise ValueError("shape/dtype mismatch between target, draft, draft_tokens and hidden")
    dev = target.device
    hs = _head_struct(head)
    L = lib()
    ws_bytes = L.cospec_verify_block_workspace_size(B, K, V, ctypes.byref(hs))
    if ws_bytes == 0 and B > 0:
        raise CospecError("invalid sizes for cospec_verify_block")
    workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    outputs = dict(accept_len=torch.empty(B, dtype=torch.int32, device=dev),
                   tokens=torch.empty((B, K + 1), dtype=torch.int32, device=dev))
    feats, fst = _features(features, dev, B, K + 1, K, K)
    args = (_ptr(target), _ptr(draft) if K > 0 else None, _dtype_code(target), ld,
            _ptr(draft_tokens) if K > 0 else None, _ptr(hidden) if K > 0 else None,
            ctypes.byref(hs), float(lam), B, K, V, _ptr(outputs["accept_len"]),
            _ptr(outputs["tokens"]))
    p = Prepared(L.cospec_verify_block, args, outputs, feats, fst, workspace, splits,
                 _uniforms(sample_u, B, K + 1), _policy_uniforms(policy_u, B, K),
                 _rl(correct, alpha, beta, B, K, dev))
    if hidden_row0 is not None:
        p.hidden_row0, p.hidden_rows = hidden_row0, hidden.shape[0]
    p._keep = [hs, target, draft, draft_tokens, hidden, head]
    return p


def prepare_tree(target, draft, parent, node_tokens, hidden, head, lam: float,
                 features: bool = True, splits: int = 0,
                 sample_u: Optional[torch.Tensor] = None,
                 policy_u: Optional[torch.Tensor] = None) -> Prepared:
    """sample_u: one uniform per target row [B, N] for temperature-1 candidates;
    policy_u: one uniform per node [B, N] for sampled arbitration."""
    B, N, V = target.shape
    ld = _row_stride(target)
    if _row_stride(draft) != ld or tuple(draft.shape) != (B, N, V):
        raise ValueError("target and draft must both be [B, N, V] with one row stride")
    for t in (parent, node_tokens):
        if tuple(t.shape) != (B, N) or t.dtype != torch.int32 or not t.is_contiguous():
            raise ValueError("parent and node_tokens must be contiguous int32 [B, N]")
    if hidden.shape[:2] != (B, N) or not hidden.is_contiguous():
        raise ValueError("hidden must be contiguous [B, N, d]")
    dev = target.device
    hs = _head_struct(head)
    L = lib()
    ws_bytes = L.cospec_verify_tree_workspace_size(B, N, V, ctypes.byref(hs))
    if ws_bytes == 0 and B > 0:
        raise CospecError("invalid sizes for cospec_verify_tree")
    workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    outputs = dict(accept_len=torch.empty(B, dtype=torch.int32, device=dev),
                   tokens=torch.empty((B, N), dtype=torch.int32, device=dev),
                   path=torch.empty((B, N), dtype=torch.int32, device=dev))
    feats, fst = _features(features, dev, B, N, N, N)
    args = (_ptr(target), _ptr(draft), _dtype_code(target), ld, _ptr(parent), _ptr(node_tokens),
            _ptr(hidden), ctypes.byref(hs), float(lam), B, N, V, _ptr(outputs["accept_len"]),
            _ptr(outputs["tokens"]), _ptr(outputs["path"]))
    p = Prepared(L.cospec_verify_tree, args, outputs, feats, fst, workspace, splits,
                 _uniforms(sample_u, B, N), _policy_uniforms(policy_u, B, N))
    p._keep = [hs, target, draft, parent, node_tokens, hidden, head]
    return p


def verify_block(target, draft, draft_tokens, hidden, head, lam: float, features: bool = True,
                 splits: int = 0,
                 sample_u: Optional[torch.Tensor] = None,
                 policy_u: Optional[torch.Tensor] = None,
                 correct: Optional[torch.Tensor] = None, alpha: float = 1.0,
                 beta: float = 0.25, hidden_row0: Optional[torch.Tensor] = None) -> dict:
    """cospec_verify_block on device tensors; returns accept_len, tokens (+ features,
    + rl_* statistics when `correct` is given)."""
    p = prepare_block(target, draft, draft_tokens, hidden, head, lam, features, splits,
                      sample_u, policy_u, correct, alpha, beta, hidden_row0)
    p.launch()
    return p.result()


def verify_block_static(target, draft, draft_tokens, hidden, head, lam: float, features: bool = True,
                        splits: int = 0, sample_u: Optional[torch.Tensor] = None) -> dict:
    """cospec_verify_block_static: the chain step on the library's static scratch buffer
    (no workspace is allocated here or in the library).  Same results as verify_block."""
    B, R, V = target.shape
    K = R - 1
    ld = _row_stride(target)
    if K > 0 and (_row_stride(draft) != ld or tuple(draft.shape) != (B, K, V)
                  or tuple(draft_tokens.shape) != (B, K) or draft_tokens.dtype != torch.int32
                  or not draft_tokens.is_contiguous() or hidden.shape[:2] != (B, K)
                  or not hidden.is_contiguous()):
        raise ValueError("shape/dtype mismatch between target, draft, draft_tokens and hidden")
    dev = target.device
    hs = _head_struct(head)
    outputs = dict(accept_len=torch.empty(B, dtype=torch.int32, device=dev),
                   tokens=torch.empty((B, K + 1), dtype=torch.int32, device=dev))
    feats, fst = _features(features, dev, B, K + 1, K, K)
    u = _uniforms(sample_u, B, K + 1)
    opts = _Options(splits=int(splits), sample_uniform=_ptr(u)) if (splits or u is not None) else None
    code = lib().cospec_verify_block_static(
        _ptr(target), _ptr(draft) if K > 0 else None, _dtype_code(target), ld,
        _ptr(draft_tokens) if K > 0 else None, _ptr(hidden) if K > 0 else None, ctypes.byref(hs), float(lam),
        B, K, V, _ptr(outputs["accept_len"]), _ptr(outputs["tokens"]),
        ctypes.byref(fst) if fst is not None else None, ctypes.byref(opts) if opts is not None else None,
        _stream())
    _check(code, "cospec_verify_block_static")
    out = dict(outputs)
    out.update(feats or {})
    return out


def verify_tree(target, draft, parent, node_tokens, hidden, head, lam: float,
                features: bool = True, splits: int = 0,
                sample_u: Optional[torch.Tensor] = None,
                policy_u: Optional[torch.Tensor] = None) -> dict:
    """cospec_verify_tree on device tensors; returns accept_len, tokens, path (+ features)."""
    p = prepare_tree(target, draft, parent, node_tokens, hidden, head, lam, features, splits,
                     sample_u, policy_u)
    p.launch()
    return p.result()


def arbitrate(hidden, head, lam: float, row_index: Optional[torch.Tensor] = None) -> dict:
    """cospec_arbitrate: head logits and threshold decisions for selected hidden rows."""
    h2 = hidden.reshape(-1, hidden.shape[-1])
    if not h2.is_contiguous():
        raise ValueError("hidden must be contiguous")
    n_rows = h2.shape[0]
    if row_index is not None and (row_index.dtype != torch.int32 or not row_index.is_contiguous()):
        raise ValueError("row_index must be contiguous int32")
    n_sel = n_rows if row_index is None else row_index.numel()
    hs = _head_struct(head)
    L = lib()
    ws = torch.empty(max(L.cospec_arbitrate_workspace_size(n_sel, ctypes.byref(hs)), 256),
                     dtype=torch.uint8, device=hidden.device)
    z = torch.empty(n_sel, dtype=torch.float32, device=hidden.device)
    acc = torch.empty(n_sel, dtype=torch.uint8, device=hidden.device)
    code = L.cospec_arbitrate(_ptr(h2), n_rows, _ptr(row_index), n_sel, ctypes.byref(hs),
                              float(lam), _ptr(z), _ptr(acc), _ptr(ws), ws.numel(), _stream())
    _check(code, "cospec_arbitrate")
    return dict(z=z, accept=acc)


class SplitBlock:
    """The chain step in two phases around the caller's arbitrator
    (cospec_verify_block_reduce, then cospec_verify_block_arbitrate).  Creating it
    enqueues phase 1; `candidates` ([B, K+1] int32) then holds the target's
    candidates the arbitrator's input needs; `arbitrate()` enqueues phase 2 on the
    hidden states and returns the results of the whole step."""

    def __init__(self, target, draft, draft_tokens, head, features: bool = True, splits: int = 0,
                 sample_u: Optional[torch.Tensor] = None):
        B, R, V = target.shape
        K = R - 1
        ld = _row_stride(target)
        if K > 0 and (_row_stride(draft) != ld or tuple(draft.shape) != (B, K, V)
                      or tuple(draft_tokens.shape) != (B, K) or draft_tokens.dtype != torch.int32
                      or not draft_tokens.is_contiguous()):
            raise ValueError("shape/dtype mismatch between target, draft and draft_tokens")
        dev = target.device
        self._hs = _head_struct(head)
        L = lib()
        ws_bytes = L.cospec_verify_block_workspace_size(B, K, V, ctypes.byref(self._hs))
        if ws_bytes == 0 and B > 0:
            raise CospecError("invalid sizes for cospec_verify_block_reduce")
        self.workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
        self.candidates = torch.empty((B, K + 1), dtype=torch.int32, device=dev)
        self.features, self._fst = _features(features, dev, B, K + 1, K, K)
        self.splits = int(splits)
        self._u = _uniforms(sample_u, B, K + 1)
        self._common = (_ptr(target), _ptr(draft) if K > 0 else None, _dtype_code(target), ld,
                        _ptr(draft_tokens) if K > 0 else None)
        self._sizes = (B, K, V)
        self._keep = [target, draft, draft_tokens, head]
        opts = _Options(splits=self.splits, sample_uniform=_ptr(self._u))
        code = L.cospec_verify_block_reduce(*self._common, ctypes.byref(self._hs), B, K, V,
                                            _ptr(self.candidates),
                                            ctypes.byref(self._fst) if self._fst is not None else None,
                                            ctypes.byref(opts), _ptr(self.workspace),
                                            self.workspace.numel(), _stream())
        _check(code, "cospec_verify_block_reduce")

    def arbitrate(self, hidden, lam: float, policy_u: Optional[torch.Tensor] = None,
                  correct: Optional[torch.Tensor] = None, alpha: float = 1.0, beta: float = 0.25,
                  hidden_row0: Optional[torch.Tensor] = None) -> dict:
        """Phase 2.  hidden: [B, K, d], or with hidden_row0 (int64 [B]) a packed
        [rows, d] array where decision i of sequence b reads row hidden_row0[b] + i - 1."""
        B, K, V = self._sizes
        dev = self.workspace.device
        if not hidden.is_contiguous():
            raise ValueError("hidden must be contiguous")
        if hidden_row0 is not None:
            if tuple(hidden_row0.shape) != (B,) or hidden_row0.dtype != torch.int64 or not hidden_row0.is_cuda:
                raise ValueError("hidden_row0 must be an int64 device tensor [B]")
            hidden_row0 = hidden_row0.contiguous()
            n_hidden = hidden.reshape(-1, hidden.shape[-1]).shape[0]
        elif K > 0 and tuple(hidden.shape[:2]) != (B, K):
            raise ValueError("hidden must be [B, K, d] without hidden_row0")
        outputs = dict(accept_len=torch.empty(B, dtype=torch.int32, device=dev),
                       tokens=torch.empty((B, K + 1), dtype=torch.int32, device=dev))
        pu = _policy_uniforms(policy_u, B, K)
        rl = _rl(correct, alpha, beta, B, K, dev)
        opts = _Options(splits=self.splits, policy_uniform=_ptr(pu),
                        rl=None if rl is None else ctypes.pointer(rl[0]),
                        hidden_row0=_ptr(hidden_row0),
                        hidden_rows=n_hidden if hidden_row0 is not None else 0)
        code = lib().cospec_verify_block_arbitrate(
            *self._common, _ptr(hidden) if K > 0 else None, ctypes.byref(self._hs), float(lam), B, K, V,
            _ptr(outputs["accept_len"]), _ptr(outputs["tokens"]),
            ctypes.byref(self._fst) if self._fst is not None else None, ctypes.byref(opts),
            _ptr(self.workspace), self.workspace.numel(), _stream())
        _check(code, "cospec_verify_block_arbitrate")
        out = dict(outputs)
        out.update(self.features or {})
        out["tgt_candidate"] = self.candidates
        if rl is not None:
            out.update({"rl_" + k: v for k, v in rl[1].items()})
        self._keep += [hidden, pu, rl, hidden_row0]
        return out


def prepare_sps(target, draft, draft_tokens, uniforms, features: bool = True,
                splits: int = 0) -> Prepared:
    """Pre-marshalled cospec_verify_block_sps (standard speculative sampling over
    chain blocks).  uniforms: float32 [B, K+1] on the device (K acceptance tests,
    then the draw of the last token).  The result holds accept_len, tokens and the
    features; `policy` holds the acceptance probabilities min(1, p_T / p_D)."""
    B, R, V = target.shape
    K = R - 1
    ld = _row_stride(target)
    if K > 0 and (_row_stride(draft) != ld or tuple(draft.shape) != (B, K, V)
                  or tuple(draft_tokens.shape) != (B, K) or draft_tokens.dtype != torch.int32
                  or not draft_tokens.is_contiguous()):
        raise ValueError("shape/dtype mismatch between target, draft and draft_tokens")
    u = _uniforms(uniforms, B, K + 1)
    if u is None:
        raise ValueError("speculative sampling needs uniforms [B, K+1]")
    dev = target.device
    L = lib()
    ws = torch.empty(max(L.cospec_verify_block_sps_workspace_size(B, K, V), 256), dtype=torch.uint8,
                     device=dev)
    outputs = dict(accept_len=torch.empty(B, dtype=torch.int32, device=dev),
                   tokens=torch.empty((B, K + 1), dtype=torch.int32, device=dev))
    feats, fst = _features(features, dev, B, K + 1, K, K)
    unwritten = {}
    if feats is not None:        # members the baseline leaves untouched (kept alive: fst points at them)
        unwritten = {k: feats.pop(k) for k in ("z_tilde", "logp_action")}
    args = (_ptr(target), _ptr(draft) if K > 0 else None, _dtype_code(target), ld,
            _ptr(draft_tokens) if K > 0 else None, _ptr(u), B, K, V, _ptr(outputs["accept_len"]),
            _ptr(outputs["tokens"]))
    p = Prepared(L.cospec_verify_block_sps, args, outputs, feats, fst, ws, splits)
    p._keep = [target, draft, draft_tokens, u, unwritten]
    return p


def sps_block(target, draft, draft_tokens, uniforms, features: bool = True, splits: int = 0) -> dict:
    """cospec_verify_block_sps on device tensors (see prepare_sps)."""
    p = prepare_sps(target, draft, draft_tokens, uniforms, features, splits)
    p.launch()
    return p.result()


def _i32(t: torch.Tensor, n: int, what: str) -> torch.Tensor:
    if tuple(t.shape) != (n,) or t.dtype != torch.int32 or not t.is_cuda:
        raise ValueError(f"{what} must be an int32 device tensor [{n}]")
    return t.contiguous()


def hybrid_mask(ctx_len: torch.Tensor, K: int, L: int) -> torch.Tensor:
    """cospec_hybrid_mask: the arbitrator's attention mask [B, L, L] (uint8, 1 = attend)."""
    B = ctx_len.shape[0]
    ctx = _i32(ctx_len, B, "ctx_len")
    out = torch.empty((B, L, L), dtype=torch.uint8, device=ctx.device)
    _check(lib().cospec_hybrid_mask(_ptr(ctx), B, int(K), int(L), _ptr(out), _stream()), "cospec_hybrid_mask")
    return out


def hybrid_attention(q, k, v, ctx_len, q_start, K: int, scale: float) -> torch.Tensor:
    """cospec_hybrid_attention: q [B, n_q, Hq, D], k and v [B, L, Hkv, D] (bf16, contiguous)
    -> [B, n_q, Hq, D] bf16, under the arbitrator's hybrid mask."""
    B, nq, Hq, D = q.shape
    L, Hkv = k.shape[1], k.shape[2]
    for t in (q, k, v):
        if t.dtype != torch.bfloat16 or not t.is_contiguous() or not t.is_cuda:
            raise ValueError("q, k and v must be contiguous bf16 device tensors")
    if tuple(k.shape) != (B, L, Hkv, D) or tuple(v.shape) != (B, L, Hkv, D):
        raise ValueError("k and v must be [B, L, Hkv, D]")
    ctx = _i32(ctx_len, B, "ctx_len")
    qs = _i32(q_start, B, "q_start")
    out = torch.empty_like(q)
    code = lib().cospec_hybrid_attention(_ptr(q), _ptr(k), _ptr(v), _ptr(ctx), _ptr(qs), B, nq, L, Hq, Hkv,
                                         D, int(K), float(scale), _ptr(out), _stream())
    _check(code, "cospec_hybrid_attention")
    return out
