"""Thin ctypes binding of libppattn.so (include/pp_attn.h).

Each function has the name of the C entry point it calls and only marshals
arguments: it takes torch tensors for device memory, passes their data pointers
and the current HIP stream, allocates outputs and the workspace with torch, and
raises PPError on a non-zero status.  Every step of the computation runs in the
library's HIP kernels; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
import torch

from .workload import Pack

_PKG = os.path.dirname(os.path.abspath(__file__))
# PP_LIB_PATH selects another build of the library (e.g. a host-sanitized one)
LIB_PATH = os.environ.get("PP_LIB_PATH") or os.path.join(_PKG, "libppattn.so")

PP_OK = 0
PP_BF16 = 0
PP_FP32 = 1
STATUS = {0: "PP_OK", 1: "PP_ERR_INVALID_ARGUMENT", 2: "PP_ERR_BAD_LAYOUT", 3: "PP_ERR_UNSUPPORTED",
          4: "PP_ERR_WORKSPACE_TOO_SMALL", 5: "PP_ERR_HIP"}

EXPORTED = [
    "pp_workspace_size", "pp_attn_fwd", "pp_attn_bwd", "pp_seq_logprob", "pp_seq_logprob_bwd", "pp_dpo_loss",
    "pp_rm_workspace_size", "pp_rm_scores", "pp_rm_scores_bwd", "pp_pack_stats",
    "pp_pack_export", "pp_tile_class_len", "pp_timing_enable", "pp_timing_select", "pp_timing_reset",
    "pp_timing_count", "pp_timing_get", "pp_status_string", "pp_last_error", "pp_version",
    "pp_rope_workspace_size", "pp_rope", "pp_attn_fwd_rope", "pp_attn_bwd_rope",
    "pp_plan_workspace_size", "pp_plan_create", "pp_plan_destroy", "pp_attn_fwd_planned", "pp_attn_bwd_planned",
    "pp_attn_fwd_noalloc", "pp_build_id", "pp_logprob_row_count", "pp_seq_logprob_bwd_rows",
    "pp_bwd_stored_ds_workspace_size",
]

NOALLOC_SCRATCH_BYTES = 4 << 20  # PP_NOALLOC_SCRATCH_BYTES


class PackStats(ctypes.Structure):
    _fields_ = [("tokens_packed", ctypes.c_int64), ("tokens_unpacked", ctypes.c_int64),
                ("tokens_padded", ctypes.c_int64), ("pairs_packed", ctypes.c_int64),
                ("pairs_unpacked", ctypes.c_int64), ("pairs_padded", ctypes.c_int64),
                ("pairs_dense_packed", ctypes.c_int64), ("eq1_cost_ratio", ctypes.c_double),
                ("eq1_memory_ratio", ctypes.c_double), ("rows_eq1_cheaper", ctypes.c_int32),
                ("rows_with_responses", ctypes.c_int32)]


class PPError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class _Desc(ctypes.Structure):
    _fields_ = [
        ("num_rows", ctypes.c_int32),
        ("max_resp", ctypes.c_int32),
        ("row_start", ctypes.POINTER(ctypes.c_int32)),
        ("prompt_len", ctypes.POINTER(ctypes.c_int32)),
        ("num_resp", ctypes.POINTER(ctypes.c_int32)),
        ("resp_off", ctypes.POINTER(ctypes.c_int32)),
        ("resp_len", ctypes.POINTER(ctypes.c_int32)),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    """Loads the built library (raises if it was not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2602_24082_amd.build` "
                          "(there is no non-HIP fallback)")
    L = ctypes.CDLL(LIB_PATH)
    L.pp_build_id.restype = ctypes.c_char_p
    from .build import source_digest
    built, want = L.pp_build_id().decode(), source_digest()
    if built != want:
        raise ImportError(f"{LIB_PATH} was built from other sources (build id {built[:12]}, sources {want[:12]}): "
                          "rebuild it with `python -m paper_2602_24082_amd.build`")
    P = ctypes.c_void_p
    i32 = ctypes.c_int32
    i = ctypes.c_int
    sz = ctypes.c_size_t
    D = ctypes.POINTER(_Desc)
    L.pp_workspace_size.argtypes = [D, i, i, i, i, i, ctypes.POINTER(sz), ctypes.POINTER(sz),
                                    ctypes.POINTER(sz), ctypes.POINTER(sz)]
    L.pp_attn_fwd.argtypes = [D, i, i, i, i, ctypes.c_float, P, P, P, P, P, P, sz, P]
    L.pp_attn_bwd.argtypes = [D, i, i, i, i, ctypes.c_float, P, P, P, P, P, P, P, P, P, P, sz, P]
    L.pp_attn_fwd_noalloc.argtypes = [D, i, i, i, ctypes.c_float, P, P, P, P, P, P]
    f32 = ctypes.c_float
    L.pp_rope_workspace_size.argtypes = [D, i, ctypes.POINTER(sz)]
    L.pp_rope.argtypes = [D, i, i, i, f32, i, P, P, P, sz, P]
    L.pp_attn_fwd_rope.argtypes = [D, i, i, i, i, f32, f32, P, P, P, P, P, P, P, P, sz, P]
    L.pp_attn_bwd_rope.argtypes = [D, i, i, i, i, f32, f32, P, P, P, P, P, P, P, P, P, P, sz, P]
    L.pp_plan_workspace_size.argtypes = [D, i, i, i, i, ctypes.POINTER(sz)]
    L.pp_bwd_stored_ds_workspace_size.argtypes = [D, i, i, i, i, ctypes.POINTER(sz), ctypes.POINTER(sz)]
    L.pp_plan_create.argtypes = [D, i, i, i, i, ctypes.POINTER(f32), P, sz, P, ctypes.POINTER(P)]
    L.pp_plan_destroy.argtypes = [P]
    L.pp_attn_fwd_planned.argtypes = [P, f32, P, P, P, P, P, P, P, P]
    L.pp_attn_bwd_planned.argtypes = [P, f32, P, P, P, P, P, P, P, P, P, P]
    L.pp_seq_logprob.argtypes = [D, i, i, P, P, P, P, P, sz, P]
    L.pp_seq_logprob_bwd.argtypes = [D, i, i, P, P, P, P, P, sz, P]
    L.pp_logprob_row_count.argtypes = [D, ctypes.POINTER(ctypes.c_int64)]
    L.pp_seq_logprob_bwd_rows.argtypes = [D, i, i, P, P, P, P, P, P, sz, P]
    L.pp_rm_workspace_size.argtypes = [D, ctypes.POINTER(sz)]
    L.pp_pack_stats.argtypes = [D, ctypes.POINTER(PackStats)]
    L.pp_rm_scores.argtypes = [D, i, i, P, P, ctypes.c_float, P, P, sz, P]
    L.pp_rm_scores_bwd.argtypes = [D, i, i, P, P, P, P, P, P, P, sz, P]
    L.pp_dpo_loss.argtypes = [i32, i32, P, P, P, ctypes.c_float, P, P, P, P, sz, P]
    L.pp_pack_export.argtypes = [D, i, i, P, P, P, sz]
    L.pp_tile_class_len.argtypes = [D, i, i, ctypes.POINTER(sz)]
    L.pp_timing_enable.argtypes = [i]
    L.pp_timing_select.argtypes = [ctypes.c_char_p]
    L.pp_timing_reset.argtypes = []
    L.pp_timing_count.argtypes = []
    L.pp_timing_count.restype = i
    L.pp_timing_get.argtypes = [i, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_double),
                                ctypes.POINTER(ctypes.c_int64)]
    L.pp_status_string.argtypes = [i]
    L.pp_status_string.restype = ctypes.c_char_p
    L.pp_last_error.argtypes = []
    L.pp_last_error.restype = ctypes.c_char_p
    L.pp_version.restype = i
    for name in ("pp_workspace_size", "pp_attn_fwd", "pp_attn_bwd", "pp_seq_logprob", "pp_dpo_loss",
                 "pp_pack_export", "pp_tile_class_len", "pp_timing_enable", "pp_timing_select",
                 "pp_timing_reset", "pp_timing_get"):
        getattr(L, name).restype = i
    _lib = L
    return L


def _check(status: int):
    if status != PP_OK:
        raise PPError(status, lib().pp_last_error().decode())


class _DescHolder:
    """Keeps the int32 arrays of a Pack alive while the C struct points at them."""

    def __init__(self, pack: Pack):
        c = lambda a: np.ascontiguousarray(a, dtype=np.int32)
        self.arrays = [c(pack.row_start), c(pack.prompt_len), c(pack.num_resp),
                       c(pack.resp_off).reshape(-1), c(pack.resp_len).reshape(-1)]
        ptr = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        self.desc = _Desc(pack.num_rows, pack.max_resp, *[ptr(a) for a in self.arrays])

    @property
    def ref(self):
        return ctypes.byref(self.desc)


def _desc_of(pack: Pack) -> _DescHolder:
    """The C descriptor of a pack, built on first use and kept on the pack (a
    pack is usually passed to many calls: every layer's attention, the
    log-probs, the loss); rebuilt whenever the pack's arrays have changed."""
    key = (pack.num_rows, pack.max_resp) + tuple(
        np.asarray(a).tobytes() for a in (pack.row_start, pack.prompt_len, pack.num_resp, pack.resp_off, pack.resp_len))
    h = getattr(pack, "_pp_desc", None)
    if h is None or h.key != key:
        h = _DescHolder(pack)
        h.key = key
        try:
            pack._pp_desc = h
        except AttributeError:  # a pack type that takes no new attributes: no caching
            pass
    return h


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return PP_BF16
    if t.dtype == torch.float32:
        return PP_FP32
    raise TypeError(f"unsupported dtype {t.dtype} (bf16 or fp32)")


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def pp_workspace_size(pack: Pack, hq: int = 1, hkv: int = 1, head_dim: int = 64, vocab: int = 0,
                      fwd=True, bwd=True, logprob=False, loss=True, dtype: int = PP_BF16):
    """Workspace bytes (fwd, bwd, logprob, loss); entries not asked for are None.
    dtype is the attention input dtype code (PP_BF16 or PP_FP32)."""
    h = _desc_of(pack)
    vals = [ctypes.c_size_t(0) for _ in range(4)]
    want = [fwd, bwd, logprob, loss]
    args = [ctypes.byref(v) if w else None for v, w in zip(vals, want)]
    _check(lib().pp_workspace_size(h.ref, dtype, hq, hkv, head_dim, vocab, *args))
    return tuple(int(v.value) if w else None for v, w in zip(vals, want))


def pp_bwd_stored_ds_workspace_size(pack: Pack, hq: int, hkv: int, head_dim: int, dtype: int = PP_BF16):
    """(bwd, plan) workspace bytes that select the backward's stored-dS mode."""
    h = _desc_of(pack)
    b, p = ctypes.c_size_t(0), ctypes.c_size_t(0)
    _check(lib().pp_bwd_stored_ds_workspace_size(h.ref, dtype, hq, hkv, head_dim, ctypes.byref(b), ctypes.byref(p)))
    return int(b.value), int(p.value)


def _bwd_workspace_bytes(pack: Pack, hq: int, hkv: int, d: int, dtype: int, store_ds: bool) -> int:
    if store_ds:
        return pp_bwd_stored_ds_workspace_size(pack, hq, hkv, d, dtype)[0]
    return pp_workspace_size(pack, hq, hkv, d, fwd=False, bwd=True, loss=False, dtype=dtype)[1]


def pp_attn_fwd(pack: Pack, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, scale: float = 0.0,
                out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                ws: Optional[torch.Tensor] = None):
    """Packed attention forward; returns (o [sumT,hq,d], lse [hq,sumT] fp32)."""
    T, hq, d = q.shape
    hkv = k.shape[1]
    h = _desc_of(pack)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty(hq, T, dtype=torch.float32, device=q.device)
    if ws is None:
        nb, = pp_workspace_size(pack, hq, hkv, d, fwd=True, bwd=False, loss=False, dtype=_dtype_code(q))[:1]
        ws = _workspace(nb, q.device)
    _check(lib().pp_attn_fwd(h.ref, _dtype_code(q), hq, hkv, d, float(scale), _ptr(q), _ptr(k), _ptr(v),
                             _ptr(out), _ptr(lse), _ptr(ws), ws.numel(), _stream(q.device)))
    return out, lse


def pp_attn_bwd(pack: Pack, q, k, v, o, lse, dout, scale: float = 0.0, dq=None, dk=None, dv=None,
                ws=None, store_ds: bool = False):
    """Packed attention backward; returns (dq, dk, dv) in the input dtype.  The
    library picks its mode from the workspace size: a workspace allocated here
    holds the stored dS when store_ds is set (else the dQ pass recomputes)."""
    T, hq, d = q.shape
    hkv = k.shape[1]
    h = _desc_of(pack)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    if ws is None:
        ws = _workspace(_bwd_workspace_bytes(pack, hq, hkv, d, _dtype_code(q), store_ds), q.device)
    _check(lib().pp_attn_bwd(h.ref, _dtype_code(q), hq, hkv, d, float(scale), _ptr(q), _ptr(k), _ptr(v),
                             _ptr(o), _ptr(lse), _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(ws),
                             ws.numel(), _stream(q.device)))
    return dq, dk, dv


def pp_rope_workspace_size(pack: Pack, head_dim: int) -> int:
    h = _desc_of(pack)
    n = ctypes.c_size_t(0)
    _check(lib().pp_rope_workspace_size(h.ref, head_dim, ctypes.byref(n)))
    return n.value


def pp_rope(pack: Pack, x: torch.Tensor, rope_base: float, inverse: bool = False, out=None, ws=None):
    """Rotary embedding of x [sumT, heads, d] on the packed position IDs; out may be x."""
    T, H, d = x.shape
    h = _desc_of(pack)
    out = torch.empty_like(x) if out is None else out
    if ws is None:
        ws = _workspace(pp_rope_workspace_size(pack, d), x.device)
    _check(lib().pp_rope(h.ref, _dtype_code(x), H, d, float(rope_base), int(bool(inverse)), _ptr(x), _ptr(out),
                         _ptr(ws), ws.numel(), _stream(x.device)))
    return out


def pp_attn_fwd_noalloc(pack: Pack, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, scale: float = 0.0,
                        out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None):
    """pp_attn_fwd (bf16) with the plan in the library's static device scratch
    instead of a workspace; returns (o, lse).  Allocates o and lse here only
    when they are not given."""
    T, hq, d = q.shape
    hkv = k.shape[1]
    h = _desc_of(pack)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty(hq, T, dtype=torch.float32, device=q.device)
    _check(lib().pp_attn_fwd_noalloc(h.ref, hq, hkv, d, float(scale), _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                     _ptr(lse), _stream(q.device)))
    return out, lse


def pp_attn_fwd_rope(pack: Pack, q, k, v, rope_base: float, scale: float = 0.0, want_q_rot: bool = True,
                     out=None, lse=None, q_rot=None, k_rot=None, ws=None):
    """Attention of rotated q, k (rotation fused into the forward); returns
    (o, lse, q_rot or None, k_rot)."""
    T, hq, d = q.shape
    hkv = k.shape[1]
    h = _desc_of(pack)
    out = torch.empty_like(q) if out is None else out
    if lse is None:
        lse = torch.empty(hq, T, dtype=torch.float32, device=q.device)
    if want_q_rot and q_rot is None:
        q_rot = torch.empty_like(q)
    k_rot = torch.empty_like(k) if k_rot is None else k_rot
    if ws is None:
        nb = pp_workspace_size(pack, hq, hkv, d, fwd=True, bwd=False, loss=False, dtype=_dtype_code(q))[0]
        ws = _workspace(nb, q.device)
    _check(lib().pp_attn_fwd_rope(h.ref, _dtype_code(q), hq, hkv, d, float(scale), float(rope_base), _ptr(q),
                                  _ptr(k), _ptr(v), _ptr(out), _ptr(lse), _ptr(q_rot), _ptr(k_rot), _ptr(ws),
                                  ws.numel(), _stream(q.device)))
    return out, lse, q_rot, k_rot


def pp_attn_bwd_rope(pack: Pack, q_rot, k_rot, v, o, lse, dout, rope_base: float, scale: float = 0.0,
                     dq=None, dk=None, dv=None, ws=None, store_ds: bool = False):
    """Backward of pp_attn_fwd_rope: (dq, dk) with respect to the un-rotated q, k, and dv
    (workspace and mode as pp_attn_bwd)."""
    T, hq, d = q_rot.shape
    hkv = k_rot.shape[1]
    h = _desc_of(pack)
    dq = torch.empty_like(q_rot) if dq is None else dq
    dk = torch.empty_like(k_rot) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    if ws is None:
        ws = _workspace(_bwd_workspace_bytes(pack, hq, hkv, d, _dtype_code(q_rot), store_ds), q_rot.device)
    _check(lib().pp_attn_bwd_rope(h.ref, _dtype_code(q_rot), hq, hkv, d, float(scale), float(rope_base),
                                  _ptr(q_rot), _ptr(k_rot), _ptr(v), _ptr(o), _ptr(lse), _ptr(dout), _ptr(dq),
                                  _ptr(dk), _ptr(dv), _ptr(ws), ws.numel(), _stream(q_rot.device)))
    return dq, dk, dv


class PlanHandle:
    """A pp_plan handle and the workspace tensor it was staged into (kept alive
    with it).  Free it with pp_plan_destroy (also done when it is collected)."""

    def __init__(self, handle: ctypes.c_void_p, ws: torch.Tensor, hq: int, hkv: int, head_dim: int,
                 rope_base: Optional[float]):
        self.handle, self.ws = handle, ws
        self.hq, self.hkv, self.head_dim, self.rope_base = hq, hkv, head_dim, rope_base

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.pp_plan_destroy(self.handle)
            self.handle = None


def pp_plan_workspace_size(pack: Pack, hq: int, hkv: int, head_dim: int, dtype: int = PP_BF16) -> int:
    h = _desc_of(pack)
    n = ctypes.c_size_t(0)
    _check(lib().pp_plan_workspace_size(h.ref, dtype, hq, hkv, head_dim, ctypes.byref(n)))
    return n.value


def pp_plan_create(pack: Pack, hq: int, hkv: int, head_dim: int, dtype: int = PP_BF16,
                   rope_base: Optional[float] = None, ws: Optional[torch.Tensor] = None,
                   device="cuda:0", store_ds: bool = False) -> PlanHandle:
    """Plans the pack once and stages the metadata into ws on the current stream
    (a workspace allocated here holds the stored dS when store_ds is set)."""
    h = _desc_of(pack)
    if ws is None:
        nb = (pp_bwd_stored_ds_workspace_size(pack, hq, hkv, head_dim, dtype)[1] if store_ds
              else pp_plan_workspace_size(pack, hq, hkv, head_dim, dtype))
        ws = _workspace(nb, device)
    base = ctypes.c_float(rope_base) if rope_base is not None else None
    out = ctypes.c_void_p(None)
    _check(lib().pp_plan_create(h.ref, dtype, hq, hkv, head_dim, ctypes.byref(base) if base is not None else None,
                                _ptr(ws), ws.numel(), _stream(ws.device), ctypes.byref(out)))
    return PlanHandle(out, ws, hq, hkv, head_dim, rope_base)


def pp_plan_destroy(plan: PlanHandle):
    if plan.handle:
        _check(lib().pp_plan_destroy(plan.handle))
        plan.handle = None


def pp_attn_fwd_planned(plan: PlanHandle, q, k, v, scale: float = 0.0, out=None, lse=None, q_rot=None, k_rot=None):
    """pp_attn_fwd (pp_attn_fwd_rope for a rotary plan) on a plan; returns
    (o, lse) or, for a rotary plan, (o, lse, q_rot, k_rot)."""
    T, hq, d = q.shape
    out = torch.empty_like(q) if out is None else out
    if lse is None:
        lse = torch.empty(hq, T, dtype=torch.float32, device=q.device)
    if plan.rope_base is not None and k_rot is None:
        k_rot = torch.empty_like(k)
    _check(lib().pp_attn_fwd_planned(plan.handle, float(scale), _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse),
                                     _ptr(q_rot), _ptr(k_rot), _stream(q.device)))
    return (out, lse) if plan.rope_base is None else (out, lse, q_rot, k_rot)


def pp_attn_bwd_planned(plan: PlanHandle, q, k, v, o, lse, dout, scale: float = 0.0, dq=None, dk=None, dv=None):
    """pp_attn_bwd (pp_attn_bwd_rope for a rotary plan, q and k rotated) on a plan."""
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    _check(lib().pp_attn_bwd_planned(plan.handle, float(scale), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse),
                                     _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), _stream(q.device)))
    return dq, dk, dv


def pp_seq_logprob(pack: Pack, logits: torch.Tensor, tokens: torch.Tensor, want_tok: bool = False,
                   seq=None, tok=None, ws=None):
    """Per-response summed log-probs [B, K_max] (and per-token [sumT] if asked)."""
    V = logits.shape[1]
    h = _desc_of(pack)
    dev = logits.device
    if seq is None:
        seq = torch.empty(pack.num_rows, max(pack.max_resp, 1), dtype=torch.float32, device=dev)
    if want_tok and tok is None:
        tok = torch.empty(logits.shape[0], dtype=torch.float32, device=dev)
    if ws is None:
        nb = pp_workspace_size(pack, vocab=V, fwd=False, bwd=False, logprob=True, loss=False)[2]
        ws = _workspace(nb, dev)
    if tokens.dtype != torch.int32:
        raise TypeError("tokens must be int32")
    _check(lib().pp_seq_logprob(h.ref, _dtype_code(logits), V, _ptr(logits), _ptr(tokens), _ptr(seq),
                                _ptr(tok), _ptr(ws), ws.numel(), _stream(dev)))
    return (seq, tok) if want_tok else seq


def pp_seq_logprob_bwd(pack: Pack, logits: torch.Tensor, tokens: torch.Tensor, dseq: torch.Tensor,
                       dlogits=None, ws=None):
    """Gradient of sum(dseq * seq_logp) w.r.t. the logits: [sumT, V] in the logits' dtype."""
    V = logits.shape[1]
    h = _desc_of(pack)
    dev = logits.device
    if dlogits is None:
        dlogits = torch.empty_like(logits)
    if ws is None:
        nb = pp_workspace_size(pack, vocab=V, fwd=False, bwd=False, logprob=True, loss=False)[2]
        ws = _workspace(nb, dev)
    if tokens.dtype != torch.int32:
        raise TypeError("tokens must be int32")
    if dseq.dtype != torch.float32 or not dseq.is_contiguous():
        raise TypeError("dseq must be contiguous float32 [B, K_max]")
    _check(lib().pp_seq_logprob_bwd(h.ref, _dtype_code(logits), V, _ptr(logits), _ptr(tokens), _ptr(dseq),
                                    _ptr(dlogits), _ptr(ws), ws.numel(), _stream(dev)))
    return dlogits


def pp_logprob_row_count(pack: Pack) -> int:
    """Number of logit rows that predict a response token."""
    h = _desc_of(pack)
    n = ctypes.c_int64(0)
    _check(lib().pp_logprob_row_count(h.ref, ctypes.byref(n)))
    return int(n.value)


def pp_seq_logprob_bwd_rows(pack: Pack, logits: torch.Tensor, tokens: torch.Tensor, dseq: torch.Tensor,
                            dlogits_rows=None, row_index=None, ws=None):
    """Gradient of sum(dseq * seq_logp) on the predicting logit rows only:
    (dlogits_rows [n, V] in the logits' dtype, row_index [n] int32)."""
    V = logits.shape[1]
    h = _desc_of(pack)
    dev = logits.device
    n = pp_logprob_row_count(pack)
    if dlogits_rows is None:
        dlogits_rows = torch.empty(n, V, dtype=logits.dtype, device=dev)
    if row_index is None:
        row_index = torch.empty(n, dtype=torch.int32, device=dev)
    if ws is None:
        nb = pp_workspace_size(pack, vocab=V, fwd=False, bwd=False, logprob=True, loss=False)[2]
        ws = _workspace(nb, dev)
    if tokens.dtype != torch.int32:
        raise TypeError("tokens must be int32")
    if dseq.dtype != torch.float32 or not dseq.is_contiguous():
        raise TypeError("dseq must be contiguous float32 [B, K_max]")
    _check(lib().pp_seq_logprob_bwd_rows(h.ref, _dtype_code(logits), V, _ptr(logits), _ptr(tokens), _ptr(dseq),
                                         _ptr(dlogits_rows), _ptr(row_index), _ptr(ws), ws.numel(), _stream(dev)))
    return dlogits_rows, row_index


def pp_rm_workspace_size(pack: Pack) -> int:
    h = _desc_of(pack)
    n = ctypes.c_size_t(0)
    _check(lib().pp_rm_workspace_size(h.ref, ctypes.byref(n)))
    return n.value


def pp_rm_scores(pack: Pack, hidden: torch.Tensor, w: torch.Tensor, bias: float = 0.0, scores=None, ws=None):
    """Reward-model head scores [B, K_max] (float32) on each response's last token."""
    H = hidden.shape[1]
    if w.dtype != hidden.dtype or w.numel() != H:
        raise TypeError("w must be [hidden_dim] in the dtype of hidden")
    h = _desc_of(pack)
    dev = hidden.device
    if scores is None:
        scores = torch.empty(pack.num_rows, max(pack.max_resp, 1), dtype=torch.float32, device=dev)
    if ws is None:
        ws = _workspace(pp_rm_workspace_size(pack), dev)
    _check(lib().pp_rm_scores(h.ref, _dtype_code(hidden), H, _ptr(hidden), _ptr(w), float(bias), _ptr(scores),
                              _ptr(ws), ws.numel(), _stream(dev)))
    return scores


def pp_rm_scores_bwd(pack: Pack, hidden: torch.Tensor, w: torch.Tensor, dscores: torch.Tensor, ws=None):
    """(dhidden [sumT, H] in hidden's dtype, dw [H] float32, dbias [1] float32)."""
    H = hidden.shape[1]
    h = _desc_of(pack)
    dev = hidden.device
    if dscores.dtype != torch.float32 or not dscores.is_contiguous():
        raise TypeError("dscores must be contiguous float32 [B, K_max]")
    dh = torch.empty_like(hidden)
    dw = torch.empty(H, dtype=torch.float32, device=dev)
    db = torch.empty(1, dtype=torch.float32, device=dev)
    if ws is None:
        ws = _workspace(pp_rm_workspace_size(pack), dev)
    _check(lib().pp_rm_scores_bwd(h.ref, _dtype_code(hidden), H, _ptr(hidden), _ptr(w), _ptr(dscores), _ptr(dh),
                                  _ptr(dw), _ptr(db), _ptr(ws), ws.numel(), _stream(dev)))
    return dh, dw, db


def pp_dpo_loss(num_resp, logp_pol: torch.Tensor, logp_ref: Optional[torch.Tensor], beta: float,
                want_rows: bool = True, want_grad: bool = True, ws=None):
    """Ranked-pair DPO / BT loss; returns (loss [1], row_loss [B] or None, dlogp [B,K] or None)."""
    nr = np.ascontiguousarray(num_resp, dtype=np.int32)
    B, K = logp_pol.shape
    dev = logp_pol.device
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    rows = torch.empty(B, dtype=torch.float32, device=dev) if want_rows else None
    grad = torch.empty(B, K, dtype=torch.float32, device=dev) if want_grad else None
    if ws is None:
        ws = _workspace((B * 4 + 255) // 256 * 256, dev)
    _check(lib().pp_dpo_loss(B, K, ctypes.c_void_p(nr.ctypes.data), _ptr(logp_pol), _ptr(logp_ref),
                             float(beta), _ptr(loss), _ptr(rows), _ptr(grad), _ptr(ws), ws.numel(),
                             _stream(dev)))
    return loss, rows, grad


def pp_pack_stats(pack: Pack) -> dict:
    """Host-only packed-versus-unpacked accounting (tokens, pairs, Eq. (1) ratios)."""
    h = _desc_of(pack)
    out = PackStats()
    _check(lib().pp_pack_stats(h.ref, ctypes.byref(out)))
    return {name: getattr(out, name) for name, _ in PackStats._fields_}


def pp_pack_export(pack: Pack, block_q: int = 128, block_k: int = 64, tiles: bool = True):
    """Host-only integer export: (position_ids, segment_ids, tile_class) numpy arrays."""
    h = _desc_of(pack)
    T = max(0, pack.total_tokens)  # a broken descriptor is the library's to report
    pos = np.zeros(T, np.int32)
    seg = np.zeros(T, np.int32)
    n = ctypes.c_size_t(0)
    tc = None
    if tiles:
        _check(lib().pp_tile_class_len(h.ref, block_q, block_k, ctypes.byref(n)))
        tc = np.zeros(n.value, np.uint8)
    _check(lib().pp_pack_export(h.ref, block_q, block_k, ctypes.c_void_p(pos.ctypes.data),
                                ctypes.c_void_p(seg.ctypes.data),
                                ctypes.c_void_p(tc.ctypes.data) if tiles else None, n.value))
    return pos, seg, tc


# ---------------------------------------------------------------- timing


def pp_timing_enable(on: bool = True):
    _check(lib().pp_timing_enable(1 if on else 0))


def pp_timing_select(names=None):
    """Time only the named launches (iterable of names, or None for all)."""
    arg = None if not names else ",".join(names).encode()
    _check(lib().pp_timing_select(arg))


def pp_timing_reset():
    _check(lib().pp_timing_reset())


def pp_timing_get() -> dict:
    """{kernel name: (total ms, launches)} since the last reset (waits for events)."""
    L = lib()
    out = {}
    for idx in range(L.pp_timing_count()):
        name = ctypes.c_char_p()
        ms = ctypes.c_double()
        n = ctypes.c_int64()
        _check(L.pp_timing_get(idx, ctypes.byref(name), ctypes.byref(ms), ctypes.byref(n)))
        out[name.value.decode()] = (ms.value, n.value)
    return out
