"""k-MIP self-attention for MI355X (gfx950): Python front end of libkmip.so.

Every function marshals torch tensors into the C ABI of include/kmip.h and
launches on the current HIP stream; all arithmetic runs in the library's HIP
kernels.  Tensors: Q, K are bf16 [N, H, d] (d = d_K), V and dOut bf16
[N, H, dv] (dv = d_V, the value width; dv = d unless the caller's V is
narrower or wider) on the GPU; out and dV are float32 [N, H, dv], dQ and dK
float32 [N, H, d]; topk_idx is int32 [N, H, k]; lse is float32 [N, H].
Attention dropout: ``keep`` is a uint8 [N, H, k] tensor of draws aligned
with the index slots (nonzero keeps a slot's weight, scaled by
1/(1 - drop_rate)), drawn by the caller.
``graph_offsets`` is a host-side int32 sequence [G+1] (or None for one graph).
"""
from __future__ import annotations

import ctypes
from typing import Optional, Sequence

import numpy as np

from ._lib import KmipError, MAX_K, MAX_K_WIDE, NOALLOC_SCRATCH_BYTES, check, load

__all__ = [
    "KmipError", "MAX_K", "MAX_K_WIDE", "NOALLOC_SCRATCH_BYTES", "topk", "topk_prefilter", "topk_prefilter_workspace_size", "attend", "fwd", "fwd_noalloc", "bwd",
    "attention", "topk_workspace_size", "bwd_workspace_size", "Workspace", "load", "KMIPAttention",
    "linear_k_schedule",
]


def _torch():
    import torch
    return torch


def _stream_ptr():
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _validate(*specs):
    """Checks (tensor, name, dtype, shape) specs before anything is allocated
    or launched: every tensor must have its dtype and shape (None: any) and
    be contiguous, and then all must sit on the same GPU.  The C ABI cannot
    see buffer sizes, so a size mismatch has to be caught here, before a
    kernel would read or write out of bounds."""
    torch = _torch()
    for t, name, dtype, shape in specs:
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a torch tensor")
        if t.dtype != dtype:
            raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
        if shape is not None and tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    dev = specs[0][0].device
    for t, name, _, _ in specs:
        if not t.is_cuda:
            raise TypeError(f"{name} must be a CUDA (HIP) tensor")
        if t.device != dev:
            raise ValueError(f"{name} is on {t.device}, expected {dev} (the device of {specs[0][1]})")


def _ptr(t):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def _offsets(graph_offsets):
    if graph_offsets is None:
        return None, None, 1
    o = np.ascontiguousarray(np.asarray(graph_offsets), dtype=np.int32)
    return o, o.ctypes.data_as(ctypes.c_void_p), len(o) - 1


def topk_workspace_size(N: int, H: int, d: int, k: int, num_graphs: int = 1) -> int:
    return int(load().kmip_topk_workspace_size(N, H, d, k, num_graphs))


def bwd_workspace_size(N: int, H: int, d: int, k: int, variant: int = 0, dv: Optional[int] = None) -> int:
    return int(load().kmip_bwd_ex_workspace_size(N, H, d, d if dv is None else dv, k, variant))


def _keep_spec(keep, N, H, kk):
    torch = _torch()
    return [] if keep is None else [(keep, "keep", torch.uint8, (N, H, kk))]


class Workspace:
    """A reusable device workspace (uint8 tensor) grown on demand."""

    def __init__(self, device=None):
        self.buf = None
        self.device = device

    def get(self, nbytes: int):
        torch = _torch()
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(max(nbytes, 256), dtype=torch.uint8,
                                   device=self.device or "cuda")
        return self.buf


def _nhd(q, name="Q"):
    torch = _torch()
    if not isinstance(q, torch.Tensor) or q.dim() != 3:
        raise ValueError(f"{name} must be a tensor [N, H, d]")
    return tuple(int(x) for x in q.shape)


def _dv(v, N, H, name="V"):
    """Value width of v, which must be [N, H, dv]."""
    torch = _torch()
    if not isinstance(v, torch.Tensor) or v.dim() != 3 or tuple(v.shape[:2]) != (N, H):
        raise ValueError(f"{name} must be a tensor [N, H, d_V] with N={N}, H={H}")
    return int(v.shape[2])


def _kk(idx, name="topk_idx"):
    torch = _torch()
    if not isinstance(idx, torch.Tensor) or idx.dim() != 3:
        raise ValueError(f"{name} must be a tensor [N, H, k]")
    return int(idx.shape[-1])


def _workspace(ws, nbytes, device):
    """Device buffer of at least nbytes from ws (a Workspace, or None for a
    fresh one), or None when nbytes is 0."""
    if nbytes == 0:
        return None
    buf = (ws or Workspace(device)).get(nbytes)
    _validate((buf, "workspace", _torch().uint8, None))
    if buf.device != device:
        raise ValueError(f"workspace is on {buf.device}, expected {device}")
    return buf


def topk(q, k_, kk: int, graph_offsets: Optional[Sequence[int]] = None, idx=None,
         workspace: Optional[Workspace] = None, select_events=None):
    """Score + select: returns topk_idx int32 [N, H, kk].

    select_events: optional pair of torch.cuda.Event, recorded on the current
    stream right before and after the score+select kernel (not the pre-passes).
    """
    torch = _torch()
    N, H, d = _nhd(q)
    kk = int(kk)
    specs = [(q, "Q", torch.bfloat16, None), (k_, "K", torch.bfloat16, (N, H, d))]
    if idx is not None:
        specs.append((idx, "topk_idx", torch.int32, (N, H, kk)))
    _validate(*specs)
    o, optr, G = _offsets(graph_offsets)
    if o is not None and (o.ndim != 1 or len(o) < 2):
        raise ValueError("graph_offsets must be a 1-D sequence of at least two entries")
    if idx is None:
        idx = torch.empty((N, H, kk), dtype=torch.int32, device=q.device)
    buf = _workspace(workspace, topk_workspace_size(N, H, d, kk, G), q.device)
    args = (_ptr(q), _ptr(k_), optr, G, N, H, d, kk, _ptr(idx), _ptr(buf),
            0 if buf is None else buf.numel(), _stream_ptr())
    if select_events is None:
        check(load().kmip_topk(*args))
    else:
        handles = []
        for ev in select_events:
            if not ev.cuda_event:
                ev.record()   # the event object exists only once recorded
            handles.append(ctypes.c_void_p(ev.cuda_event))
        check(load().kmip_topk_with_events(*args, *handles))
    return idx


def topk_prefilter_workspace_size(N: int, H: int, d: int, k: int) -> int:
    return int(load().kmip_topk_prefilter_workspace_size(N, H, d, k))


def topk_prefilter(q, k_, kk: int, idx=None, workspace: Optional[Workspace] = None, redone=None):
    """Score + select of one graph through the int8 prefilter with a provable
    bound and an exact re-rank (k <= 32): the same topk_idx as topk().
    redone: optional int32 tensor of one element on the device, set to the
    number of query blocks the select kernel redid."""
    torch = _torch()
    N, H, d = _nhd(q)
    kk = int(kk)
    specs = [(q, "Q", torch.bfloat16, None), (k_, "K", torch.bfloat16, (N, H, d))]
    if idx is not None:
        specs.append((idx, "topk_idx", torch.int32, (N, H, kk)))
    if redone is not None:
        specs.append((redone, "redone", torch.int32, (1,)))
    _validate(*specs)
    if idx is None:
        idx = torch.empty((N, H, kk), dtype=torch.int32, device=q.device)
    buf = _workspace(workspace, topk_prefilter_workspace_size(N, H, d, kk), q.device)
    check(load().kmip_topk_prefilter(_ptr(q), _ptr(k_), N, H, d, kk, _ptr(idx), _ptr(redone), _ptr(buf),
                                     0 if buf is None else buf.numel(), _stream_ptr()))
    return idx


def attend(q, k_, v, idx, scale: float, out=None, lse=None, keep=None, drop_rate: float = 0.0):
    """Gather-softmax-aggregate on a given index set: returns (out, lse)."""
    torch = _torch()
    N, H, d = _nhd(q)
    dv = _dv(v, N, H)
    kk = _kk(idx)
    specs = [(q, "Q", torch.bfloat16, None), (k_, "K", torch.bfloat16, (N, H, d)),
             (v, "V", torch.bfloat16, (N, H, dv)), (idx, "topk_idx", torch.int32, (N, H, kk))]
    specs += _keep_spec(keep, N, H, kk)
    if out is not None:
        specs.append((out, "out", torch.float32, (N, H, dv)))
    if lse is not None:
        specs.append((lse, "lse", torch.float32, (N, H)))
    _validate(*specs)
    if out is None:
        out = torch.empty((N, H, dv), dtype=torch.float32, device=q.device)
    if lse is None:
        lse = torch.empty((N, H), dtype=torch.float32, device=q.device)
    check(load().kmip_attend_ex(_ptr(q), _ptr(k_), _ptr(v), N, H, d, dv, kk, float(scale), _ptr(idx),
                                _ptr(keep), float(drop_rate), _ptr(out), _ptr(lse), _stream_ptr()))
    return out, lse


def _event_handles(events):
    handles = []
    for ev in events:
        if ev is None:
            handles.append(ctypes.c_void_p(0))
            continue
        if not ev.cuda_event:
            ev.record()   # the event object exists only once recorded
        handles.append(ctypes.c_void_p(ev.cuda_event))
    return handles


def fwd(q, k_, v, kk: int, scale: float, graph_offsets=None, workspace=None, keep=None,
        drop_rate: float = 0.0, out=None, idx=None, lse=None, events=None):
    """Full forward: returns (out, topk_idx, lse).

    out, idx, lse: optional outputs to write into.  events: optional triple
    of torch.cuda.Event (or None entries) recorded around the score+select
    kernel and right before the aggregate."""
    torch = _torch()
    N, H, d = _nhd(q)
    dv = _dv(v, N, H)
    kk = int(kk)
    specs = [(q, "Q", torch.bfloat16, None), (k_, "K", torch.bfloat16, (N, H, d)),
             (v, "V", torch.bfloat16, (N, H, dv)), *_keep_spec(keep, N, H, kk)]
    for t, name, dt, shp in ((out, "out", torch.float32, (N, H, dv)), (idx, "topk_idx", torch.int32, (N, H, kk)),
                             (lse, "lse", torch.float32, (N, H))):
        if t is not None:
            specs.append((t, name, dt, shp))
    _validate(*specs)
    o, optr, G = _offsets(graph_offsets)
    if o is not None and (o.ndim != 1 or len(o) < 2):
        raise ValueError("graph_offsets must be a 1-D sequence of at least two entries")
    if out is None:
        out = torch.empty((N, H, dv), dtype=torch.float32, device=q.device)
    if idx is None:
        idx = torch.empty((N, H, kk), dtype=torch.int32, device=q.device)
    if lse is None:
        lse = torch.empty((N, H), dtype=torch.float32, device=q.device)
    buf = _workspace(workspace, topk_workspace_size(N, H, d, kk, G), q.device)
    args = (_ptr(q), _ptr(k_), _ptr(v), optr, G, N, H, d, dv, kk, float(scale), _ptr(keep), float(drop_rate),
            _ptr(out), _ptr(idx), _ptr(lse), _ptr(buf), 0 if buf is None else buf.numel(), _stream_ptr())
    if events is None:
        check(load().kmip_fwd_ex(*args))
    else:
        if len(events) != 3:
            raise ValueError("events must be (select_start, select_stop, attend_start)")
        check(load().kmip_fwd_ex_with_events(*args, *_event_handles(events)))
    return out, idx, lse


def fwd_noalloc(q, k_, v, kk: int, scale: float, out, idx, lse):
    """Forward of one graph into caller-allocated out [N, H, d] float32,
    idx [N, H, kk] int32 and lse [N, H] float32, through kmip_fwd_noalloc:
    the library allocates nothing (its working data lives in a fixed
    per-device array).  Calls that overlap on one GPU race."""
    torch = _torch()
    N, H, d = _nhd(q)
    kk = int(kk)
    _validate((q, "Q", torch.bfloat16, None), (k_, "K", torch.bfloat16, (N, H, d)),
              (v, "V", torch.bfloat16, (N, H, d)), (out, "out", torch.float32, (N, H, d)),
              (idx, "topk_idx", torch.int32, (N, H, kk)), (lse, "lse", torch.float32, (N, H)))
    check(load().kmip_fwd_noalloc(_ptr(q), _ptr(k_), _ptr(v), N, H, d, kk, float(scale), _ptr(out),
                                  _ptr(idx), _ptr(lse), _stream_ptr()))
    return out, idx, lse


def bwd(q, k_, v, dout, idx, lse, scale: float, variant: int = 0, dq=None, dk=None, dv=None,
        workspace=None, keep=None, drop_rate: float = 0.0):
    """Backward with the index set held fixed: returns (dQ, dK, dV) float32."""
    torch = _torch()
    N, H, d = _nhd(q)
    wv = _dv(v, N, H)
    kk = _kk(idx)
    nd, nv = (N, H, d), (N, H, wv)
    specs = [(q, "Q", torch.bfloat16, None), (k_, "K", torch.bfloat16, nd), (v, "V", torch.bfloat16, nv),
             (dout, "dOut", torch.bfloat16, nv), (idx, "topk_idx", torch.int32, (N, H, kk)),
             (lse, "lse", torch.float32, (N, H))] + _keep_spec(keep, N, H, kk)
    for t, name, shp in ((dq, "dQ", nd), (dk, "dK", nd), (dv, "dV", nv)):
        if t is not None:
            specs.append((t, name, torch.float32, shp))
    _validate(*specs)
    dev = q.device
    dq = dq if dq is not None else torch.empty(nd, dtype=torch.float32, device=dev)
    dk = dk if dk is not None else torch.empty(nd, dtype=torch.float32, device=dev)
    dv = dv if dv is not None else torch.empty(nv, dtype=torch.float32, device=dev)
    buf = _workspace(workspace, bwd_workspace_size(N, H, d, kk, variant, dv=wv), dev)
    check(load().kmip_bwd_ex(_ptr(q), _ptr(k_), _ptr(v), _ptr(dout), _ptr(idx), _ptr(lse), _ptr(keep),
                             float(drop_rate), N, H, d, wv, kk, float(scale), _ptr(dq), _ptr(dk), _ptr(dv),
                             int(variant), _ptr(buf), 0 if buf is None else buf.numel(), _stream_ptr()))
    return dq, dk, dv


def attention(q, k_, v, kk: int, scale: float, graph_offsets=None, variant: int = 0, workspace=None,
              keep=None, drop_rate: float = 0.0):
    """Differentiable k-MIP attention for training: returns out (float32 [N, H, d_V]).

    The forward is ``fwd``; autograd's backward calls ``bwd`` with the saved
    (topk_idx, lse), so the index set is held fixed and no gradient flows
    through the selection (Section 3.1 and Appendix E of arXiv 2604.03815).
    The incoming output gradient is rounded to bf16, the type the library's
    backward reads, and dQ, dK, dV are returned in the dtype of Q, K, V.
    keep / drop_rate: attention dropout draws uint8 [N, H, kk] and rate,
    used by the forward and again by the backward.
    """
    torch = _torch()

    class _Attention(torch.autograd.Function):
        @staticmethod
        def forward(ctx, q_, k2, v_):
            out, idx, lse = fwd(q_, k2, v_, kk, scale, graph_offsets=graph_offsets, workspace=workspace,
                                keep=keep, drop_rate=drop_rate)
            ctx.save_for_backward(q_, k2, v_, idx, lse)
            return out

        @staticmethod
        def backward(ctx, dout):
            q_, k2, v_, idx, lse = ctx.saved_tensors
            dq, dk, dv = bwd(q_, k2, v_, dout.to(torch.bfloat16).contiguous(), idx, lse, scale,
                             variant=variant, workspace=workspace, keep=keep, drop_rate=drop_rate)
            return dq.to(q_.dtype), dk.to(k2.dtype), dv.to(v_.dtype)

    return _Attention.apply(q, k_, v)


from .layer import KMIPAttention, linear_k_schedule  # noqa: E402
