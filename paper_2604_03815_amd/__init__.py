"""k-MIP self-attention for MI355X (gfx950): Python front end of libkmip.so.

Every function marshals torch tensors into the C ABI of include/kmip.h and
launches on the current HIP stream; all arithmetic runs in the library's HIP
kernels.  Tensors: Q, K, V, dOut are bf16 [N, H, d] on the GPU; out, dQ, dK,
dV are float32 [N, H, d]; topk_idx is int32 [N, H, k]; lse is float32 [N, H].
``graph_offsets`` is a host-side int32 sequence [G+1] (or None for one graph).
"""
from __future__ import annotations

import ctypes
from typing import Optional, Sequence

import numpy as np

from ._lib import KmipError, MAX_K, check, load

__all__ = [
    "KmipError", "MAX_K", "topk", "attend", "fwd", "bwd", "attention", "topk_workspace_size",
    "bwd_workspace_size", "Workspace", "load",
]


def _torch():
    import torch
    return torch


def _stream_ptr():
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t, dtype, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _offsets(graph_offsets):
    if graph_offsets is None:
        return None, None, 1
    o = np.ascontiguousarray(np.asarray(graph_offsets), dtype=np.int32)
    return o, o.ctypes.data_as(ctypes.c_void_p), len(o) - 1


def topk_workspace_size(N: int, H: int, d: int, k: int, num_graphs: int = 1) -> int:
    return int(load().kmip_topk_workspace_size(N, H, d, k, num_graphs))


def bwd_workspace_size(N: int, H: int, d: int, k: int, variant: int = 0) -> int:
    return int(load().kmip_bwd_workspace_size(N, H, d, k, variant))


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


def _shape(q):
    if q.dim() != 3:
        raise ValueError("Q must be [N, H, d]")
    return q.shape


def topk(q, k_, kk: int, graph_offsets: Optional[Sequence[int]] = None, idx=None,
         workspace: Optional[Workspace] = None, select_events=None):
    """Score + select: returns topk_idx int32 [N, H, kk].

    select_events: optional pair of torch.cuda.Event, recorded on the current
    stream right before and after the score+select kernel (not the pre-passes).
    """
    torch = _torch()
    N, H, d = _shape(q)
    if idx is None:
        idx = torch.empty((N, H, kk), dtype=torch.int32, device=q.device)
    o, optr, G = _offsets(graph_offsets)
    ws = workspace or Workspace(q.device)
    nbytes = topk_workspace_size(N, H, d, kk, G)
    buf = ws.get(nbytes)
    args = (_dev(q, torch.bfloat16, "Q"), _dev(k_, torch.bfloat16, "K"), optr, G, N, H, d, kk,
            _dev(idx, torch.int32, "topk_idx"), ctypes.c_void_p(buf.data_ptr()), buf.numel(),
            _stream_ptr())
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


def attend(q, k_, v, idx, scale: float, out=None, lse=None):
    """Gather-softmax-aggregate on a given index set: returns (out, lse)."""
    torch = _torch()
    N, H, d = _shape(q)
    kk = idx.shape[-1]
    if out is None:
        out = torch.empty((N, H, d), dtype=torch.float32, device=q.device)
    if lse is None:
        lse = torch.empty((N, H), dtype=torch.float32, device=q.device)
    check(load().kmip_attend(_dev(q, torch.bfloat16, "Q"), _dev(k_, torch.bfloat16, "K"),
                             _dev(v, torch.bfloat16, "V"), N, H, d, kk, float(scale),
                             _dev(idx, torch.int32, "topk_idx"), _dev(out, torch.float32, "out"),
                             _dev(lse, torch.float32, "lse"), _stream_ptr()))
    return out, lse


def fwd(q, k_, v, kk: int, scale: float, graph_offsets=None, workspace=None):
    """Full forward: returns (out, topk_idx, lse)."""
    torch = _torch()
    N, H, d = _shape(q)
    out = torch.empty((N, H, d), dtype=torch.float32, device=q.device)
    idx = torch.empty((N, H, kk), dtype=torch.int32, device=q.device)
    lse = torch.empty((N, H), dtype=torch.float32, device=q.device)
    o, optr, G = _offsets(graph_offsets)
    ws = workspace or Workspace(q.device)
    buf = ws.get(topk_workspace_size(N, H, d, kk, G))
    check(load().kmip_fwd(_dev(q, torch.bfloat16, "Q"), _dev(k_, torch.bfloat16, "K"),
                          _dev(v, torch.bfloat16, "V"), optr, G, N, H, d, kk, float(scale),
                          _dev(out, torch.float32, "out"), _dev(idx, torch.int32, "topk_idx"),
                          _dev(lse, torch.float32, "lse"), ctypes.c_void_p(buf.data_ptr()),
                          buf.numel(), _stream_ptr()))
    return out, idx, lse


def bwd(q, k_, v, dout, idx, lse, scale: float, variant: int = 0, dq=None, dk=None, dv=None,
        workspace=None):
    """Backward with the index set held fixed: returns (dQ, dK, dV) float32."""
    torch = _torch()
    N, H, d = _shape(q)
    kk = idx.shape[-1]
    dq = dq if dq is not None else torch.empty((N, H, d), dtype=torch.float32, device=q.device)
    dk = dk if dk is not None else torch.empty((N, H, d), dtype=torch.float32, device=q.device)
    dv = dv if dv is not None else torch.empty((N, H, d), dtype=torch.float32, device=q.device)
    nbytes = bwd_workspace_size(N, H, d, kk, variant)
    buf = (workspace or Workspace(q.device)).get(nbytes) if nbytes else None
    check(load().kmip_bwd(_dev(q, torch.bfloat16, "Q"), _dev(k_, torch.bfloat16, "K"),
                          _dev(v, torch.bfloat16, "V"), _dev(dout, torch.bfloat16, "dOut"),
                          _dev(idx, torch.int32, "topk_idx"), _dev(lse, torch.float32, "lse"),
                          N, H, d, kk, float(scale), _dev(dq, torch.float32, "dQ"),
                          _dev(dk, torch.float32, "dK"), _dev(dv, torch.float32, "dV"),
                          int(variant), ctypes.c_void_p(buf.data_ptr() if buf is not None else 0),
                          0 if buf is None else buf.numel(), _stream_ptr()))
    return dq, dk, dv


def attention(q, k_, v, kk: int, scale: float, graph_offsets=None, variant: int = 0, workspace=None):
    """Differentiable k-MIP attention for training: returns out (float32 [N, H, d]).

    The forward is ``fwd``; autograd's backward calls ``bwd`` with the saved
    (topk_idx, lse), so the index set is held fixed and no gradient flows
    through the selection (Section 3.1 and Appendix E of arXiv 2604.03815).
    The incoming output gradient is rounded to bf16, the type the library's
    backward reads, and dQ, dK, dV are returned in the dtype of Q, K, V.
    """
    torch = _torch()

    class _Attention(torch.autograd.Function):
        @staticmethod
        def forward(ctx, q_, k2, v_):
            out, idx, lse = fwd(q_, k2, v_, kk, scale, graph_offsets=graph_offsets, workspace=workspace)
            ctx.save_for_backward(q_, k2, v_, idx, lse)
            return out

        @staticmethod
        def backward(ctx, dout):
            q_, k2, v_, idx, lse = ctx.saved_tensors
            dq, dk, dv = bwd(q_, k2, v_, dout.to(torch.bfloat16).contiguous(), idx, lse, scale,
                             variant=variant, workspace=workspace)
            return dq.to(q_.dtype), dk.to(k2.dtype), dv.to(v_.dtype)

    return _Attention.apply(q, k_, v)
