"""Multi-head k-MIP self-attention layer around the library's kernels.

Eq. 2 of arXiv 2604.03815 and Algorithm 1 (Appendix E): for input features
X [N, d_model] and heads h = 1..H,

    Q^h = X W_Q^h,  K^h = X W_K^h  (d_K wide),   V^h = X W_V^h  (d_V wide),
    O^h = softmax(T_k(Q^h K^h^T) / sqrt(d_K)) V^h,
    k-MIP(X) = sum_h O^h W_O^h.

The projections and the head sum are dense GEMMs that stay with the caller
(torch): the per-head weights are stored side by side, so one GEMM gives the
[N, H, d_K] layout the library takes, and O [N, H, d_V] flattened times
W_O [H d_V, d_model] is the sum over heads.  Selection, softmax, aggregation
and their backward run in the library (``attention``).

Two training-side options:
  * ``k_schedule``: a callable step -> k (e.g. ``linear_k_schedule``) for
    annealing k, starting large so that every query sees many keys early in
    training and narrowing to the final k (the mitigation of supervision
    starvation proposed in the Conclusion, "Limitations");
  * ``attn_dropout``: dropout on the attention weights (the experimental
    details list an attention-dropout rate), with the keep mask drawn here by
    torch and passed to the kernels.
"""
from __future__ import annotations

import math
from typing import Callable, Optional

import torch

from . import attention


def linear_k_schedule(k_start: int, k_end: int, steps: int) -> Callable[[int], int]:
    """k annealed linearly from k_start to k_end over `steps` calls, then held."""
    if k_start < 1 or k_end < 1 or steps < 1:
        raise ValueError("k_start, k_end and steps must be >= 1")

    def k_at(step: int) -> int:
        t = min(max(step, 0), steps) / steps
        return int(round(k_start + (k_end - k_start) * t))

    return k_at


class KMIPAttention(torch.nn.Module):
    """One layer of multi-head k-MIP self-attention (Eq. 1-2, Algorithm 1).

    d_model: input and output width; heads: H; d_k, d_v: per-head widths of
    queries/keys and of values (each in {16, 32, 64, 128}); k: keys kept per
    query (or k_schedule).  forward(x [N, d_model], graph_offsets=None)
    returns [N, d_model] float32; graph_offsets (host int sequence [G+1])
    makes the attention block-diagonal over a batch of graphs.
    """

    def __init__(self, d_model: int, heads: int, d_k: int, d_v: Optional[int] = None, k: int = 16,
                 k_schedule: Optional[Callable[[int], int]] = None, attn_dropout: float = 0.0,
                 variant: int = 0, device=None, generator: Optional[torch.Generator] = None):
        super().__init__()
        d_v = d_k if d_v is None else d_v
        if not 0.0 <= attn_dropout < 1.0:
            raise ValueError("attn_dropout must lie in [0, 1)")
        self.d_model, self.heads, self.d_k, self.d_v = d_model, heads, d_k, d_v
        self.k, self.k_schedule, self.attn_dropout, self.variant = k, k_schedule, attn_dropout, variant
        self.scale = 1.0 / math.sqrt(d_k)
        self.step = 0
        std = 1.0 / math.sqrt(d_model)

        def param(rows, cols, s):
            w = torch.empty(rows, cols, device=device)
            w.normal_(0.0, s, generator=generator)
            return torch.nn.Parameter(w)

        self.w_q = param(d_model, heads * d_k, std)
        self.w_k = param(d_model, heads * d_k, std)
        self.w_v = param(d_model, heads * d_v, std)
        self.w_o = param(heads * d_v, d_model, 1.0 / math.sqrt(heads * d_v))

    def current_k(self) -> int:
        return int(self.k_schedule(self.step)) if self.k_schedule is not None else int(self.k)

    def project(self, x):
        """Q, K, V [N, H, width] in bf16, the library's input type."""
        N = x.shape[0]
        q = (x @ self.w_q).to(torch.bfloat16).view(N, self.heads, self.d_k)
        k = (x @ self.w_k).to(torch.bfloat16).view(N, self.heads, self.d_k)
        v = (x @ self.w_v).to(torch.bfloat16).view(N, self.heads, self.d_v)
        return q, k, v

    def forward(self, x, graph_offsets=None, keep=None):
        """keep: optional uint8 [N, H, k] dropout keep mask (1 keeps a kept
        key's weight, scaled by 1/(1 - attn_dropout)); drawn here when
        training with attn_dropout > 0 and none is given."""
        if x.dim() != 2 or x.shape[1] != self.d_model:
            raise ValueError(f"x must be [N, {self.d_model}]")
        kk = self.current_k()
        if self.training:
            self.step += 1
        q, k, v = self.project(x.float())
        rate = self.attn_dropout if self.training else 0.0
        if rate > 0.0 and keep is None:
            keep = (torch.rand(q.shape[0], self.heads, kk, device=q.device) >= rate).to(torch.uint8)
        o = attention(q, k, v, kk, self.scale, graph_offsets=graph_offsets, variant=self.variant,
                      keep=keep if rate > 0.0 else None, drop_rate=rate)
        return o.reshape(x.shape[0], self.heads * self.d_v) @ self.w_o
