"""The dense-attention comparator (bench.py --compare-dense) on the GPU.

Dense softmax attention is what k-MIP attention reduces to when k covers the
whole graph (Section 3.1: T_k keeps every entry when k = N).  The comparator
is torch's scaled_dot_product_attention restricted to its flash and
memory-efficient kernels; these tests pin it to the float64 oracle at k = N
(forward and gradients), and check the library at k = N against both.
"""
import numpy as np
import pytest

import oracle
import workloads
from parity import allclose_report

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import torch.nn.functional as F  # noqa: E402
from torch.nn.attention import SDPBackend, sdpa_kernel  # noqa: E402

import paper_2604_03815_amd as kmip  # noqa: E402

DEV = torch.device("cuda:0")


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)


def _sdpa(w, backward):
    """Dense attention of one graph [N, 1, d] with torch SDPA (flash or
    memory-efficient kernels only); returns out (and dQ, dK, dV)."""
    q, k, v = (_dev(getattr(w, n)).view(w.N, w.d)[None, None] for n in ("q", "kk", "v"))
    with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
        if not backward:
            with torch.no_grad():
                return F.scaled_dot_product_attention(q, k, v, scale=w.scale), None
        qg, kg, vg = (x.clone().requires_grad_() for x in (q, k, v))
        o = F.scaled_dot_product_attention(qg, kg, vg, scale=w.scale)
        o.backward(_dev(w.dout).view(w.N, w.d)[None, None])
    torch.cuda.synchronize()
    return o.detach(), (qg.grad, kg.grad, vg.grad)


def _dense_report(name, got, ref):
    """The comparator's own precision: its kernels round the softmax weights
    and the score gradients to bf16 (unit roundoff 2^-8) before the matrix
    products of the backward, so errors scale with the largest entry of the
    tensor, not with each entry: |x - r| <= 1e-3 + 2e-2 |r| + 1e-2 max|r|."""
    ref = np.asarray(ref, np.float64)
    allclose_report(name, got, ref, atol=1e-3 + 1e-2 * float(np.abs(ref).max()), rtol=2e-2)


@pytest.mark.parametrize("N", [100, 300, 1000])
def test_dense_comparator_matches_oracle_full_attention(N):
    w = workloads.iid(N, 1, 16, N, seed=N)
    print(f"[case] sdpa N={N} d=16", flush=True)
    out, grads = _sdpa(w, backward=True)
    Qd, Kd, Vd, dOd = (oracle.from_bf16(getattr(w, n)) for n in ("q", "kk", "v", "dout"))
    ref_out, ref_idx, _ = oracle.forward(Qd, Kd, Vd, N, w.scale)
    # bf16 outputs: one rounding of 2^-9 relative on top of the tolerance
    _dense_report("dense out", out.float().cpu().numpy().reshape(N, 1, 16), ref_out.reshape(N, 1, 16))
    rq, rk, rv = oracle.backward(Qd, Kd, Vd, dOd, ref_idx, w.scale)
    for name, g, r in (("dQ", grads[0], rq), ("dK", grads[1], rk), ("dV", grads[2], rv)):
        _dense_report("dense " + name, g.float().cpu().numpy().reshape(r.shape), r)


@pytest.mark.parametrize("N", [64, 128])
def test_kmip_with_k_equal_n_is_dense_attention(N):
    w = workloads.iid(N, 1, 16, N, seed=7 + N)
    print(f"[case] kmip k=N={N}", flush=True)
    q, k, v, g = (_dev(getattr(w, n)) for n in ("q", "kk", "v", "dout"))
    out, idx, lse = kmip.fwd(q, k, v, N, w.scale)
    dq, dk, dv = kmip.bwd(q, k, v, g, idx, lse, w.scale)
    dout, dgrads = _sdpa(w, backward=True)
    torch.cuda.synchronize()
    assert (torch.sort(idx, -1).values == torch.arange(N, device=DEV, dtype=torch.int32)).all()
    # the library against the oracle at the usual bar, against the dense
    # kernels at theirs
    Qd, Kd, Vd, dOd = (oracle.from_bf16(getattr(w, n)) for n in ("q", "kk", "v", "dout"))
    ref_out, _ = oracle.attend(Qd, Kd, Vd, idx.cpu().numpy(), w.scale)
    allclose_report("kmip out", out.cpu().numpy().reshape(N, 16), ref_out)
    rq, rk, rv = oracle.backward(Qd, Kd, Vd, dOd, idx.cpu().numpy(), w.scale)
    for name, a, r in (("dQ", dq, rq), ("dK", dk, rk), ("dV", dv, rv)):
        allclose_report("kmip " + name, a.cpu().numpy(), r)
    _dense_report("kmip vs dense out", out.cpu().numpy().reshape(N, 16), dout.float().cpu().numpy().reshape(N, 16))
    for name, a, b in (("dQ", dq, dgrads[0]), ("dK", dk, dgrads[1]), ("dV", dv, dgrads[2])):
        _dense_report("kmip vs dense " + name, a.cpu().numpy().reshape(N, 16),
                      b.float().cpu().numpy().reshape(N, 16))
