"""Training-side features on the GPU against the float64 oracle.

  * attention dropout: the caller's keep draws go to the forward and the
    backward; every backward variant (the bucketed one only with
    d_V = d_K) against the oracle with the same draws;
  * the multi-head layer of Eq. 2 (projections, k-MIP attention per head,
    head sum through W_O), forward and gradients, against the oracle on the
    layer's own bf16 projections;
  * k annealing: the layer's k follows its schedule.
"""
import numpy as np
import pytest

import oracle
import workloads
from parity import allclose_report, check_sets_all, check_structure

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2604_03815_amd as kmip  # noqa: E402

DEV = torch.device("cuda:0")


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)


def _f64(w):
    return tuple(oracle.from_bf16(getattr(w, n)) for n in ("q", "kk", "v", "dout"))


DROPOUT = [
    # (N, H, d, dv, k, rate, sizes)
    (2000, 2, 16, 16, 16, 0.5, [700, 1300]),
    (3000, 1, 32, 32, 32, 0.1, None),
    (1500, 3, 64, 32, 8, 0.3, [1, 0, 1499]),
    (20000, 2, 16, 16, 32, 0.5, None),     # grouped select, bucketed backward
]


@pytest.mark.parametrize("case", DROPOUT, ids=lambda c: "N%d_H%d_d%d_dv%d_k%d_r%.1f" % c[:6])
def test_dropout_matches_oracle(case):
    N, H, d, dv, k, rate, sizes = case
    w = workloads.iid(N, H, d, k, seed=N + k, sizes=sizes, dv=dv)
    rng = np.random.default_rng(N)
    keep_np = (rng.random((N, H, k)) >= rate).astype(np.uint8)
    keep = torch.from_numpy(keep_np).to(DEV)
    q, kk, v, g = (_dev(getattr(w, n)) for n in ("q", "kk", "v", "dout"))
    print(f"[case] dropout N={N} H={H} d={d} dv={dv} k={k} rate={rate}", flush=True)
    out, idx, lse = kmip.fwd(q, kk, v, k, w.scale, graph_offsets=w.offsets, keep=keep, drop_rate=rate)
    out0, idx0, lse0 = kmip.fwd(q, kk, v, k, w.scale, graph_offsets=w.offsets)
    torch.cuda.synchronize()
    # the draws touch neither the selection nor the softmax statistics
    assert torch.equal(idx, idx0) and torch.equal(lse, lse0)
    Qd, Kd, Vd, dOd = _f64(w)
    gi = idx.cpu().numpy()
    check_structure(gi, w.offsets, N, H, k)
    check_sets_all(w, Qd, Kd, gi)
    ref_out, ref_lse = oracle.attend(Qd, Kd, Vd, gi, w.scale, keep=keep_np, drop_rate=rate)
    allclose_report("out", out.cpu().numpy().reshape(-1, dv), ref_out)
    allclose_report("lse", lse.cpu().numpy().reshape(-1), ref_lse)
    rq, rk, rv = oracle.backward(Qd, Kd, Vd, dOd, gi, w.scale, keep=keep_np, drop_rate=rate)
    for variant in ((0, 1, 2, 3, 4) if dv == d else (0, 1, 2, 4)):
        dq, dk, dvg = kmip.bwd(q, kk, v, g, idx, lse, w.scale, variant=variant, keep=keep, drop_rate=rate)
        torch.cuda.synchronize()
        allclose_report(f"dQ v{variant}", dq.cpu().numpy(), rq)
        allclose_report(f"dK v{variant}", dk.cpu().numpy(), rk)
        allclose_report(f"dV v{variant}", dvg.cpu().numpy(), rv)


def _norm_report(name, got, ref):
    """Outside the library the layer's GEMMs run in the caller's precision
    (bf16 projections, fp32 head sum; gradients rounded to bf16 where they
    pass through bf16 tensors), so the layer's figures are held to a bound
    relative to the largest entry of each tensor:
    |x - r| <= 1e-3 + 2e-2 |r| + 2e-2 max|r|."""
    ref = np.asarray(ref, np.float64)
    allclose_report(name, got, ref, atol=1e-3 + 2e-2 * float(np.abs(ref).max()), rtol=2e-2)


@pytest.mark.parametrize("d_model,H,dk,dv,k,sizes", [
    (48, 3, 16, 32, 16, [120, 1, 179]),
    (64, 2, 32, 32, 24, None),
])
def test_layer_matches_oracle(d_model, H, dk, dv, k, sizes):
    N = 300 if sizes else 2500
    gen = torch.Generator(device=DEV)
    gen.manual_seed(5)
    layer = kmip.KMIPAttention(d_model, H, dk, dv, k=k, device=DEV, generator=gen)
    offsets = None if sizes is None else np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    rng = np.random.default_rng(d_model)
    x = torch.from_numpy(rng.standard_normal((N, d_model)).astype(np.float32)).to(DEV).requires_grad_()
    gy = torch.from_numpy(rng.standard_normal((N, d_model)).astype(np.float32)).to(DEV)
    print(f"[case] layer N={N} d_model={d_model} H={H} dk={dk} dv={dv} k={k}", flush=True)
    y = layer(x, graph_offsets=offsets)
    (y * gy).sum().backward()
    torch.cuda.synchronize()
    assert y.shape == (N, d_model)
    # the oracle on the layer's own bf16 projections
    with torch.no_grad():
        q, kk, v = layer.project(x.detach())
    Qd, Kd, Vd = (oracle.from_bf16(t.cpu().view(torch.int16).numpy().view(np.uint16)) for t in (q, kk, v))
    o, idx, _ = oracle.forward(Qd, Kd, Vd, k, 1.0 / np.sqrt(dk), offsets=offsets)
    Wq, Wk, Wv, Wo = (p.detach().double().cpu().numpy() for p in (layer.w_q, layer.w_k, layer.w_v, layer.w_o))
    X, GY = x.detach().double().cpu().numpy(), gy.double().cpu().numpy()
    _norm_report("layer out", y.detach().cpu().numpy(), o.reshape(N, H * dv) @ Wo)
    # backward: dO = gY W_O^T, rounded to bf16 as the attention's backward reads it
    dO = oracle.from_bf16(workloads.bf16_round((GY @ Wo.T).astype(np.float32))).reshape(N, H, dv)
    dQ, dK, dV = oracle.backward(Qd, Kd, Vd, dO, idx, 1.0 / np.sqrt(dk))
    dX = (dQ.reshape(N, -1) @ Wq.T + dK.reshape(N, -1) @ Wk.T + dV.reshape(N, -1) @ Wv.T)
    _norm_report("dX", x.grad.cpu().numpy(), dX)
    _norm_report("dW_Q", layer.w_q.grad.cpu().numpy(), X.T @ dQ.reshape(N, -1))
    _norm_report("dW_K", layer.w_k.grad.cpu().numpy(), X.T @ dK.reshape(N, -1))
    _norm_report("dW_V", layer.w_v.grad.cpu().numpy(), X.T @ dV.reshape(N, -1))
    _norm_report("dW_O", layer.w_o.grad.cpu().numpy(), o.reshape(N, H * dv).T @ GY)


def test_layer_k_annealing_and_dropout():
    N, d_model, H, dk = 1000, 32, 2, 16
    sched = kmip.linear_k_schedule(64, 8, 4)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(1)
    layer = kmip.KMIPAttention(d_model, H, dk, k_schedule=sched, attn_dropout=0.5, device=DEV, generator=gen)
    x = torch.randn(N, d_model, device=DEV, generator=gen)
    seen = []
    layer.train()
    for _ in range(6):
        kk = layer.current_k()
        seen.append(kk)
        y = layer(x)
        y.sum().backward()
        # in evaluation (no dropout, the schedule's next k): equal to the
        # library's forward at that k
        layer.eval()
        ke = layer.current_k()
        with torch.no_grad():
            q, k_, v = layer.project(x)
            o, _, _ = kmip.fwd(q, k_, v, ke, layer.scale)
            ye = layer(x)
        layer.train()
        torch.cuda.synchronize()
        assert torch.allclose(ye, o.reshape(N, -1) @ layer.w_o, rtol=1e-5, atol=1e-6)
        # dropout in training changes the output, not its shape
        assert y.shape == ye.shape and not torch.equal(y, ye)
    assert seen == [64, 50, 36, 22, 8, 8]
