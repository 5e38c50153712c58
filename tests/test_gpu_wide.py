"""Larger k (up to 512) and wider heads (d_K = 128) on the GPU against the
float64 oracle.

k > 128 gives the select kernel loser trees of 256 or 512 leaves (8 or 9
levels, up to 132 KB of LDS per wave); d_K = 128 streams key tiles of eight
16-dimension chunks.  Every case compares the index set of every query-head
with the oracle, out and lse on every query-head, and every backward variant
built for the sizes (the bucketed one is not: it must refuse them).
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
from paper_2604_03815_amd import _lib  # noqa: E402

DEV = torch.device("cuda:0")


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)


WIDE = [
    # (N, H, d, dv, k, sizes)
    (3000, 1, 16, 16, 129, None),                              # trees of 256 leaves
    (5000, 2, 32, 32, 256, None),
    (4000, 1, 64, 64, 512, None),                              # 512 leaves, 132 KB of LDS
    (9000, 2, 16, 16, 200, None),                              # grouped, pruned, lower-bound pass
    (10000, 1, 32, 32, 400, None),                             # grouped, pruned
    (2000, 2, 16, 32, 300, [1, 299, 300, 301, 480, 619]),      # batch: n < k graphs, small graphs streamed
    (3000, 1, 128, 128, 16, None),
    (12000, 1, 128, 64, 128, None),                            # N >= 8192 but not grouped at d = 128
    (1500, 2, 128, 16, 100, [100, 400, 1000]),
    (2500, 3, 128, 128, 1, None),
]


@pytest.mark.parametrize("case", WIDE, ids=lambda c: "N%d_H%d_d%d_dv%d_k%d" % c[:5])
def test_wide_sizes_full(case):
    N, H, d, dv, k, sizes = case
    w = workloads.iid(N, H, d, k, seed=N + k + d, sizes=sizes, dv=dv)
    q, kk, v, g = (_dev(getattr(w, n)) for n in ("q", "kk", "v", "dout"))
    print(f"[case] wide N={N} H={H} d={d} dv={dv} k={k} sizes={sizes}", flush=True)
    out, idx, lse = kmip.fwd(q, kk, v, k, w.scale, graph_offsets=w.offsets)
    torch.cuda.synchronize()
    Qd, Kd, Vd, dOd = (oracle.from_bf16(getattr(w, n)) for n in ("q", "kk", "v", "dout"))
    gi = idx.cpu().numpy()
    check_structure(gi, w.offsets, N, H, k)
    exact, strict, loose = check_sets_all(w, Qd, Kd, gi)
    print(f"[sets] {exact} exact by scores, {strict} well-separated, {loose} near-tied", flush=True)
    ref_out, ref_lse = oracle.attend(Qd, Kd, Vd, gi, w.scale)
    allclose_report("out", out.cpu().numpy().reshape(-1, dv), ref_out)
    allclose_report("lse", lse.cpu().numpy().reshape(-1), ref_lse)
    rq, rk, rv = oracle.backward(Qd, Kd, Vd, dOd, gi, w.scale)
    for variant in (0, _lib.BWD_ATOMIC, _lib.BWD_SEGMENTED, _lib.BWD_KEY_AGGREGATED):
        print(f"[case] wide backward variant {variant}", flush=True)
        dq, dk, dvg = kmip.bwd(q, kk, v, g, idx, lse, w.scale, variant=variant)
        torch.cuda.synchronize()
        allclose_report(f"dQ v{variant}", dq.cpu().numpy(), rq)
        allclose_report(f"dK v{variant}", dk.cpu().numpy(), rk)
        allclose_report(f"dV v{variant}", dvg.cpu().numpy(), rv)
    with pytest.raises(kmip.KmipError):
        kmip.bwd(q, kk, v, g, idx, lse, w.scale, variant=_lib.BWD_BUCKETED)


@pytest.mark.parametrize("N,d,k,sizes", [
    (6000, 16, 300, [5000, 600, 400]),   # k > 128: the tie rule in trees of 512 leaves
    (3000, 128, 128, None),
])
def test_wide_integer_ties_exact(N, d, k, sizes):
    # Scores in a small integer range tie everywhere: every row, order
    # included, must be the oracle's (score descending, index ascending).
    rng = np.random.default_rng(N + d + k)
    H = 2
    q = rng.integers(-2, 3, size=(N, H, d)).astype(np.float32)
    kk = rng.integers(-1, 2, size=(N, H, d)).astype(np.float32)
    v = rng.standard_normal((N, H, d)).astype(np.float32)
    offsets = None if sizes is None else np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    w = workloads.Workload("wide_ties", N, H, d, k, 0.25, offsets, workloads.bf16_round(q),
                           workloads.bf16_round(kk), workloads.bf16_round(v), None, False)
    print(f"[case] wide ties N={N} d={d} k={k} sizes={sizes}", flush=True)
    idx = kmip.topk(_dev(w.q), _dev(w.kk), k, graph_offsets=offsets)
    torch.cuda.synchronize()
    gi = idx.cpu().numpy().reshape(N * H, k)
    o_idx, _, _ = oracle.topk(oracle.from_bf16(w.q), oracle.from_bf16(w.kk), k, offsets=offsets)
    np.testing.assert_array_equal(gi, o_idx)


def test_wide_refusals():
    q = torch.zeros((64, 1, 128), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(kmip.KmipError):
        kmip.topk(q, q, 129)                      # d = 128 takes k <= 128
    q16 = torch.zeros((1024, 1, 16), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(kmip.KmipError):
        kmip.topk(q16, q16, 513)
    idx = kmip.topk(q16, q16, 512)                # every score 0: keys 0 .. 511 in order
    torch.cuda.synchronize()
    assert (idx.cpu().numpy() == np.arange(512, dtype=np.int32)).all()
