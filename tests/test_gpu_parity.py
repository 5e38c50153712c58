"""GPU parity: the HIP path (through the C ABI) against the float64 oracle.

Small and medium cases, config 2 and config 3 (N = 100k) have the index set
of every query-head compared; configs 4 and 5 (N = 500k, 262k) the sets of
65,536 and 16,384 query-heads spread over heads and directions.  Structure,
out/lse and the gradients (the oracle evaluated on the GPU's own index sets)
are compared on every query-head of every case.
"""
import numpy as np
import pytest

import oracle
import workloads
from parity import (allclose_report, check_sets_all, check_structure, sample_rows, stratified_rows)

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2604_03815_amd as kmip  # noqa: E402

DEV = torch.device("cuda:0")


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)


def _f64(w):
    return tuple(oracle.from_bf16(getattr(w, n)) if getattr(w, n) is not None else None
                 for n in ("q", "kk", "v", "dout"))


def _run(w, backward=True, variant=0):
    q, k, v = _dev(w.q), _dev(w.kk), _dev(w.v)
    print(f"[case] {w.name} N={w.N} H={w.H} d={w.d} k={w.k} graphs={w.num_graphs} bwd variant {variant}",
          flush=True)
    out, idx, lse = kmip.fwd(q, k, v, w.k, w.scale, graph_offsets=w.offsets)
    grads = None
    if backward and w.dout is not None:
        grads = kmip.bwd(q, k, v, _dev(w.dout), idx, lse, w.scale, variant=variant)
    torch.cuda.synchronize()
    res = {"out": out.cpu().numpy(), "idx": idx.cpu().numpy(), "lse": lse.cpu().numpy()}
    if grads is not None:
        res.update(dq=grads[0].cpu().numpy(), dk=grads[1].cpu().numpy(), dv=grads[2].cpu().numpy())
    return res


def _check_all(w, res, sample=None):
    """Index sets of every query-head (sample=None) or of `sample` query-heads
    spread over heads and directions; structure, out, lse and every gradient
    on every query-head against the oracle on the GPU's own sets."""
    Qd, Kd, Vd, dOd = _f64(w)
    check_structure(res["idx"], w.offsets, w.N, w.H, w.k)
    sel = None if sample is None else stratified_rows(Qd, sample, seed=123)
    exact, strict, loose = check_sets_all(w, Qd, Kd, res["idx"], sel=sel)
    print(f"[sets] {w.name}: {exact} exact by scores, {strict} well-separated, {loose} near-tied "
          f"query-heads of {w.N * w.H if sel is None else len(sel)} checked", flush=True)
    ref_out, ref_lse = oracle.attend(Qd, Kd, Vd, res["idx"], w.scale)
    allclose_report("out", res["out"].reshape(-1, Vd.shape[2]), ref_out)
    allclose_report("lse", res["lse"].reshape(-1), ref_lse)
    if "dq" in res:
        rq, rk, rv = oracle.backward(Qd, Kd, Vd, dOd, res["idx"], w.scale)
        allclose_report("dQ", res["dq"], rq)
        allclose_report("dK", res["dk"], rk)
        allclose_report("dV", res["dv"], rv)
    return exact + strict, loose


SMALL = [
    # (N, H, d, k, sizes)
    (1, 1, 16, 1, None),
    (33, 1, 16, 4, None),
    (1000, 2, 16, 32, None),
    (777, 3, 32, 16, [1, 31, 33, 0, 100, 612]),
    (2049, 1, 64, 128, None),
    (300, 2, 32, 128, [50, 250]),
    (5000, 1, 16, 100, None),
    (4097, 2, 64, 1, None),
    (3000, 1, 32, 64, [3000]),
    (130, 4, 16, 8, [0, 65, 0, 65, 0]),
]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: "N%d_H%d_d%d_k%d" % c[:4])
def test_small_cases_full(case):
    N, H, d, k, sizes = case
    w = workloads.iid(N, H, d, k, seed=N + 7 * k + d, sizes=sizes)
    _check_all(w, _run(w))


@pytest.mark.parametrize("n,d,k", [(8193, 16, 32), (12345, 32, 16), (9001, 64, 128)])
def test_key_tree_odd_sizes_full(n, d, k):
    # Single graphs just above the size from which the keys are stored in
    # tree order: nodes of odd sizes, a partial last superblock, and both the
    # per-level splits and the levels finished in LDS.  Full comparison.
    w = workloads.iid(n, 2, d, k, seed=n + d)
    _check_all(w, _run(w))


def test_identical_keys_tree():
    # Every key row equal: every projection ties, so each split of the key
    # tree is decided by the tie count alone, and every score of a query
    # ties, so every query keeps keys 0 .. k-1 in that order.
    N, H, d, k = 20000, 2, 32, 16
    rng = np.random.default_rng(3)
    row = rng.standard_normal((1, H, d)).astype(np.float32)
    w = workloads.Workload("same_keys", N, H, d, k, 0.25, None,
                           workloads.bf16_round(rng.standard_normal((N, H, d)).astype(np.float32)),
                           workloads.bf16_round(np.repeat(row, N, axis=0)),
                           workloads.bf16_round(rng.standard_normal((N, H, d)).astype(np.float32)),
                           None, False)
    res = _run(w, backward=False)
    assert (res["idx"] == np.arange(k, dtype=np.int32)).all()


def test_config1_full():
    w = workloads.make(1)
    strict, loose = _check_all(w, _run(w, backward=False))
    print(f"c1: {strict} with the oracle's set, {loose} near-tied query-heads")


@pytest.mark.parametrize("variant", [1, 2, 3, 4])
def test_config2_full_fwd_bwd(variant):
    w = workloads.make(2)
    strict, loose = _check_all(w, _run(w, variant=variant))
    print(f"c2: {strict} with the oracle's set, {loose} near-tied query-heads")


@pytest.mark.parametrize("d,k", [(16, 32), (32, 16), (64, 128)])
def test_backward_hub_keys(d, k):
    # Queries that all point the same way select the same few keys: the
    # key-aggregated scatter then sums nearly all pairs in LDS.  Both
    # backward variants must match the oracle on the GPU's own index sets.
    rng = np.random.default_rng(d + k)
    N, H = 20_000, 2
    base = rng.standard_normal((1, H, d)).astype(np.float32)
    q = base + 0.1 * rng.standard_normal((N, H, d)).astype(np.float32)
    kk = rng.standard_normal((N, H, d)).astype(np.float32)
    w = workloads.Workload("hubs", N, H, d, k, 1.0 / np.sqrt(d), None, workloads.bf16_round(q),
                           workloads.bf16_round(kk),
                           workloads.bf16_round(rng.standard_normal((N, H, d)).astype(np.float32)),
                           workloads.bf16_round(rng.standard_normal((N, H, d)).astype(np.float32)),
                           True)
    Qd, Kd, Vd, dOd = _f64(w)
    for variant in (1, 2, 3, 4):
        res = _run(w, variant=variant)
        rq, rk, rv = oracle.backward(Qd, Kd, Vd, dOd, res["idx"], w.scale)
        allclose_report("dQ", res["dq"], rq)
        allclose_report("dK", res["dk"], rk)
        allclose_report("dV", res["dv"], rv)


@pytest.mark.parametrize("d", [16, 32, 64])
def test_exact_ties_integer_inputs(d):
    # Integer inputs make every fp32 score exact, so the GPU must reproduce
    # the tie rule (score desc, index asc) bit for bit, order included.
    rng = np.random.default_rng(d)
    N, H, k = 700, 2, 24
    q = rng.integers(-1, 2, size=(N, H, d)).astype(np.float32)
    kk = rng.integers(-1, 2, size=(N, H, d)).astype(np.float32)
    v = rng.standard_normal((N, H, d)).astype(np.float32)
    w = workloads.Workload("ties", N, H, d, k, 0.5, np.array([0, 13, 13, 400, 700], np.int32),
                           workloads.bf16_round(q), workloads.bf16_round(kk),
                           workloads.bf16_round(v), None, False)
    res = _run(w, backward=False)
    Qd, Kd, Vd, _ = _f64(w)
    _, o_idx, _ = oracle.forward(Qd, Kd, Vd, k, w.scale, offsets=w.offsets)
    np.testing.assert_array_equal(res["idx"], o_idx)


# Block-diagonal batches of graphs of at most 480 nodes go to the small-graph
# select (scores of a whole graph in LDS, threshold by bisection, order by
# rank); larger graphs of the same batch to the streaming kernel.  Integer
# inputs make ties everywhere, so rows must match the oracle's index for
# index (tie rule and order included).
SMALL_GRAPH_BATCHES = [
    # (d, k, sizes)
    (16, 1, [480, 481, 3, 0, 200]),
    (32, 7, [5, 480, 1, 64, 479]),
    (64, 32, [33, 31, 300, 0, 2]),
    (16, 128, [128, 127, 129, 480, 90]),
    (32, 16, [450] * 6 + [100] * 5),
]


@pytest.mark.parametrize("d,k,sizes", SMALL_GRAPH_BATCHES, ids=lambda c: str(c))
def test_small_graph_batches_integer_ties(d, k, sizes):
    rng = np.random.default_rng(sum(sizes) + d + k)
    N, H = sum(sizes), 2
    q = rng.integers(-2, 3, size=(N, H, d)).astype(np.float32)
    kk = rng.integers(-1, 2, size=(N, H, d)).astype(np.float32)
    v = rng.standard_normal((N, H, d)).astype(np.float32)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    w = workloads.Workload("small_ties", N, H, d, k, 0.25, offsets, workloads.bf16_round(q),
                           workloads.bf16_round(kk), workloads.bf16_round(v), None, False)
    res = _run(w, backward=False)
    Qd, Kd, Vd, _ = _f64(w)
    _, o_idx, _ = oracle.forward(Qd, Kd, Vd, k, w.scale, offsets=offsets)
    np.testing.assert_array_equal(res["idx"], o_idx)
    ref_out, _ = oracle.attend(Qd, Kd, Vd, res["idx"], w.scale)
    allclose_report("out", res["out"].reshape(-1, d), ref_out)


def test_small_graph_batch_normal_rows():
    # i.i.d. normal rows in graphs around the size limit: full protocol
    sizes = [480, 479, 481, 250, 17, 0, 480]
    w = workloads.iid(sum(sizes), 3, 32, 24, seed=480, sizes=sizes)
    _check_all(w, _run(w))


def test_all_scores_tied():
    # Q = 0: every score is 0, so each query keeps the k lowest indices of its graph.
    N, H, d, k = 200, 1, 32, 16
    rng = np.random.default_rng(0)
    w = workloads.Workload("zeroq", N, H, d, k, 0.25, np.array([0, 10, 200], np.int32),
                           workloads.bf16_round(np.zeros((N, H, d), np.float32)),
                           workloads.bf16_round(rng.standard_normal((N, H, d)).astype(np.float32)),
                           workloads.bf16_round(rng.standard_normal((N, H, d)).astype(np.float32)),
                           None, False)
    res = _run(w, backward=False)
    idx = res["idx"][:, 0, :]
    np.testing.assert_array_equal(idx[:10, :10], np.tile(np.arange(10), (10, 1)))
    assert (idx[:10, 10:] == -1).all()
    np.testing.assert_array_equal(idx[10:], np.tile(np.arange(10, 26), (190, 1)))
    V = oracle.from_bf16(w.v)[:, 0, :]
    allclose_report("out", res["out"][10:, 0, :], np.tile(V[10:26].mean(axis=0), (190, 1)))


# One graph of 100k nodes and two heads: enough items that the grouped path
# runs with seeded thresholds and scans that start mid-graph and wrap.
GROUPED_N, GROUPED_H = 100_000, 2


@pytest.mark.parametrize("d,k", [(16, 32), (32, 16), (64, 128)])
def test_exact_ties_grouped_seeded(d, k):
    # Scores in a small integer range tie everywhere: the set, its order and
    # the tie rule must match the oracle exactly on a sample of query-heads,
    # however the keys were streamed and whatever threshold seeded them.
    rng = np.random.default_rng(100 + d + k)
    N, H = GROUPED_N, GROUPED_H
    q = rng.integers(-2, 3, size=(N, H, d)).astype(np.float32)
    kk = rng.integers(-1, 2, size=(N, H, d)).astype(np.float32)
    v = rng.standard_normal((N, H, d)).astype(np.float32)
    w = workloads.Workload("ties_grouped", N, H, d, k, 0.25, None, workloads.bf16_round(q),
                           workloads.bf16_round(kk), workloads.bf16_round(v), None, False)
    res = _run(w, backward=False)
    check_structure(res["idx"], None, N, H, k)
    sel = sample_rows(N, H, 512, seed=5)
    Qd, Kd, _, _ = _f64(w)
    o_idx, _, _ = oracle.topk(Qd, Kd, k, sel=sel)
    np.testing.assert_array_equal(res["idx"].reshape(N * H, k)[sel], o_idx)


def test_all_scores_tied_grouped():
    # Q = 0 on a large graph: every score is 0, so every query keeps keys
    # 0 .. k-1, in that order, even though scans start mid-graph.
    N, H, d, k = GROUPED_N, GROUPED_H, 16, 32
    rng = np.random.default_rng(1)
    w = workloads.Workload("zeroq_grouped", N, H, d, k, 0.25, None,
                           workloads.bf16_round(np.zeros((N, H, d), np.float32)),
                           workloads.bf16_round(rng.standard_normal((N, H, d)).astype(np.float32)),
                           workloads.bf16_round(rng.standard_normal((N, H, d)).astype(np.float32)),
                           None, False)
    res = _run(w, backward=False)
    assert (res["idx"] == np.arange(k, dtype=np.int32)).all()


def test_deterministic_and_overwrites():
    w = workloads.iid(3000, 2, 32, 16, seed=5, sizes=[1000, 2000])
    q, k, v, g = _dev(w.q), _dev(w.kk), _dev(w.v), _dev(w.dout)
    a = kmip.fwd(q, k, v, w.k, w.scale, graph_offsets=w.offsets)
    idx = torch.full_like(a[1], 12345)
    out = torch.full_like(a[0], float("nan"))
    lse = torch.full_like(a[2], -7.0)
    kmip.topk(q, k, w.k, graph_offsets=w.offsets, idx=idx)
    kmip.attend(q, k, v, idx, w.scale, out=out, lse=lse)
    torch.cuda.synchronize()
    assert torch.equal(a[1], idx)
    assert torch.equal(a[0], out)
    assert torch.equal(a[2], lse)
    dq = torch.full_like(a[0], 3.0)
    dk = torch.full_like(a[0], 3.0)
    dv = torch.full_like(a[0], 3.0)
    g1 = kmip.bwd(q, k, v, g, idx, lse, w.scale)
    kmip.bwd(q, k, v, g, idx, lse, w.scale, dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    assert torch.equal(g1[0], dq)
    # dK/dV are atomic scatters: equal up to summation order
    allclose_report("dK rerun", dk.cpu().numpy(), g1[1].cpu().numpy(), atol=1e-6, rtol=1e-5)
    allclose_report("dV rerun", dv.cpu().numpy(), g1[2].cpu().numpy(), atol=1e-6, rtol=1e-5)


def test_guard_canaries():
    # Outputs live inside larger buffers; the guard regions must stay untouched.
    w = workloads.iid(515, 3, 16, 20, seed=9, sizes=[515])
    q, k, v, g = _dev(w.q), _dev(w.kk), _dev(w.v), _dev(w.dout)
    N, H, d, kk = w.N, w.H, w.d, w.k
    pad = 4096
    ibuf = torch.full((N * H * kk + 2 * pad,), -77, dtype=torch.int32, device=DEV)
    obuf = torch.full((N * H * d + 2 * pad,), 5.5, dtype=torch.float32, device=DEV)
    lbuf = torch.full((N * H + 2 * pad,), 6.5, dtype=torch.float32, device=DEV)
    gbufs = [torch.full((N * H * d + 2 * pad,), 7.5, dtype=torch.float32, device=DEV) for _ in range(3)]
    idx = ibuf[pad:pad + N * H * kk].view(N, H, kk)
    out = obuf[pad:pad + N * H * d].view(N, H, d)
    lse = lbuf[pad:pad + N * H].view(N, H)
    kmip.topk(q, k, kk, idx=idx)
    kmip.attend(q, k, v, idx, w.scale, out=out, lse=lse)
    views = [b[pad:pad + N * H * d].view(N, H, d) for b in gbufs]
    kmip.bwd(q, k, v, g, idx, lse, w.scale, dq=views[0], dk=views[1], dv=views[2])
    torch.cuda.synchronize()
    for b, fill in [(ibuf, -77), (obuf, 5.5), (lbuf, 6.5)] + [(x, 7.5) for x in gbufs]:
        assert (b[:pad] == fill).all() and (b[-pad:] == fill).all()
    assert (idx >= 0).all()


def test_invalid_arguments_leave_outputs_untouched():
    w = workloads.iid(64, 1, 16, 4, seed=3)
    q, k, v = _dev(w.q), _dev(w.kk), _dev(w.v)
    idx = torch.full((64, 1, 4), -9, dtype=torch.int32, device=DEV)
    with pytest.raises(kmip.KmipError) as e:
        kmip.topk(q, k, 4, graph_offsets=[0, 30, 20, 64], idx=idx)
    assert e.value.status == 1
    with pytest.raises(kmip.KmipError) as e:
        kmip.topk(q, k, 513, idx=torch.empty((64, 1, 513), dtype=torch.int32, device=DEV))
    assert e.value.status == 2
    with pytest.raises(kmip.KmipError):
        kmip.attend(q, k, v, idx, -1.0)
    torch.cuda.synchronize()
    assert (idx == -9).all()


# Full sizes, in the launch configuration bench.py times.  Config 3: the
# index set of every one of its 400,000 query-heads.  Configs 4 and 5: 65,536
# and 16,384 query-heads spread over heads and directions.  Structure, out,
# lse and the gradients: every query-head.
@pytest.mark.parametrize("cfg,sample", [(3, None), (4, 65536), (5, 16384)])
def test_full_size(cfg, sample):
    w = workloads.make(cfg)
    sets, loose = _check_all(w, _run(w), sample=sample)
    print(f"c{cfg}: {sets} query-heads with the oracle's set, {loose} near-tied with a valid set")


# The select shape bench.py times at N=500k (two query blocks of 32 per wave,
# four candidate slots per lane) is the one the library picks when k <= 32,
# ceil(N/64)*H >= 8192 and there is one graph.  These graphs reach it at
# sizes where every query-head can be compared: point-cloud features (keys
# stored in tree order, pruned by bounds, seeded thresholds) and i.i.d.
# normal rows (most superblocks scanned).
TWO_BLOCK = [
    ("points", 8192, 64, 32), ("points", 12288, 48, 16), ("iid", 8192, 64, 32), ("iid", 12288, 48, 16),
]


@pytest.mark.parametrize("kind,n,h,k", TWO_BLOCK, ids=lambda c: str(c))
def test_two_block_shape_full(kind, n, h, k):
    assert k <= 32 and (n + 63) // 64 * h >= 8192
    if kind == "points":
        w = workloads.make(4, n=n, heads=h)
        w.k = k
    else:
        w = workloads.iid(n, h, 16, k, seed=n + k)
    _check_all(w, _run(w))


def test_two_block_shape_integer_ties():
    # Integer rows: every fp32 score is exact and ties abound, so the two-block
    # shape must give the oracle's rows index for index (tie rule included).
    N, H, d, k = 8192, 64, 16, 32
    rng = np.random.default_rng(8192)
    q = rng.integers(-2, 3, size=(N, H, d)).astype(np.float32)
    kk = rng.integers(-1, 2, size=(N, H, d)).astype(np.float32)
    v = rng.standard_normal((N, H, d)).astype(np.float32)
    w = workloads.Workload("ties_two_block", N, H, d, k, 0.25, None, workloads.bf16_round(q),
                           workloads.bf16_round(kk), workloads.bf16_round(v), None, False)
    res = _run(w, backward=False)
    Qd, Kd, _, _ = _f64(w)
    o_idx, _, _ = oracle.topk(Qd, Kd, k)
    np.testing.assert_array_equal(res["idx"].reshape(N * H, k), o_idx)


def test_pruning_margin_far_clusters():
    # Keys in 64 tight clusters far from the origin: centre components
    # ~ N(0, 20^2) (|c| about 80), spread 0.004 before rounding to bf16, so a
    # superblock's ball radius is dominated by the |c| 2^-12 term of its
    # rounding margin rather than by the spread of its keys.  Full comparison
    # of every query-head; ties inside a cluster leave many near-tied rows.
    N, H, d, k = 16384, 2, 16, 32
    rng = np.random.default_rng(64)
    cen = rng.standard_normal((64, H, d)).astype(np.float32) * np.float32(20.0)
    lab = rng.integers(0, 64, size=N)
    kk = cen[lab] + np.float32(0.004) * rng.standard_normal((N, H, d)).astype(np.float32)
    q = rng.standard_normal((N, H, d)).astype(np.float32)
    v = rng.standard_normal((N, H, d)).astype(np.float32)
    g = rng.standard_normal((N, H, d)).astype(np.float32)
    w = workloads.Workload("far_clusters", N, H, d, k, 0.25, None, workloads.bf16_round(q),
                           workloads.bf16_round(kk), workloads.bf16_round(v), workloads.bf16_round(g),
                           True)
    _check_all(w, _run(w))


@pytest.mark.parametrize("n,h,d,k", [(600_000, 4, 16, 32), (70_000, 32, 64, 16)])
def test_backward_wide_buckets(n, h, d, k):
    # N*H above 8192 * 4096/d key rows: the bucketed backward (the default
    # variant) widens its buckets to 512 key rows.  Index sets on sampled
    # query-heads, structure on all; out, lse and every gradient on every
    # query-head against the oracle on the GPU's own sets.
    w = workloads.make(4, n=n) if d == 16 else workloads.iid(n, h, d, k, seed=11)
    assert w.N * w.H > 8192 * 4096 // w.d
    res = _run(w)
    strict, loose = _check_all(w, res, sample=4096)
    print(f"N={w.N} H={w.H} d={w.d}: sampled {strict} with the oracle's set, {loose} near-tied query-heads")


def test_autograd_wrapper_matches_backward_and_oracle():
    # kmip.attention under torch autograd: the loss sum(out * dO) gives
    # Q, K, V gradients equal to kmip.bwd's rounded to bf16, the inputs'
    # dtype (dQ bit for bit; dK and dV sum with atomics, so to within a bf16
    # rounding), and within tolerance of the oracle's on the GPU's index sets.
    w = workloads.iid(300, 2, 32, 16, seed=3, sizes=[120, 1, 179])
    q, k, v = (_dev(a).requires_grad_() for a in (w.q, w.kk, w.v))
    g = _dev(w.dout)
    out = kmip.attention(q, k, v, w.k, w.scale, graph_offsets=w.offsets)
    (out * g.float()).sum().backward()
    out2, idx, lse = kmip.fwd(q.detach(), k.detach(), v.detach(), w.k, w.scale, graph_offsets=w.offsets)
    dq, dk, dv = kmip.bwd(q.detach(), k.detach(), v.detach(), g, idx, lse, w.scale)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), out2)
    assert q.grad.dtype == k.grad.dtype == v.grad.dtype == torch.bfloat16
    assert torch.equal(q.grad, dq.to(torch.bfloat16))
    for got, ref in ((k.grad, dk), (v.grad, dv)):
        assert torch.allclose(got.float(), ref, rtol=2.0 ** -7, atol=1e-6)
    Qd, Kd, Vd, dOd = _f64(w)
    rq, rk, rv = oracle.backward(Qd, Kd, Vd, dOd, idx.cpu().numpy(), w.scale)
    for name, got, ref in (("dQ", q.grad, rq), ("dK", k.grad, rk), ("dV", v.grad, rv)):
        allclose_report(name, got.float().cpu().numpy(), ref)


# Value rows of another width than the query/key rows (Section 3.1: W_V maps
# to d_V dimensions).  The index sets depend on Q and K only; out, lse and
# the gradients are compared with the oracle on every query-head, for every
# backward variant that takes d_V != d_K (the bucketed one needs them equal;
# the library's choice then is the segmented one).
VALUE_WIDTH = [
    # (N, H, d, dv, k, sizes)
    (3000, 2, 16, 32, 16, [1000, 7, 1993]),
    (2500, 3, 32, 64, 32, None),
    (1800, 2, 64, 16, 24, [900, 0, 900]),
    (2100, 1, 32, 16, 128, [2100]),
    (20000, 2, 16, 64, 32, None),       # one graph above the grouping size
]


@pytest.mark.parametrize("case", VALUE_WIDTH, ids=lambda c: "N%d_H%d_d%d_dv%d_k%d" % c[:5])
def test_value_width_full(case):
    N, H, d, dv, k, sizes = case
    w = workloads.iid(N, H, d, k, seed=N + dv, sizes=sizes, dv=dv)
    for variant in (0, 1, 2, 4):
        res = _run(w, variant=variant)
        assert res["out"].shape == (N, H, dv) and res["dv"].shape == (N, H, dv) and res["dk"].shape == (N, H, d)
        _check_all(w, res)


def test_value_width_bucketed_refused():
    w = workloads.iid(500, 1, 16, 8, seed=1, dv=32)
    q, k, v, g = _dev(w.q), _dev(w.kk), _dev(w.v), _dev(w.dout)
    out, idx, lse = kmip.fwd(q, k, v, w.k, w.scale)
    with pytest.raises(kmip.KmipError) as e:
        kmip.bwd(q, k, v, g, idx, lse, w.scale, variant=3)
    assert e.value.status == 2


def test_stale_workspace_does_not_change_selection():
    # The library clears every counter it reads (work counters, dense-mode
    # votes, seed slots) at the start of each call, whatever the workspace
    # held before: a workspace filled with 0x7f bytes (counters reading as
    # huge values) gives the same index sets as a zeroed one, and the select
    # kernel takes about as long.  A one-head graph takes the per-head
    # counters' shortest fill (one entry).
    w = workloads.make(5, n=65536)
    q, k = _dev(w.q), _dev(w.kk)
    ws = kmip.Workspace(DEV)
    buf = ws.get(kmip.topk_workspace_size(w.N, w.H, w.d, w.k, 1))
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    times, sets = {}, {}
    for fill in (0, 0x7F, 0, 0x7F):
        idx = torch.empty((w.N, w.H, w.k), dtype=torch.int32, device=DEV)
        buf.fill_(fill)
        kmip.topk(q, k, w.k, graph_offsets=w.offsets, idx=idx, workspace=ws, select_events=evs)
        torch.cuda.synchronize()
        times.setdefault(fill, []).append(evs[0].elapsed_time(evs[1]))
        sets[fill] = torch.sort(idx, -1).values.cpu()
    print(f"select ms, zeroed workspace {times[0]}, 0x7f-filled {times[0x7F]}", flush=True)
    assert torch.equal(sets[0], sets[0x7F])
    assert min(times[0x7F]) < 1.5 * min(times[0]) + 0.1


def test_peak_memory_linear_in_n():
    # Peak device memory of a forward+backward step (inputs, outputs and the
    # library's workspaces) grows linearly with N: the bytes per node at the
    # 500k-node configuration stay within 10% of those at a quarter of it.
    per_node = {}
    for n in (125_000, 500_000):
        w = workloads.make(4, n=n)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats(DEV)
        base = torch.cuda.memory_allocated(DEV)
        res = _run(w)
        del res
        torch.cuda.synchronize()
        per_node[n] = (torch.cuda.max_memory_allocated(DEV) - base) / n
        print(f"N={n}: {per_node[n]:.0f} peak bytes per node", flush=True)
    assert per_node[500_000] <= 1.1 * per_node[125_000]
    assert per_node[500_000] < 8192


def test_fwd_grouped_order_matches_separate_calls():
    # kmip_fwd on one grouped graph takes the aggregate in the grouped query
    # order; the rows must be those of kmip_topk + kmip_attend, bit for bit,
    # and the recorded events must bracket the select kernel and the
    # aggregate in that order.
    w = workloads.iid(12000, 2, 16, 16, seed=12)
    q, k, v = _dev(w.q), _dev(w.kk), _dev(w.v)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    out, idx, lse = kmip.fwd(q, k, v, w.k, w.scale, events=ev)
    end = torch.cuda.Event(enable_timing=True)
    end.record()
    idx2 = kmip.topk(q, k, w.k)
    out2, lse2 = kmip.attend(q, k, v, idx2, w.scale)
    torch.cuda.synchronize()
    assert torch.equal(idx, idx2) and torch.equal(out, out2) and torch.equal(lse, lse2)
    assert ev[0].elapsed_time(ev[1]) > 0 and ev[1].elapsed_time(ev[2]) >= 0 and ev[2].elapsed_time(end) > 0


@pytest.mark.parametrize("k", [1, 8, 16])
def test_small_graph_lists_and_full_rows_in_one_wave(k):
    # The small-graph select lists, per query, the keys that reach a lower
    # bound of its k-th best (k <= 16) and selects on the list when at most
    # 112 keys do; otherwise it searches all of the row.  Here a quarter of
    # the queries are zero (every score ties at 0: all n keys reach the
    # bound, so n > 112 takes the full row) next to queries with integer
    # rows (short lists), so the four queries of a wave mix both paths.
    # Integer inputs make the scores exact: every row, order included, must
    # be the oracle's.
    rng = np.random.default_rng(77 + k)
    sizes = [480, 113, 112, 300, 17, 479, 250]
    N, H, d = sum(sizes), 2, 32
    q = rng.integers(-2, 3, size=(N, H, d)).astype(np.float32)
    q[rng.random(N) < 0.25] = 0.0
    kk = rng.integers(-2, 3, size=(N, H, d)).astype(np.float32)
    v = rng.standard_normal((N, H, d)).astype(np.float32)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    w = workloads.Workload("small_mixed", N, H, d, k, 0.25, offsets, workloads.bf16_round(q),
                           workloads.bf16_round(kk), workloads.bf16_round(v), None, False)
    print(f"[case] small-graph lists k={k} sizes={sizes}", flush=True)
    res = _run(w, backward=False)
    Qd, Kd, Vd, _ = _f64(w)
    _, o_idx, _ = oracle.forward(Qd, Kd, Vd, k, w.scale, offsets=offsets)
    np.testing.assert_array_equal(res["idx"], o_idx)
    ref_out, ref_lse = oracle.attend(Qd, Kd, Vd, res["idx"], w.scale)
    allclose_report("out", res["out"].reshape(-1, d), ref_out)
    allclose_report("lse", res["lse"].reshape(-1), ref_lse)
