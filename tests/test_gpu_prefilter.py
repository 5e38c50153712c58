"""The int8 prefilter with a provable bound (kmip_topk_prefilter) on the GPU.

Its result must be kmip_topk's, row for row and in order: the re-rank forms
the same fp32 scores with the same MFMA, and the bound makes every key of
the exact top-k a candidate.  Each case also reports how many blocks of 32
queries the select kernel redid (lists that would overflow), and is checked
against the float64 oracle.
"""
import numpy as np
import pytest

import oracle
import workloads
from parity import check_sets_all, check_structure

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2604_03815_amd as kmip  # noqa: E402

DEV = torch.device("cuda:0")


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)


def _both(w, k):
    q, kk = _dev(w.q), _dev(w.kk)
    redone = torch.zeros(1, dtype=torch.int32, device=DEV)
    print(f"[case] prefilter {w.name} N={w.N} H={w.H} d={w.d} k={k}", flush=True)
    got = kmip.topk_prefilter(q, kk, k, redone=redone)
    ref = kmip.topk(q, kk, k)
    torch.cuda.synchronize()
    nblocks = (w.N + 31) // 32
    r = int(redone.item())
    print(f"[redo] {r} of {nblocks} query blocks redone by the select kernel", flush=True)
    return got.cpu().numpy(), ref.cpu().numpy(), r, nblocks


CASES = [
    # (name, N, H, d, k)
    ("iid", 6000, 2, 16, 8),
    ("iid", 6000, 1, 32, 32),
    ("iid", 4000, 2, 64, 16),
    ("iid", 3000, 1, 128, 32),
    ("iid", 4097, 3, 32, 1),
    ("iid", 100, 1, 32, 32),     # fewer keys than the list holds
    ("iid", 33, 2, 16, 32),      # graph smaller than k: -1 padding
    ("iid", 1, 1, 16, 1),
    ("fourier", 20000, 2, 32, 32),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "%s_N%d_H%d_d%d_k%d" % c)
def test_prefilter_equals_select(case):
    name, N, H, d, k = case
    if name == "fourier":
        w = workloads.make(3, n=N, heads=H)
        w.k = k
    else:
        w = workloads.iid(N, H, d, k, seed=N + d + k)
    got, ref, r, nblocks = _both(w, k)
    np.testing.assert_array_equal(got, ref)
    check_structure(got, None, N, H, k)
    Qd, Kd = oracle.from_bf16(w.q), oracle.from_bf16(w.kk)
    check_sets_all(w, Qd, Kd, got)
    if name == "iid" and N >= 3000:
        # the int8 path, not the redo, decides most rows of generic data
        assert r < nblocks // 2


@pytest.mark.parametrize("distinct", [4, 400])
def test_prefilter_ties(distinct):
    # Integer inputs: the int8 scores are exact, so the lists hold the keys
    # that tie with the k-th best score and a few more.  With 4 distinct key
    # rows a quarter of the keys tie at the top: no list holds them, every
    # block is redone by the select kernel.  With 400 the lists fit.  Both
    # give the oracle's rows, tie order included.
    rng = np.random.default_rng(9 + distinct)
    N, H, d, k = 3000, 2, 16, 16
    rows = rng.integers(-1, 2, size=(distinct, H, d)).astype(np.float32)
    kk = rows[rng.integers(0, distinct, size=N)]
    w = workloads.Workload("ties", N, H, d, k, 0.25, None,
                           workloads.bf16_round(rng.integers(-2, 3, size=(N, H, d)).astype(np.float32)),
                           workloads.bf16_round(kk),
                           workloads.bf16_round(rng.standard_normal((N, H, d)).astype(np.float32)), None, False)
    got, ref, r, nblocks = _both(w, k)
    np.testing.assert_array_equal(got, ref)
    o_idx, _, _ = oracle.topk(oracle.from_bf16(w.q), oracle.from_bf16(w.kk), k)
    np.testing.assert_array_equal(got.reshape(N * H, k), o_idx)
    if distinct == 4:
        assert r == nblocks
    else:
        assert r < nblocks


def test_prefilter_mixed_blocks():
    # Queries 0 .. 1599 are zero (all scores tie: their blocks are redone);
    # the others are generic and go through the re-rank.
    rng = np.random.default_rng(4)
    N, H, d, k = 4000, 1, 32, 8
    q = rng.standard_normal((N, H, d)).astype(np.float32)
    q[:1600] = 0.0
    w = workloads.Workload("mixed", N, H, d, k, 0.25, None, workloads.bf16_round(q),
                           workloads.bf16_round(rng.standard_normal((N, H, d)).astype(np.float32)),
                           workloads.bf16_round(rng.standard_normal((N, H, d)).astype(np.float32)), None, False)
    got, ref, r, nblocks = _both(w, k)
    np.testing.assert_array_equal(got, ref)
    assert (got[:1600] == np.arange(k, dtype=np.int32)).all()
    assert 50 <= r < nblocks


def test_prefilter_refuses_large_k():
    q = torch.zeros((64, 1, 16), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(kmip.KmipError):
        kmip.topk_prefilter(q, q, 33)
