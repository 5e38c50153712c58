"""The parity checker itself, on the CPU: index sets the oracle produced pass,
and sets with a planted mistake fail (the GPU tests rely on it to reject a
wrong set without sorting every row)."""
import numpy as np
import pytest

import oracle
import workloads
from parity import check_sets, check_sets_all, stratified_rows


def _wl(seed=0):
    return workloads.iid(3000, 2, 16, 8, seed=seed, sizes=[1000, 7, 1993])


def test_oracle_sets_pass_without_sorting_most_rows():
    w = _wl()
    Qd, Kd = oracle.from_bf16(w.q), oracle.from_bf16(w.kk)
    _, idx, _ = oracle.forward(Qd, Kd, oracle.from_bf16(w.v), w.k, w.scale, offsets=w.offsets)
    exact, strict, loose = check_sets_all(w, Qd, Kd, idx)
    assert exact + strict + loose == w.N * w.H
    assert exact > 0.95 * w.N * w.H     # i.i.d. scores seldom tie at the k-th place
    sel = stratified_rows(Qd, 500, seed=1)
    assert sum(check_sets_all(w, Qd, Kd, idx, sel=sel)) == 500


def _swap_in_outsider(w, Qd, Kd, idx, row):
    """Replaces the last member of `row` by the graph's lowest-scoring key:
    a wrong set of a well-separated row."""
    bad = idx.reshape(w.N * w.H, w.k).copy()
    o, sc, _ = oracle.topk(Qd, Kd, w.N, offsets=w.offsets, sel=np.array([row]))
    worst = o[0][o[0] >= 0][-1]
    bad[row, w.k - 1] = worst
    return bad


@pytest.mark.parametrize("checker", [check_sets, check_sets_all])
def test_planted_wrong_member_fails(checker):
    w = _wl(1)
    Qd, Kd = oracle.from_bf16(w.q), oracle.from_bf16(w.kk)
    _, idx, _ = oracle.forward(Qd, Kd, oracle.from_bf16(w.v), w.k, w.scale, offsets=w.offsets)
    bad = _swap_in_outsider(w, Qd, Kd, idx, row=2 * 1500 + 1)
    with pytest.raises(AssertionError):
        checker(w, Qd, Kd, bad)


def test_planted_duplicate_fails():
    w = _wl(2)
    Qd, Kd = oracle.from_bf16(w.q), oracle.from_bf16(w.kk)
    _, idx, _ = oracle.forward(Qd, Kd, oracle.from_bf16(w.v), w.k, w.scale, offsets=w.offsets)
    bad = idx.reshape(w.N * w.H, w.k).copy()
    bad[10, 1] = bad[10, 0]
    with pytest.raises(AssertionError):
        check_sets_all(w, Qd, Kd, bad)


def test_equally_good_tied_set_passes():
    # Integer rows tie often: trading a member for a non-member of exactly the
    # same score is another correct set, accepted by the tolerant rule.
    rng = np.random.default_rng(5)
    N, H, d, k = 400, 1, 16, 6
    q = workloads.bf16_round(rng.integers(-1, 2, size=(N, H, d)).astype(np.float32))
    kk = workloads.bf16_round(rng.integers(-1, 2, size=(N, H, d)).astype(np.float32))
    w = workloads.Workload("ties", N, H, d, k, 0.5, None, q, kk, q, None, False)
    Qd, Kd = oracle.from_bf16(q), oracle.from_bf16(kk)
    o, sc, nx = oracle.topk(Qd, Kd, k)
    rows = np.nonzero(sc[:, k - 1] == nx)[0]
    assert rows.size > 0
    alt = o.copy()
    for r in rows:
        full, fsc, _ = oracle.topk(Qd, Kd, N, sel=np.array([r]))
        alt[r, k - 1] = full[0, k]      # the (k+1)-th key scores the same as the k-th
    assert sum(check_sets_all(w, Qd, Kd, alt)[1:]) >= rows.size


def test_stratified_rows_cover_heads():
    w = workloads.make(4, n=5000)
    Qd = oracle.from_bf16(w.q)
    sel = stratified_rows(Qd, 1000, seed=3)
    assert sel.size == 1000 and np.unique(sel).size == 1000
    assert np.all(np.bincount(sel % w.H, minlength=w.H) == 250)
