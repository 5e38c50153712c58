"""GPU-vs-oracle parity protocol (helpers for the gpu tests, smoke and bench).

Index sets.  For each query-head the oracle's exact scores (float64 on the
same bf16 inputs) give the k-th and (k+1)-th best scores s_k and s_k1.  When
  gap = (s_k - s_k1) / max(|s_k|, |s_k1|) > 1e-3   and   s_k - s_k1 > eps
the top-k set is well separated and the GPU set must equal the oracle's set
exactly.  eps = 8 * d * 2^-24 * sum_t |q_t| * max|K| bounds the float32
accumulation error of any score of that query, so it only matters when the
scores are near zero.  Otherwise several sets are correct, and the GPU set
must be a valid top-k within tau = 1e-3 * max(|s_k|, |s_k1|) + eps:
  min over the GPU set >= max over the rest - tau,
with distinct in-graph indices and min(k, n) of them.

Values.  out and lse are compared with the oracle evaluated on the GPU's own
index set; gradients with the oracle backward on the GPU's index set.  The
bar is |x - r| <= 1e-3 + 2e-2 |r| elementwise.
"""
from __future__ import annotations

import numpy as np

import oracle

REL_GAP = 1e-3
ATOL = 1e-3
RTOL = 2e-2


def allclose_report(name, got, ref, atol=ATOL, rtol=RTOL):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    err = np.abs(got - ref)
    bad = err > atol + rtol * np.abs(ref)
    both_inf = np.isinf(got) & np.isinf(ref) & (np.sign(got) == np.sign(ref))
    bad &= ~both_inf
    if bad.any():
        i = np.argmax(np.where(bad, err, -1))
        raise AssertionError(
            f"{name}: {int(bad.sum())} of {bad.size} elements outside "
            f"{atol}+{rtol}|r|; worst at flat {i}: got {got.flat[i]!r} ref {ref.flat[i]!r}")


def graph_bounds(offsets, N):
    """lo[i], hi[i] for every node i."""
    if offsets is None:
        return np.zeros(N, np.int64), np.full(N, N, np.int64)
    o = np.asarray(offsets, np.int64)
    sizes = np.diff(o)
    lo = np.repeat(o[:-1], sizes)
    hi = np.repeat(o[1:], sizes)
    return lo, hi


def check_structure(idx, offsets, N, H, k):
    """Every row: indices inside the query's graph, distinct, min(k, n) valid
    ones first and -1 after.  Vectorised; runs at any size."""
    idx = np.asarray(idx).reshape(N, H, k)
    lo, hi = graph_bounds(offsets, N)
    n = (hi - lo)[:, None, None]
    want = np.minimum(n, k)
    slot = np.arange(k)[None, None, :]
    valid = idx >= 0
    assert np.array_equal(valid, np.broadcast_to(slot < want, idx.shape)), "padding layout"
    inside = (idx >= lo[:, None, None]) & (idx < hi[:, None, None])
    assert np.all(inside | ~valid), "index outside its graph"
    srt = np.sort(np.where(valid, idx, -1 - slot), axis=2)
    assert not np.any((np.diff(srt, axis=2) == 0) & (srt[:, :, 1:] >= 0)), "duplicate index"


def check_sets(w, Qd, Kd, idx_gpu, sel=None):
    """Parity of GPU index sets with the oracle on the selected query-heads
    (all if sel is None).  Returns (n_strict, n_tolerant)."""
    N, H, d, k = w.N, w.H, w.d, w.k
    g = np.asarray(idx_gpu).reshape(N * H, k)
    rows = np.arange(N * H) if sel is None else np.asarray(sel, np.int64)
    o_idx, o_sc, o_next = oracle.topk(Qd, Kd, k, offsets=w.offsets, sel=rows)
    lo, hi = graph_bounds(w.offsets, N)
    i_node = rows // H
    n = (hi - lo)[i_node]
    kk = np.minimum(n, k)
    s_k = o_sc[np.arange(len(rows)), np.maximum(kk - 1, 0)]
    s_k1 = o_next
    # float32 accumulation bound of any score of the query
    kmax = np.abs(Kd).max() if Kd.size else 0.0
    qabs = np.abs(Qd.reshape(N * H, d)[rows]).sum(axis=1)
    eps = 8.0 * d * 2.0 ** -24 * qabs * kmax
    denom = np.maximum(np.abs(s_k), np.abs(s_k1))
    with np.errstate(invalid="ignore", divide="ignore"):
        gap_rel = np.where(np.isinf(s_k1), np.inf, (s_k - s_k1) / np.where(denom > 0, denom, 1.0))
    strict = (gap_rel > REL_GAP) & ((s_k - s_k1) > eps)
    gsub = g[rows]
    differ = np.any(np.sort(gsub, axis=1) != np.sort(o_idx, axis=1), axis=1) & strict
    mism = rows[differ].tolist()
    assert not mism, f"{len(mism)} well-separated query-heads differ, e.g. {mism[:5]}"
    loose = np.nonzero(~strict)[0]
    if loose.size:
        mn, mx, fl = oracle.check_set(Qd, Kd, gsub[loose], offsets=w.offsets, sel=rows[loose])
        assert np.all(fl == 0), "structurally invalid set among near-tied queries"
        tau = REL_GAP * denom[loose] + eps[loose]
        ok = (mn >= mx - tau) | np.isinf(mx)
        assert np.all(ok), f"{int((~ok).sum())} near-tied query-heads hold an invalid top-k"
    return int(strict.sum()), int(loose.size)


def sample_rows(N, H, m, seed=0):
    rng = np.random.default_rng(seed)
    m = min(m, N * H)
    return np.sort(rng.choice(N * H, size=m, replace=False))


def check_sets_all(w, Qd, Kd, idx_gpu, sel=None):
    """Parity of GPU index sets with the oracle on the selected query-heads
    (all if sel is None), without sorting every row.

    The oracle's exact-score check gives, per query-head, the lowest score
    inside the GPU set (min_in) and the highest score of a graph key outside
    it (max_out).  A structurally valid set with min_in > max_out holds
    exactly the keys that score above every other key of the graph: it is
    the unique top-k set, the oracle's.  Only the remaining query-heads (a
    tie or a near-tie at the k-th place, or a wrong set) go through the full
    protocol of check_sets, whose sort settles which case it is.  Rows are
    checked head by head on contiguous copies of that head's Q and K, so the
    keys stream through the host's caches once per row.
    Returns (n_exact, n_strict, n_tolerant)."""
    N, H, d, k = w.N, w.H, w.d, w.k
    g = np.asarray(idx_gpu).reshape(N * H, k)
    rows = np.arange(N * H, dtype=np.int64) if sel is None else np.asarray(sel, np.int64)
    mn = np.empty(rows.size)
    mx = np.empty(rows.size)
    fl = np.empty(rows.size, np.int32)
    for h in range(H):
        m = (rows % H) == h
        if not m.any():
            continue
        q1 = np.ascontiguousarray(Qd[:, h:h + 1, :])
        k1 = np.ascontiguousarray(Kd[:, h:h + 1, :])
        mn[m], mx[m], fl[m] = oracle.check_set(q1, k1, g[rows[m]], offsets=w.offsets, sel=rows[m] // H)
    bad = np.nonzero(fl != 0)[0]
    assert bad.size == 0, f"{bad.size} structurally invalid sets, e.g. query-heads {rows[bad[:5]].tolist()}"
    exact = mn > mx
    rest = rows[~exact]
    n_strict = n_loose = 0
    if rest.size:
        n_strict, n_loose = check_sets(w, Qd, Kd, idx_gpu, sel=rest)
    return int(exact.sum()), n_strict, n_loose


def stratified_rows(Qd, m, seed=0, directions=64):
    """m query-heads spread evenly over heads and over direction labels (the
    nearest of `directions` seeded random unit vectors per head): the rows
    sorted by (head, label, node) are sampled at evenly spaced positions with
    a seeded offset, so every head and every sizeable label gets its share."""
    N, H, d = Qd.shape
    rng = np.random.default_rng(seed)
    u = rng.standard_normal((H, directions, d))
    u /= np.linalg.norm(u, axis=2, keepdims=True)
    lab = np.einsum("nhd,hcd->nhc", Qd, u).argmax(axis=2)            # [N, H]
    qh = np.arange(N * H, dtype=np.int64)
    order = np.lexsort((qh // H, lab.reshape(-1), qh % H))
    m = min(m, N * H)
    pos = (np.arange(m) * (N * H / m) + rng.random() * (N * H / m)).astype(np.int64)
    return np.sort(order[np.minimum(pos, N * H - 1)])
