"""Pins for the CPU oracle: each test ties it to something other than itself.

The paper prints no worked numerical example, so the oracle is pinned by what
the definition and the mathematics fix:
  * brute-force enumeration of k-subsets on tiny integer inputs with
    deliberate ties (RowwiseTopK of Algorithm 1, ties to the lower index);
  * a hand-derived example with ties (tests/golden/tiny_ties.json);
  * k = n reduces to textbook softmax attention (torch CPU float64
    scaled_dot_product_attention and its autograd);
  * k = 1 reduces to argmax (numpy, first occurrence = lower index);
  * k < n on tie-free inputs matches a masked dense attention built from
    torch CPU float64 primitives (topk, softmax, logsumexp) and its autograd;
  * permutation equivariance (assumption A3 of Appendix B, and the tie
    footnote of Section 4.2);
  * block-diagonal batches equal separate per-graph runs;
  * selection invariances (positive rescaling, per-query score shifts);
  * softmax weights sum to one, value shifts, the hardmax limit used in the
    proof of Theorem 2 (Appendix C);
  * central finite differences of the oracle's own forward for the backward,
    plus gradient invariants that follow from the invariances above.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _int_inputs(rng, N, H, d, lo=-2, hi=2):
    return rng.integers(lo, hi + 1, size=(N, H, d)).astype(np.float64)


def _graphs(offsets, N):
    if offsets is None:
        return [(0, N)]
    return [(int(offsets[g]), int(offsets[g + 1])) for g in range(len(offsets) - 1)]


def _brute_force_set(scores_row, lo, hi, k):
    """The unique k-subset whose members all beat all non-members under
    (score desc, index asc), found by enumerating every subset."""
    keys = list(range(lo, hi))
    kk = min(k, len(keys))

    def beats(a, b):
        return scores_row[a] > scores_row[b] or (scores_row[a] == scores_row[b] and a < b)

    found = []
    for S in itertools.combinations(keys, kk):
        Sset = set(S)
        if all(beats(a, b) for a in S for b in keys if b not in Sset):
            found.append(S)
    assert len(found) == 1
    return set(found[0])


@pytest.mark.parametrize("seed", range(40))
def test_brute_force_subsets_with_ties(seed):
    rng = np.random.default_rng(1000 + seed)
    H = int(rng.integers(1, 3))
    d = int(rng.integers(1, 4))
    sizes = [int(x) for x in rng.integers(0, 7, size=int(rng.integers(1, 3)))]
    if sum(sizes) == 0:
        sizes[0] = 3
    N = sum(sizes)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    k = int(rng.integers(1, 5))
    Q = _int_inputs(rng, N, H, d, -1, 1)   # small range -> many exact ties
    K = _int_inputs(rng, N, H, d, -1, 1)
    idx, sc, nxt = oracle.topk(Q, K, k, offsets=offsets)
    idx = idx.reshape(N, H, k)
    sc = sc.reshape(N, H, k)
    for (lo, hi) in _graphs(offsets, N):
        for i in range(lo, hi):
            for h in range(H):
                # exact integer scores, computed without the oracle
                row = {j: int(sum(int(Q[i, h, t]) * int(K[j, h, t]) for t in range(d)))
                       for j in range(lo, hi)}
                want = _brute_force_set(row, lo, hi, k)
                got = [int(x) for x in idx[i, h] if x >= 0]
                assert set(got) == want
                assert len(got) == min(k, hi - lo)
                assert all(x == -1 for x in idx[i, h][len(got):])
                # kept in (score desc, index asc) order, with their exact scores
                assert got == sorted(got, key=lambda j: (-row[j], j))
                assert [float(s) for s in sc[i, h][:len(got)]] == [float(row[j]) for j in got]


def test_golden_tiny_ties():
    with open(os.path.join(GOLDEN, "tiny_ties.json")) as f:
        g = json.load(f)
    Q = np.array(g["Q"], np.float64)[:, None, :]
    K = np.array(g["K"], np.float64)[:, None, :]
    V = np.array(g["V"], np.float64)[:, None, :]
    out, idx, lse = oracle.forward(Q, K, V, g["k"], g["scale"])
    assert idx[:, 0, :].tolist() == g["expected_idx"]
    e = math.e
    want_out = np.array([[3.0, 4.0], [4.0, 5.0],
                         [(e * 5 + 1) / (e + 1), (e * 6 + 2) / (e + 1)],
                         [(e * 1 + 5) / (e + 1), (e * 2 + 6) / (e + 1)]])
    want_lse = np.array([1 + math.log(2), 1 + math.log(2), 1 + math.log(e + 1),
                         1 + math.log(e + 1)])
    np.testing.assert_allclose(out[:, 0, :], want_out, rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(lse[:, 0], want_lse, rtol=1e-14)
    _, sc, _ = oracle.topk(Q, K, g["k"])
    assert sc.tolist() == [[float(x) for x in r] for r in g["expected_kept_scores"]]


def _sdpa_per_graph(Q, K, V, offsets, scale):
    N, H, d = Q.shape
    out = np.zeros((N, H, V.shape[2]))
    lse = np.zeros((N, H))
    for (lo, hi) in _graphs(offsets, N):
        if hi == lo:
            continue
        q = torch.from_numpy(Q[lo:hi]).permute(1, 0, 2).contiguous()
        kk = torch.from_numpy(K[lo:hi]).permute(1, 0, 2).contiguous()
        v = torch.from_numpy(V[lo:hi]).permute(1, 0, 2).contiguous()
        o = torch.nn.functional.scaled_dot_product_attention(q, kk, v, scale=scale)
        out[lo:hi] = o.permute(1, 0, 2).numpy()
        logits = scale * torch.matmul(q, kk.transpose(1, 2).contiguous())
        lse[lo:hi] = torch.logsumexp(logits, dim=-1).T.numpy()
    return out, lse


@pytest.mark.parametrize("seed", range(4))
def test_k_equals_n_is_softmax_attention(seed):
    rng = np.random.default_rng(seed)
    sizes = [5, 9, 1, 12]
    N, H, d = sum(sizes), 2, 4
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    Q, K, V = (rng.standard_normal((N, H, d)) for _ in range(3))
    scale = 0.37
    out, idx, lse = oracle.forward(Q, K, V, max(sizes), scale, offsets=offsets)
    want_out, want_lse = _sdpa_per_graph(Q, K, V, offsets, scale)
    np.testing.assert_allclose(out, want_out, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, want_lse, rtol=1e-12, atol=1e-12)
    # graphs smaller than k: every key kept, unused slots padded with -1
    for (lo, hi) in _graphs(offsets, N):
        for i in range(lo, hi):
            for h in range(H):
                got = idx[i, h]
                assert sorted(got[: hi - lo].tolist()) == list(range(lo, hi))
                assert (got[hi - lo:] == -1).all()


def test_k1_is_argmax():
    rng = np.random.default_rng(7)
    N, H, d = 40, 3, 3
    Q = _int_inputs(rng, N, H, d)
    K = _int_inputs(rng, N, H, d)
    V = rng.standard_normal((N, H, d))
    out, idx, lse = oracle.forward(Q, K, V, 1, 1.0)
    for h in range(H):
        S = Q[:, h, :] @ K[:, h, :].T
        am = np.argmax(S, axis=1)   # first occurrence on ties = lower index
        np.testing.assert_array_equal(idx[:, h, 0], am)
        np.testing.assert_allclose(out[:, h, :], V[am, h, :], rtol=0, atol=0)
        np.testing.assert_allclose(lse[:, h], S[np.arange(N), am], rtol=1e-15)


def _masked_dense_torch(Q, K, V, k, scale):
    """Textbook top-k masked attention from torch primitives (tie-free inputs)."""
    q = Q.permute(1, 0, 2)
    kk = K.permute(1, 0, 2)
    v = V.permute(1, 0, 2).contiguous()
    S = torch.matmul(q, kk.transpose(1, 2).contiguous())
    top = torch.topk(S, k, dim=-1).indices
    mask = torch.full_like(S, float("-inf"))
    mask.scatter_(-1, top, 0.0)
    logits = scale * S + mask
    A = torch.softmax(logits, dim=-1)
    out = torch.matmul(A, v).permute(1, 0, 2)
    lse = torch.logsumexp(logits, dim=-1).T
    return out, lse, top


@pytest.mark.parametrize("seed", range(3))
def test_k_less_than_n_matches_masked_dense(seed):
    rng = np.random.default_rng(100 + seed)
    N, H, d, k = 37, 2, 5, 6
    Qn, Kn, Vn = (rng.standard_normal((N, H, d)) for _ in range(3))
    scale = 0.61
    out, idx, lse = oracle.forward(Qn, Kn, Vn, k, scale)
    Q, K, V = (torch.from_numpy(x) for x in (Qn, Kn, Vn))
    want_out, want_lse, top = _masked_dense_torch(Q, K, V, k, scale)
    np.testing.assert_allclose(out, want_out.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, want_lse.numpy(), rtol=1e-12, atol=1e-12)
    for h in range(H):
        for i in range(N):
            assert set(idx[i, h].tolist()) == set(top[h, i].tolist())


@pytest.mark.parametrize("seed", range(3))
def test_backward_matches_torch_autograd(seed):
    rng = np.random.default_rng(200 + seed)
    N, H, d, k = 29, 2, 4, 5
    Qn, Kn, Vn, dOn = (rng.standard_normal((N, H, d)) for _ in range(4))
    scale = 0.8
    _, idx, _ = oracle.forward(Qn, Kn, Vn, k, scale)
    dQ, dK, dV = oracle.backward(Qn, Kn, Vn, dOn, idx, scale)
    Q, K, V = (torch.from_numpy(x).clone().requires_grad_(True) for x in (Qn, Kn, Vn))
    out, _, _ = _masked_dense_torch(Q, K, V, k, scale)
    (out * torch.from_numpy(dOn)).sum().backward()
    np.testing.assert_allclose(dQ, Q.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dK, K.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dV, V.grad.numpy(), rtol=1e-11, atol=1e-12)


def test_backward_k_equals_n_matches_sdpa_autograd():
    rng = np.random.default_rng(5)
    N, H, d = 17, 3, 4
    Qn, Kn, Vn, dOn = (rng.standard_normal((N, H, d)) for _ in range(4))
    scale = 0.5
    _, idx, _ = oracle.forward(Qn, Kn, Vn, N, scale)
    dQ, dK, dV = oracle.backward(Qn, Kn, Vn, dOn, idx, scale)
    Q, K, V = (torch.from_numpy(x).permute(1, 0, 2).contiguous().requires_grad_(True)
               for x in (Qn, Kn, Vn))
    o = torch.nn.functional.scaled_dot_product_attention(Q, K, V, scale=scale)
    (o * torch.from_numpy(dOn).permute(1, 0, 2)).sum().backward()
    np.testing.assert_allclose(dQ, Q.grad.permute(1, 0, 2).numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dK, K.grad.permute(1, 0, 2).numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dV, V.grad.permute(1, 0, 2).numpy(), rtol=1e-11, atol=1e-12)


def _loss(Q, K, V, dO, k, scale, offsets=None):
    out, _, _ = oracle.forward(Q, K, V, k, scale, offsets=offsets)
    return float((out * dO).sum())


def test_backward_finite_differences():
    rng = np.random.default_rng(11)
    sizes = [6, 8]
    N, H, d, k = sum(sizes), 2, 3, 3
    offsets = np.array([0, 6, 14], np.int32)
    Q, K, V, dO = (rng.standard_normal((N, H, d)) for _ in range(4))
    scale = 0.9
    _, idx, _ = oracle.forward(Q, K, V, k, scale, offsets=offsets)
    # keep away from selection ties: the k-th/k+1-th gap must be large enough
    _, _, nxt = oracle.topk(Q, K, k, offsets=offsets)
    dQ, dK, dV = oracle.backward(Q, K, V, dO, idx, scale)
    eps = 1e-6
    for name, X, G in (("Q", Q, dQ), ("K", K, dK), ("V", V, dV)):
        num = np.zeros_like(X)
        for pos in np.ndindex(X.shape):
            Xp, Xm = X.copy(), X.copy()
            Xp[pos] += eps
            Xm[pos] -= eps
            args_p = {"Q": Q, "K": K, "V": V}
            args_m = {"Q": Q, "K": K, "V": V}
            args_p[name], args_m[name] = Xp, Xm
            num[pos] = (_loss(args_p["Q"], args_p["K"], args_p["V"], dO, k, scale, offsets)
                        - _loss(args_m["Q"], args_m["K"], args_m["V"], dO, k, scale, offsets)) / (2 * eps)
        np.testing.assert_allclose(G, num, rtol=1e-6, atol=1e-7, err_msg=name)


def test_permutation_equivariance():
    rng = np.random.default_rng(3)
    N, H, d, k = 50, 2, 4, 7
    Q, K, V = (rng.standard_normal((N, H, d)) for _ in range(3))
    out, idx, lse = oracle.forward(Q, K, V, k, 0.7)
    perm = rng.permutation(N)          # new node a holds old node perm[a]
    inv = np.argsort(perm)             # old node j sits at inv[j]
    out2, idx2, lse2 = oracle.forward(Q[perm], K[perm], V[perm], k, 0.7)
    np.testing.assert_allclose(out2, out[perm], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(lse2, lse[perm], rtol=1e-13)
    for a in range(N):
        for h in range(H):
            assert set(idx2[a, h].tolist()) == set(inv[idx[perm[a], h]].tolist())


def test_block_diagonal_equals_separate_graphs():
    rng = np.random.default_rng(4)
    sizes = [13, 0, 1, 21, 8]
    N, H, d, k = sum(sizes), 2, 3, 5
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    Q, K, V = (rng.standard_normal((N, H, d)) for _ in range(3))
    out, idx, lse = oracle.forward(Q, K, V, k, 0.4, offsets=offsets)
    for (lo, hi) in _graphs(offsets, N):
        if hi == lo:
            continue
        o, ix, l = oracle.forward(Q[lo:hi], K[lo:hi], V[lo:hi], k, 0.4)
        np.testing.assert_allclose(out[lo:hi], o, rtol=0, atol=0)
        np.testing.assert_allclose(lse[lo:hi], l, rtol=0, atol=0)
        shifted = np.where(ix >= 0, ix + lo, -1)
        np.testing.assert_array_equal(idx[lo:hi], shifted)
        valid = idx[lo:hi][idx[lo:hi] >= 0]
        assert valid.min() >= lo and valid.max() < hi


def test_selection_invariances():
    rng = np.random.default_rng(9)
    N, H, d, k = 30, 2, 3, 4
    Q = _int_inputs(rng, N, H, d, -3, 3)
    K = _int_inputs(rng, N, H, d, -3, 3)
    _, idx, _ = oracle.forward(Q, K, Q, k, 1.0)
    # positive rescaling of Q and of K
    _, idx_a, _ = oracle.forward(3 * Q, 2 * K, Q, k, 1.0)
    np.testing.assert_array_equal(idx_a, idx)
    # K -> K + c adds q_i . c to every score of query i: the set cannot change
    c = rng.integers(-2, 3, size=(1, H, d)).astype(np.float64)
    _, idx_b, _ = oracle.forward(Q, K + c, Q, k, 1.0)
    np.testing.assert_array_equal(idx_b, idx)


def test_weights_sum_to_one_and_value_shift():
    rng = np.random.default_rng(12)
    N, H, d, k = 40, 2, 4, 6
    Q, K, V = (rng.standard_normal((N, H, d)) for _ in range(3))
    out1, idx, _ = oracle.forward(Q, K, np.ones_like(V), k, 0.5)
    np.testing.assert_allclose(out1, 1.0, rtol=0, atol=1e-14)
    out, _, _ = oracle.forward(Q, K, V, k, 0.5)
    c = rng.standard_normal((1, H, d))
    out_c, _, _ = oracle.forward(Q, K, V + c, k, 0.5)
    np.testing.assert_allclose(out_c, out + c, rtol=1e-13, atol=1e-13)
    # convex hull of the selected value rows, per coordinate
    for i in range(N):
        for h in range(H):
            rows = V[idx[i, h], h, :]
            assert (out[i, h] >= rows.min(axis=0) - 1e-13).all()
            assert (out[i, h] <= rows.max(axis=0) + 1e-13).all()


def test_hardmax_limit():
    rng = np.random.default_rng(13)
    N, H, d, k = 25, 1, 4, 5
    Q, K, V = (rng.standard_normal((N, H, d)) for _ in range(3))
    S = Q[:, 0, :] @ K[:, 0, :].T
    srt = np.sort(S, axis=1)
    gap = (srt[:, -1] - srt[:, -2]).min()
    lam = 60.0 / gap   # exp(-60) ~ 1e-26 leak from the runner-up
    out, idx, lse = oracle.forward(Q, K, V, k, lam)
    am = np.argmax(S, axis=1)
    np.testing.assert_allclose(out[:, 0, :], V[am, 0, :], rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse[:, 0], lam * S[np.arange(N), am], rtol=1e-12)


def test_gradient_invariants():
    rng = np.random.default_rng(14)
    sizes = [11, 17]
    N, H, d, k = sum(sizes), 2, 4, 5
    offsets = np.array([0, 11, 28], np.int32)
    Q, K, V, dO = (rng.standard_normal((N, H, d)) for _ in range(4))
    _, idx, _ = oracle.forward(Q, K, V, k, 0.6, offsets=offsets)
    dQ, dK, dV = oracle.backward(Q, K, V, dO, idx, 0.6)
    for (lo, hi) in _graphs(offsets, N):
        # shifting all keys of a graph by c shifts each query's scores by a constant
        np.testing.assert_allclose(dK[lo:hi].sum(axis=0), 0.0, atol=1e-12)
        # the weights of every query sum to one
        np.testing.assert_allclose(dV[lo:hi].sum(axis=0), dO[lo:hi].sum(axis=0), atol=1e-12)
        # Q -> tQ, K -> K/t leaves every score unchanged
        for h in range(H):
            a = (dQ[lo:hi, h] * Q[lo:hi, h]).sum()
            b = (dK[lo:hi, h] * K[lo:hi, h]).sum()
            assert abs(a - b) < 1e-11


def test_check_set_detects_bad_sets():
    rng = np.random.default_rng(15)
    N, H, d, k = 20, 1, 3, 4
    Q, K = (rng.standard_normal((N, H, d)) for _ in range(2))
    idx, sc, nxt = oracle.topk(Q, K, k)
    mn, mx, fl = oracle.check_set(Q, K, idx)
    assert (fl == 0).all()
    np.testing.assert_allclose(mn, sc[:, -1], rtol=0, atol=0)
    np.testing.assert_allclose(mx, nxt, rtol=0, atol=0)
    bad = idx.copy()
    bad[0, 1] = bad[0, 0]           # duplicate
    bad[1, 0] = -1                  # pad before a valid entry, and a short set
    bad[2, 0] = N + 3               # outside the graph
    _, _, fl = oracle.check_set(Q, K, bad)
    assert fl[0] & 2 and fl[0] & 4
    assert fl[1] & 8 and fl[1] & 4
    assert fl[2] & 1


# ---- value rows of another width than the query/key rows (Section 3.1:
# W_Q, W_K map to d_K dimensions, W_V to d_V) ----

@pytest.mark.parametrize("d,dv", [(4, 7), (6, 2)])
def test_value_width_k_equals_n_is_softmax_attention(d, dv):
    rng = np.random.default_rng(d * 10 + dv)
    sizes = [5, 9, 1, 12]
    N, H = sum(sizes), 2
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    Q, K = (rng.standard_normal((N, H, d)) for _ in range(2))
    V = rng.standard_normal((N, H, dv))
    out, idx, lse = oracle.forward(Q, K, V, max(sizes), 0.45, offsets=offsets)
    assert out.shape == (N, H, dv)
    want_out, want_lse = _sdpa_per_graph(Q, K, V, offsets, 0.45)
    np.testing.assert_allclose(out, want_out, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, want_lse, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("d,dv", [(5, 3), (3, 8)])
def test_value_width_masked_dense_and_autograd(d, dv):
    rng = np.random.default_rng(300 + d + dv)
    N, H, k = 31, 2, 6
    Qn, Kn = (rng.standard_normal((N, H, d)) for _ in range(2))
    Vn, dOn = (rng.standard_normal((N, H, dv)) for _ in range(2))
    scale = 0.7
    out, idx, lse = oracle.forward(Qn, Kn, Vn, k, scale)
    dQ, dK, dV = oracle.backward(Qn, Kn, Vn, dOn, idx, scale)
    assert dQ.shape == dK.shape == (N, H, d) and dV.shape == (N, H, dv)
    Q, K, V = (torch.from_numpy(x).clone().requires_grad_(True) for x in (Qn, Kn, Vn))
    want_out, want_lse, top = _masked_dense_torch(Q, K, V, k, scale)
    np.testing.assert_allclose(out, want_out.detach().numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, want_lse.detach().numpy(), rtol=1e-12, atol=1e-12)
    (want_out * torch.from_numpy(dOn)).sum().backward()
    np.testing.assert_allclose(dQ, Q.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dK, K.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dV, V.grad.numpy(), rtol=1e-11, atol=1e-12)


def test_value_width_backward_finite_differences():
    rng = np.random.default_rng(21)
    N, H, d, dv, k = 12, 1, 3, 5, 3
    offsets = np.array([0, 5, 12], np.int32)
    Q, K = (rng.standard_normal((N, H, d)) for _ in range(2))
    V, dO = (rng.standard_normal((N, H, dv)) for _ in range(2))
    scale = 0.9
    _, idx, _ = oracle.forward(Q, K, V, k, scale, offsets=offsets)
    dQ, dK, dV = oracle.backward(Q, K, V, dO, idx, scale)
    eps = 1e-6
    for name, X, G in (("Q", Q, dQ), ("K", K, dK), ("V", V, dV)):
        num = np.zeros_like(X)
        for pos in np.ndindex(X.shape):
            args = [{"Q": Q, "K": K, "V": V} for _ in range(2)]
            for a, sgn in zip(args, (1.0, -1.0)):
                Xs = X.copy()
                Xs[pos] += sgn * eps
                a[name] = Xs
            num[pos] = (_loss(args[0]["Q"], args[0]["K"], args[0]["V"], dO, k, scale, offsets)
                        - _loss(args[1]["Q"], args[1]["K"], args[1]["V"], dO, k, scale, offsets)) / (2 * eps)
        np.testing.assert_allclose(G, num, rtol=1e-6, atol=1e-7, err_msg=name)


def test_value_columns_split_and_gradient_invariants():
    # out and dV are linear in the value columns: splitting V (and dO) into
    # column blocks gives the column blocks of the full result, while dQ and
    # dK add up over the blocks (dp sums over the value dimensions)
    rng = np.random.default_rng(22)
    N, H, d, dv, k = 26, 2, 4, 9, 5
    offsets = np.array([0, 10, 26], np.int32)
    Q, K = (rng.standard_normal((N, H, d)) for _ in range(2))
    V, dO = (rng.standard_normal((N, H, dv)) for _ in range(2))
    out, idx, _ = oracle.forward(Q, K, V, k, 0.6, offsets=offsets)
    dQ, dK, dV = oracle.backward(Q, K, V, dO, idx, 0.6)
    parts = [(0, 4), (4, 9)]
    sq = np.zeros_like(dQ)
    sk = np.zeros_like(dK)
    for a, b in parts:
        o, ix, _ = oracle.forward(Q, K, V[:, :, a:b], k, 0.6, offsets=offsets)
        np.testing.assert_array_equal(ix, idx)
        np.testing.assert_allclose(o, out[:, :, a:b], rtol=1e-13, atol=1e-13)
        pq, pk, pv = oracle.backward(Q, K, V[:, :, a:b], dO[:, :, a:b], idx, 0.6)
        np.testing.assert_allclose(pv, dV[:, :, a:b], rtol=1e-13, atol=1e-13)
        sq += pq
        sk += pk
    np.testing.assert_allclose(sq, dQ, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(sk, dK, rtol=1e-11, atol=1e-12)
    for (lo, hi) in _graphs(offsets, N):
        np.testing.assert_allclose(dK[lo:hi].sum(axis=0), 0.0, atol=1e-12)
        np.testing.assert_allclose(dV[lo:hi].sum(axis=0), dO[lo:hi].sum(axis=0), atol=1e-12)


# ---- attention dropout (inverted dropout on the kept weights, the keep
# draws given) ----

def _dropout_dense_torch(Q, K, V, k, scale, keep_dense, rate):
    """Top-k masked dense attention with dropout on its weights, from torch
    primitives: A = softmax(scale S + mask), out = (A * keep / (1 - rate)) V."""
    q = Q.permute(1, 0, 2)
    kk = K.permute(1, 0, 2)
    v = V.permute(1, 0, 2).contiguous()
    S = torch.matmul(q, kk.transpose(1, 2).contiguous())
    top = torch.topk(S, k, dim=-1).indices
    mask = torch.full_like(S, float("-inf"))
    mask.scatter_(-1, top, 0.0)
    A = torch.softmax(scale * S + mask, dim=-1)
    out = torch.matmul(A * keep_dense / (1.0 - rate), v).permute(1, 0, 2)
    return out


def _dense_keep(idx, keep, N):
    """The per-slot keep draws [N, H, k] scattered onto the dense [H, N, N] grid."""
    Nq, H, k = idx.shape
    dense = np.zeros((H, Nq, N))
    for i in range(Nq):
        for h in range(H):
            for t in range(k):
                if idx[i, h, t] >= 0:
                    dense[h, i, idx[i, h, t]] = keep[i, h, t]
    return torch.from_numpy(dense)


@pytest.mark.parametrize("d,dv,rate", [(4, 4, 0.5), (3, 6, 0.25)])
def test_dropout_matches_torch_autograd(d, dv, rate):
    rng = np.random.default_rng(400 + d + dv)
    N, H, k = 23, 2, 6
    Qn, Kn = (rng.standard_normal((N, H, d)) for _ in range(2))
    Vn, dOn = (rng.standard_normal((N, H, dv)) for _ in range(2))
    scale = 0.7
    _, idx, _ = oracle.forward(Qn, Kn, Vn, k, scale)
    keep = (rng.random((N, H, k)) >= rate).astype(np.uint8)
    out, lse = oracle.attend(Qn, Kn, Vn, idx, scale, keep=keep, drop_rate=rate)
    dQ, dK, dV = oracle.backward(Qn, Kn, Vn, dOn, idx, scale, keep=keep, drop_rate=rate)
    Q, K, V = (torch.from_numpy(x).clone().requires_grad_(True) for x in (Qn, Kn, Vn))
    want = _dropout_dense_torch(Q, K, V, k, scale, _dense_keep(idx, keep, N), rate)
    np.testing.assert_allclose(out, want.detach().numpy().reshape(N * H, dv), rtol=1e-12, atol=1e-12)
    # lse is that of the weights before dropout
    _, lse0 = oracle.attend(Qn, Kn, Vn, idx, scale)
    np.testing.assert_array_equal(lse, lse0)
    (want * torch.from_numpy(dOn)).sum().backward()
    np.testing.assert_allclose(dQ, Q.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dK, K.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dV, V.grad.numpy(), rtol=1e-11, atol=1e-12)


def test_dropout_keep_all_is_no_dropout_and_finite_differences():
    rng = np.random.default_rng(31)
    N, H, d, k, rate = 11, 1, 3, 4, 0.3
    Q, K, V, dO = (rng.standard_normal((N, H, d)) for _ in range(4))
    _, idx, _ = oracle.forward(Q, K, V, k, 0.8)
    ones = np.ones((N, H, k), np.uint8)
    np.testing.assert_array_equal(oracle.attend(Q, K, V, idx, 0.8, keep=ones)[0], oracle.attend(Q, K, V, idx, 0.8)[0])
    for a, b in zip(oracle.backward(Q, K, V, dO, idx, 0.8, keep=ones), oracle.backward(Q, K, V, dO, idx, 0.8)):
        np.testing.assert_array_equal(a, b)
    keep = (rng.random((N, H, k)) >= rate).astype(np.uint8)
    dQ, dK, dV = oracle.backward(Q, K, V, dO, idx, 0.8, keep=keep, drop_rate=rate)

    def loss(xs):
        # the index set and the draws held fixed, as in the backward
        o, _ = oracle.attend(xs["Q"], xs["K"], xs["V"], idx, 0.8, keep=keep, drop_rate=rate)
        return float((o.reshape(N, H, d) * dO).sum())

    eps = 1e-6
    for name, X, G in (("Q", Q, dQ), ("K", K, dK), ("V", V, dV)):
        num = np.zeros_like(X)
        for pos in np.ndindex(X.shape):
            vals = []
            for sgn in (1.0, -1.0):
                xs = {"Q": Q, "K": K, "V": V}
                xs[name] = X.copy()
                xs[name][pos] += sgn * eps
                vals.append(loss(xs))
            num[pos] = (vals[0] - vals[1]) / (2 * eps)
        np.testing.assert_allclose(G, num, rtol=1e-6, atol=1e-7, err_msg=name)
