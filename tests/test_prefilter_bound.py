"""The bound behind the int8 prefilter, checked on the CPU (no GPU).

The prefilter (kmip_topk_prefilter) keeps, per query, every key whose exact
int8 score I_j = q8 . k8_j reaches T = M - ceil(2 (E + delta) / (s_q s_K)),
where M is the k-th largest of 64 group maxima of I and E = |q| e_max +
e_q n_max bounds the quantisation error (Cauchy-Schwarz).  The claim is
recall 1: every key that scores at least the query's k-th best score (ties
included) is kept.  This file states the rule in float64 / exact integers
from that description and checks the claim against the exact top-k of the
bf16 inputs on random, clustered and adversarial data (keys placed half a
quantisation step off the grid, where rounding errs most), with delta = 0:
the float64 scores here are exact, so the fp32 term is not needed.
"""
import math

import numpy as np
import pytest


def pow2_scale(m):
    """Smallest power of two s with m / s <= 127 (1 for m = 0)."""
    if m <= 0:
        return 1.0
    return 2.0 ** math.ceil(math.log2(m / 127.0))


def bf16(x):
    x = np.ascontiguousarray(x, np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint32) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def candidates(Q, K, k):
    """Candidate mask [nq, n] of the prefilter rule for one head."""
    sK = pow2_scale(np.abs(K).max())
    k8 = np.clip(np.rint(K / sK), -127, 127)
    e = np.linalg.norm(K - sK * k8, axis=1)
    nk = np.linalg.norm(sK * k8, axis=1)
    n = K.shape[0]
    groups = (np.arange(n) // 32 % 2) * 32 + np.arange(n) % 32
    out = np.zeros((Q.shape[0], n), bool)
    for i, q in enumerate(Q):
        sq = pow2_scale(np.abs(q).max())
        q8 = np.clip(np.rint(q / sq), -127, 127)
        eq = np.linalg.norm(q - sq * q8)
        E = np.linalg.norm(q) * e.max() + eq * nk.max()
        I = (k8 @ q8).astype(np.int64)
        gmax = np.full(64, np.iinfo(np.int64).min)
        np.maximum.at(gmax, groups, I)
        M = np.sort(gmax)[::-1][k - 1]
        T = M - math.ceil(2 * E / (sq * sK)) if M > np.iinfo(np.int64).min else np.iinfo(np.int64).min
        out[i] = I >= T
    return out


def assert_recall_one(Q, K, k):
    cand = candidates(Q, K, k)
    S = Q @ K.T
    kth = np.sort(S, axis=1)[:, ::-1][:, k - 1]
    must = S >= kth[:, None]
    missed = must & ~cand
    assert not missed.any(), f"{int(missed.sum())} keys of an exact top-k not kept"
    return cand.sum(axis=1)


@pytest.mark.parametrize("d,k", [(16, 1), (16, 32), (32, 8), (64, 32), (128, 16)])
def test_recall_one_gaussian(d, k):
    rng = np.random.default_rng(d + k)
    Q = bf16(rng.standard_normal((40, d)))
    K = bf16(rng.standard_normal((3000, d)))
    kept = assert_recall_one(Q, K, k)
    # the bound is useful: far fewer than all keys survive
    assert np.median(kept) < 3000 / 4


def test_recall_one_clustered_and_scaled():
    rng = np.random.default_rng(1)
    d, k = 32, 32
    mu = rng.standard_normal((16, d)) * 4.0
    K = bf16(mu[rng.integers(0, 16, 4000)] + 0.05 * rng.standard_normal((4000, d)))
    Q = bf16(mu[rng.integers(0, 16, 30)] * rng.uniform(0.01, 100.0, (30, 1)))
    assert_recall_one(Q, K, k)


def test_recall_one_adversarial_rounding():
    # Keys half a quantisation step off the grid in every dimension, and a
    # query that lines up with the rounding errors; plus near-ties at the
    # k-th best score.
    rng = np.random.default_rng(2)
    d, k = 16, 8
    sK = pow2_scale(127.0)
    base = rng.integers(-100, 100, size=(2000, d)).astype(np.float64)
    K = bf16((base + 0.5) * sK)
    K[:50] = K[50]                       # exact ties
    Q = bf16(np.vstack([np.sign(rng.standard_normal((10, d))) * 0.75,
                        rng.standard_normal((10, d))]))
    assert_recall_one(Q, K, k)


def test_rule_breaks_without_the_bound():
    # The same rule with the error term dropped loses keys of the exact top-k
    # on off-grid data: the bound is what makes the recall 1.
    rng = np.random.default_rng(3)
    d, k = 16, 32
    Q = bf16(rng.standard_normal((200, d)))
    K = bf16(rng.standard_normal((4000, d)) * 1e-2 + 0.3)
    sK = pow2_scale(np.abs(K).max())
    k8 = np.clip(np.rint(K / sK), -127, 127)
    S = Q @ K.T
    kth = np.sort(S, axis=1)[:, ::-1][:, k - 1]
    lost = 0
    for i, q in enumerate(Q):
        sq = pow2_scale(np.abs(q).max())
        I = k8 @ np.clip(np.rint(q / sq), -127, 127)
        lost += int(((S[i] >= kth[i]) & (I < np.sort(I)[::-1][k - 1])).sum())
    assert lost > 0
