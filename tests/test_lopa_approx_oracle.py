"""Pins of the LoPA-approximation oracle (CPU only): facts that hold independently of it.

* exact recovery of a planted M + rank-r product (the error reaches 0 and M, U V come back);
* the error never rises from one half step to the next (each step solves its subproblem);
* the M step against brute force over every position and sign of a row;
* the UV step reaches the Eckart-Young bound: no rank-r matrix from a perturbed SVD, or
  from a projection onto random subspaces, does better;
* a rank-deficient W - M is reproduced exactly.
"""
import itertools

import numpy as np
import pytest

from oracle import lopa_approx as la


def planted(seed, H, D, r, small=0.05):
    rng = np.random.default_rng(seed)
    idx = rng.integers(0, D, size=H).astype(np.int32)
    sgn = np.where(rng.random(H) < 0.5, -1, 1).astype(np.int8)
    U = rng.standard_normal((H, r)) * small
    V = rng.standard_normal((r, D)) * small
    return la.dense_m(idx, sgn, D) + U @ V, idx, sgn, U @ V


@pytest.mark.parametrize("H,D,r", [(40, 24, 3), (64, 32, 8), (30, 30, 1)])
def test_planted_exact_recovery(H, D, r):
    W, idx, sgn, UV = planted(1, H, D, r)
    res = la.lopa_approx(W, r)
    assert np.array_equal(res.g_idx, idx) and np.array_equal(res.g_sign, sgn)
    assert np.allclose(res.U @ res.V, UV, atol=1e-12)
    assert res.history[-1] < 1e-20
    assert res.iters <= 2


@pytest.mark.parametrize("seed", [2, 3, 4])
def test_error_never_rises(seed):
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((80, 48))
    res = la.lopa_approx(W, 6, max_iters=30)
    h = np.array(res.history)
    assert np.all(np.diff(h) <= 1e-9 * h[:-1]), h
    assert res.iters >= 1
    # stopped because M stood still (or hit the cap)
    assert res.iters < 30 or h[-1] == h[-2]


def test_m_step_is_optimal_by_brute_force():
    rng = np.random.default_rng(5)
    R = rng.standard_normal((6, 5))
    R[2, 1] = R[2, 3] = 4.0          # a tie: the lower column wins
    R[3, :] = 0.0                    # a zero row: column 0, sign +1
    idx, sgn = la.m_step(R)
    for i in range(R.shape[0]):
        best = min(np.sum((R[i] - s * np.eye(5)[j]) ** 2) for j, s in itertools.product(range(5), (1, -1)))
        got = np.sum((R[i] - sgn[i] * np.eye(5)[idx[i]]) ** 2)
        assert got == pytest.approx(best)
    assert idx[2] == 1 and sgn[2] == 1 and idx[3] == 0 and sgn[3] == 1


def test_uv_step_reaches_the_eckart_young_bound():
    rng = np.random.default_rng(6)
    A = rng.standard_normal((50, 30))
    r = 5
    U, V = la.truncated_svd(A, r)
    best = np.sum((A - U @ V) ** 2)
    for _ in range(20):   # projections onto other rank-r subspaces do worse
        Q, _ = np.linalg.qr(rng.standard_normal((30, r)))
        P = A @ Q @ Q.T
        assert np.sum((A - P) ** 2) >= best - 1e-9
    # the bound itself: the sum of the discarded squared singular values
    s = np.linalg.svd(A, compute_uv=False)
    assert best == pytest.approx(np.sum(s[r:] ** 2))


def test_rank_deficient_residual():
    W, idx, sgn, UV = planted(7, 36, 20, 2, small=0.1)
    res = la.lopa_approx(W, 4)      # r above the planted rank: the extra directions are zero
    assert res.history[-1] < 1e-20
    assert np.allclose(res.U @ res.V, UV, atol=1e-12)


def test_bad_rank():
    with pytest.raises(ValueError):
        la.lopa_approx(np.zeros((4, 3)), 4)


@pytest.mark.parametrize("seed", [8, 9])
def test_factor_convention(seed):
    """The factors' convention (reading: U carries the singular values): V has orthonormal
    rows, U = (W - M) V^T, and U's columns are orthogonal with norms equal to the top r
    singular values of W - M, largest first.  Moving the singular values onto V fails the
    first two; a transposed or unsorted V fails the last."""
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((60, 36))
    r = 7
    res = la.lopa_approx(W, r)
    R = W - la.dense_m(res.g_idx, res.g_sign, W.shape[1])
    assert np.allclose(res.V @ res.V.T, np.eye(r), atol=1e-12)
    assert np.allclose(res.U, R @ res.V.T, atol=1e-12)
    s = np.linalg.svd(R, compute_uv=False)
    gram = res.U.T @ res.U
    assert np.allclose(gram, np.diag(s[:r] ** 2), atol=1e-9 * s[0] ** 2)
