"""Reference oracle of the LoPA approximation (test infrastructure, not product).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import this module.  It shares nothing with the GPU library.

What it computes (Section 3.3, "LoPA approximation"): for a gate matrix W (H x D) and a
rank r, an approximation W ~ M + U V with M in C (one nonzero per row, +1 or -1, the
fixed term G of Eq. (lopaapprox)), U (H x r) and V (r x D), by alternating minimization
of the squared Frobenius error ||W - M - U V||^2:

* M step (U, V fixed): each row of M holds the sign of the largest-magnitude entry of
  that row of W - U V, at that entry's column (for one +-1 per row this minimizes the
  row's error: ||R_i - s e_j||^2 = ||R_i||^2 - 2 s R_ij + 1);
* UV step (M fixed): U V is the rank-r truncated SVD of W - M (Eckart-Young);
* start from U = V = 0 with an M step; stop when an M step leaves M unchanged (C is
  finite and no step raises the error, so this happens after finitely many steps) or
  after max_iters UV steps.

Readings (the paper does not fix them): among equal magnitudes the lowest column wins,
and a zero entry gets the sign +1; U carries the singular values (U = left vectors
scaled by them, V = right vectors), the largest first.

Plain fp64 numpy; the SVD is numpy's (LAPACK), used as one step.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass
class ApproxResult:
    g_idx: np.ndarray      # [H] int32, M's column per row
    g_sign: np.ndarray     # [H] int8, M's value per row (+1 / -1)
    U: np.ndarray          # [H, r] fp64 (LoPA's B)
    V: np.ndarray          # [r, D] fp64 (LoPA's A)
    iters: int             # UV steps taken
    history: list = field(default_factory=list)  # the error after every half step, in order


def m_step(R: np.ndarray):
    """The optimal one-+-1-per-row M for the residual R = W - U V."""
    j = np.argmax(np.abs(R), axis=1)              # first index among ties
    v = R[np.arange(R.shape[0]), j]
    s = np.where(v >= 0, 1, -1).astype(np.int8)
    return j.astype(np.int32), s


def dense_m(g_idx, g_sign, D):
    M = np.zeros((len(g_idx), D))
    M[np.arange(len(g_idx)), g_idx] = g_sign
    return M


def error(W, g_idx, g_sign, UV):
    """||W - M - U V||_F^2."""
    return float(np.sum((W - dense_m(g_idx, g_sign, W.shape[1]) - UV) ** 2))


def truncated_svd(A: np.ndarray, r: int):
    """The rank-r truncated SVD of A as (U scaled by the singular values, V)."""
    Uf, s, Vt = np.linalg.svd(A, full_matrices=False)
    return Uf[:, :r] * s[:r], Vt[:r]


def lopa_approx(W, r: int, max_iters: int = 20) -> ApproxResult:
    W = np.asarray(W, np.float64)
    H, D = W.shape
    if not (1 <= r <= min(H, D)):
        raise ValueError("need 1 <= r <= min(H, D)")
    UV = np.zeros_like(W)
    g_idx, g_sign = m_step(W - UV)                 # U = V = 0: M first
    hist = [error(W, g_idx, g_sign, UV)]
    U = np.zeros((H, r))
    V = np.zeros((r, D))
    it = 0
    while it < max_iters:
        U, V = truncated_svd(W - dense_m(g_idx, g_sign, D), r)
        UV = U @ V
        it += 1
        hist.append(error(W, g_idx, g_sign, UV))
        ni, ns = m_step(W - UV)
        hist.append(error(W, ni, ns, UV))
        if np.array_equal(ni, g_idx) and np.array_equal(ns, g_sign):
            break
        g_idx, g_sign = ni, ns
    return ApproxResult(g_idx=g_idx, g_sign=g_sign, U=U, V=V, iters=it, history=hist)
