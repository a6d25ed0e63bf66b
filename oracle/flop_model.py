"""The paper's FLOP cost model, in closed form (test infrastructure, not product).

Each function restates one formula of the paper; counts are multiply-adds per token.

* Section 3.1, Eq. (flops_ratio): a dense gated FFN costs 3HD; with standard gating
  and sparsity s the gate still costs HD and each of the other two matrices costs
  (1 - s)HD, so FLOP-ratio = 3 / (3 - 2s).
* Section 3.3, "Adaptive hidden dimension": with LoPA of rank r the hidden size that
  keeps the parameter count at 3HD is H' = D(3H - r) / (r + 2D).
* Section 3.3, "FLOP-ratio for LoPA": ignoring the fixed matrix G, the gate costs
  r(D + H') and the other two (1 - s)DH' each.
* Section 3.4, architecture casting: the hidden size is not adapted (H' = H), while the
  baseline stays the dense 3HD.
"""
from __future__ import annotations


def standard_cost(D: int, H: int, n_active: float) -> float:
    """Multiply-adds of the sparse method with standard gating: HD for W1, n*D for each of W3, W2."""
    return H * D + 2 * n_active * D


def lopa_cost(D: int, H: int, r: int, n_active: float) -> float:
    """Multiply-adds with LoPA gating (G omitted): r(D + H) for V then U, n*D for each of W3, W2."""
    return r * (D + H) + 2 * n_active * D


def dense_cost(D: int, H: int) -> float:
    """Multiply-adds of the dense gated FFN: three H x D products."""
    return 3 * H * D


def flop_ratio_standard(s: float) -> float:
    """Eq. (flops_ratio) with standard gating: 3 / (3 - 2s)."""
    return 3.0 / (3.0 - 2.0 * s)


def lopa_hidden_dim(D: float, H: float, r: float) -> float:
    """H' that keeps r(H' + D) + 2H'D equal to 3HD."""
    return D * (3.0 * H - r) / (r + 2.0 * D)


def flop_ratio_lopa(D: float, Hp: float, r: float, s: float) -> float:
    """LoPA FLOP-ratio at hidden size H' (Section 3.3): (r(D+H') + 2DH') / (r(D+H') + 2(1-s)DH')."""
    gate = r * (D + Hp)
    return (gate + 2.0 * D * Hp) / (gate + 2.0 * (1.0 - s) * D * Hp)


def flop_ratio_lopa_cast(D: float, H: float, alpha: float, s: float) -> float:
    """LoPA casting: rank r = alpha*D, hidden size adapted to H' so the numerator is 3HD."""
    r = alpha * D
    return flop_ratio_lopa(D, lopa_hidden_dim(D, H, r), r, s)


def flop_ratio_arch_cast(D: float, H: float, r: float, s: float) -> float:
    """Architecture casting: W1 replaced by rank-r LoPA at the original H, against the dense 3HD."""
    return 3.0 * H * D / (r * (D + H) + 2.0 * (1.0 - s) * D * H)
