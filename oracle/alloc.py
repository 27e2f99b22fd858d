"""Fixed-total per-layer capacity allocation (Section 3.3, Eq. 3).

Test infrastructure only (see the package docstring).

Steps, in the paper's order:
  1. transform the layer score: identity for attention entropy, a cap at the
     across-layer 95th percentile for PPL degradation;
  2. if the smallest transformed value is not positive, shift every value by
     (-min + 1e-6);
  3. normalise to weights w_l and form the provisional budgets B * w_l (Eq. 3);
  4. repeatedly fix layers whose provisional budget falls below b_min at b_min
     and share the remaining total among the other layers by weight;
  5. round to integers: floor, then hand the residual units to the largest
     fractional remainders (the same vector as nearest-integer rounding with the
     residual assigned by fractional remainder, up to ties).
Readings: equal remainders go to the lower layer index; the percentile is the
linear-interpolation one.
"""
from __future__ import annotations

import numpy as np

IDENTITY = 0
PPL_CAP = 1


def transform(scores, kind: int = IDENTITY) -> np.ndarray:
    """T(s): identity, or min(s, Q_0.95(s)) with linear-interpolation percentile."""
    s = np.asarray(scores, dtype=np.float64)
    if kind == IDENTITY:
        return s.copy()
    if kind == PPL_CAP:
        return np.minimum(s, np.percentile(s, 95.0))
    raise ValueError("unknown transform")


def shift_nonpositive(t) -> np.ndarray:
    """If min t <= 0, shift every value by (-min t + 1e-6)."""
    t = np.asarray(t, dtype=np.float64)
    if t.min() <= 0.0:
        t = t - t.min() + 1e-6
    return t


def clamped_shares(weights, total: float, b_min: float) -> np.ndarray:
    """Provisional real-valued budgets of Eq. 3 with the iterative b_min clamp."""
    w = np.asarray(weights, dtype=np.float64)
    n = w.size
    fixed = np.zeros(n, dtype=bool)
    share = np.zeros(n)
    while True:
        free = ~fixed
        remaining = total - b_min * fixed.sum()
        share[free] = remaining * w[free] / w[free].sum()
        share[fixed] = b_min
        newly = free & (share < b_min)
        if not newly.any():
            return share
        fixed |= newly


def largest_remainder(share, total: int) -> np.ndarray:
    """Floor, then +1 to the (total - sum floor) largest fractional parts (ties: lower index)."""
    share = np.asarray(share, dtype=np.float64)
    base = np.floor(share).astype(np.int64)
    frac = share - base
    residual = int(total - base.sum())
    order = sorted(range(share.size), key=lambda i: (-frac[i], i))
    for i in order[:residual]:
        base[i] += 1
    return base


def allocate(weights, total: int, b_min: int) -> np.ndarray:
    """Integer budgets with sum == total and every budget >= b_min (steps 3-5)."""
    w = np.asarray(weights, dtype=np.float64)
    if w.size * b_min > total:
        raise ValueError("total below n_layers * b_min")
    if (w <= 0).any():
        raise ValueError("weights must be positive (apply the shift first)")
    return largest_remainder(clamped_shares(w, float(total), float(b_min)), int(total))


def allocate_from_scores(scores, kind: int, total: int, b_min: int) -> np.ndarray:
    """Steps 1-5 from raw layer scores."""
    return allocate(shift_nonpositive(transform(scores, kind)), total, b_min)


def compacted_kv_bytes(budgets, n_kv_heads: int, head_dim: int, elem_bytes: int) -> int:
    """Bytes of retained K and V for one sequence: sum_l b_l * Hkv * d * 2 (K and V) * elem."""
    return int(np.sum(budgets)) * n_kv_heads * head_dim * 2 * elem_bytes
