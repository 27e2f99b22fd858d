"""Attention-entropy layer score for capacity allocation (Section 3.3).

Test infrastructure only (see the package docstring).

The paper scores layer l by H_l, the expectation over calibration sequences,
heads and queries of the Shannon entropy of the full (uncompressed) attention
row of each query; entropy allocation then feeds H_l through the identity
transform into Eq. 3 with b_min = 32.

Readings taken where the paper is silent:
  * the row of the query at position t is the causal softmax of
    q_t . k_j / sqrt(d) over keys j = 0..t, per query head; query head hq reads
    KV head hq // G (as in the prefill rules);
  * entropy in natural-log units (nats);
  * the expectation is the plain mean over sequences, query heads and the
    profiled query positions; the profiled positions are the last n_q positions
    of each calibration sequence (n_q = L: every query).
"""
from __future__ import annotations

import numpy as np

from .prefill import bf16_to_f64


def row_entropies(q_bits, k_bits) -> np.ndarray:
    """Entropy (nats) of every profiled query row of one sequence and layer.

    q_bits: bf16 bits [Hq, n_q, d] for positions L - n_q .. L - 1; k_bits: bf16 bits [Hkv, L, d].
    Returns float64 [Hq, n_q].
    """
    q = bf16_to_f64(q_bits)
    k = bf16_to_f64(k_bits)
    Hq, n_q, d = q.shape
    Hkv, L, _ = k.shape
    G = Hq // Hkv
    out = np.empty((Hq, n_q))
    for hq in range(Hq):
        kh = k[hq // G]
        z = (q[hq] @ kh.T) / np.sqrt(d)                  # [n_q, L]
        for i in range(n_q):
            t = L - n_q + i
            row = z[i, :t + 1]
            p = np.exp(row - row.max())
            p /= p.sum()
            nz = p[p > 0]
            out[hq, i] = -np.sum(nz * np.log(nz))
    return out


def layer_score(q_list, k_list) -> float:
    """H_l: mean row entropy over the calibration sequences (lists of per-sequence arrays)."""
    return float(np.mean([row_entropies(q, k) for q, k in zip(q_list, k_list)]))
