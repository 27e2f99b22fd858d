"""Helpers shared by the GPU parity tests: run the HIP path and the oracle on the same seeded
bf16 inputs and apply the acceptance rule.

Acceptance (per sequence, layer, KV head):
  * scores: |S_gpu - S_oracle| <= 1e-3 * |S_oracle| (+1e-30) on the candidate range;
  * retained set: n_keep distinct ascending positions in [0, L); the forced part (window,
    recent tail, sinks) identical; outside the ambiguity band {j : |S_oracle[j] - tau| <=
    1e-3 * tau} around the oracle's k-th score tau, the selected positions identical;
  * gathered K / V rows bitwise equal to the input rows at the GPU's positions.
"""
from __future__ import annotations

import numpy as np

from oracle import prefill as OP

RTOL = 1e-3
ATOL = 1e-30


def bits_to_torch(bits, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(torch.bfloat16)


def torch_to_bits(t):
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def check_scores(s_gpu, s_ora, what=""):
    s_gpu = np.asarray(s_gpu, dtype=np.float64)
    err = np.abs(s_gpu - s_ora)
    bad = err > RTOL * np.abs(s_ora) + ATOL
    assert not bad.any(), (f"{what}: {bad.sum()} scores outside 1e-3 rel; worst rel "
                           f"{np.max(err / (np.abs(s_ora) + ATOL)):.3e} at {np.argmax(err / (np.abs(s_ora) + ATOL))}")


def check_retained(idx_gpu, ora: dict, h: int, L: int, what=""):
    """Acceptance rule for one KV head.  Returns the number of positions in the ambiguity band."""
    idx_gpu = np.asarray(idx_gpu, dtype=np.int64)
    idx_ora = ora["idx"][h]
    assert idx_gpu.shape == idx_ora.shape, what
    assert (idx_gpu >= 0).all() and (idx_gpu < L).all(), f"{what}: positions out of range"
    assert (np.diff(idx_gpu) > 0).all(), f"{what}: positions not strictly ascending"
    lay = ora["layout"]
    if lay is None:
        assert np.array_equal(idx_gpu, idx_ora), f"{what}: retain-all mismatch"
        return 0
    cand_end, k, lo, hi = lay
    assert np.array_equal(idx_gpu[k:], idx_ora[k:]), f"{what}: forced part differs"
    if ora["scores"] is None or k == 0:
        assert np.array_equal(idx_gpu, idx_ora), f"{what}: closed-form set differs"
        return 0
    tau = np.sort(ora["scores"][h])[::-1][k - 1]
    amb = set(np.flatnonzero(np.abs(ora["scores"][h] - tau) <= RTOL * tau).tolist())
    sel_g = set(idx_gpu[:k].tolist())
    sel_o = set(idx_ora[:k].tolist())
    assert all(j < cand_end for j in sel_g), f"{what}: selected position outside candidates"
    diff = (sel_g ^ sel_o) - amb
    assert not diff, f"{what}: selections differ outside the tie band at {sorted(diff)[:10]}"
    return len(amb)


def check_gather(k_out_bits, v_out_bits, k_bits, v_bits, idx_gpu, what=""):
    assert np.array_equal(k_out_bits, k_bits[idx_gpu]), f"{what}: gathered K differs"
    assert np.array_equal(v_out_bits, v_bits[idx_gpu]), f"{what}: gathered V differs"


def oracle_unpooled(q_bits, k_bits):
    """Unpooled group-mean window score over all positions, [Hkv, L] (seeds decode H2O)."""
    q = OP.bf16_to_f64(q_bits)
    k = OP.bf16_to_f64(k_bits)
    return OP.group_mean(OP.window_scores(q, k), q.shape[0] // k.shape[0])
