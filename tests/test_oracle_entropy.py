"""Pins for the oracle's attention-entropy layer score (Section 3.3)."""
import math

import numpy as np
import pytest

from oracle import entropy as E
from synth import f32_to_bf16_bits


def bits(x):
    return f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def test_zero_queries_give_uniform_rows():
    # q = 0: every visible key has the same logit, so row t has entropy ln(t + 1) exactly
    rng = np.random.default_rng(0)
    Hq, Hkv, L, n_q, d = 4, 2, 37, 11, 16
    q = np.zeros((Hq, n_q, d), dtype=np.uint16)
    k = bits(rng.standard_normal((Hkv, L, d)))
    h = E.row_entropies(q, k)
    expect = np.log(np.arange(L - n_q, L) + 1.0)
    np.testing.assert_allclose(h, np.broadcast_to(expect, (Hq, n_q)), rtol=1e-13)
    assert E.layer_score([q], [k]) == pytest.approx(expect.mean(), rel=1e-13)


def test_two_keys_binary_entropy():
    # L = 2, the query at position 1 sees keys 0 and 1 with logits 0 and 2 (d = 4, 1/sqrt(d) = 1/2)
    d = 4
    q = bits(np.array([[[2.0, 0, 0, 0]]]))
    k = bits(np.array([[[0.0, 0, 0, 0], [2.0, 0, 0, 0]]]))
    p = 1.0 / (1.0 + math.exp(-2.0))
    expect = -(p * math.log(p) + (1 - p) * math.log(1 - p))
    assert E.row_entropies(q, k)[0, 0] == pytest.approx(expect, rel=1e-13)


def test_dominant_key_gives_zero_entropy():
    d, L = 8, 20
    k = np.zeros((1, L, d), dtype=np.float32)
    k[0, 5, 0] = 64.0
    q = np.zeros((1, 1, d), dtype=np.float32)
    q[0, 0, 0] = 64.0                       # logit 64 * 64 / sqrt(8) ~ 1448 on key 5, 0 elsewhere
    h = E.row_entropies(bits(q), bits(k))
    assert 0.0 <= h[0, 0] < 1e-300


def test_entropy_bounds_and_group_mapping():
    rng = np.random.default_rng(1)
    Hq, Hkv, L, n_q, d = 6, 3, 50, 50, 8
    q = bits(2.0 * rng.standard_normal((Hq, n_q, d)))
    k = bits(rng.standard_normal((Hkv, L, d)))
    h = E.row_entropies(q, k)
    # 0 <= H(row t) <= ln(t + 1), the uniform row's entropy
    assert (h >= 0).all()
    assert (h <= np.log(np.arange(1, L + 1))[None, :] + 1e-12).all()
    # query head hq reads KV head hq // G: each head alone against its KV head agrees
    G = Hq // Hkv
    for hq in range(Hq):
        alone = E.row_entropies(q[hq:hq + 1], k[hq // G:hq // G + 1])
        np.testing.assert_allclose(alone[0], h[hq], rtol=1e-14)
