"""Pins for two oracle outputs: the per-position score carried into decode (`acc`) and the
TOVA prompt-compression rule.

`acc` is the unpooled group-mean score of every retained position (window and recent
positions included), the seed of H2O's decode-phase accumulated attention.  It is checked
against explicit loops over queries and keys (math.exp, no oracle helper), against the
harmonic closed form for equal keys, and against a plateau neighbour whose pooled and
unpooled scores differ.

TOVA in prefill ranks every prompt position by the group-mean attention of the last prompt
query.  It is pinned by the uniform-key closed form (every position 1/L, ties keep the
lowest positions), explicit loops, the one-step reduction to the decode rule (keeping L-1 of
L positions drops exactly the entry a TOVA decode step over the same keys evicts) and its
independence from the other window rows.
"""
import math

import numpy as np
import pytest

from oracle import decode as D
from oracle import prefill as P
from synth import f32_to_bf16_bits


def bits(x):
    return f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def harmonic(n):
    return sum(1.0 / t for t in range(1, n + 1))


def loop_scores(q, k, rows, G):
    """Group-mean attention per key from the query rows `rows` (explicit loops, math.exp).

    q [Hq, R, d] and k [Hkv, L, d] float64; query row r sits at position pos[r] and sees keys
    0..pos[r]; `rows` maps row index -> position."""
    Hq, _, d = q.shape
    Hkv, L, _ = k.shape
    S = np.zeros((Hkv, L))
    for hq in range(Hq):
        h = hq // G
        for r, t in rows:
            logits = [sum(q[hq, r, c] * k[h, j, c] for c in range(d)) / math.sqrt(d) for j in range(t + 1)]
            m = max(logits)
            ex = [math.exp(x - m) for x in logits]
            tot = sum(ex)
            for j in range(t + 1):
                S[h, j] += ex[j] / tot / G
    return S


def small_inputs(Hq=4, Hkv=2, L=14, w=4, d=4, seed=11, scale=1.5):
    rng = np.random.default_rng(seed)
    q = bits(scale * rng.standard_normal((Hq, w, d)))
    k = bits(rng.standard_normal((Hkv, L, d)))
    v = bits(rng.standard_normal((Hkv, L, d)))
    return q, k, v


# ----------------------------------------------------------------------------- acc

@pytest.mark.parametrize("rule,b", [(P.SNAPKV, 9), (P.SNAPKV, 3), (P.H2O, 7), (P.H2O, 13), (P.TOVA, 5),
                                    (P.SNAPKV, 14), (P.H2O, 20)])
def test_acc_is_the_unpooled_score_of_every_retained_position(rule, b):
    L, w, G = 14, 4, 2
    q, k, v = small_inputs(L=L, w=w)
    out = P.evict_layer(rule, b, q, k, v, window=w, pool_kernel=3)
    qf, kf = P.bf16_to_f64(q), P.bf16_to_f64(k)
    if rule == P.TOVA:
        S = loop_scores(qf[:, w - 1:], kf, [(0, L - 1)], G)
    else:
        S = loop_scores(qf, kf, [(i, L - w + i) for i in range(w)], G)
    for h in range(2):
        np.testing.assert_allclose(out["acc"][h], S[h, out["idx"][h]], rtol=1e-12, atol=1e-300)


def test_acc_of_full_span_h2o_is_the_full_span_score():
    L, d, b = 10, 4, 6
    rng = np.random.default_rng(5)
    q = bits(rng.standard_normal((4, L, d)))
    k = bits(rng.standard_normal((2, L, d)))
    v = bits(rng.standard_normal((2, L, d)))
    out = P.evict_layer(P.H2O_FULL, b, q, k, v, window=1)
    S = loop_scores(P.bf16_to_f64(q), P.bf16_to_f64(k), [(t, t) for t in range(L)], 2)
    for h in range(2):
        np.testing.assert_allclose(out["acc"][h], S[h, out["idx"][h]], rtol=1e-12)


@pytest.mark.parametrize("rule", [P.FULL, P.STREAMING])
def test_acc_of_unscored_rules_is_zero(rule):
    q, k, v = small_inputs()
    out = P.evict_layer(rule, 6, q, k, v, window=4)
    assert (out["acc"] == 0).all() and out["acc"].shape == out["idx"].shape


def test_acc_uniform_keys_harmonic_including_window_and_recent():
    """Equal keys: position j gets H_L - H_max(j, L-w) from the window rows; acc carries that
    value at every retained position, window (SnapKV) and recent (H2O) positions included."""
    L, w, d = 40, 6, 4
    rng = np.random.default_rng(2)
    q = bits(rng.standard_normal((4, w, d)))
    k = bits(np.tile(rng.standard_normal(d), (2, L, 1)))
    v = bits(rng.standard_normal((2, L, d)))
    expect = np.array([harmonic(L) - harmonic(max(j, L - w)) for j in range(L)])
    for rule, b in ((P.SNAPKV, 15), (P.H2O, 16)):
        out = P.evict_layer(rule, b, q, k, v, window=w, pool_kernel=7)
        for h in range(2):
            np.testing.assert_allclose(out["acc"][h], expect[out["idx"][h]], rtol=1e-12)
        # H2O keeps r = 8 recent positions; their acc differs from the prefix value
        if rule == P.H2O:
            assert out["acc"][0][-1] == pytest.approx(1.0 / L, rel=1e-12)


def test_acc_of_a_plateau_neighbour_is_its_unpooled_score():
    """One key with logit +50 for every window row: its +-3 neighbours share its pooled score
    (about w) and are retained, but their acc is their own unpooled score (about 0)."""
    L, w, d = 64, 8, 8
    qa = np.zeros(d); qa[0] = 1.0
    q = bits(np.tile(qa, (4, w, 1)))
    k = np.zeros((2, L, d), dtype=np.float32)
    k[:, 30] = 50.0 * math.sqrt(d) * qa
    v = np.zeros((2, L, d), dtype=np.float32)
    out = P.evict_layer(P.SNAPKV, w + 3, q, bits(k), bits(v), window=w, pool_kernel=7)
    idx = out["idx"][0].tolist()
    assert idx[:3] == [27, 28, 29]
    # pooled score about w, unpooled score w * e^-50 / (1 + ...) for the neighbours
    assert out["scores"][0][27] == pytest.approx(w, rel=1e-12)
    unpooled = w * math.exp(-50.0) / (1.0 + (L - w) * math.exp(-50.0))
    assert out["acc"][0][0] == pytest.approx(unpooled, rel=1e-6)
    assert out["acc"][0][0] < 1e-20


# ----------------------------------------------------------------------------- TOVA prefill

def test_tova_uniform_keys_keep_the_lowest_positions():
    L, w, d, b = 30, 4, 4, 7
    rng = np.random.default_rng(8)
    q = bits(rng.standard_normal((4, w, d)))
    k = bits(np.tile(rng.standard_normal(d), (2, L, 1)))
    v = bits(rng.standard_normal((2, L, d)))
    out = P.evict_layer(P.TOVA, b, q, k, v, window=w)
    np.testing.assert_allclose(out["scores"], 1.0 / L, rtol=1e-12)
    for h in range(2):
        assert out["idx"][h].tolist() == list(range(b))
    assert out["layout"] == (L, b, L, L)


def test_tova_scores_and_selection_against_loops():
    L, w, G, b = 14, 4, 2, 6
    q, k, v = small_inputs(L=L, w=w)
    out = P.evict_layer(P.TOVA, b, q, k, v, window=w)
    S = loop_scores(P.bf16_to_f64(q)[:, w - 1:], P.bf16_to_f64(k), [(0, L - 1)], G)
    np.testing.assert_allclose(out["scores"], S, rtol=1e-12)
    np.testing.assert_allclose(S.sum(axis=1), 1.0, rtol=1e-12)   # one query: a distribution
    for h in range(2):
        keep = sorted(sorted(range(L), key=lambda j: (-S[h, j], j))[:b])
        assert out["idx"][h].tolist() == keep
        np.testing.assert_array_equal(out["k_out"][h], k[h, keep])
        np.testing.assert_array_equal(out["v_out"][h], v[h, keep])


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_tova_keeping_all_but_one_drops_the_decode_step_victim(seed):
    """A TOVA decode step whose cache holds positions 0..L-2 and whose new token is position
    L-1 (query q_{L-1}) scores the same L entries with the same softmax and evicts the minimum;
    prefill TOVA with capacity L-1 must drop exactly that position (random inputs: no ties)."""
    L, w, d, Hq, Hkv = 24, 4, 8, 4, 2
    G = Hq // Hkv
    rng = np.random.default_rng(100 + seed)
    q = bits(rng.standard_normal((Hq, w, d)))
    k = bits(rng.standard_normal((Hkv, L, d)))
    v = bits(rng.standard_normal((Hkv, L, d)))
    out = P.evict_layer(P.TOVA, L - 1, q, k, v, window=w)
    qf, kf = P.bf16_to_f64(q), P.bf16_to_f64(k)
    for h in range(Hkv):
        _, victim = D.tova_step(kf[h, :L - 1], np.arange(L - 1), qf[h * G:(h + 1) * G, w - 1], kf[h, L - 1], L - 1)
        dropped = sorted(set(range(L)) - set(out["idx"][h].tolist()))
        assert dropped == [victim]


def test_tova_reads_only_the_last_query_row():
    q, k, v = small_inputs(L=20, w=5)
    q2 = q.copy()
    q2[:, :4] = bits(np.random.default_rng(9).standard_normal(q[:, :4].shape))
    a = P.evict_layer(P.TOVA, 8, q, k, v, window=5)
    b = P.evict_layer(P.TOVA, 8, q2, k, v, window=5)
    np.testing.assert_array_equal(a["idx"], b["idx"])
    np.testing.assert_array_equal(a["scores"], b["scores"])


def test_tova_dominant_key_is_kept_and_budget_at_least_context_keeps_all():
    L, w, d = 32, 4, 8
    qa = np.zeros(d); qa[2] = 1.0
    q = bits(np.tile(qa, (4, w, 1)))
    k = np.zeros((2, L, d), dtype=np.float32)
    k[0, 11] = 50.0 * math.sqrt(d) * qa
    k[1, 5] = 50.0 * math.sqrt(d) * qa
    v = np.zeros((2, L, d), dtype=np.float32)
    out = P.evict_layer(P.TOVA, 1, q, bits(k), bits(v), window=w)
    assert out["idx"][:, 0].tolist() == [11, 5]
    full = P.evict_layer(P.TOVA, L, q, bits(k), bits(v), window=w)
    np.testing.assert_array_equal(full["idx"], np.tile(np.arange(L), (2, 1)))
