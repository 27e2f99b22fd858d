"""Pins for the oracle's prefill compression (window scoring, pooling, group mean, top-k, rules).

Each check is fixed by something other than the oracle's own formulas: closed
forms (harmonic numbers, the logistic function), invariants (softmax rows sum
to 1), brute force (explicit window maxima, rank counting, exhaustive subset
search) or hand-computed values.
"""
import itertools
import math

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import prefill as P
from synth import f32_to_bf16_bits, prefill_layer


def bits(x):
    return f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def harmonic(n):
    return sum(1.0 / t for t in range(1, n + 1))


# ----------------------------------------------------------------------------- scale

def test_two_key_logistic_pins_the_logit_scale():
    # d = 4, q = (1,1,1,1), k0 = 0, k1 = (1,1,0,0): q.k1 = 2, scaled by 1/sqrt(4) -> logit 1
    q = np.ones((1, 1, 4))
    k = np.array([[[0, 0, 0, 0], [1, 1, 0, 0]]], dtype=float)
    A = P.window_scores(q, k)
    s = 1.0 / (1.0 + math.exp(-1.0))
    np.testing.assert_allclose(A[0], [1 - s, s], rtol=1e-14)


# ----------------------------------------------------------------------------- softmax / window sum

@settings(max_examples=30, deadline=None)
@given(st.integers(1, 3), st.integers(1, 3), st.integers(2, 40), st.data())
def test_rows_sum_to_one_and_window_totals_w(hkv, G, L, data):
    w = data.draw(st.integers(1, L))
    rng = np.random.default_rng(L * 7 + w)
    q = rng.standard_normal((hkv * G, w, 8))
    k = rng.standard_normal((hkv, L, 8))
    Pm = P.softmax_rows(P.window_logits(q, k))
    np.testing.assert_allclose(Pm.sum(axis=-1), 1.0, rtol=0, atol=1e-12)
    A = P.window_scores(q, k)
    np.testing.assert_allclose(A.sum(axis=-1), w, rtol=1e-12)
    assert (A >= 0).all()


def test_uniform_keys_give_harmonic_window_scores():
    """Equal keys: row i (position L-w+i) spreads 1/(L-w+i+1) over its visible keys, so
    A[j] = H_L - H_max(j, L-w).  Pins the causal mask (diagonal included) and the window sum."""
    L, w, d = 50, 8, 4
    rng = np.random.default_rng(0)
    q = rng.standard_normal((2, w, d))
    k = np.tile(rng.standard_normal(d), (1, L, 1))
    A = P.window_scores(q, k)
    expect = np.array([harmonic(L) - harmonic(max(j, L - w)) for j in range(L)])
    np.testing.assert_allclose(A[0], expect, rtol=1e-12)
    np.testing.assert_allclose(A[1], expect, rtol=1e-12)


# ----------------------------------------------------------------------------- pooling / group mean

def test_max_pool_hand_values_and_prefix_clip():
    a = np.array([0, 5, 0, 0, 0, 0, 0, 0, 0, 3], dtype=float)
    np.testing.assert_array_equal(P.max_pool_prefix(a, 3, 10), [5, 5, 5, 0, 0, 0, 0, 0, 3, 3])
    # pooled over the prefix [0, 8) only: position 7 must not see index 8 or 9
    np.testing.assert_array_equal(P.max_pool_prefix(a, 3, 8), [5, 5, 5, 0, 0, 0, 0, 0])
    np.testing.assert_array_equal(P.max_pool_prefix(a, 7, 6), [5, 5, 5, 5, 5, 0])


@settings(max_examples=50, deadline=None)
@given(st.lists(st.floats(0, 10), min_size=1, max_size=30), st.sampled_from([1, 3, 5, 7]), st.data())
def test_max_pool_brute_force(vals, kernel, data):
    a = np.array(vals)
    n = data.draw(st.integers(1, len(vals)))
    out = P.max_pool_prefix(a, kernel, n)
    half = kernel // 2
    for j in range(n):
        window = [vals[t] for t in range(j - half, j + half + 1) if 0 <= t < n]
        assert out[j] == max(window)


def test_pool_then_group_mean_order():
    # G = 2, kernel 3; pooling each head first gives [3,3,1,0]; the reverse order
    # (mean then pool) would give [2,2,1,0].
    A = np.array([[4.0, 0, 0, 0], [0, 2.0, 0, 0]])
    S = P.group_mean(P.max_pool_prefix(A, 3, 4), 2)
    np.testing.assert_array_equal(S, [[3, 3, 1, 0]])


def test_gqa_mapping_and_group_mean():
    """Query heads 0,1 read KV head 0 and 2,3 read KV head 1 (hq // G, not hq % Hkv).

    KV head 0 has one key aligned with the direction of query heads 0,1 (logit 50),
    KV head 1 one key aligned with query heads 2,3; the directions are orthogonal."""
    L, w, d = 40, 4, 8
    qa = np.zeros(d); qa[0] = 1.0
    qb = np.zeros(d); qb[1] = 1.0
    q = np.stack([np.tile(qa, (w, 1)), np.tile(qa, (w, 1)), np.tile(qb, (w, 1)), np.tile(qb, (w, 1))])
    k = np.zeros((2, L, d))
    k[0, 10] = 50.0 * math.sqrt(d) * qa
    k[1, 20] = 50.0 * math.sqrt(d) * qb
    A = P.window_scores(q, k)
    S = P.group_mean(A, 2)
    # every window row puts all but ~L*exp(-50) of its mass on the planted key
    assert S[0, 10] == pytest.approx(w, rel=1e-15, abs=1e-15 * w)
    assert S[1, 20] == pytest.approx(w, rel=1e-15, abs=1e-15 * w)
    assert S[0, 20] < 1e-15 and S[1, 10] < 1e-15


# ----------------------------------------------------------------------------- top-k

def rank_count_select(s, k):
    """j is kept iff (#strictly larger) + (#equal at a smaller position) < k."""
    n = len(s)
    keep = [j for j in range(n)
            if sum(s[i] > s[j] for i in range(n)) + sum(s[i] == s[j] for i in range(j)) < k]
    return keep


def best_subset(s, k):
    """Exhaustive: maximum score sum, then the lexicographically smallest position tuple."""
    best = None
    for c in itertools.combinations(range(len(s)), k):
        key = (-sum(s[i] for i in c), c)
        if best is None or key < best:
            best = key
    return list(best[1])


@settings(max_examples=150, deadline=None)
@given(st.lists(st.integers(0, 4), min_size=1, max_size=9), st.data())
def test_topk_against_brute_force(vals, data):
    # small integer scores -> many exact ties
    s = np.array(vals, dtype=float)
    k = data.draw(st.integers(0, len(vals)))
    got = P.topk_positions(s, k).tolist()
    assert got == rank_count_select(vals, k)
    if len(vals) <= 8:
        assert got == sorted(best_subset(vals, k))


# ----------------------------------------------------------------------------- rules

def layer_inputs(L=96, w=8, Hq=4, Hkv=2, d=16, seed=3):
    rng = np.random.default_rng(seed)
    return (bits(rng.standard_normal((Hq, w, d))), bits(rng.standard_normal((Hkv, L, d))),
            bits(rng.standard_normal((Hkv, L, d))))


@pytest.mark.parametrize("b", [0, 1, 3, 4, 5, 20, 95])
def test_streaming_closed_form(b):
    q, k, v = layer_inputs()
    L = k.shape[1]
    out = P.evict_layer(P.STREAMING, b, q, k, v, window=8)
    for h in range(2):
        r = out["idx"][h].tolist()
        assert len(r) == b and r == sorted(set(r))
        s0 = min(4, b)
        # sinks are the first s0 positions, the rest are the last b - s0 positions
        assert r[:s0] == list(range(s0))
        assert all(x >= L - (b - s0) for x in r[s0:])
        dropped = sorted(set(range(L)) - set(r))
        # what is dropped is one contiguous block right after the sinks
        assert dropped == list(range(s0, s0 + len(dropped)))


@pytest.mark.parametrize("rule", [P.FULL, P.STREAMING, P.SNAPKV, P.H2O])
@pytest.mark.parametrize("extra", [0, 1, 500])
def test_budget_at_least_context_keeps_everything(rule, extra):
    q, k, v = layer_inputs()
    L = k.shape[1]
    out = P.evict_layer(rule, L + extra, q, k, v, window=8)
    np.testing.assert_array_equal(out["idx"], np.tile(np.arange(L), (2, 1)))
    np.testing.assert_array_equal(out["k_out"], k)
    np.testing.assert_array_equal(out["v_out"], v)


def test_full_keeps_everything_at_any_budget():
    q, k, v = layer_inputs()
    out = P.evict_layer(P.FULL, 3, q, k, v, window=8)
    np.testing.assert_array_equal(out["k_out"], k)


def uniform_key_inputs(L=64, w=8, d=8):
    rng = np.random.default_rng(1)
    q = bits(rng.standard_normal((4, w, d)))
    k = bits(np.tile(rng.standard_normal(d), (2, L, 1)))
    v = bits(rng.standard_normal((2, L, d)))
    return q, k, v


def test_uniform_keys_snapkv_keeps_prefix_head_and_window():
    # constant prefix scores -> ties -> lowest positions first
    L, w, b = 64, 8, 20
    q, k, v = uniform_key_inputs(L, w)
    out = P.evict_layer(P.SNAPKV, b, q, k, v, window=w, pool_kernel=7)
    expect = list(range(b - w)) + list(range(L - w, L))
    for h in range(2):
        assert out["idx"][h].tolist() == expect
    np.testing.assert_allclose(out["scores"], harmonic(L) - harmonic(L - w), rtol=1e-12)


def test_uniform_keys_h2o_split():
    # b = 11: r = 5 recent, 6 heavy from [0, L-5); window positions 56..58 score lower
    L, w, b = 64, 8, 11
    q, k, v = uniform_key_inputs(L, w)
    out = P.evict_layer(P.H2O, b, q, k, v, window=w)
    expect = list(range(6)) + list(range(L - 5, L))
    for h in range(2):
        assert out["idx"][h].tolist() == expect
    S = out["scores"][0]
    assert S.shape == (L - 5,)
    np.testing.assert_allclose(S[57], harmonic(L) - harmonic(57), rtol=1e-12)


def test_one_hot_key_plateau_and_tie_break():
    """A key with logit +50 for every window row: its pooled score ~w spreads to its +-3
    neighbours (kernel 7); with room for 3 picks the three lowest plateau positions win."""
    L, w, d = 64, 8, 8
    qa = np.zeros(d); qa[0] = 1.0
    q = bits(np.tile(qa, (4, w, 1)))
    k = np.zeros((2, L, d), dtype=np.float32)
    k[:, 30] = 50.0 * math.sqrt(d) * qa
    v = np.zeros((2, L, d), dtype=np.float32)
    out = P.evict_layer(P.SNAPKV, w + 3, q, bits(k), bits(v), window=w, pool_kernel=7)
    for h in range(2):
        assert out["idx"][h].tolist() == [27, 28, 29] + list(range(L - w, L))
        assert (out["scores"][h][27:34] == out["scores"][h][30]).all()
        assert out["scores"][h][30] == pytest.approx(w, rel=1e-12)
    # room for 9: the whole plateau, then the two lowest positions of the equal rest
    out = P.evict_layer(P.SNAPKV, w + 9, q, bits(k), bits(v), window=w, pool_kernel=7)
    assert out["idx"][0].tolist() == [0, 1] + list(range(27, 34)) + list(range(L - w, L))


def test_snapkv_budget_not_above_window_keeps_last_b():
    q, k, v = layer_inputs()
    out = P.evict_layer(P.SNAPKV, 5, q, k, v, window=8)
    assert out["idx"][0].tolist() == list(range(91, 96))


def test_gather_is_a_bit_copy_of_the_retained_rows():
    q, k, v = layer_inputs()
    out = P.evict_layer(P.SNAPKV, 30, q, k, v, window=8)
    for h in range(2):
        np.testing.assert_array_equal(out["k_out"][h], k[h, out["idx"][h]])
        np.testing.assert_array_equal(out["v_out"][h], v[h, out["idx"][h]])


@settings(max_examples=40, deadline=None)
@given(st.sampled_from([P.STREAMING, P.SNAPKV, P.H2O, P.FULL]), st.integers(0, 120), st.integers(1, 16))
def test_rule_outputs_are_valid_sets(rule, b, w):
    q, k, v = layer_inputs(w=w)
    L = k.shape[1]
    out = P.evict_layer(rule, b, q, k, v, window=w)
    b_eff = L if rule == P.FULL else min(b, L)
    for h in range(2):
        r = out["idx"][h]
        assert len(r) == b_eff
        assert (np.diff(r) > 0).all() and (r >= 0).all() and (r < L).all()
        lay = out["layout"]
        if lay is not None:
            cand_end, kk, lo, hi = lay
            assert set(range(lo, hi)) <= set(r.tolist())
            if rule in (P.SNAPKV, P.H2O):
                # the selected part is exactly the rank-count top-k of the float64 scores
                sel = [x for x in r.tolist() if x < cand_end]
                assert sel == rank_count_select(out["scores"][h].tolist(), kk)


def test_planted_structure_is_found_on_the_single_layer_workload():
    """Plausibility only: on the 1K single-layer workload the sink and most planted
    heavy hitters survive SnapKV at budget 128."""
    x = prefill_layer(1, 0, 0, seq_len=1024, window=32, n_hh=16)
    out = P.evict_layer(P.SNAPKV, 128, x["q"], x["k"], x["v"], window=32, pool_kernel=7)
    for h in range(8):
        kept = set(out["idx"][h].tolist())
        assert 0 in kept
        assert len(kept & set(x["hh"][h].tolist())) >= 12


# ----------------------------------------------------------------------------- H2O, full span

def test_full_span_uniform_keys_harmonic_and_total():
    """H2O_FULL with equal keys: query t spreads 1/(t+1) over keys 0..t, so key j receives
    H_L - H_j; the scores of a head total L (one unit per query)."""
    L, d = 40, 4
    rng = np.random.default_rng(3)
    q = bits(rng.standard_normal((8, L, d)))
    k = bits(np.tile(rng.standard_normal(d), (2, L, 1)))
    v = bits(rng.standard_normal((2, L, d)))
    out = P.evict_layer(P.H2O_FULL, 10, q, k, v, window=1)
    expect = np.array([harmonic(L) - harmonic(j) for j in range(L)])
    r = P.h2o_recent(10, 1, 2)
    np.testing.assert_allclose(out["scores"], np.tile(expect[:L - r], (2, 1)), rtol=1e-12)
    full = P.evict_layer(P.H2O_FULL, L, q, k, v, window=1)
    np.testing.assert_allclose(full["scores"].sum(axis=1), L, rtol=1e-12)


def test_full_span_brute_force_and_h2o_selection():
    """Explicit loops over queries and keys (math.exp, no oracle helper) against the oracle's
    full-span scores, and the selection: r recent plus the top-(b-r) of [0, L-r)."""
    L, d, Hq, Hkv, b = 12, 4, 4, 2, 7
    rng = np.random.default_rng(4)
    q = bits(1.5 * rng.standard_normal((Hq, L, d)))
    k = bits(rng.standard_normal((Hkv, L, d)))
    v = bits(rng.standard_normal((Hkv, L, d)))
    out = P.evict_layer(P.H2O_FULL, b, q, k, v, window=1)
    qf, kf = P.bf16_to_f64(q), P.bf16_to_f64(k)
    G = Hq // Hkv
    S = np.zeros((Hkv, L))
    for hq in range(Hq):
        for t in range(L):
            logits = [sum(qf[hq, t, c] * kf[hq // G, j, c] for c in range(d)) / math.sqrt(d) for j in range(t + 1)]
            m = max(logits)
            ex = [math.exp(x - m) for x in logits]
            tot = sum(ex)
            for j in range(t + 1):
                S[hq // G, j] += ex[j] / tot / G
    r = b // 2
    np.testing.assert_allclose(out["scores"], S[:, :L - r], rtol=1e-12)
    for h in range(Hkv):
        order = sorted(range(L - r), key=lambda j: (-S[h, j], j))[:b - r]
        assert out["idx"][h].tolist() == sorted(order) + list(range(L - r, L))
    with pytest.raises(ValueError):
        P.evict_layer(P.H2O_FULL, b, q[:, :5], k, v, window=5)   # needs every position's query
