"""Pins for the oracle's decode-phase H2O and TOVA updates."""
import math

import numpy as np
import pytest

from oracle import decode as D


def run(C=12, d=8, G=2, recent=4, steps=20, seed=0):
    rng = np.random.default_rng(seed)
    k_cache = rng.standard_normal((C, d))
    v_cache = rng.standard_normal((C, d))
    L0 = 50
    pos = np.sort(rng.choice(L0, C, replace=False))
    acc = rng.random(C)
    total0 = acc.sum()
    evicted = 0.0
    for t in range(steps):
        p = L0 + t
        q = rng.standard_normal((G, d))
        kt, vt = rng.standard_normal(d), rng.standard_normal(d)
        acc_all, victim, cand = D.h2o_step(k_cache, pos, acc, q, kt, p, recent)
        # every query head's probabilities sum to 1, so the group mean adds exactly 1
        assert acc_all.sum() == pytest.approx(acc.sum() + 1.0, rel=1e-12)
        pos_all = np.concatenate([pos, [p]])
        # the recent positions p-recent+1..p are never candidates
        assert not cand[pos_all > p - recent].any()
        # brute force: no candidate has a smaller (acc, pos) pair than the victim
        for e in np.flatnonzero(cand):
            assert (acc_all[e], pos_all[e]) >= (acc_all[victim], pos_all[victim])
        evicted += acc_all[victim]
        D.apply_step(k_cache, v_cache, pos, acc, acc_all, victim, kt, vt, p)
        assert len(pos) == C and len(set(pos.tolist())) == C
        # live + evicted accumulated mass = initial mass + one per step
        assert acc.sum() + evicted == pytest.approx(total0 + t + 1, rel=1e-12)
    return pos


def test_decode_invariants():
    run()
    run(C=6, G=4, recent=3, steps=40, seed=1)


def test_equal_logits_evict_the_oldest_lowest_score():
    # q orthogonal to every key: all C+1 probabilities are 1/(C+1)
    C, d = 4, 4
    k_cache = np.zeros((C, d)); k_cache[:, 1] = 1.0
    q = np.zeros((1, d)); q[0, 0] = 1.0
    pos = np.array([3, 7, 9, 10])
    acc = np.array([0.5, 0.2, 0.2, 0.9])
    acc_all, victim, cand = D.h2o_step(k_cache, pos, acc, q, k_cache[0], p=11, recent=2)
    np.testing.assert_allclose(acc_all, np.r_[acc, 0.0] + 0.2, rtol=1e-15)
    # candidates: pos <= 9 -> slots 0,1,2; slots 1 and 2 tie at 0.4 -> smaller position (7)
    assert cand.tolist() == [True, True, True, False, False]
    assert victim == 1


def test_two_entry_logistic():
    # C = 1 cached key with logit 0 and a new key with logit 1 (scale 1/sqrt(4))
    d = 4
    k_cache = np.zeros((1, d))
    q = np.ones((1, d))
    kt = np.array([1.0, 1.0, 0.0, 0.0])
    acc_all, victim, _ = D.h2o_step(k_cache, np.array([0]), np.array([0.0]), q, kt, p=5, recent=0)
    s = 1.0 / (1.0 + math.exp(-1.0))
    np.testing.assert_allclose(acc_all, [1 - s, s], rtol=1e-14)
    assert victim == 0   # recent=0: both are candidates, the cached key has less mass


# ---- TOVA: eviction by the current query's attention (Section 2.1), decode only

def test_tova_single_head_evicts_the_smallest_logit():
    # with one query head the softmax is monotone in the logit, so the victim is the entry with
    # the smallest q.k (ties: smallest position) -- decided here without any softmax
    rng = np.random.default_rng(3)
    for trial in range(50):
        C, d = int(rng.integers(1, 20)), 8
        k_cache = rng.standard_normal((C, d))
        q = rng.standard_normal((1, d))
        kt = rng.standard_normal(d)
        pos = np.sort(rng.choice(100, C, replace=False))
        p = 100 + trial
        score, victim = D.tova_step(k_cache, pos, q, kt, p)
        dots = np.r_[k_cache @ q[0], kt @ q[0]]
        pos_all = np.r_[pos, p]
        expect = min(range(C + 1), key=lambda e: (dots[e], pos_all[e]))
        assert victim == expect
        assert score.sum() == pytest.approx(1.0, rel=1e-12)


def test_tova_identical_heads_reduce_to_one_head():
    rng = np.random.default_rng(4)
    C, d = 9, 8
    k_cache = rng.standard_normal((C, d))
    q1 = rng.standard_normal((1, d))
    kt = rng.standard_normal(d)
    pos = np.arange(C) * 3
    s1, v1 = D.tova_step(k_cache, pos, q1, kt, 40)
    s4, v4 = D.tova_step(k_cache, pos, np.repeat(q1, 4, axis=0), kt, 40)
    np.testing.assert_allclose(s4, s1, rtol=1e-14)
    assert v1 == v4


def test_tova_equal_keys_evict_the_smallest_position_and_the_new_token_can_lose():
    C, d = 5, 4
    k_cache = np.zeros((C, d)); k_cache[:, 1] = 1.0
    q = np.zeros((2, d)); q[:, 0] = 1.0          # orthogonal to every key: all scores 1/(C+1)
    pos = np.array([12, 4, 30, 8, 21])
    score, victim = D.tova_step(k_cache, pos, q, k_cache[0], 40)
    np.testing.assert_allclose(score, 1.0 / (C + 1), rtol=1e-15)
    assert victim == 1                            # position 4
    # a new key the query heads dislike is itself the victim; the cache then stays as it was
    kt = np.array([-5.0, 0.0, 0.0, 0.0])
    score, victim = D.tova_step(k_cache, pos, q, kt, 40)
    assert victim == C
    kc, vc, ps = k_cache.copy(), k_cache.copy(), pos.copy()
    D.apply_tova(kc, vc, ps, victim, kt, kt, 40)
    assert np.array_equal(kc, k_cache) and np.array_equal(ps, pos)


def test_tova_two_entry_logistic_group_mean():
    # C = 1; two query heads see logit gaps +1 and -3 between the new and the cached key
    d = 4
    k_cache = np.zeros((1, d))
    kt = np.array([2.0, 0.0, 0.0, 0.0])          # q.kt / sqrt(4) = q[0]
    q = np.array([[1.0, 0, 0, 0], [-3.0, 0, 0, 0]])
    score, victim = D.tova_step(k_cache, np.array([0]), q, kt, 7)
    sig = lambda x: 1.0 / (1.0 + math.exp(-x))
    new = 0.5 * (sig(1.0) + sig(-3.0))
    np.testing.assert_allclose(score, [1.0 - new, new], rtol=1e-14)
    assert victim == (1 if new < 1.0 - new else 0)
