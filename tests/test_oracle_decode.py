"""Pins for the oracle's decode-phase H2O update."""
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
