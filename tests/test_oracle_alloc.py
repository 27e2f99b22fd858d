"""Pins for the oracle's capacity allocator (Section 3.3, Eq. 3).

Each case is fixed by hand arithmetic or by an invariant the paper states
(sum of budgets equals the total, every budget at least b_min), not by
re-running the allocator's own formula.
"""
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import alloc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_equal_weights_tie_goes_to_lower_layer():
    # 10 / 3 = 3.33 each: floors 3,3,3, one residual unit, equal remainders -> layer 0
    assert list(alloc.allocate([1, 1, 1], 10, 0)) == [4, 3, 3]


def test_single_clamp_round():
    # shares 30*[10,1,1]/12 = [25, 2.5, 2.5]; layers 1,2 fixed at 8; layer 0 gets 30 - 16
    assert list(alloc.allocate([10, 1, 1], 30, 8)) == [14, 8, 8]


def test_clamp_needs_several_passes():
    # pass 1: 24*[10,3,1]/14 = [17.1, 5.14, 1.71] -> fix layer 2 at 5
    # pass 2: 19*[10,3]/13 = [14.6, 4.38] -> fix layer 1 at 5
    # pass 3: layer 0 takes the remaining 14
    assert list(alloc.allocate([10, 3, 1], 24, 5)) == [14, 5, 5]


def test_residual_goes_to_largest_remainders():
    # shares 20*[0.55, 0.3, 0.15] = [11, 6, 3] exact; 21*[..] = [11.55, 6.3, 3.15]
    assert list(alloc.allocate([0.55, 0.3, 0.15], 20, 0)) == [11, 6, 3]
    # floors 11,6,3 = 20; one unit to the largest remainder (0.55, layer 0)
    assert list(alloc.allocate([0.55, 0.3, 0.15], 21, 0)) == [12, 6, 3]
    # 22: two units -> remainders 0.55 (l0), 0.3 (l1)
    assert list(alloc.allocate([0.55, 0.3, 0.15], 22, 0)) == [12, 7, 3]


def test_shift_rule_for_nonpositive_scores():
    t = alloc.shift_nonpositive([-1.0, 0.0, 1.0])
    np.testing.assert_allclose(t, [1e-6, 1.0 + 1e-6, 2.0 + 1e-6], rtol=0, atol=1e-15)
    # positive scores are left alone
    np.testing.assert_array_equal(alloc.shift_nonpositive([0.5, 2.0]), [0.5, 2.0])


def test_ppl_cap_at_95th_percentile():
    s = np.arange(1, 21, dtype=float)            # 1..20
    # linear-interpolation percentile: rank 0.95 * 19 = 18.05 -> 19 + 0.05 * (20 - 19) = 19.05
    t = alloc.transform(s, alloc.PPL_CAP)
    assert t[-1] == pytest.approx(19.05)
    assert t[-2] == 19.0
    np.testing.assert_array_equal(t[:-1], s[:-1])
    np.testing.assert_array_equal(alloc.transform(s, alloc.IDENTITY), s)


def test_paper_kv_byte_identity():
    """Appendix E: 32 layers x 512 retained positions = 16,384 positions = 64.00 MiB of K and V."""
    g = json.load(open(os.path.join(GOLDEN, "paper_system_bytes.json")))
    budgets = alloc.allocate(np.ones(g["n_layers"]), g["n_layers"] * g["budget_per_layer"], 48)
    assert int(budgets.sum()) == g["layer_token_positions"]
    assert set(budgets.tolist()) == {g["budget_per_layer"]}
    m = g["model_shape"]
    nbytes = alloc.compacted_kv_bytes(budgets, m["n_kv_heads"], m["head_dim"], m["elem_bytes"])
    assert nbytes / 2 ** 20 == pytest.approx(g["kv_state_mib"], abs=0.005)


def test_stored_budget_vectors_hold_the_invariants():
    g = json.load(open(os.path.join(GOLDEN, "budgets.json")))
    b = np.array(g["pyramid_512"])
    assert b.sum() == 32 * 512 and b.min() >= 48
    assert (np.diff(b) <= 0).all()          # the ramp decreases
    for avg, vec in g["sweep"].items():
        v = np.array(vec)
        assert v.sum() == 32 * int(avg) and v.min() >= 48


@settings(max_examples=200, deadline=None)
@given(st.lists(st.floats(0.01, 100.0), min_size=1, max_size=40),
       st.integers(0, 64), st.integers(0, 5000))
def test_allocation_invariants(weights, b_min, extra):
    w = np.array(weights)
    total = len(w) * b_min + extra
    b = alloc.allocate(w, total, b_min)
    assert b.sum() == total
    assert (b >= b_min).all()
    share = alloc.clamped_shares(w, float(total), float(b_min))
    # rounding moves no layer by a full unit
    assert (np.abs(b - share) < 1.0).all()
    # unclamped layers keep the weight order (up to one unit from rounding)
    free = share > b_min
    idx = np.flatnonzero(free)
    for i in idx:
        for j in idx:
            if w[i] > w[j]:
                assert b[i] >= b[j] - 1
