"""Pins for the oracle's per-group reward statistics and seed ordering:
a hand-worked fixture, Python's statistics module, brute-force sorting and
the invariants (zero-sum advantages, a permutation with non-increasing
values, ties by index, constant rewards)."""
import json
import math
import os
import statistics

import numpy as np

from oracle import dit_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "reward_stats_worked.json")


def test_hand_worked_fixture():
    g = json.load(open(GOLDEN))
    r = np.array(g["rewards"])
    for k, key in ((2, "selected_k2"), (3, "selected_k3")):
        out = O.group_reward_stats(r, 1e-4, k)
        np.testing.assert_allclose(out["mean"], g["mean"], rtol=1e-15)
        np.testing.assert_allclose(out["std"], np.sqrt(g["std_squared"]), rtol=1e-12, atol=1e-15)
        np.testing.assert_array_equal(out["order"], g["order"])
        np.testing.assert_array_equal(out["selected"], g[key])
        want = np.array(g["adv_numerators"]) / (np.sqrt(g["std_squared"])[:, None] + 1e-4)
        np.testing.assert_allclose(out["adv"], want, rtol=1e-12, atol=1e-12)


def test_against_statistics_module(rng):
    r = rng.uniform(size=(20, 16))
    out = O.group_reward_stats(r, 1e-4, 4)
    for g in range(20):
        assert math.isclose(out["mean"][g], statistics.fmean(r[g]), rel_tol=1e-14)
        assert math.isclose(out["std"][g], statistics.pstdev(r[g]), rel_tol=1e-12)
    np.testing.assert_allclose(out["adv"].sum(axis=1), 0.0, atol=1e-12)


def test_order_is_sorted_permutation_with_index_ties(rng):
    r = rng.integers(0, 4, size=(50, 12)).astype(np.float64) / 4    # many ties
    out = O.group_reward_stats(r, 1e-4, 5)
    for g in range(50):
        o = out["order"][g]
        assert sorted(o.tolist()) == list(range(12))
        vals = r[g][o]
        assert np.all(np.diff(vals) <= 0)
        for i in range(11):
            if vals[i] == vals[i + 1]:
                assert o[i] < o[i + 1]
        np.testing.assert_array_equal(out["selected"][g], np.r_[o[:3], o[-2:]])


def test_constant_rewards():
    out = O.group_reward_stats(np.full((3, 8), 0.25), 1e-4, 2)
    np.testing.assert_array_equal(out["std"], 0.0)
    np.testing.assert_array_equal(out["adv"], 0.0)
    np.testing.assert_array_equal(out["order"], np.tile(np.arange(8), (3, 1)))


def test_select_none_and_all(rng):
    r = rng.uniform(size=(4, 6))
    assert O.group_reward_stats(r, 1e-4, 0)["selected"].shape == (4, 0)
    out = O.group_reward_stats(r, 1e-4, 6)
    np.testing.assert_array_equal(out["selected"], out["order"])
