"""Pins for the planner / seed-bank oracle (section 4.3 and section 5).

Pinned against things other than the oracle's own code:
  * a hand-worked eight-round run (tests/golden/planner_worked.json) with the eligible sets,
    the choices, the UCB values and the fallback when nothing fits;
  * invariants: the first |A| choices visit every eligible action once in order of planned
    cost; with beta = 0 the choice is the action with the best window mean (greedy); the
    window mean equals the mean of the last W_b feedbacks; eligibility is monotone in d and s
    and includes the boundary T_plan == W; equal planned costs fall to fewer steps;
  * the feedback ratio's closed form for constant per-set sigma, and its error cases;
  * seed bank: the hand-worked example and a brute-force property check on small inputs;
  * planted mistakes (ln N instead of ln(N+1), N_i instead of n_i) fail the worked example.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import planner_oracle as P

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "planner_worked.json")))


def _run_worked(planner_cls=P.Planner):
    g = GOLD
    pl = planner_cls(g["d_values"], g["s_values"], g["beta"], g["window"], g["prompts"])
    for rd in g["rounds"]:
        assert pl.eligible(g["t_train"], rd["n_spot"], g["t_step"]) == rd["eligible"]
        if "ucb_before" in rd:
            for i, u in zip(rd["eligible"], rd["ucb_before"]):
                assert abs(pl.ucb(i) - u) < 1e-9, (i, pl.ucb(i), u)
        i, fits = pl.select(g["t_train"], rd["n_spot"], g["t_step"])
        assert (i, fits) == (rd["chosen"], rd["fits"])
        if "feedback" in rd:
            pl.update(i, rd["feedback"])
    return pl


def test_worked_example():
    _run_worked()


def test_planted_mistakes_fail_worked_example(monkeypatch):
    def ucb_ln_n(self, i):       # ln N instead of ln(N + 1)
        n_i = min(self.count[i], self.window)
        if n_i == 0:
            return math.inf
        return sum(self.history[i][-n_i:]) / n_i + self.beta * math.sqrt(math.log(max(sum(self.count), 1)) / n_i)

    def ucb_total(self, i):      # N_i (all feedbacks) instead of the window
        if self.count[i] == 0:
            return math.inf
        return sum(self.history[i]) / self.count[i] + self.beta * math.sqrt(math.log(sum(self.count) + 1) / self.count[i])

    for bad in (ucb_ln_n, ucb_total):
        monkeypatch.setattr(P.Planner, "ucb", bad)
        with pytest.raises(AssertionError):
            _run_worked()
        monkeypatch.undo()


def test_unobserved_first_in_cost_order():
    rng = np.random.default_rng(0)
    pl = P.Planner([4, 8, 16, 32], [12, 14, 16, 18, 20], 0.5, 8, 16)
    elig = pl.eligible(100.0, 8, 0.01)
    want = sorted(elig, key=lambda i: (pl.actions[i][0] * pl.actions[i][1], pl.actions[i][1], pl.actions[i][0]))
    got = []
    for _ in elig:
        i, fits = pl.select(100.0, 8, 0.01)
        assert fits
        got.append(i)
        pl.update(i, rng.uniform(0.5, 2.0))
    assert got == want


def test_beta_zero_is_greedy_on_window_means():
    rng = np.random.default_rng(1)
    pl = P.Planner([8, 16], [12, 16, 20], 0.0, 3, 8)
    for _ in range(40):
        i, _ = pl.select(1e9, 1, 1.0)
        pl.update(i, rng.uniform(0, 1))
        means = {j: np.mean(pl.history[j][-3:]) for j in range(len(pl.actions)) if pl.history[j]}
        if len(means) == len(pl.actions):
            nxt, _ = pl.select(1e9, 1, 1.0)
            best = max(means.values())
            assert means[nxt] == best


def test_window_mean_is_last_wb_feedbacks():
    pl = P.Planner([8], [12], 1.0, 4, 1)
    vals = [3.0, 1.0, 4.0, 1.0, 5.0, 9.0, 2.0, 6.0]
    for v in vals:
        pl.update(0, v)
    # single action: N = 8, n = 4, mean of 5, 9, 2, 6 = 5.5
    assert abs(pl.ucb(0) - (5.5 + math.sqrt(math.log(9) / 4))) < 1e-12


def test_eligibility_boundary_and_monotone():
    pl = P.Planner([1, 2, 3, 4], [1, 2, 3], 0.5, 2, 5)
    # T_plan = d * 5 * s * 0.5; W = 10 * 3 = 30: eligible iff d * s <= 12
    e = set(pl.eligible(10.0, 3, 0.5))
    for i, (d, s) in enumerate(pl.actions):
        assert (i in e) == (d * s <= 12)
    assert pl.actions.index((4, 3)) in e          # boundary: T_plan == W is eligible
    for i, (d, s) in enumerate(pl.actions):
        for j, (d2, s2) in enumerate(pl.actions):
            if i in e and d2 <= d and s2 <= s:
                assert j in e


def test_equal_cost_prefers_fewer_steps_then_fewer_sequences():
    pl = P.Planner([8, 16], [8, 16], 0.5, 2, 1)   # (8,16) and (16,8) have equal cost
    i, _ = pl.select(1e9, 1, 1.0)
    assert pl.actions[i] == (8, 8)
    pl.update(i, 1.0)
    i, _ = pl.select(1e9, 1, 1.0)
    assert pl.actions[i] == (16, 8)                # fewer steps beats fewer sequences


def test_feedback_closed_form_and_errors():
    fe = GOLD["feedback_example"]
    assert P.feedback(fe["sigma"], fe["explored"]) == pytest.approx(fe["r"], rel=1e-15)
    rng = np.random.default_rng(2)
    for _ in range(20):
        m, u = rng.integers(1, 30), rng.integers(1, 8)
        a, b = rng.uniform(0.1, 3), rng.uniform(0.1, 3)
        r = P.feedback([a] * m + [b] * u, [1] * m + [0] * u)
        assert r == pytest.approx((m * a + u * b) / (m + u) / b, rel=1e-12)
    with pytest.raises(ValueError):
        P.feedback([1.0, 2.0], [1, 1])
    with pytest.raises(ValueError):
        P.feedback([1.0, 0.0], [1, 0])


def test_seed_bank_worked_example():
    s = GOLD["seed_bank_example"]
    assert P.seed_bank_keep(s["seeds"], s["rewards"], s["k"]) == s["kept"]
    bank = P.SeedBank(s["k"])
    bank.put(7, s["seeds"], s["rewards"])
    assert bank.get(7) == s["kept"] and bank.get(8) == []


def test_seed_bank_brute_force_property():
    rng = np.random.default_rng(3)
    for _ in range(200):
        d = int(rng.integers(1, 7))
        k = int(rng.integers(0, d + 1))
        rew = list(rng.integers(0, 4, d) / 4.0)        # many ties
        seeds = list(range(100, 100 + d))
        kept = P.seed_bank_keep(seeds, rew, k)
        top, bottom = kept[:(k + 1) // 2], kept[(k + 1) // 2:]
        pos = {sd: j for j, sd in enumerate(seeds)}
        key = lambda sd: (-rew[pos[sd]], pos[sd])   # noqa: E731
        rank = sorted(seeds, key=key)
        # the top part is the first ceil(k/2) of the ranking, the bottom part its last floor(k/2)
        assert top == rank[:len(top)]
        assert bottom == (rank[d - len(bottom):] if bottom else [])
        assert len(set(kept)) == len(kept)
        for combo in itertools.combinations(range(d), len(top)):      # no better top set exists
            assert sorted(rew[j] for j in combo) <= sorted(rew[pos[sd]] for sd in top) or \
                sum(rew[j] for j in combo) <= sum(rew[pos[sd]] for sd in top) + 1e-12
