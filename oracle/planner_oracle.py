"""Oracle: the exploration planner (section 4.3) and the seed bank (section 5), plain Python.

TEST INFRASTRUCTURE ONLY. Only ``tests/`` may import or run this module. It shares no code with
the native library (``paper_2606_19004_amd``) and imports nothing from it.

What it computes, in the paper's notation:
  * action a = (d, s): d sequences per prompt, s effective denoising steps (section 4.3.1);
  * planned time T_plan(a) = d * C * s * t_step for C prompts; exploration window
    W = T_train * N_spot; eligible set = {a : T_plan(a) <= W} (section 4.3.1, action space);
  * feedback r = sigma_all / sigma_unc, the mean per-group reward std over all groups
    divided by the mean over the unexplored groups (section 4.3.2, bandit feedback);
  * UCB(a_i) = mu_i + beta * sqrt(ln(N + 1) / n_i) with mu_i the mean of the W_b most
    recent feedbacks of a_i, n_i = min(N_i, W_b), N = sum of N_i, and UCB = +inf when
    n_i = 0; a* = argmax over the eligible set, ties to lower planned cost, then fewer
    effective steps, then fewer sequences (section 4.3.3);
  * seed bank: per prompt, keep the top ceil(k/2) and bottom floor(k/2) seeds of the
    exploration rewards (section 5, dynamic exploration), order = descending reward
    with ties by ascending position.
Readings where the paper is silent: W_b is a parameter (no value is printed); when no action
fits the window the planner falls back to the cheapest action overall (the overflowing part
of exploration then continues after the model update, as section 4.3.4 describes) and says
that it did not fit; the feedback is undefined (ValueError) without unexplored groups or
when their mean std is 0.
"""
from __future__ import annotations

import math


class Planner:
    def __init__(self, d_values, s_values, beta, window, prompts):
        if not d_values or not s_values or window < 1 or prompts < 1 or beta < 0:
            raise ValueError("bad planner parameters")
        # action index = i_d * len(s_values) + i_s
        self.actions = [(int(d), int(s)) for d in d_values for s in s_values]
        self.beta, self.window, self.prompts = float(beta), int(window), int(prompts)
        self.history = [[] for _ in self.actions]
        self.count = [0] * len(self.actions)

    def planned_time(self, i, t_step):
        d, s = self.actions[i]
        return float(d * self.prompts * s) * t_step

    def eligible(self, t_train, n_spot, t_step):
        w = t_train * n_spot
        return [i for i in range(len(self.actions)) if self.planned_time(i, t_step) <= w]

    def ucb(self, i):
        n_i = min(self.count[i], self.window)
        if n_i == 0:
            return math.inf
        recent = self.history[i][-n_i:]
        mu = sum(recent) / n_i
        n_total = sum(self.count)
        return mu + self.beta * math.sqrt(math.log(n_total + 1) / n_i)

    def _tie_key(self, i):
        d, s = self.actions[i]
        return (d * s, s, d)          # planned cost is proportional to d * s

    def select(self, t_train, n_spot, t_step):
        """(action index, fits): argmax UCB over the eligible set with the paper's tie-breaks."""
        cand = self.eligible(t_train, n_spot, t_step)
        if not cand:
            return min(range(len(self.actions)), key=self._tie_key), False
        best = cand[0]
        for i in cand[1:]:
            ui, ub = self.ucb(i), self.ucb(best)
            if ui > ub or (ui == ub and self._tie_key(i) < self._tie_key(best)):
                best = i
        return best, True

    def update(self, i, r):
        self.history[i].append(float(r))
        self.count[i] += 1


def feedback(sigma, explored):
    """r = mean(sigma over all groups) / mean(sigma over unexplored groups)."""
    sig = [float(x) for x in sigma]
    unc = [x for x, e in zip(sig, explored) if not e]
    if not sig or not unc:
        raise ValueError("feedback needs at least one unexplored group")
    s_unc = sum(unc) / len(unc)
    if s_unc == 0.0:
        raise ValueError("unexplored groups have zero reward std")
    return (sum(sig) / len(sig)) / s_unc


def seed_bank_keep(seeds, rewards, k):
    """The top ceil(k/2) then the bottom floor(k/2) seeds by reward (descending, ties by position)."""
    d = len(seeds)
    if not 0 <= k <= d:
        raise ValueError("need 0 <= k <= number of seeds")
    order = sorted(range(d), key=lambda j: (-float(rewards[j]), j))
    top, bottom = (k + 1) // 2, k // 2
    keep = order[:top] + (order[d - bottom:] if bottom else [])
    return [seeds[j] for j in keep]


class SeedBank:
    def __init__(self, k):
        self.k = int(k)
        self.bank = {}

    def put(self, prompt_id, seeds, rewards):
        self.bank[int(prompt_id)] = seed_bank_keep(list(seeds), list(rewards), min(self.k, len(seeds)))

    def get(self, prompt_id):
        return list(self.bank.get(int(prompt_id), []))
