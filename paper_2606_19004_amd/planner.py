"""ctypes binding of the exploration planner and seed bank (include/ditplan.h).

Argument marshalling only: every decision is made by the native library.
"""
from __future__ import annotations

import ctypes as C
import math

from .ditstep import DitError, lib

_lib = lib()
EXPORTS = ("dit_planner_create", "dit_planner_destroy", "dit_planner_num_actions", "dit_planner_action",
           "dit_planner_eligible", "dit_planner_select", "dit_planner_update", "dit_planner_stats",
           "dit_planner_feedback", "dit_seed_bank_create", "dit_seed_bank_destroy", "dit_seed_bank_put",
           "dit_seed_bank_put_selected", "dit_seed_bank_get", "dit_seed_bank_size")

_i32, _i64, _f64, _vp = C.c_int32, C.c_int64, C.c_double, C.c_void_p
_pi32, _pi64, _pf64, _pf32 = C.POINTER(_i32), C.POINTER(_i64), C.POINTER(_f64), C.POINTER(C.c_float)
_sigs = {
    "dit_planner_create": ([_pi32, _i32, _pi32, _i32, _f64, _i32, _i32, C.POINTER(_vp)], _i32),
    "dit_planner_destroy": ([_vp], None),
    "dit_planner_num_actions": ([_vp], _i32),
    "dit_planner_action": ([_vp, _i32, _pi32, _pi32], _i32),
    "dit_planner_eligible": ([_vp, _f64, _i32, _f64, _pi32, _pi32], _i32),
    "dit_planner_select": ([_vp, _f64, _i32, _f64, _pi32, _pi32, _pf64], _i32),
    "dit_planner_update": ([_vp, _i32, _f64], _i32),
    "dit_planner_stats": ([_vp, _i32, _pi32, _pi32, _pf64, _pf64], _i32),
    "dit_planner_feedback": ([_pf32, _pi32, _i32, _pf64], _i32),
    "dit_seed_bank_create": ([_i32, C.POINTER(_vp)], _i32),
    "dit_seed_bank_destroy": ([_vp], None),
    "dit_seed_bank_put": ([_vp, _i64, _pi64, _pf32, _i32], _i32),
    "dit_seed_bank_put_selected": ([_vp, _pi64, _i32, _pi64, _i32, _pi32, _i32], _i32),
    "dit_seed_bank_get": ([_vp, _i64, _pi64, _i32, _pi32], _i32),
    "dit_seed_bank_size": ([_vp], _i32),
}
for _name, (_args, _res) in _sigs.items():
    _fn = getattr(_lib, _name)
    _fn.argtypes = _args
    _fn.restype = _res


def _check(status):
    if status != 0:
        raise DitError(status, _lib.dit_last_error_message().decode())


def _arr(ctype, values):
    values = list(values)
    return (ctype * max(len(values), 1))(*values)


class Planner:
    """Bandit planner over actions (d, s); index = i_d * len(s_values) + i_s."""

    def __init__(self, d_values, s_values, beta=0.5, window=10, prompts=32):
        h = _vp()
        _check(_lib.dit_planner_create(_arr(_i32, d_values), len(d_values), _arr(_i32, s_values), len(s_values),
                                       float(beta), int(window), int(prompts), C.byref(h)))
        self._h = h

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            _lib.dit_planner_destroy(h)
            self._h = None

    @property
    def num_actions(self):
        return _lib.dit_planner_num_actions(self._h)

    def action(self, i):
        d, s = _i32(), _i32()
        _check(_lib.dit_planner_action(self._h, i, C.byref(d), C.byref(s)))
        return d.value, s.value

    def eligible(self, t_train, n_spot, t_step):
        n = self.num_actions
        mask, cnt = (_i32 * n)(), _i32()
        _check(_lib.dit_planner_eligible(self._h, float(t_train), int(n_spot), float(t_step), mask, C.byref(cnt)))
        return [i for i in range(n) if mask[i]]

    def select(self, t_train, n_spot, t_step):
        """(index, fits, ucb)."""
        i, f, u = _i32(), _i32(), _f64()
        _check(_lib.dit_planner_select(self._h, float(t_train), int(n_spot), float(t_step), C.byref(i), C.byref(f),
                                       C.byref(u)))
        return i.value, bool(f.value), u.value

    def update(self, i, r):
        _check(_lib.dit_planner_update(self._h, int(i), float(r)))

    def stats(self, i):
        """(N_i, n_i, window mean, UCB)."""
        tot, win, mean, ucb = _i32(), _i32(), _f64(), _f64()
        _check(_lib.dit_planner_stats(self._h, int(i), C.byref(tot), C.byref(win), C.byref(mean), C.byref(ucb)))
        return tot.value, win.value, mean.value, ucb.value


def feedback(sigma, explored):
    """r = mean sigma over all groups / mean sigma over unexplored groups (sigma: host floats)."""
    sig = [float(x) for x in sigma]
    r = _f64()
    _check(_lib.dit_planner_feedback(_arr(C.c_float, sig), _arr(_i32, [int(bool(e)) for e in explored]), len(sig),
                                     C.byref(r)))
    return r.value


class SeedBank:
    def __init__(self, k):
        h = _vp()
        _check(_lib.dit_seed_bank_create(int(k), C.byref(h)))
        self._h = h

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            _lib.dit_seed_bank_destroy(h)
            self._h = None

    def put(self, prompt_id, seeds, rewards):
        seeds, rewards = list(seeds), [float(r) for r in rewards]
        _check(_lib.dit_seed_bank_put(self._h, int(prompt_id), _arr(_i64, seeds), _arr(C.c_float, rewards),
                                      len(seeds)))

    def put_selected(self, prompt_ids, seeds, selected):
        """seeds: [groups][d] ints, selected: [groups][k] positions (group_reward_stats' output)."""
        g = len(prompt_ids)
        d = len(seeds[0]) if g else 0
        k = len(selected[0]) if g else 0
        _check(_lib.dit_seed_bank_put_selected(self._h, _arr(_i64, prompt_ids), g,
                                               _arr(_i64, [s for row in seeds for s in row]), d,
                                               _arr(_i32, [s for row in selected for s in row]), k))

    def get(self, prompt_id, capacity=64):
        out, cnt = (_i64 * capacity)(), _i32()
        _check(_lib.dit_seed_bank_get(self._h, int(prompt_id), out, capacity, C.byref(cnt)))
        return list(out[:min(cnt.value, capacity)])

    def __len__(self):
        return _lib.dit_seed_bank_size(self._h)


INF = math.inf
