"""Pins for the oracle's flow-matching update.

The strongest pin is distributional: for Gaussian data x0 ~ N(0, s^2) the
rectified-flow marginal at time t is N(0, (1-t)^2 s^2 + t^2) and the exact
velocity field is linear, so a correct reverse-time SDE step (and the ODE
step) must carry exact samples of the time-t marginal to the time-t' marginal.
A wrong sign, coefficient or dropped term in the drift changes the variance
it ends at; the test below plants such mistakes to show it notices."""
import math

import numpy as np
import pytest

from oracle import dit_oracle as O


def test_ode_closed_form(rng):
    x, v = rng.standard_normal(100), rng.standard_normal(100)
    np.testing.assert_allclose(O.flow_step(x, v, None, 0.7, 0.65, 0.0), x - 0.05 * v, rtol=1e-13, atol=1e-14)


def test_constant_velocity_over_steps(rng):
    x0, v = rng.standard_normal(64), rng.standard_normal(64)
    ts = np.linspace(0.9, 0.1, 17)
    x = x0
    for t, tn in zip(ts[:-1], ts[1:]):
        x = O.flow_step(x, v, None, t, tn, 0.0)
    np.testing.assert_allclose(x, x0 + (0.1 - 0.9) * v, rtol=1e-13, atol=1e-14)


def test_sde_with_zero_level_is_ode(rng):
    x, v, e = rng.standard_normal(50), rng.standard_normal(50), rng.standard_normal(50)
    np.testing.assert_array_equal(O.flow_step(x, v, e, 0.6, 0.55, 0.0), O.flow_step(x, v, None, 0.6, 0.55, 0.0))


def test_sde_noise_scale(rng):
    """x' minus its noise-free value is sigma*sqrt(-h)*eps with sigma = a sqrt(t/(1-t))."""
    x, v, e = rng.standard_normal(1000), rng.standard_normal(1000), rng.standard_normal(1000)
    t, tn, a = 0.8, 0.75, 0.7
    diff = O.flow_step(x, v, e, t, tn, a) - O.flow_step(x, v, np.zeros(1000), t, tn, a)
    np.testing.assert_allclose(diff, a * math.sqrt(t / (1 - t)) * math.sqrt(0.05) * e, rtol=1e-12)


def _gaussian_run(step, a, s=0.5, t0=0.8, t1=0.5, n_steps=300, n=400_000, seed=7):
    rng = np.random.default_rng(seed)
    var = lambda t: (1 - t) ** 2 * s * s + t * t  # noqa: E731
    x = (1 - t0) * s * rng.standard_normal(n) + t0 * rng.standard_normal(n)
    ts = np.linspace(t0, t1, n_steps + 1)
    for t, tn in zip(ts[:-1], ts[1:]):
        v = (t - (1 - t) * s * s) / var(t) * x        # E[eps - x0 | x_t = x]
        x = step(x, v, rng.standard_normal(n), t, tn, a)
    return x.var(), var(t1)


@pytest.mark.parametrize("a", [0.0, 0.7, 1.0])
def test_marginal_preserved_for_gaussian_data(a):
    got, want = _gaussian_run(O.flow_step, a)
    assert abs(got / want - 1) < 0.01, (got, want)


def test_marginal_pin_detects_planted_mistakes():
    """Plant plausible mistakes in a copy of the SDE step on the CPU: each must miss the marginal."""
    def wrong(kind):
        def step(x, v, eps, t, tn, a):
            h = tn - t
            sig = a * math.sqrt(t / (1 - t))
            if kind == "drift_coef":      # sigma^2/t instead of sigma^2/(2t)
                return x + h * (v + sig * sig / t * (x + (1 - t) * v)) + sig * math.sqrt(-h) * eps
            if kind == "drift_sign":      # score added with the wrong sign
                return x + h * (v - sig * sig / (2 * t) * (x + (1 - t) * v)) + sig * math.sqrt(-h) * eps
            if kind == "dropped_v":       # (1-t) v term dropped from the score
                return x + h * (v + sig * sig / (2 * t) * x) + sig * math.sqrt(-h) * eps
            raise ValueError(kind)
        return step
    for kind in ("drift_coef", "drift_sign", "dropped_v"):
        got, want = _gaussian_run(wrong(kind), 0.7)
        assert abs(got / want - 1) > 0.03, (kind, got, want)
