"""Pins for the oracle's flow_logprob (Gaussian transition density of the SDE step).

Pinned against things other than the oracle's own formula:
  * scipy's normal log-pdf summed over elements, with the mean taken as the
    noise-free SDE step (flow_step with eps = 0) and the scale sigma sqrt(-h);
  * the closed form for x' drawn by flow_step itself: the residual is exactly
    sigma sqrt(-h) eps, so logp = -|eps|^2/2 - n log(sigma sqrt(-h)) - n/2 log(2 pi);
  * a Monte-Carlo check that exp(logp) integrates like a density: the sample mean of
    -2 logp over draws matches n log(2 pi var) + n (chi-square mean);
  * error cases (a = 0, t outside (0,1), t_next >= t);
  * planted mistakes (variance sigma^2 |h| replaced by sigma^2, mean without the
    score term) fail the closed-form pin.
"""
import math

import numpy as np
import pytest
from scipy import stats

from oracle import dit_oracle as O


def _draw(seed, b=3, n=257):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((b, n)), rng.standard_normal((b, n)), rng.standard_normal((b, n))


@pytest.mark.parametrize("t,tn,a", [(0.8, 0.75, 0.7), (0.3, 0.1, 1.0), (0.06, 0.01, 0.7), (0.94, 0.5, 0.2)])
def test_logprob_matches_scipy_normal(t, tn, a):
    x, v, xn = _draw(1)
    mean = O.flow_step(x, v, np.zeros_like(x), t, tn, a)
    scale = O.sde_sigma(t, a) * math.sqrt(t - tn)
    ref = stats.norm.logpdf(xn, loc=mean, scale=scale).sum(axis=1)
    np.testing.assert_allclose(O.flow_logprob(x, v, xn, t, tn, a), ref, rtol=1e-12, atol=1e-9)


@pytest.mark.parametrize("t,tn,a", [(0.8, 0.75, 0.7), (0.5, 0.45, 0.3)])
def test_logprob_of_own_sample_closed_form(t, tn, a):
    x, v, eps = _draw(2, b=4, n=1000)
    xn = O.flow_step(x, v, eps, t, tn, a)
    s = O.sde_sigma(t, a) * math.sqrt(t - tn)
    n = x.shape[1]
    want = -0.5 * (eps * eps).sum(axis=1) - n * math.log(s) - 0.5 * n * math.log(2 * math.pi)
    np.testing.assert_allclose(O.flow_logprob(x, v, xn, t, tn, a), want, rtol=1e-11)


def test_logprob_monte_carlo_mean():
    t, tn, a, n = 0.7, 0.65, 0.7, 64
    rng = np.random.default_rng(3)
    x, v = rng.standard_normal((1, n)), rng.standard_normal((1, n))
    var = O.sde_sigma(t, a) ** 2 * (t - tn)
    eps = rng.standard_normal((20000, n))
    xn = O.flow_step(np.repeat(x, 20000, 0), np.repeat(v, 20000, 0), eps, t, tn, a)
    lp = O.flow_logprob(np.repeat(x, 20000, 0), np.repeat(v, 20000, 0), xn, t, tn, a)
    # E[-2 logp] = n log(2 pi var) + n, standard error sqrt(2n / 20000)
    assert abs(np.mean(-2 * lp) - (n * math.log(2 * math.pi * var) + n)) < 5 * math.sqrt(2 * n / 20000)


@pytest.mark.parametrize("t,tn,a", [(0.8, 0.75, 0.0), (1.0, 0.9, 0.7), (0.0, -0.1, 0.7), (0.5, 0.5, 0.7),
                                    (0.5, 0.6, 0.7)])
def test_logprob_domain_errors(t, tn, a):
    x, v, xn = _draw(4)
    with pytest.raises(ValueError):
        O.flow_logprob(x, v, xn, t, tn, a)


def test_planted_mistakes_fail_the_closed_form(monkeypatch):
    t, tn, a = 0.8, 0.75, 0.7
    x, v, eps = _draw(5, b=2, n=500)
    xn = O.flow_step(x, v, eps, t, tn, a)
    s = O.sde_sigma(t, a) * math.sqrt(t - tn)
    n = x.shape[1]
    want = -0.5 * (eps * eps).sum(axis=1) - n * math.log(s) - 0.5 * n * math.log(2 * math.pi)
    good = O.flow_logprob(x, v, xn, t, tn, a)
    np.testing.assert_allclose(good, want, rtol=1e-11)
    # mean without the score (drift) correction
    monkeypatch.setattr(O, "flow_mean", lambda x, v, t, tn, a: x + (tn - t) * v)
    assert not np.allclose(O.flow_logprob(x, v, xn, t, tn, a), want, rtol=1e-6)
    monkeypatch.undo()
    # variance sigma^2 instead of sigma^2 |h|
    monkeypatch.setattr(O, "sde_sigma", lambda t, a: a * math.sqrt(t / (1 - t)) / math.sqrt(t - tn))
    xn2 = xn  # same sample, density evaluated with the wrong variance
    assert not np.allclose(O.flow_logprob(x, v, xn2, t, tn, a), want, rtol=1e-6)
