"""Pins for the oracle's elementwise pieces: SiLU, GELU-tanh, LayerNorm,
modulation split, 2D RoPE and the timestep sinusoid.  Each is checked against
an independent library routine, a closed form or an invariant."""
import math

import numpy as np
import torch
import torch.nn.functional as F

from oracle import dit_oracle as O


def test_silu_matches_torch(rng):
    z = rng.standard_normal(1000) * 6
    np.testing.assert_allclose(O.silu(z), F.silu(torch.from_numpy(z)).numpy(), rtol=1e-14, atol=1e-15)


def test_gelu_tanh_matches_torch_and_erf(rng):
    z = rng.standard_normal(1000) * 4
    np.testing.assert_allclose(O.gelu_tanh(z), F.gelu(torch.from_numpy(z), approximate="tanh").numpy(),
                               rtol=1e-13, atol=1e-15)
    # the tanh form approximates the exact erf GELU to ~1e-3
    exact = np.array([0.5 * x * (1 + math.erf(x / math.sqrt(2))) for x in z])
    assert np.max(np.abs(O.gelu_tanh(z) - exact)) < 1e-3


def test_layer_norm_matches_torch_and_moments(rng):
    x = rng.standard_normal((7, 96)) * 3 + 1.5
    ref = F.layer_norm(torch.from_numpy(x), (96,), eps=1e-6).numpy()
    y = O.layer_norm(x)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y.mean(-1), 0, atol=1e-12)
    np.testing.assert_allclose((y ** 2).mean(-1), 1, atol=1e-5)   # eps shifts it slightly


def test_modulate_reduces_to_layer_norm(rng):
    x = rng.standard_normal((2, 5, 32))
    zero = np.zeros((2, 32))
    np.testing.assert_array_equal(O.modulate(x, zero, zero), O.layer_norm(x))
    # scale = -1 kills the normalised term, leaving the shift
    shift = rng.standard_normal((2, 32))
    np.testing.assert_allclose(O.modulate(x, shift, -np.ones((2, 32))), np.broadcast_to(shift[:, None], x.shape),
                               atol=1e-15)


def test_modulation_chunks(rng):
    d = 8
    temb = rng.standard_normal((3, d))
    w = np.zeros((6 * d, d))
    b = np.arange(6 * d, dtype=np.float64)
    m = O.modulation(temb, w, b)
    for i, name in enumerate(O.MOD_CHUNKS):
        np.testing.assert_array_equal(m[name], np.broadcast_to(np.arange(i * d, (i + 1) * d), (3, d)))
    # the linear part uses SiLU(temb): one nonzero weight picks one input
    w2 = np.zeros((6 * d, d))
    w2[5, 2] = 1.0
    m2 = O.modulation(temb, w2, np.zeros(6 * d))
    np.testing.assert_allclose(m2["shift1"][:, 5], temb[:, 2] / (1 + np.exp(-temb[:, 2])), rtol=1e-15)


def _rope_tokens(q, grid_h, grid_w):
    """Place vector q at every image token and rotate."""
    n = grid_h * grid_w
    x = np.broadcast_to(q, (n, 1, q.shape[-1])).copy()
    return O.rope_2d(x, grid_h, grid_w)[:, 0, :]


def test_rope_origin_identity_and_norms(rng):
    gh, gw, d = 5, 7, 16
    x = rng.standard_normal((gh * gw, 3, d))
    y = O.rope_2d(x, gh, gw)
    np.testing.assert_array_equal(y[0], x[0])               # token (0,0): no rotation
    pn = lambda a: a[..., 0::2] ** 2 + a[..., 1::2] ** 2   # noqa: E731
    np.testing.assert_allclose(pn(y), pn(x), rtol=1e-12)     # each pair keeps its norm


def test_rope_first_pair_angle_is_position():
    # pair 0 of each half has frequency theta^0 = 1: rotation angle = row (dims 0,1) or column (d/2, d/2+1)
    gh, gw, d = 4, 6, 16
    q = np.zeros(d)
    q[0] = 1.0
    q[d // 2] = 1.0
    y = _rope_tokens(q, gh, gw)
    for n in range(gh * gw):
        r, c = divmod(n, gw)
        np.testing.assert_allclose(y[n, [0, 1]], [math.cos(r), math.sin(r)], atol=1e-15)
        np.testing.assert_allclose(y[n, [d // 2, d // 2 + 1]], [math.cos(c), math.sin(c)], atol=1e-15)
    # pair 1 of the row half rotates by r * theta^(-2/m), m = d/2
    q = np.zeros(d)
    q[2] = 1.0
    y = _rope_tokens(q, gh, gw)
    f1 = 10000.0 ** (-2.0 / (d // 2))
    for n in range(gh * gw):
        r = n // gw
        np.testing.assert_allclose(y[n, [2, 3]], [math.cos(r * f1), math.sin(r * f1)], atol=1e-15)


def test_rope_relative_position(rng):
    """<R(p) q, R(p') k> depends only on p' - p along each axis."""
    gh, gw, d = 6, 6, 32
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    rq, rk = _rope_tokens(q, gh, gw), _rope_tokens(k, gh, gw)
    tok = lambda r, c: r * gw + c  # noqa: E731
    base = rq[tok(1, 2)] @ rk[tok(3, 1)]
    for dr, dc in [(1, 0), (0, 3), (2, 2), (-1, 1)]:
        np.testing.assert_allclose(rq[tok(1 + dr, 2 + dc)] @ rk[tok(3 + dr, 1 + dc)], base, rtol=1e-11)
    assert abs(rq[tok(1, 2)] @ rk[tok(3, 2)] - base) > 1e-3   # and it does depend on the offset


def test_rope_matches_complex_rotation(rng):
    """Interleaved pairs (2i, 2i+1) as complex numbers multiplied by exp(i*angle)."""
    gh, gw, d = 3, 4, 8
    x = rng.standard_normal((gh * gw, 2, d))
    y = O.rope_2d(x, gh, gw)
    m = d // 2
    for n in range(gh * gw):
        pos = divmod(n, gw)
        for half in range(2):
            for i in range(m // 2):
                ang = pos[half] * 10000.0 ** (-2.0 * i / m)
                z = complex(x[n, 1, half * m + 2 * i], x[n, 1, half * m + 2 * i + 1]) * complex(math.cos(ang), math.sin(ang))
                np.testing.assert_allclose(y[n, 1, half * m + 2 * i:half * m + 2 * i + 2], [z.real, z.imag], atol=1e-14)


def test_timestep_sinusoid():
    e0 = O.timestep_sinusoid(np.array([0.0]))[0]
    np.testing.assert_array_equal(e0, np.r_[np.ones(128), np.zeros(128)])
    f = O.timestep_frequencies()
    assert f[0] == 1.0
    np.testing.assert_allclose(f[1:] / f[:-1], 10.0 ** (-4.0 / 128), rtol=1e-13)   # geometric ladder
    t = 0.37
    e = O.timestep_sinusoid(np.array([t]))[0]
    np.testing.assert_allclose(e[:128] ** 2 + e[128:] ** 2, 1.0, rtol=1e-14)
    np.testing.assert_allclose(e[[0, 128]], [math.cos(1000 * t), math.sin(1000 * t)], rtol=1e-13)
