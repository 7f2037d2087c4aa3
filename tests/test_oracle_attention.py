"""Pins for the oracle's joint attention: torch's scaled_dot_product_attention
(an independent library routine), a pure-Python brute force on tiny inputs,
and the invariants softmax attention must satisfy."""
import math

import numpy as np
import torch
import torch.nn.functional as F

from oracle import dit_oracle as O


def test_attention_matches_torch_sdpa(rng):
    for nq, s, d in [(5, 9, 8), (33, 70, 64), (17, 17, 128)]:
        q, k, v = rng.standard_normal((nq, d)) * 2, rng.standard_normal((s, d)) * 2, rng.standard_normal((s, d))
        ref = F.scaled_dot_product_attention(torch.from_numpy(q)[None], torch.from_numpy(k)[None],
                                             torch.from_numpy(v)[None])[0].numpy()
        np.testing.assert_allclose(O.attention(q, k, v), ref, rtol=1e-11, atol=1e-12)


def test_attention_brute_force(rng):
    q, k, v = rng.standard_normal((3, 4)), rng.standard_normal((6, 4)), rng.standard_normal((6, 4))
    out = O.attention(q, k, v)
    for i in range(3):
        s = [sum(q[i][c] * k[j][c] for c in range(4)) / 2.0 for j in range(6)]   # 1/sqrt(4)
        e = [math.exp(x) for x in s]
        z = sum(e)
        ref = [sum(e[j] / z * v[j][c] for j in range(6)) for c in range(4)]
        np.testing.assert_allclose(out[i], ref, rtol=1e-13)


def test_attention_probabilities_rows_sum_to_one(rng):
    s = 12
    q, k = rng.standard_normal((4, s)) * 3, rng.standard_normal((s, s)) * 3
    p = O.attention(q, k, np.eye(s))          # V = I exposes P itself
    assert np.all(p > 0)
    np.testing.assert_allclose(p.sum(-1), 1.0, rtol=1e-14)


def test_attention_invariants(rng):
    q, k, v = rng.standard_normal((10, 16)), rng.standard_normal((25, 16)), rng.standard_normal((25, 16))
    # constant V -> constant output
    c = rng.standard_normal(16)
    np.testing.assert_allclose(O.attention(q, k, np.broadcast_to(c, (25, 16))), np.broadcast_to(c, (10, 16)),
                               rtol=1e-13)
    # permuting keys and values together leaves the output unchanged
    perm = rng.permutation(25)
    np.testing.assert_allclose(O.attention(q, k[perm], v[perm]), O.attention(q, k, v), rtol=1e-12)
    # permuting queries permutes the output rows
    qp = rng.permutation(10)
    np.testing.assert_allclose(O.attention(q[qp], k, v), O.attention(q, k, v)[qp], rtol=1e-12)
    # large logits: max subtraction keeps the result finite
    assert np.all(np.isfinite(O.attention(q * 1e3, k, v)))


def test_joint_attention_heads_are_independent(rng):
    q, k, v = rng.standard_normal((6, 3, 8)), rng.standard_normal((11, 3, 8)), rng.standard_normal((11, 3, 8))
    o = O.joint_attention(q, k, v)
    ref = F.scaled_dot_product_attention(torch.from_numpy(q).permute(1, 0, 2), torch.from_numpy(k).permute(1, 0, 2),
                                         torch.from_numpy(v).permute(1, 0, 2)).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-11, atol=1e-12)
