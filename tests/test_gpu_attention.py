"""GPU parity: joint_attention against the oracle's softmax attention."""
import math

import numpy as np
import pytest
import torch

import seeded_inputs as si
from oracle import dit_oracle as O
from tests.gpu_util import dev, host64, rel_err

pytestmark = pytest.mark.gpu

# bf16 inputs, bf16 P before the PV product and a bf16 output: ~2^-8 relative per
# rounding, averaged over many keys; 1e-2 leaves a wide margin, a layout bug gives O(1).
TOL_BF16 = 1e-2
TOL_F32 = 1e-5


@pytest.fixture(scope="module")
def d():
    from paper_2606_19004_amd import ditstep
    return ditstep


def _packed(rng, b, s, h, hd, dtype):
    """A packed [B][S][3][H][d] buffer like the block's QKV output."""
    x = rng.standard_normal((b, s, 3, h, hd)).astype(np.float32)
    return si.stored(x, dtype)


def _run(d, qkv_store, b, s, h, hd, dtype):
    buf = dev(qkv_store, dtype)
    o = torch.zeros((b, s, h * hd), dtype=buf.dtype, device="cuda")
    D = h * hd
    flat = buf.view(-1)
    d.joint_attention(flat[0:], flat[D:], flat[2 * D:], o, b, h, s, hd, (s * 3 * D, 3 * D, hd), (s * D, D, hd),
                      dtype=dtype)
    return host64(o).reshape(b, s, h, hd)


@pytest.mark.parametrize("b,s,h,hd", [(2, 200, 3, 128), (1, 64, 2, 128), (3, 77, 5, 64), (1, 1, 1, 128),
                                      (2, 385, 2, 64)])
def test_attention_bf16_small(d, b, s, h, hd):
    rng = np.random.default_rng(s * 7 + hd)
    st = _packed(rng, b, s, h, hd, "bf16")
    got = _run(d, st, b, s, h, hd, "bf16")
    x = si.as_f64(st, "bf16")
    for bi in range(b):
        ref = O.joint_attention(x[bi, :, 0], x[bi, :, 1], x[bi, :, 2])
        assert rel_err(got[bi], ref) <= TOL_BF16


@pytest.mark.parametrize("dtype,hd", [("bf16", 128), ("bf16", 64), ("f32", 64)])
def test_attention_separate_tensors_head_major_output(d, dtype, hd):
    """The general-stride boundary: q, k and v as three separate [B][S][H][d] tensors (not slices of
    one packed buffer) and the output written head-major, [B][H][S][d], through its strides."""
    rng = np.random.default_rng(29 + hd)
    b, s, h = 2, 150, 3
    qkv = [si.stored(rng.standard_normal((b, s, h, hd)).astype(np.float32), dtype) for _ in range(3)]
    q, k, v = (dev(x, dtype) for x in qkv)
    o = torch.full((b, h, s, hd), 7.0, dtype=q.dtype, device="cuda")
    d.joint_attention(q, k, v, o, b, h, s, hd, (s * h * hd, h * hd, hd), (h * s * hd, hd, s * hd), dtype=dtype)
    got = host64(o)
    xs = [si.as_f64(x, dtype) if dtype == "bf16" else x.astype(np.float64) for x in qkv]
    for bi in range(b):
        ref = O.joint_attention(xs[0][bi], xs[1][bi], xs[2][bi])        # [S][H][d]
        assert rel_err(got[bi].transpose(1, 0, 2), ref) <= (TOL_BF16 if dtype == "bf16" else TOL_F32)


@pytest.mark.parametrize("b,s,h,hd", [(2, 80, 4, 64), (1, 45, 2, 128)])
def test_attention_f32(d, b, s, h, hd):
    rng = np.random.default_rng(s)
    st = _packed(rng, b, s, h, hd, "f32")
    got = _run(d, st, b, s, h, hd, "f32")
    for bi in range(b):
        ref = O.joint_attention(st[bi, :, 0].astype(np.float64), st[bi, :, 1].astype(np.float64),
                                st[bi, :, 2].astype(np.float64))
        assert rel_err(got[bi], ref) <= TOL_F32


def test_attention_large_logits_stay_finite(d):
    rng = np.random.default_rng(5)
    x = rng.standard_normal((1, 300, 3, 2, 128)).astype(np.float32)
    x[:, :, 0] *= 30.0       # scores of several hundred
    st = si.stored(x, "bf16")
    got = _run(d, st, 1, 300, 2, 128, "bf16")
    xs = si.as_f64(st, "bf16")
    ref = O.joint_attention(xs[0, :, 0], xs[0, :, 1], xs[0, :, 2])
    assert np.all(np.isfinite(got))
    assert rel_err(got[0], ref) <= TOL_BF16


@pytest.mark.parametrize("name", ["block_1280", "headslice_1280"])
def test_attention_full_size_sampled(d, name):
    """Full 6912-token shapes; the oracle evaluates sampled query rows of a few (sample, head) pairs."""
    cfg = si.CONFIGS[name]
    b, s, h, hd = cfg.batch, cfg.seq, cfg.heads, cfg.head_dim
    q = si.stored(si.normal(f"{name}/attn_qkv", (b, s, 3, h, hd)), "bf16")
    got = _run(d, q, b, s, h, hd, "bf16")
    rng = np.random.default_rng(11)
    rows = np.r_[0, s - 1, rng.choice(s, 30, replace=False)]
    for bi, hi in [(0, 0), (b - 1, h - 1), (b // 2, h // 2)]:
        x = si.as_f64(q[bi, :, :, hi], "bf16")        # [S][3][d]
        ref = O.attention(x[rows, 0], x[:, 1], x[:, 2])
        assert rel_err(got[bi, rows, hi], ref) <= TOL_BF16


@pytest.mark.parametrize("step,hd", [(10.0, 128), (3.0, 128), (10.0, 64), (-6.0, 128)])
def test_attention_running_max_moves_across_tiles(d, step, hd):
    """Scores that grow (or shrink) steadily along the key sequence: the row max in the exp2
    domain moves by `step` per 64-key tile, so the kernel's running max is raised on many tiles
    (step > 8, the lazy-rescale threshold), only every few tiles with probabilities up to 2^8
    in between (step 3), or never after the first tile (step < 0)."""
    rng = np.random.default_rng(int(abs(step) * 10) + hd)
    b, s, h = 2, 450, 2
    e = np.ones(hd) / math.sqrt(hd)
    ab = step * math.sqrt(hd) / math.log2(math.e)      # q.k/sqrt(d) in log2 units grows by `step` per tile
    x = np.empty((b, s, 3, h, hd), np.float32)
    x[:, :, 0] = 4.0 * e + 0.05 * rng.standard_normal((b, s, h, hd))
    ramp = (np.arange(s) / 64.0)[None, :, None, None] * (ab / 4.0)
    x[:, :, 1] = ramp * e + 0.05 * rng.standard_normal((b, s, h, hd))
    x[:, :, 2] = rng.standard_normal((b, s, h, hd))
    st = si.stored(x, "bf16")
    got = _run(d, st, b, s, h, hd, "bf16")
    xs = si.as_f64(st, "bf16")
    assert np.all(np.isfinite(got))
    for bi in range(b):
        ref = O.joint_attention(xs[bi, :, 0], xs[bi, :, 1], xs[bi, :, 2])
        assert rel_err(got[bi], ref) <= TOL_BF16
