"""GPU pin of the bf16 MFMA GEMM: with integer-valued operands the result is exact, so the kernel
must reproduce an exact integer product bit for bit.

The plain GEMM of the C ABI is the patch embedding, x_img = latent W_in^T + b_in, whose reduction
depth K is the latent width (any multiple of 64). Latent entries are 0 or +-1 with at most 100
nonzeros per row, weights are in {-1, 0, 1} and biases in {-2, ..., 2}: every partial sum is an
integer of magnitude at most 102, so the fp32 accumulation, the bias add and the bf16 output (exact
for integers up to 256) are all exact, whatever the accumulation order. The expected values are
computed in float64, exact for such integers."""
import dataclasses

import numpy as np
import pytest
import torch

import seeded_inputs as si
from tests.gpu_util import block_cfg, dev, host64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def d():
    from paper_2606_19004_amd import ditstep
    return ditstep


def _bf16_bits(a):
    return si.to_bf16_bits(np.asarray(a, np.float32))


# (configuration, latent width K): the step's launch shape on 256 x 256 tiles with one, two, three
# and ten 64-deep k-tiles; ragged row and column tiles on the smaller tile paths
CASES = [("step_512_k16", 64), ("step_512_k16", 128), ("step_512_k16", 192), ("step_512_k16", 640),
         ("small_bf16_d64", 192), ("small_bf16", 320), ("mlp_short_k128", 256)]


@pytest.mark.parametrize("name,k", CASES)
def test_patch_embed_integer_operands_bit_exact(d, name, k):
    cfg = dataclasses.replace(si.CONFIGS[name], latent_dim=k)
    B, N, D = cfg.batch, cfg.n_img, cfg.hidden
    rng = np.random.default_rng(1000 + k + D)
    nz = min(100, k)                                         # <= 100 entries of +-1 per row
    pos = np.argsort(rng.random((B * N, k)), axis=1)[:, :nz]
    lat = np.zeros((B * N, k), np.float32)
    np.put_along_axis(lat, pos, rng.choice(np.array([-1.0, 1.0], np.float32), (B * N, nz)), axis=1)
    w_in = rng.integers(-1, 2, (D, k)).astype(np.float32)
    b_in = rng.integers(-2, 3, D).astype(np.float32)
    sw = {n: np.zeros(shp, np.float32) for n, shp in si.step_weight_shapes(cfg).items()}
    sw["in_w"], sw["in_b"] = w_in, b_in
    swd = {n: dev(_bf16_bits(a), "bf16") for n, a in sw.items()}
    c = block_cfg(d, cfg)
    ws = d.workspace(d.dit_denoise_workspace_bytes(c, B, k))
    x = torch.full((B, N, D), 3.0, dtype=torch.bfloat16, device="cuda")
    d.dit_patch_embed(c, d.step_weights(swd), dev(lat.reshape(B, N, k)), x, ws)
    got = host64(x).reshape(B * N, D)
    # every 256-row tile and every column is checked: the first and last row of each row tile
    # plus random rows
    rows = np.unique(np.r_[np.arange(0, B * N, 256), np.minimum(np.arange(255, B * N + 255, 256), B * N - 1),
                           rng.choice(B * N, min(64, B * N), replace=False)])
    want = lat[rows].astype(np.float64) @ w_in.T.astype(np.float64) + b_in
    assert np.max(np.abs(want)) <= 256
    np.testing.assert_array_equal(got[rows], want)
