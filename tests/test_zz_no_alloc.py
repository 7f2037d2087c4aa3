"""dit_timestep_embed_noalloc (scratch in the library's fixed device array) against
dit_timestep_embed (scratch in a caller workspace): the same kernels, so the results must be
equal bit for bit. Two calls in a row, the second with a smaller batch (the array keeps the
first call's contents), in the bf16 and fp32 configurations; and the size limit."""
import dataclasses

import numpy as np
import pytest
import torch

import seeded_inputs as si
from tests.gpu_util import block_cfg, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def d():
    from paper_2606_19004_amd import ditstep
    return ditstep


@pytest.mark.parametrize("name,batches", [("step_512_k16", (16, 5)), ("tiny_f32", (7, 2)), ("step_512_k16", (156, 1))])
def test_noalloc_timestep_embed_matches_workspace_version(d, name, batches):
    cfg = si.CONFIGS[name]
    inp = si.step_inputs(dataclasses.replace(cfg, blocks=0))
    c = block_cfg(d, cfg)
    sw_t = {k: dev(v, cfg.dtype) for k, v in inp["step_weights"].items()}   # kept alive: sw holds raw pointers
    sw = d.step_weights(sw_t)
    for call, B in enumerate(batches):
        tt = np.linspace(0.03 + 0.01 * call, 0.97, B).astype(np.float32)
        t = dev(tt)
        want = torch.full((B, cfg.hidden), float("nan"), device="cuda")
        got = torch.full((B, cfg.hidden), float("nan"), device="cuda")
        ws = d.workspace(d.dit_denoise_workspace_bytes(c, B, cfg.latent_dim))
        d.dit_timestep_embed(c, sw, t, want, ws)
        d.dit_timestep_embed_noalloc(c, sw, t, got)
        torch.cuda.synchronize()
        assert torch.isfinite(want).all()
        assert torch.equal(got, want), (name, call, B)


def test_noalloc_rejects_batches_beyond_the_array(d):
    cfg = si.CONFIGS["step_512_k16"]
    inp = si.step_inputs(dataclasses.replace(cfg, blocks=0))
    c = block_cfg(d, cfg)
    sw_t = {k: dev(v, cfg.dtype) for k, v in inp["step_weights"].items()}
    sw = d.step_weights(sw_t)
    B = 400
    t = dev(np.full(B, 0.5, np.float32))
    out = torch.zeros((B, cfg.hidden), device="cuda")
    with pytest.raises(d.DitError) as ei:
        d.dit_timestep_embed_noalloc(c, sw, t, out)
    assert ei.value.name == "DIT_ERR_UNSUPPORTED" and "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert torch.count_nonzero(out) == 0
