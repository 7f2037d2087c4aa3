"""The denoise step captured into a HIP graph (torch.cuda.CUDAGraph over the library's launches on
the capturing stream) and replayed: every replay matches the eager call bit for bit. The step
records only kernels and one device-to-device copy (no memset nodes), so it can be replayed by
callers that run the step in a captured loop. Between replays the test runs eager work of its own
and synchronises, and the in-place latent is restored from a saved copy before each replay."""
import dataclasses

import numpy as np
import pytest
import torch

import seeded_inputs as si
from tests.gpu_util import block_cfg, dev, upload_block

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def d():
    from paper_2606_19004_amd import ditstep
    return ditstep


def setup_step(d, cfg):
    inp = si.step_inputs(cfg)
    c = block_cfg(d, cfg)
    swd = {k: dev(v, cfg.dtype) for k, v in inp["step_weights"].items()}
    bws = [upload_block(b, cfg.dtype) for b in inp["blocks"]]
    blocks = [d.block_weights(b["img"], b["txt"]) for b in bws]
    lat0 = dev(inp["latent"])
    bufs = dict(lat=lat0.clone(), xt=dev(inp["x_txt"], cfg.dtype), eps=dev(inp["eps"]),
                v=torch.zeros_like(lat0),
                ws=d.workspace(d.dit_denoise_workspace_bytes(c, cfg.batch, cfg.latent_dim)))
    keep = (swd, bws)   # device tensors the weight structs point to

    def call():
        a = cfg.noise_level
        d.dit_denoise_step(c, d.step_weights(swd), blocks, inp["t"], inp["t_next"], a, bufs["lat"], bufs["xt"],
                           bufs["eps"] if a > 0 else None, bufs["v"], bufs["ws"])
    return call, bufs, lat0, keep


@pytest.mark.parametrize("name,a", [("small_step_bf16", 0.7), ("small_step_bf16", 0.0), ("tiny_f32", 0.7)])
def test_step_graph_replay_matches_eager(d, name, a):
    cfg = dataclasses.replace(si.CONFIGS[name], noise_level=a)
    call, bufs, lat0, keep = setup_step(d, cfg)
    call()   # eager: also sets the library's per-device state before the capture
    torch.cuda.synchronize()
    lat_e, v_e = bufs["lat"].clone(), bufs["v"].clone()
    assert torch.isfinite(lat_e).all() and torch.isfinite(v_e).all()

    g = torch.cuda.CUDAGraph()
    bufs["lat"].copy_(lat0)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    other = torch.randn(1 << 20, device="cuda")
    for r in range(3):
        bufs["lat"].copy_(lat0)
        bufs["v"].zero_()
        other.mul_(1.0001).add_(0.5)   # eager work of the caller's own between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(bufs["v"], v_e), f"replay {r}: velocity differs from the eager call"
        assert torch.equal(bufs["lat"], lat_e), f"replay {r}: latent differs from the eager call"
    del g, keep
