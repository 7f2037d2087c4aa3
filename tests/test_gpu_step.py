"""GPU parity: the full K-seed denoise step (timestep MLP, patch embedding,
block stack, velocity head, flow update) and its pieces against the oracle."""
import dataclasses

import numpy as np
import pytest
import torch

import seeded_inputs as si
from oracle import dit_oracle as O
from tests.conftest import weights_f64
from tests.gpu_util import block_cfg, dev, host64, rel_err, upload_block

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def d():
    from paper_2606_19004_amd import ditstep
    return ditstep


def step_f64(inp, cfg):
    sw = {k: si.as_f64(v, cfg.dtype) for k, v in inp["step_weights"].items()}
    blocks = [weights_f64(b, cfg.dtype) for b in inp["blocks"]]
    return sw, blocks


def run_step(d, cfg, inp):
    c = block_cfg(d, cfg)
    swd = {k: dev(v, cfg.dtype) for k, v in inp["step_weights"].items()}
    up = {}   # blocks that share one weight set are uploaded once
    for b in inp["blocks"]:
        if id(b) not in up:
            up[id(b)] = upload_block(b, cfg.dtype)
    bws = [up[id(b)] for b in inp["blocks"]]
    blocks = [d.block_weights(b["img"], b["txt"]) for b in bws]
    lat = dev(inp["latent"])
    xt = dev(inp["x_txt"], cfg.dtype)
    eps = dev(inp["eps"])
    v = torch.zeros_like(lat)
    ws = d.workspace(d.dit_denoise_workspace_bytes(c, cfg.batch, cfg.latent_dim))
    a = cfg.noise_level
    d.dit_denoise_step(c, d.step_weights(swd), blocks, inp["t"], inp["t_next"], a, lat, xt,
                       eps if a > 0 else None, v, ws)
    torch.cuda.synchronize()
    return lat.cpu().numpy().astype(np.float64), v.cpu().numpy().astype(np.float64)


def oracle_step(cfg, inp, batches=None):
    sw, blocks = step_f64(inp, cfg)
    sel = slice(None) if batches is None else batches
    lat = inp["latent"][sel].astype(np.float64)
    xt = si.as_f64(inp["x_txt"], cfg.dtype)[sel]
    eps = inp["eps"][sel].astype(np.float64)
    t, tn = float(np.float32(inp["t"])), float(np.float32(inp["t_next"]))
    new, v, _ = O.denoise_step(cfg, sw, blocks, lat, xt, t, tn, eps, float(np.float32(cfg.noise_level)))
    return new, v


def check_step(cfg, inp, new, v, ref_new, ref_v, lat0):
    t = 2e-2 if cfg.dtype == "bf16" else 1e-4
    assert rel_err(v, ref_v) <= t, rel_err(v, ref_v)
    assert rel_err(new - lat0, ref_new - lat0) <= t, rel_err(new - lat0, ref_new - lat0)
    assert rel_err(new, ref_new) <= (1e-5 if cfg.dtype == "f32" else 2e-3)


@pytest.mark.parametrize("name,a", [("tiny_f32", 0.0), ("tiny_f32", 0.7), ("small_step_bf16", 0.7),
                                    ("small_step_bf16", 0.0)])
def test_step_small_full_compare(d, name, a):
    cfg = dataclasses.replace(si.CONFIGS[name], noise_level=a)
    inp = si.step_inputs(cfg)
    new, v = run_step(d, cfg, inp)
    ref_new, ref_v = oracle_step(cfg, inp)
    check_step(cfg, inp, new, v, ref_new, ref_v, inp["latent"].astype(np.float64))


def test_step_full_shape_two_blocks_one_seed(d):
    """The K=16, 1024 + 256 token launch shape with 2 blocks; seed 3 compared in full."""
    cfg = dataclasses.replace(si.CONFIGS["step_512_k16"], blocks=2)
    inp = si.step_inputs(cfg)
    new, v = run_step(d, cfg, inp)
    ref_new, ref_v = oracle_step(cfg, inp, batches=[3])
    check_step(cfg, inp, new[[3]], v[[3]], ref_new, ref_v, inp["latent"][[3]].astype(np.float64))
    # the K seeds are independent: identical inputs give identical outputs
    assert np.all(np.isfinite(new)) and np.all(np.isfinite(v))


def test_step_nine_blocks_small(d):
    """Nine blocks: the modulation of the first eight is computed in one batched launch (sixteen weight
    slots) and the ninth in a group of its own, and the RoPE table is filled once for the stack;
    compared in full against the oracle."""
    cfg = dataclasses.replace(si.CONFIGS["small_step_bf16"], blocks=9)
    inp = si.step_inputs(cfg)
    new, v = run_step(d, cfg, inp)
    ref_new, ref_v = oracle_step(cfg, inp)
    check_step(cfg, inp, new, v, ref_new, ref_v, inp["latent"].astype(np.float64))


def test_step_full_shape_eight_blocks_seed_permutation(d):
    """The step in the launch configuration bench.py times (8 blocks, K=16, 1024 + 256 tokens, SDE),
    checked through a property that holds at any size: the K seeds are processed independently, so
    permuting the seeds of the inputs permutes the outputs, bit for bit. The 8 blocks reuse the two
    blocks' weights of the 2-block test (the oracle check of that shape is there)."""
    cfg = dataclasses.replace(si.CONFIGS["step_512_k16"], blocks=2)
    inp = si.step_inputs(cfg)
    inp["blocks"] = [inp["blocks"][i % 2] for i in range(8)]
    cfg = dataclasses.replace(cfg, blocks=8)
    new1, v1 = run_step(d, cfg, inp)
    perm = np.random.default_rng(5).permutation(cfg.batch)
    pinp = dict(inp, latent=inp["latent"][perm], eps=inp["eps"][perm], x_txt=inp["x_txt"][perm])
    new2, v2 = run_step(d, cfg, pinp)
    assert np.all(np.isfinite(new1)) and np.all(np.isfinite(v1))
    np.testing.assert_array_equal(v2, v1[perm])
    np.testing.assert_array_equal(new2, new1[perm])


def test_step_pieces_full_shape(d):
    cfg = si.CONFIGS["step_512_k16"]
    inp = si.step_inputs(dataclasses.replace(cfg, blocks=0))
    c = block_cfg(d, cfg)
    sw = {k: dev(v, "bf16") for k, v in inp["step_weights"].items()}
    sw64 = {k: si.as_f64(v, "bf16") for k, v in inp["step_weights"].items()}
    B = cfg.batch
    ws = d.workspace(d.dit_denoise_workspace_bytes(c, B, 64))
    # timestep embedding for distinct t per sample
    tt = np.linspace(0.02, 0.98, B).astype(np.float32)
    temb = torch.zeros((B, cfg.hidden), device="cuda")
    d.dit_timestep_embed(c, d.step_weights(sw), dev(tt), temb, ws)
    ref_temb = O.timestep_embed(tt.astype(np.float64), sw64)
    assert rel_err(temb.cpu().numpy(), ref_temb) <= 1e-3
    # patch embedding: bf16 latent x bf16 weights, fp32 accumulate, bf16 out
    lat = dev(inp["latent"])
    ximg = torch.zeros((B, cfg.n_img, cfg.hidden), dtype=torch.bfloat16, device="cuda")
    d.dit_patch_embed(c, d.step_weights(sw), lat, ximg, ws)
    lat_b = si.as_f64(si.to_bf16_bits(inp["latent"]), "bf16")
    assert rel_err(host64(ximg), O.patch_embed(lat_b, sw64)) <= 2e-2
    # final layer on a random hidden state
    x = si.stored(si.normal("final/x", (B, cfg.n_img, cfg.hidden)), "bf16")
    t64 = ref_temb
    v = torch.zeros((B, cfg.n_img, 64), device="cuda")
    d.dit_final_layer(c, d.step_weights(sw), dev(t64.astype(np.float32)), dev(x, "bf16"), v, ws)
    ref_v = O.final_layer(si.as_f64(x, "bf16"), t64.astype(np.float32).astype(np.float64), sw64)
    assert rel_err(v.cpu().numpy(), ref_v) <= 2e-2


def _blocks_f64_lazy(inp, cfg):
    """The blocks' weights as float64, one block at a time (8 blocks at hidden 3072 would take
    22 GB at once); the oracle walks the stack once."""
    for b in inp["blocks"]:
        yield weights_f64(b, cfg.dtype)


@pytest.mark.timeout(900)
def test_step_headline_eight_distinct_blocks_against_oracle(d):
    """The configuration bench.py times, as it times it: 8 distinct blocks, K=16 seeds, 1024 image +
    256 text tokens, SDE a=0.7, then the reward statistics of 64 groups x 16 seeds. Two seeds of the
    step are compared in full with the oracle (velocity and latent delta 2e-2, latent 2e-3); the
    statistics' order and selection are compared bit for bit."""
    cfg = si.CONFIGS["step_512_k16"]
    assert cfg.blocks == 8 and cfg.batch == 16 and cfg.noise_level == 0.7
    print(f"[headline] generating {cfg.blocks} blocks of seeded weights", flush=True)
    inp = si.step_inputs(cfg)
    assert len({id(b) for b in inp["blocks"]}) == 8
    new, v = run_step(d, cfg, inp)
    assert np.all(np.isfinite(new)) and np.all(np.isfinite(v))
    rw = dev(inp["rewards"])
    G, n, k = cfg.reward_groups, cfg.reward_n, cfg.reward_k
    outs = [torch.empty(G, device="cuda"), torch.empty(G, device="cuda"), torch.empty((G, n), device="cuda"),
            torch.empty((G, n), dtype=torch.int32, device="cuda"), torch.empty((G, k), dtype=torch.int32, device="cuda")]
    d.group_reward_stats(rw, 1e-4, k, *outs)
    ref_stats = O.group_reward_stats(inp["rewards"].astype(np.float64), 1e-4, k)
    np.testing.assert_array_equal(outs[3].cpu().numpy(), ref_stats["order"])
    np.testing.assert_array_equal(outs[4].cpu().numpy(), ref_stats["selected"])
    seeds = [0, 13]
    print(f"[headline] oracle for seeds {seeds}", flush=True)
    sw = {k_: si.as_f64(a, cfg.dtype) for k_, a in inp["step_weights"].items()}
    lat = inp["latent"][seeds].astype(np.float64)
    xt = si.as_f64(inp["x_txt"], cfg.dtype)[seeds]
    eps = inp["eps"][seeds].astype(np.float64)
    t, tn = float(np.float32(inp["t"])), float(np.float32(inp["t_next"]))
    ref_new, ref_v, _ = O.denoise_step(cfg, sw, _blocks_f64_lazy(inp, cfg), lat, xt, t, tn, eps,
                                       float(np.float32(cfg.noise_level)))
    check_step(cfg, inp, new[seeds], v[seeds], ref_new, ref_v, lat)
