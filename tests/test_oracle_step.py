"""Pins for the oracle's full-step pieces: timestep MLP, patch embedding,
final (velocity) layer and their composition with the flow update."""
import numpy as np
import torch
import torch.nn.functional as F

import seeded_inputs as si
from oracle import dit_oracle as O

CFG = si.Shape("pinstep", hidden=32, heads=2, head_dim=16, grid_h=2, grid_w=3, n_txt=4, batch=3,
               dtype="f32", blocks=1, latent_dim=8)


def step_weights(rng):
    return {t: rng.standard_normal(shp) * 0.3 for t, shp in si.step_weight_shapes(CFG).items()}


def T(a):
    return torch.from_numpy(np.ascontiguousarray(a))


def test_timestep_mlp_against_torch(rng):
    sw = step_weights(rng)
    t = np.array([0.0, 0.25, 0.9])
    e = O.timestep_sinusoid(t)
    ref = F.linear(F.silu(F.linear(T(e), T(sw["t1_w"]), T(sw["t1_b"]))), T(sw["t2_w"]), T(sw["t2_b"]))
    np.testing.assert_allclose(O.timestep_embed(t, sw), ref.numpy(), rtol=1e-12, atol=1e-13)


def test_final_layer_shift_scale_form(rng):
    sw = step_weights(rng)
    d = CFG.hidden
    x = rng.standard_normal((3, CFG.n_img, d))
    temb = rng.standard_normal((3, d))
    sw["fmod_w"][:] = 0.0
    sw["fmod_b"][:d] = 0.0       # shift_f = 0
    sw["fmod_b"][d:] = -1.0      # scale_f = -1  ->  LN(x)(1 + scale) = 0
    np.testing.assert_allclose(O.final_layer(x, temb, sw), np.broadcast_to(sw["fout_b"], (3, CFG.n_img, 8)),
                               atol=1e-15)
    sw = step_weights(rng)
    m = F.linear(F.silu(T(temb)), T(sw["fmod_w"]), T(sw["fmod_b"]))
    h = F.layer_norm(T(x), (d,), eps=1e-6) * (1 + m[:, None, d:]) + m[:, None, :d]
    ref = F.linear(h, T(sw["fout_w"]), T(sw["fout_b"]))
    np.testing.assert_allclose(O.final_layer(x, temb, sw), ref.numpy(), rtol=1e-12, atol=1e-13)


def test_patch_embed_is_linear(rng):
    sw = step_weights(rng)
    lat = rng.standard_normal((3, CFG.n_img, 8))
    ref = F.linear(T(lat), T(sw["in_w"]), T(sw["in_b"]))
    np.testing.assert_allclose(O.patch_embed(lat, sw), ref.numpy(), rtol=1e-13, atol=1e-14)


def test_denoise_step_composition(rng):
    sw = step_weights(rng)
    blocks = [{s: {t: rng.standard_normal(shp) * 0.1 for t, shp in si.block_weight_shapes(CFG).items()}
               for s in ("img", "txt")}]
    lat = rng.standard_normal((3, CFG.n_img, 8))
    txt = rng.standard_normal((3, CFG.n_txt, CFG.hidden))
    eps = rng.standard_normal(lat.shape)
    new, v, temb = O.denoise_step(CFG, sw, blocks, lat, txt, 0.6, 0.55, eps, 0.7)
    temb2 = O.timestep_embed(np.full(3, 0.6), sw)
    xi, _ = O.block_forward(CFG, blocks[0], temb2, O.patch_embed(lat, sw), txt)
    v2 = O.final_layer(xi, temb2, sw)
    np.testing.assert_allclose(v, v2, rtol=1e-13)
    np.testing.assert_allclose(new, O.flow_step(lat, v2, eps, 0.6, 0.55, 0.7), rtol=1e-13)
