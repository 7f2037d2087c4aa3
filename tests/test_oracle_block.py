"""Pins for the oracle's MMDiT block.

Each case reduces the block to something fixed independently of the oracle's
own code: the adaLN-Zero identity, a uniform-attention closed form, a
per-token MLP built from torch modules, torch's SDPA for the attention half,
and the symmetries (image-token permutation, text/image exchange) the block
must have when RoPE is off."""
import dataclasses

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import seeded_inputs as si
from oracle import dit_oracle as O

CFG = si.Shape("pin", hidden=32, heads=2, head_dim=16, grid_h=3, grid_w=4, n_txt=5, batch=2, dtype="f32")


def rand_weights(rng, cfg=CFG, std=0.2):
    return {s: {t: rng.standard_normal(shp) * std for t, shp in si.block_weight_shapes(cfg).items()}
            for s in ("img", "txt")}


def rand_inputs(rng, cfg=CFG):
    return (rng.standard_normal((cfg.batch, cfg.hidden)),
            rng.standard_normal((cfg.batch, cfg.n_img, cfg.hidden)),
            rng.standard_normal((cfg.batch, cfg.n_txt, cfg.hidden)))


def zero_chunk(w, chunk):
    d = CFG.hidden
    i = O.MOD_CHUNKS.index(chunk)
    for s in w:
        w[s]["mod_w"][i * d:(i + 1) * d] = 0.0
        w[s]["mod_b"][i * d:(i + 1) * d] = 0.0


def test_adaln_zero_is_identity(rng):
    w = rand_weights(rng)
    zero_chunk(w, "gate1")
    zero_chunk(w, "gate2")
    temb, xi, xt = rand_inputs(rng)
    oi, ot = O.block_forward(CFG, w, temb, xi, xt)
    np.testing.assert_array_equal(oi, xi)
    np.testing.assert_array_equal(ot, xt)


def test_uniform_attention_closed_form(rng):
    """W_q = b_q = 0: every score is 0, attention averages V over all S joint tokens."""
    w = rand_weights(rng)
    d = CFG.hidden
    for s in w:
        w[s]["qkv_w"][:d] = 0.0
        w[s]["qkv_b"][:d] = 0.0
    zero_chunk(w, "gate2")
    temb, xi, xt = rand_inputs(rng)
    oi, ot = O.block_forward(CFG, w, temb, xi, xt)
    x = {"img": xi, "txt": xt}
    for b in range(CFG.batch):
        vals, mods = [], {}
        for s in ("txt", "img"):
            mods[s] = O.modulation(temb[b:b + 1], w[s]["mod_w"], w[s]["mod_b"])
            h = O.modulate(x[s][b:b + 1], mods[s]["shift1"], mods[s]["scale1"])[0]
            vals.append(h @ w[s]["qkv_w"][2 * d:].T + w[s]["qkv_b"][2 * d:])
        mean_v = np.concatenate(vals).mean(axis=0)          # one vector for all queries
        for s, out in (("img", oi), ("txt", ot)):
            y = w[s]["out_w"] @ mean_v + w[s]["out_b"]
            np.testing.assert_allclose(out[b], x[s][b] + mods[s]["gate1"][0] * y, rtol=1e-12, atol=1e-12)


def test_mlp_half_against_torch_modules(rng):
    """gate1 = 0 leaves only the per-token MLP branch."""
    w = rand_weights(rng)
    zero_chunk(w, "gate1")
    temb, xi, xt = rand_inputs(rng)
    oi, ot = O.block_forward(CFG, w, temb, xi, xt)
    d = CFG.hidden
    for s, x, out in (("img", xi, oi), ("txt", xt, ot)):
        T = lambda a: torch.from_numpy(np.ascontiguousarray(a))  # noqa: E731
        m = F.linear(F.silu(T(temb)), T(w[s]["mod_w"]), T(w[s]["mod_b"]))
        shift2, scale2, gate2 = m[:, 3 * d:4 * d], m[:, 4 * d:5 * d], m[:, 5 * d:6 * d]
        h2 = F.layer_norm(T(x), (d,), eps=1e-6) * (1 + scale2[:, None]) + shift2[:, None]
        u = F.gelu(F.linear(h2, T(w[s]["mlp1_w"]), T(w[s]["mlp1_b"])), approximate="tanh")
        ref = T(x) + gate2[:, None] * F.linear(u, T(w[s]["mlp2_w"]), T(w[s]["mlp2_b"]))
        np.testing.assert_allclose(out, ref.numpy(), rtol=1e-11, atol=1e-12)


def _attn_half_torch(cfg, w, temb, xi, xt, rope):
    """gate2 = 0: x + gate1 * W_o SDPA(q, k, v) over [text; image], with torch primitives."""
    d, H, hd = cfg.hidden, cfg.heads, cfg.head_dim
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a))  # noqa: E731
    outs = {}
    q, k, v, g = {}, {}, {}, {}
    for s, x in (("txt", xt), ("img", xi)):
        m = F.linear(F.silu(T(temb)), T(w[s]["mod_w"]), T(w[s]["mod_b"]))
        shift1, scale1, g[s] = m[:, :d], m[:, d:2 * d], m[:, 2 * d:3 * d]
        h = F.layer_norm(T(x), (d,), eps=1e-6) * (1 + scale1[:, None]) + shift1[:, None]
        qkv = F.linear(h, T(w[s]["qkv_w"]), T(w[s]["qkv_b"]))
        n = x.shape[1]
        q[s], k[s], v[s] = [qkv[..., i * d:(i + 1) * d].reshape(cfg.batch, n, H, hd) for i in range(3)]
        if s == "img" and rope:
            q[s] = T(np.stack([O.rope_2d(a.numpy(), cfg.grid_h, cfg.grid_w) for a in q[s]]))
            k[s] = T(np.stack([O.rope_2d(a.numpy(), cfg.grid_h, cfg.grid_w) for a in k[s]]))
    Q = torch.cat([q["txt"], q["img"]], 1).transpose(1, 2)
    K = torch.cat([k["txt"], k["img"]], 1).transpose(1, 2)
    V = torch.cat([v["txt"], v["img"]], 1).transpose(1, 2)
    o = F.scaled_dot_product_attention(Q, K, V).transpose(1, 2).reshape(cfg.batch, -1, d)
    nt = xt.shape[1]
    for s, x, sl in (("txt", xt, slice(0, nt)), ("img", xi, slice(nt, None))):
        y = F.linear(o[:, sl], T(w[s]["out_w"]), T(w[s]["out_b"]))
        outs[s] = (T(x) + g[s][:, None] * y).numpy()
    return outs["img"], outs["txt"]


def test_attention_half_against_torch_sdpa(rng):
    for rope in (False, True):
        w = rand_weights(rng)
        zero_chunk(w, "gate2")
        temb, xi, xt = rand_inputs(rng)
        oi, ot = O.block_forward(CFG, w, temb, xi, xt, rope=rope)
        ri, rt = _attn_half_torch(CFG, w, temb, xi, xt, rope)
        np.testing.assert_allclose(oi, ri, rtol=1e-10, atol=1e-11)
        np.testing.assert_allclose(ot, rt, rtol=1e-10, atol=1e-11)


def test_image_token_permutation_equivariance_without_rope(rng):
    w = rand_weights(rng)
    temb, xi, xt = rand_inputs(rng)
    perm = rng.permutation(CFG.n_img)
    oi, ot = O.block_forward(CFG, w, temb, xi, xt, rope=False)
    pi, pt = O.block_forward(CFG, w, temb, xi[:, perm], xt, rope=False)
    np.testing.assert_allclose(pi, oi[:, perm], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(pt, ot, rtol=1e-11, atol=1e-12)
    # with RoPE on the same permutation is NOT an equivariance (positions are tied to the grid)
    ri, _ = O.block_forward(CFG, w, temb, xi, xt, rope=True)
    qi, _ = O.block_forward(CFG, w, temb, xi[:, perm], xt, rope=True)
    assert np.max(np.abs(qi - ri[:, perm])) > 1e-6


def test_stream_exchange_symmetry_without_rope(rng):
    """Same weights in both streams and no RoPE: which tokens are 'text' does not matter."""
    w = rand_weights(rng)
    w["txt"] = {t: a.copy() for t, a in w["img"].items()}
    temb, xi, xt = rand_inputs(rng)
    oi, ot = O.block_forward(CFG, w, temb, xi, xt, rope=False)
    # move the first 7 image tokens into the text stream (5 + 7 = 12 text, 5 image)
    cfg2 = dataclasses.replace(CFG, grid_h=1, grid_w=5, n_txt=12)
    xt2 = np.concatenate([xt, xi[:, :7]], axis=1)
    xi2 = xi[:, 7:]
    oi2, ot2 = O.block_forward(cfg2, w, temb, xi2, xt2, rope=False)
    np.testing.assert_allclose(ot2[:, :5], ot, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(ot2[:, 5:], oi[:, :7], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(oi2, oi[:, 7:], rtol=1e-11, atol=1e-12)


def test_sampled_rows_equal_full(rng):
    w = rand_weights(rng)
    temb, xi, xt = rand_inputs(rng)
    oi, ot = O.block_forward(CFG, w, temb, xi, xt)
    ri, rt = [3, 0, 11], [4, 1]
    si_, st_ = O.block_forward_sample(CFG, w, temb[1], xi[1], xt[1], img_rows=ri, txt_rows=rt)
    np.testing.assert_allclose(si_, oi[1][ri], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(st_, ot[1][rt], rtol=1e-13, atol=1e-14)


def _mlp_half_torch(w_s, temb_b, x_b):
    """The MLP half of one stream for one sample from torch primitives: the modulation chunks are
    sliced out of F.linear(F.silu(temb)) by position (shift2, scale2, gate2 = chunks 3, 4, 5)."""
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a))  # noqa: E731
    d = x_b.shape[-1]
    m = F.linear(F.silu(T(temb_b)), T(w_s["mod_w"]), T(w_s["mod_b"]))
    shift2, scale2, gate2 = m[3 * d:4 * d], m[4 * d:5 * d], m[5 * d:6 * d]
    h2 = F.layer_norm(T(x_b), (d,), eps=1e-6) * (1 + scale2) + shift2
    u = F.gelu(F.linear(h2, T(w_s["mlp1_w"]), T(w_s["mlp1_b"])), approximate="tanh")
    return (T(x_b) + gate2 * F.linear(u, T(w_s["mlp2_w"]), T(w_s["mlp2_b"]))).numpy()


def _mod_row(w_s, temb_b):
    return {k: v[0] for k, v in O.modulation(temb_b[None, :], w_s["mod_w"], w_s["mod_b"]).items()}


def test_mlp_half_function_against_torch_and_block(rng):
    """O.mlp_half (the reference of the GPU MLP-half tests) equals a torch composition of the same
    step, and equals the whole block with gate1 = 0 (only the MLP branch left)."""
    w = rand_weights(rng)
    temb, xi, xt = rand_inputs(rng)
    for s, x in (("img", xi), ("txt", xt)):
        for b in range(CFG.batch):
            got = O.mlp_half(w[s], _mod_row(w[s], temb[b]), x[b])
            np.testing.assert_allclose(got, _mlp_half_torch(w[s], temb[b], x[b]), rtol=1e-11, atol=1e-12)
    zero_chunk(w, "gate1")
    oi, ot = O.block_forward(CFG, w, temb, xi, xt)
    for s, x, out in (("img", xi, oi), ("txt", xt, ot)):
        for b in range(CFG.batch):
            np.testing.assert_allclose(O.mlp_half(w[s], _mod_row(w[s], temb[b]), x[b]), out[b],
                                       rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("swap", [("scale2", "scale1"), ("shift2", "shift1"), ("gate2", "gate1")])
def test_mlp_half_planted_chunk_mistake_fails_the_pin(rng, swap):
    """A version of mlp_half that reads the pre-attention chunk instead of the MLP one (e.g. scale1
    for scale2) is caught by the torch comparison above."""
    w = rand_weights(rng)
    temb, xi, _ = rand_inputs(rng)
    m = _mod_row(w["img"], temb[0])
    bad = dict(m)
    bad[swap[0]] = m[swap[1]]
    ref = _mlp_half_torch(w["img"], temb[0], xi[0])
    assert not np.allclose(O.mlp_half(w["img"], bad, xi[0]), ref, rtol=1e-11, atol=1e-12)
