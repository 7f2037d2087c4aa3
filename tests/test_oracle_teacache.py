"""Pins for the oracle's TeaCache gate.

Pinned against things other than the oracle's own code:
  * the relative L1 distance on hand-computed arrays, its scale invariance and its value 0 for
    equal inputs;
  * a hand-worked gate sequence (threshold 0.3, identity rescale): distances 0.1, 0.15, 0.1,
    0.02, 0.25 accumulate to 0.1, 0.25, 0.35 -> run and reset, 0.02, 0.27: skip, skip, run,
    skip, skip; a forced step runs and resets; a rescale polynomial 2x doubles the distances;
  * the step: threshold 0 runs the blocks every time and equals denoise_step exactly; a huge
    threshold reuses the first step's residual, which equals the blocks' output minus input
    recomputed independently; planted mistakes (residual not refreshed, h_prev not updated on
    skipped steps) fail those checks.
"""
import dataclasses

import numpy as np
import pytest

import seeded_inputs as si
from oracle import dit_oracle as O


def test_rel_l1_hand_values():
    prev = np.array([[1.0, -2.0], [3.0, 0.0]])
    now = np.array([[1.5, -2.0], [2.0, 1.0]])
    # |diff| = 0.5 + 0 + 1 + 1 = 2.5 ; sum |prev| = 6
    assert O.teacache_rel_l1(now, prev) == pytest.approx(2.5 / 6.0, rel=1e-15)
    assert O.teacache_rel_l1(7.0 * now, 7.0 * prev) == pytest.approx(2.5 / 6.0, rel=1e-14)
    assert O.teacache_rel_l1(prev, prev) == 0.0


def test_gate_hand_sequence():
    st = O.TeaCacheState(0.3)
    st.h_prev, st.residual = 1, 1          # past the first step
    runs = [st.gate(r) for r in (0.1, 0.15, 0.1, 0.02, 0.25)]
    assert runs == [False, False, True, False, False]
    assert st.accumulated == pytest.approx(0.27)
    assert st.gate(0.01, force=True) is True and st.accumulated == 0.0
    st2 = O.TeaCacheState(0.3, coef=[2.0, 0.0])   # rescale r -> 2 r
    st2.h_prev, st2.residual = 1, 1
    assert [st2.gate(r) for r in (0.1, 0.1, 0.05)] == [False, True, False]
    fresh = O.TeaCacheState(100.0)
    assert fresh.gate(0.0) is True                 # no previous input: run


def _setup(name="small_step_bf16"):
    cfg = si.CONFIGS[name]
    inp = si.step_inputs(cfg)
    f = lambda a: si.as_f64(a, cfg.dtype)  # noqa: E731
    sw = {k: f(a) for k, a in inp["step_weights"].items()}
    bw = [{s: {k: f(a) for k, a in b[s].items()} for s in b} for b in inp["blocks"]]
    return cfg, inp, sw, bw, f


def test_threshold_zero_equals_plain_step():
    cfg, inp, sw, bw, f = _setup()
    st = O.TeaCacheState(0.0)
    lat = inp["latent"].astype(np.float64)
    xt = f(inp["x_txt"])
    eps = inp["eps"].astype(np.float64)
    t = 0.8
    for k in range(3):
        want, wv, _ = O.denoise_step(cfg, sw, bw, lat, xt, t, t - 0.05, eps, 0.7)
        got, gv, ran, rel = O.denoise_step_teacache(cfg, sw, bw, lat, xt, t, t - 0.05, eps, 0.7, st)
        assert ran and (rel is None) == (k == 0)
        assert np.array_equal(got, want) and np.array_equal(gv, wv)
        lat, t = want, t - 0.05


def test_large_threshold_reuses_first_residual(monkeypatch):
    cfg, inp, sw, bw, f = _setup()
    lat0 = inp["latent"].astype(np.float64)
    xt = f(inp["x_txt"])
    eps = inp["eps"].astype(np.float64)
    st = O.TeaCacheState(1e9)
    lat1, _, ran, _ = O.denoise_step_teacache(cfg, sw, bw, lat0, xt, 0.8, 0.75, eps, 0.7, st)
    assert ran
    # residual of step 1, recomputed directly
    temb = O.timestep_embed(np.full(lat0.shape[0], 0.8), sw)
    x0 = O.patch_embed(lat0, sw)
    x = x0
    xtt = xt
    for w in bw:
        x, xtt = O.block_forward(cfg, w, temb, x, xtt)
    np.testing.assert_allclose(st.residual, x - x0, rtol=0, atol=1e-12)
    lat2, v2, ran2, rel2 = O.denoise_step_teacache(cfg, sw, bw, lat1, xt, 0.75, 0.7, eps, 0.7, st)
    assert not ran2 and rel2 > 0
    temb2 = O.timestep_embed(np.full(lat0.shape[0], 0.75), sw)
    x2 = O.patch_embed(lat1, sw) + (x - x0)
    v_want = O.final_layer(x2, temb2, sw)
    np.testing.assert_allclose(v2, v_want, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lat2, O.flow_step(lat1, v_want, eps, 0.75, 0.7, 0.7), rtol=0, atol=1e-12)
    # h_prev follows every step, skipped or not
    np.testing.assert_allclose(st.h_prev, O.block0_modulated_input(bw[0], temb2, O.patch_embed(lat1, sw)), atol=1e-12)


def test_planted_mistake_stale_h_prev_changes_distances():
    cfg, inp, sw, bw, f = _setup()
    lat = inp["latent"].astype(np.float64)
    xt = f(inp["x_txt"])
    eps = inp["eps"].astype(np.float64)
    good, bad = O.TeaCacheState(1e9), O.TeaCacheState(1e9)
    rels_good, rels_bad = [], []
    lg = lb = lat
    for k, t in enumerate((0.8, 0.75, 0.7, 0.65)):
        lg, _, _, rg = O.denoise_step_teacache(cfg, sw, bw, lg, xt, t, t - 0.05, eps, 0.7, good)
        keep = bad.h_prev
        lb, _, _, rb = O.denoise_step_teacache(cfg, sw, bw, lb, xt, t, t - 0.05, eps, 0.7, bad)
        if k >= 1:
            bad.h_prev = keep          # mistake: the cached input is only refreshed on computed steps
        rels_good.append(rg)
        rels_bad.append(rb)
    assert rels_good[:2] == rels_bad[:2]
    assert rels_good[2] != rels_bad[2]


def _block0_input_torch(w0, temb, x_img):
    """LN(x_img)(1 + scale1) + shift1 from torch primitives, with the image stream's modulation
    sliced by position (shift1 = chunk 0, scale1 = chunk 1)."""
    import torch
    import torch.nn.functional as F
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a))  # noqa: E731
    d = x_img.shape[-1]
    m = F.linear(F.silu(T(temb)), T(w0["img"]["mod_w"]), T(w0["img"]["mod_b"]))
    shift1, scale1 = m[:, :d], m[:, d:2 * d]
    return (F.layer_norm(T(x_img), (d,), eps=1e-6) * (1 + scale1[:, None]) + shift1[:, None]).numpy()


def _block0_case():
    rng = np.random.default_rng(77)
    cfg = si.Shape("pin_b0", hidden=32, heads=2, head_dim=16, grid_h=3, grid_w=4, n_txt=5, batch=3, dtype="f32")
    w0 = {s: {t: rng.standard_normal(shp) * 0.3 for t, shp in si.block_weight_shapes(cfg).items()}
          for s in ("img", "txt")}
    temb = rng.standard_normal((cfg.batch, cfg.hidden))
    x = rng.standard_normal((cfg.batch, cfg.n_img, cfg.hidden)) * 2.0 + 0.5
    return w0, temb, x


def test_block0_modulated_input_against_torch():
    w0, temb, x = _block0_case()
    np.testing.assert_allclose(O.block0_modulated_input(w0, temb, x), _block0_input_torch(w0, temb, x),
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("mistake", ["chunks_2", "text_stream"])
def test_block0_modulated_input_planted_mistakes_fail_the_pin(mistake):
    """Reading the pre-MLP chunks (shift2, scale2) or the text stream's modulation weights instead of
    the image stream's shift1/scale1 gives a different value, which the torch comparison catches."""
    w0, temb, x = _block0_case()
    ref = _block0_input_torch(w0, temb, x)
    if mistake == "chunks_2":
        m = O.modulation(temb, w0["img"]["mod_w"], w0["img"]["mod_b"])
        bad = O.modulate(x, m["shift2"], m["scale2"])
    else:
        bad = O.block0_modulated_input({"img": w0["txt"]}, temb, x)
    assert not np.allclose(bad, ref, rtol=1e-12, atol=1e-12)
