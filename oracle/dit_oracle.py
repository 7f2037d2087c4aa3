"""Oracle: plain float64 definitions of one K-seed DiT denoise step.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import or run this module. It shares
no code with the HIP library (``paper_2606_19004_amd``) and imports nothing
from it; the only common module is ``seeded_inputs`` (draws and shapes, no
arithmetic of the method).

What is computed, and where it comes from. The paper (Spotlight, arXiv
2606.19004) is a scheduling system; it fixes *what* runs per request but not
the model internals:
  * rollout = K samples per prompt with distinct seeds (a "prompt group"),
    section 2.1 and Fig. "fig:grpo";
  * each denoising step is one full forward pass of the DiT backbone
    (Qwen-Image), section 2.1;
  * the sampler backbone is FlowGRPO, section 5 (SDE window: Table
    "tab:convergence_hyperparams", appendix);
  * per-sample scalar rewards r_k are aggregated per prompt group; the planner
    uses the per-group reward standard deviation sigma_g (section 4.3.2) and
    seed selection keeps the top-k / bottom-k seeds by reward (section 5,
    "Dynamic Exploration"; DanceGRPO's top and bottom K/2, section 2.2).
The MMDiT block itself (adaLN-modulated LayerNorm, QKV, 2D RoPE, joint
text+image attention, gated residuals, GELU-tanh MLP), the timestep embedding
and the SDE formula are not given by the paper; the readings used here are
the public dual-stream MMDiT / rectified-flow conventions, listed one by one
in the design notes and next to each function below.

Every function works on float64 arrays holding exactly the (bf16- or
fp32-representable) inputs, and keeps float64 throughout: no intermediate is
rounded. Pins for each function live in tests/test_oracle_*.py.
"""
from __future__ import annotations

import math

import numpy as np

LN_EPS = 1e-6
ROPE_THETA = 10000.0
ADV_EPS = 1e-4
TIME_FREQ_DIM = 256
TIME_SCALE = 1000.0
TIME_MAX_PERIOD = 10000.0


# ---------------------------------------------------------------------------
# elementwise pieces
# ---------------------------------------------------------------------------
def silu(z):
    """SiLU(z) = z * sigmoid(z) (reading: the modulation input is SiLU(temb))."""
    return z / (1.0 + np.exp(-z))


def gelu_tanh(z):
    """GELU, tanh form: 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3)))."""
    return 0.5 * z * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (z + 0.044715 * z ** 3)))


def layer_norm(x, eps=LN_EPS):
    """LayerNorm over the last axis, biased variance, no affine (reading)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def linear(x, w, b):
    """y = x W^T + b with W stored [out][in]."""
    return x @ w.T + b


# ---------------------------------------------------------------------------
# adaLN modulation
# ---------------------------------------------------------------------------
MOD_CHUNKS = ("shift1", "scale1", "gate1", "shift2", "scale2", "gate2")


def modulation(temb, w_mod, b_mod):
    """m = W_mod SiLU(temb) + b_mod, split into six D-wide chunks in the order
    (shift1, scale1, gate1, shift2, scale2, gate2).  temb [B][D] -> dict of [B][D]."""
    m = linear(silu(temb), w_mod, b_mod)
    d = temb.shape[-1]
    return {name: m[..., i * d:(i + 1) * d] for i, name in enumerate(MOD_CHUNKS)}


def modulate(x, shift, scale, eps=LN_EPS):
    """h = LN(x) * (1 + scale) + shift; shift/scale [B][D] broadcast over tokens."""
    return layer_norm(x, eps) * (1.0 + scale[:, None, :]) + shift[:, None, :]


# ---------------------------------------------------------------------------
# 2D rotary position embedding on image tokens
# ---------------------------------------------------------------------------
def rope_angles(pos, m, theta=ROPE_THETA):
    """Angles pos * theta^(-2i/m) for the m/2 pairs of one axis half (size m)."""
    i = np.arange(m // 2, dtype=np.float64)
    return np.asarray(pos, dtype=np.float64)[..., None] * theta ** (-2.0 * i / m)


def rope_2d(x, grid_h, grid_w, theta=ROPE_THETA):
    """Axial 2D RoPE on image tokens.

    x: [..., N_i, H, d] with image token n = r * grid_w + c.  Head dims
    [0, d/2) rotate by the row r, dims [d/2, d) by the column c; inside a half
    of size m = d/2 the pairs are (2i, 2i+1) and rotate by pos * theta^(-2i/m):
    (a, b) -> (a cos - b sin, a sin + b cos)."""
    d = x.shape[-1]
    m = d // 2
    n = np.arange(grid_h * grid_w)
    out = np.array(x, dtype=np.float64, copy=True)
    for half, pos in ((0, n // grid_w), (1, n % grid_w)):
        ang = rope_angles(pos, m, theta)                     # [N_i][m/2]
        cos = np.cos(ang)[:, None, :]                         # broadcast over heads
        sin = np.sin(ang)[:, None, :]
        a = x[..., half * m + 0:half * m + m:2]
        b = x[..., half * m + 1:half * m + m:2]
        out[..., half * m + 0:half * m + m:2] = a * cos - b * sin
        out[..., half * m + 1:half * m + m:2] = a * sin + b * cos
    return out


# ---------------------------------------------------------------------------
# attention
# ---------------------------------------------------------------------------
def attention(q, k, v, scale=None):
    """Non-causal softmax attention for one (sample, head).

    q [Nq][d], k, v [S][d] -> o [Nq][d] with o_i = sum_j p_ij v_j,
    p_i = softmax_j(q_i . k_j * scale), scale = 1/sqrt(d) by default.
    Max subtraction keeps exp finite; it does not change the result."""
    if scale is None:
        scale = 1.0 / math.sqrt(q.shape[-1])
    s = (q @ k.T) * scale
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p /= p.sum(axis=-1, keepdims=True)
    return p @ v


def joint_attention(q, k, v, scale=None):
    """Multi-head attention over a joint sequence.

    q [Nq][H][d], k/v [S][H][d] -> o [Nq][H][d]; every query attends to all S
    keys (text and image, no mask)."""
    out = np.empty(q.shape, dtype=np.float64)
    for h in range(q.shape[1]):
        out[:, h, :] = attention(q[:, h, :], k[:, h, :], v[:, h, :], scale)
    return out


# ---------------------------------------------------------------------------
# one dual-stream MMDiT block
# ---------------------------------------------------------------------------
def _qkv(h, w, heads):
    qkv = linear(h, w["qkv_w"], w["qkv_b"])                 # [N][3D]
    n, d3 = qkv.shape
    d = d3 // 3
    q = qkv[:, 0 * d:1 * d].reshape(n, heads, d // heads)
    k = qkv[:, 1 * d:2 * d].reshape(n, heads, d // heads)
    v = qkv[:, 2 * d:3 * d].reshape(n, heads, d // heads)
    return q, k, v


def block_forward_sample(cfg, w, temb_b, x_img_b, x_txt_b, img_rows=None, txt_rows=None, rope=None):
    """One MMDiT block for ONE sample (seed) of the batch.

    cfg: a seeded_inputs.Shape (hidden, heads, grid, eps/theta defaults).
    w: {"img"|"txt": {tensor: float64 array}} (weights [out][in]).
    temb_b [D]; x_img_b [N_i][D]; x_txt_b [N_t][D].
    img_rows / txt_rows: which output token rows to produce (default all);
    keys and values always cover the whole joint sequence.
    Returns (x_img_out [len(img_rows)][D], x_txt_out [len(txt_rows)][D]).

    Steps: modulation per stream; h = LN(x)(1+scale1)+shift1; q,k,v = W_qkv h + b;
    2D RoPE on image q,k; joint attention over [text ; image];
    x += gate1 * (W_o o + b_o); h2 = LN(x)(1+scale2)+shift2;
    x += gate2 * (W_2 GELU_tanh(W_1 h2 + b_1) + b_2)."""
    if rope is None:
        rope = cfg.rope
    heads = cfg.heads
    n_img, n_txt = x_img_b.shape[0], x_txt_b.shape[0]
    img_rows = np.arange(n_img) if img_rows is None else np.asarray(img_rows)
    txt_rows = np.arange(n_txt) if txt_rows is None else np.asarray(txt_rows)
    x = {"img": x_img_b, "txt": x_txt_b}
    rows = {"img": img_rows, "txt": txt_rows}
    mod = {s: modulation(temb_b[None, :], w[s]["mod_w"], w[s]["mod_b"]) for s in ("img", "txt")}
    mod = {s: {c: v[0] for c, v in mod[s].items()} for s in mod}

    q, k, v = {}, {}, {}
    for s in ("img", "txt"):
        h = layer_norm(x[s]) * (1.0 + mod[s]["scale1"]) + mod[s]["shift1"]
        q[s], k[s], v[s] = _qkv(h, w[s], heads)
    if rope:
        q["img"] = rope_2d(q["img"], cfg.grid_h, cfg.grid_w)
        k["img"] = rope_2d(k["img"], cfg.grid_h, cfg.grid_w)
    k_joint = np.concatenate([k["txt"], k["img"]], axis=0)   # text first
    v_joint = np.concatenate([v["txt"], v["img"]], axis=0)

    out = {}
    for s in ("img", "txt"):
        r = rows[s]
        o = joint_attention(q[s][r], k_joint, v_joint).reshape(len(r), heads * cfg.head_dim)
        xs = x[s][r] + mod[s]["gate1"] * linear(o, w[s]["out_w"], w[s]["out_b"])
        h2 = layer_norm(xs) * (1.0 + mod[s]["scale2"]) + mod[s]["shift2"]
        u = gelu_tanh(linear(h2, w[s]["mlp1_w"], w[s]["mlp1_b"]))
        out[s] = xs + mod[s]["gate2"] * linear(u, w[s]["mlp2_w"], w[s]["mlp2_b"])
    return out["img"], out["txt"]


def block_forward(cfg, w, temb, x_img, x_txt, rope=None):
    """Batched block: temb [B][D], x_img [B][N_i][D], x_txt [B][N_t][D] -> both outputs."""
    oi, ot = [], []
    for b in range(temb.shape[0]):
        a, c = block_forward_sample(cfg, w, temb[b], x_img[b], x_txt[b], rope=rope)
        oi.append(a)
        ot.append(c)
    return np.stack(oi), np.stack(ot)


def mlp_half(w, mod_b, x_b):
    """The MLP half of a block for one sample and one stream:
    x + gate2 * (W_2 GELU_tanh(W_1 (LN(x)(1+scale2)+shift2) + b_1) + b_2)."""
    h2 = layer_norm(x_b) * (1.0 + mod_b["scale2"]) + mod_b["shift2"]
    u = gelu_tanh(linear(h2, w["mlp1_w"], w["mlp1_b"]))
    return x_b + mod_b["gate2"] * linear(u, w["mlp2_w"], w["mlp2_b"])


# ---------------------------------------------------------------------------
# full step: timestep embedding, patch embedding, final layer
# ---------------------------------------------------------------------------
def timestep_frequencies(dim=TIME_FREQ_DIM, max_period=TIME_MAX_PERIOD):
    """f_j = max_period^(-j/(dim/2)), j < dim/2 (geometric ladder from 1 down)."""
    half = dim // 2
    return np.exp(-math.log(max_period) * np.arange(half, dtype=np.float64) / half)


def timestep_sinusoid(t, dim=TIME_FREQ_DIM):
    """e(t) = [cos(1000 t f_j) ; sin(1000 t f_j)], cosine half first."""
    arg = TIME_SCALE * np.asarray(t, dtype=np.float64)[..., None] * timestep_frequencies(dim)
    return np.concatenate([np.cos(arg), np.sin(arg)], axis=-1)


def timestep_embed(t, sw):
    """temb = W_2 SiLU(W_1 e(t) + b_1) + b_2; t [B] -> [B][D]."""
    e = timestep_sinusoid(t)
    return linear(silu(linear(e, sw["t1_w"], sw["t1_b"])), sw["t2_w"], sw["t2_b"])


def patch_embed(latent, sw):
    """Packed latent tokens [B][N_i][64] -> hidden [B][N_i][D] (W_in latent + b_in)."""
    return linear(latent, sw["in_w"], sw["in_b"])


def final_layer(x_img, temb, sw):
    """Velocity head: (shift_f, scale_f) = W_f SiLU(temb) + b_f;
    v = W_out (LN(x)(1+scale_f)+shift_f) + b_out -> [B][N_i][64]."""
    d = temb.shape[-1]
    m = linear(silu(temb), sw["fmod_w"], sw["fmod_b"])
    shift, scale = m[:, :d], m[:, d:]
    return linear(modulate(x_img, shift, scale), sw["fout_w"], sw["fout_b"])


# ---------------------------------------------------------------------------
# flow-matching sampler update (FlowGRPO backbone, section 5)
# ---------------------------------------------------------------------------
def sde_sigma(t, a):
    """Noise level sigma_t = a sqrt(t / (1 - t))."""
    return a * math.sqrt(t / (1.0 - t))


def flow_step(x, v, eps, t, t_next, a):
    """One sampler step from t to t_next (< t; noise at t=1, data at t=0), h = t_next - t.

    a == 0: Euler step of the probability-flow ODE, x' = x + h v.
    a  > 0: reverse-time SDE with the same marginals.  With x_t = (1-t) x0 + t eps
    and v = eps - x0, the score is -(x + (1-t) v)/t, and the Euler-Maruyama step is
        x' = x + h (v - sigma^2/2 * score) + sigma sqrt(-h) eps,
    i.e. x' = x + h (v + sigma^2/(2t) (x + (1-t) v)) + sigma sqrt(-h) eps."""
    h = t_next - t
    if a == 0.0:
        return x + h * v
    sigma = sde_sigma(t, a)
    score = -(x + (1.0 - t) * v) / t
    return x + h * (v - 0.5 * sigma * sigma * score) + sigma * math.sqrt(-h) * eps


def flow_mean(x, v, t, t_next, a):
    """Mean of the SDE step's transition: the step above without its noise term."""
    h = t_next - t
    sigma = sde_sigma(t, a)
    score = -(x + (1.0 - t) * v) / t
    return x + h * (v - 0.5 * sigma * sigma * score)


def flow_logprob(x, v, x_next, t, t_next, a):
    """Log-density of x_next under the SDE step's Gaussian transition from x, per sample.

    The step draws x' = mean(x, v) + sigma sqrt(-h) eps with eps ~ N(0, I), so
    x' ~ N(mean, sigma^2 (-h) I); this is the per-sample likelihood that FlowGRPO's
    policy ratio is built from (section 5: FlowGRPO is the algorithm backbone).
    Reduced by summation over all latent elements of a sample (rows of the
    [batch][n] inputs): the exact log-density. The deterministic ODE step (a == 0)
    has no density; h >= 0 is not a denoising step. Both raise ValueError."""
    h = t_next - t
    if not a > 0.0:
        raise ValueError("flow_logprob needs noise_level a > 0 (the ODE step has no density)")
    if not (0.0 < t < 1.0) or not h < 0.0:
        raise ValueError("flow_logprob needs 0 < t < 1 and t_next < t")
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    v = np.atleast_2d(np.asarray(v, dtype=np.float64))
    xn = np.atleast_2d(np.asarray(x_next, dtype=np.float64))
    var = sde_sigma(t, a) ** 2 * (-h)
    r = xn - flow_mean(x, v, t, t_next, a)
    n = x.shape[1]
    return -(r * r).sum(axis=1) / (2.0 * var) - 0.5 * n * math.log(2.0 * math.pi * var)


# ---------------------------------------------------------------------------
# per prompt-group reward statistics and seed selection
# ---------------------------------------------------------------------------
def group_reward_stats(rewards, adv_eps=ADV_EPS, k_select=0):
    """Per group g of n seeds (rows of rewards [G][n]):

    mean_g, population std sigma_g (the sigma_g of section 4.3.2),
    advantages (r - mean_g) / (sigma_g + adv_eps) (GRPO normalisation; zero when
    sigma_g == 0), order = seed indices by descending reward with ties by
    ascending index, and selected = the top ceil(k/2) followed by the bottom
    floor(k/2) of that order (top/bottom seed selection, sections 2.2 and 5)."""
    r = np.asarray(rewards, dtype=np.float64)
    g, n = r.shape
    mean = r.mean(axis=1)
    std = np.sqrt(((r - mean[:, None]) ** 2).mean(axis=1))
    adv = np.where(std[:, None] > 0, (r - mean[:, None]) / (std[:, None] + adv_eps), 0.0)
    order = np.empty((g, n), dtype=np.int32)
    for i in range(g):
        order[i] = sorted(range(n), key=lambda j: (-r[i, j], j))
    top, bottom = (k_select + 1) // 2, k_select // 2
    selected = np.concatenate([order[:, :top], order[:, n - bottom:]], axis=1).astype(np.int32)
    return {"mean": mean, "std": std, "adv": adv, "order": order, "selected": selected}


# ---------------------------------------------------------------------------
# one full K-seed denoise step
# ---------------------------------------------------------------------------
def denoise_step(cfg, step_w, blocks_w, latent, x_txt, t, t_next, eps, a):
    """temb(t) -> patch embedding -> blocks -> velocity -> flow update.

    Returns (latent', v, temb). All B samples share t."""
    b = latent.shape[0]
    temb = timestep_embed(np.full(b, t), step_w)
    x_img = patch_embed(latent, step_w)
    for w in blocks_w:
        x_img, x_txt = block_forward(cfg, w, temb, x_img, x_txt)
    v = final_layer(x_img, temb, step_w)
    return flow_step(latent, v, eps, t, t_next, a), v, temb


# ---------------------------------------------------------------------------
# TeaCache gate: skip the block stack on steps whose block input barely moved
# ---------------------------------------------------------------------------
# The exploration planner lowers the effective number of denoising steps s with TeaCache
# (section 4.3.1): it caches the block stack's output residual and reuses it on steps whose
# timestep-modulated input differs little from the previous step's. Readings (the paper
# names TeaCache and does not restate it): the compared input is block 0's modulated image
# input LN(x_img)(1 + scale1) + shift1; the distance is the relative L1 distance over the
# whole batch, sum |h - h_prev| / sum |h_prev|; a caller-given polynomial rescales it
# (identity when none is given: fitted coefficients are model-specific and not printed);
# the rescaled distances accumulate across steps, and a step reuses the cached residual
# while the accumulated value stays below the threshold, otherwise it runs the blocks and
# the accumulator restarts at 0. The first step, and any step the caller forces (e.g. the
# last one), runs the blocks. The K seeds of a batch skip or run together.
def teacache_rel_l1(h_now, h_prev):
    """sum |h_now - h_prev| / sum |h_prev| over all elements."""
    h_now = np.asarray(h_now, dtype=np.float64)
    h_prev = np.asarray(h_prev, dtype=np.float64)
    return float(np.abs(h_now - h_prev).sum() / np.abs(h_prev).sum())


class TeaCacheState:
    def __init__(self, threshold, coef=()):
        self.threshold = float(threshold)
        self.coef = [float(c) for c in coef]     # highest power first; empty = identity
        self.accumulated = 0.0
        self.h_prev = None                       # block 0's modulated image input of the last step
        self.residual = None                     # x_img after the blocks minus before, last computed step

    def gate(self, rel, force=False):
        """True: run the blocks; False: reuse the cached residual. Updates the accumulator."""
        if force or self.h_prev is None or self.residual is None:
            self.accumulated = 0.0
            return True
        self.accumulated += float(np.polyval(self.coef, rel)) if self.coef else rel
        if self.accumulated < self.threshold:
            return False
        self.accumulated = 0.0
        return True


def block0_modulated_input(w0, temb, x_img):
    """LN(x_img)(1 + scale1) + shift1 with block 0's image-stream modulation, [B][N_i][D]."""
    m = modulation(temb, w0["img"]["mod_w"], w0["img"]["mod_b"])
    return modulate(x_img, m["shift1"], m["scale1"])


def denoise_step_teacache(cfg, step_w, blocks_w, latent, x_txt, t, t_next, eps, a, state, force=False):
    """denoise_step with the TeaCache gate in front of the block stack.

    Returns (latent', v, ran_blocks, rel) with rel = None on a step without a previous input."""
    b = latent.shape[0]
    temb = timestep_embed(np.full(b, t), step_w)
    x_img = patch_embed(latent, step_w)
    h0 = block0_modulated_input(blocks_w[0], temb, x_img) if blocks_w else x_img
    rel = teacache_rel_l1(h0, state.h_prev) if state.h_prev is not None else None
    run = state.gate(rel, force)
    state.h_prev = h0
    if run:
        x_in = x_img
        for w in blocks_w:
            x_img, x_txt = block_forward(cfg, w, temb, x_img, x_txt)
        state.residual = x_img - x_in
    else:
        x_img = x_img + state.residual
    v = final_layer(x_img, temb, step_w)
    return flow_step(latent, v, eps, t, t_next, a), v, run, rel
