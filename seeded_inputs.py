"""Seeded synthetic inputs for the K-seed DiT denoise step.

This module is shared by the CPU oracle and the HIP path and therefore holds
none of the method's arithmetic: only workload shapes, seeded random draws and
the bf16 storage format (round-to-nearest-even of fp32, an input-preparation
step that both sides consume as given).

Recipe (every tensor is drawn independently):
  * tensor named ``name`` under master seed ``s`` is drawn from
    ``numpy.random.default_rng([s, crc32(name)])``, so a tensor never changes
    when another one is added;
  * linear weights and biases ~ N(0, 0.02);
  * image hidden states, text hidden states and block-level temb ~ N(0, 1);
  * per-sample latent noise ~ N(0, 1), drawn per seed from ``[s, 1000 + k]``
    (one deterministic seed per sample, as the paper's evaluation assigns);
  * timestep t ~ U(0, 1) (one t per denoise step, shared by the K seeds);
  * SDE noise eps ~ N(0, 1); rewards ~ U(0, 1).

Shapes follow Qwen-Image-sized MMDiT blocks (hidden 3072, 24 heads x 128) at
512x512 (32x32 latent tokens + 256 text tokens) and 1280x1280 (80x80 + 512)
and a tiny fp32 model; the paper's benchmarks (DeepSeek-OCR, Geneval prompts
scored by reward models) are replaced by these synthetic draws.
"""
from __future__ import annotations

import dataclasses
import zlib

import numpy as np

MASTER_SEED = 42


# --------------------------------------------------------------------------
# workload shapes
# --------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class Shape:
    name: str
    hidden: int
    heads: int
    head_dim: int
    grid_h: int
    grid_w: int
    n_txt: int
    batch: int
    dtype: str = "bf16"          # "bf16" or "f32": storage/compute type
    blocks: int = 1
    mlp_ratio: int = 4
    rope: bool = True
    # full-step extras
    latent_dim: int = 64         # 16 latent channels x 2x2 patch
    noise_level: float = 0.0     # SDE noise scale a (0 = Euler ODE)
    dt: float = 0.05
    reward_groups: int = 0
    reward_n: int = 0
    reward_k: int = 0

    @property
    def n_img(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def seq(self) -> int:
        return self.n_img + self.n_txt

    @property
    def mlp_hidden(self) -> int:
        return self.mlp_ratio * self.hidden

    def gemm_flops_per_block(self) -> float:
        """2*M*N*K summed over QKV (3D), out (D), MLP up (4D) and down (4D)."""
        d, f = self.hidden, self.mlp_hidden
        m = self.batch * self.seq
        return 2.0 * m * d * (3 * d + d + f + f)

    def attn_flops_per_block(self) -> float:
        """QK^T and PV over the joint sequence, non-causal: 4*B*H*S^2*d."""
        return 4.0 * self.batch * self.heads * self.seq * self.seq * self.head_dim


CONFIGS = {
    # tiny fp32 model: one block, hidden 256, 4x64 heads, 8x8 latent grid, 16 text tokens, K=2
    "tiny_f32": Shape("tiny_f32", 256, 4, 64, 8, 8, 16, 2, dtype="f32", blocks=1, dt=0.05),
    # 512x512-shaped single block, K=8
    "block_512": Shape("block_512", 3072, 24, 128, 32, 32, 256, 8),
    # 1280x1280-shaped single block, K=4
    "block_1280": Shape("block_1280", 3072, 24, 128, 80, 80, 512, 4),
    # one sequence-parallel rank's share at 1280x1280: 6 of 24 heads over all 6912 tokens, K=8
    # (hidden is the sliced width 6*128; the MLP part uses `mlp_slice_1280`)
    "headslice_1280": Shape("headslice_1280", 768, 6, 128, 80, 80, 512, 8),
    # full-hidden MLP on a 1728-token slice of that rank: 1600 image + 128 text tokens, K=8
    "mlp_slice_1280": Shape("mlp_slice_1280", 3072, 24, 128, 40, 40, 128, 8, rope=False),
    # full denoise step: 8 blocks at 512x512 shape, K=16, SDE a=0.7, rewards 64 groups x 16 seeds
    "step_512_k16": Shape("step_512_k16", 3072, 24, 128, 32, 32, 256, 16, blocks=8,
                          noise_level=0.7, dt=0.05, reward_groups=64, reward_n=16, reward_k=4),
    # small bf16 cases for element-wise parity: several tiles plus ragged tails
    "small_bf16": Shape("small_bf16", 256, 2, 128, 7, 9, 21, 3),
    "small_bf16_d64": Shape("small_bf16_d64", 320, 5, 64, 11, 13, 37, 2),
    # MLP half with a long down-projection (K = 4*2176 = 8704) and ragged rows and columns
    # (63 + 21 tokens x 3 seeds; 2176 output features): the three-stage GEMM path with partial tiles
    "mlp_long_k": Shape("mlp_long_k", 2176, 17, 128, 7, 9, 21, 3, rope=False),
    # MLP halves with short up projections (K = 128 and 192: two and three 64-deep k-tiles) over
    # 16 x (64x64 + 100) rows, enough 256 x 256 tiles to take the large-tile GEMM path, with a
    # partial last row tile in each stream
    "mlp_short_k128": Shape("mlp_short_k128", 128, 1, 128, 64, 64, 100, 16, rope=False),
    "mlp_short_k192": Shape("mlp_short_k192", 192, 3, 64, 64, 64, 100, 16, rope=False),
    "small_step_bf16": Shape("small_step_bf16", 256, 2, 128, 8, 12, 24, 4, blocks=2,
                             noise_level=0.7, dt=0.05, reward_groups=5, reward_n=4, reward_k=2),
}


# --------------------------------------------------------------------------
# seeded draws
# --------------------------------------------------------------------------
def _rng(name: str, seed: int) -> np.random.Generator:
    return np.random.default_rng([seed, zlib.crc32(name.encode())])


def normal(name: str, shape, std: float = 1.0, seed: int = MASTER_SEED) -> np.ndarray:
    x = _rng(name, seed).standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


def uniform(name: str, shape, lo: float = 0.0, hi: float = 1.0, seed: int = MASTER_SEED) -> np.ndarray:
    return _rng(name, seed).uniform(lo, hi, size=shape).astype(np.float32)


def sample_noise(k: int, shape, seed: int = MASTER_SEED) -> np.ndarray:
    """Per-sample deterministic noise: sample k draws from seed [seed, 1000+k]."""
    return np.random.default_rng([seed, 1000 + k]).standard_normal(size=shape, dtype=np.float32)


# --------------------------------------------------------------------------
# bf16 storage format (round to nearest even), as bit patterns in uint16
# --------------------------------------------------------------------------
def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def stored(x: np.ndarray, dtype: str) -> np.ndarray:
    """fp32 draw -> storage array: uint16 bf16 bits for "bf16", float32 for "f32"."""
    return to_bf16_bits(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def as_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Storage array -> the exact values it holds, as float64."""
    if dtype == "bf16":
        return bf16_bits_to_f32(x).astype(np.float64)
    return np.asarray(x, dtype=np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# tensor sets
# --------------------------------------------------------------------------
STREAMS = ("img", "txt")
BLOCK_TENSORS = ("mod_w", "mod_b", "qkv_w", "qkv_b", "out_w", "out_b",
                 "mlp1_w", "mlp1_b", "mlp2_w", "mlp2_b")


def block_weight_shapes(cfg: Shape) -> dict:
    d, f = cfg.hidden, cfg.mlp_hidden
    return {"mod_w": (6 * d, d), "mod_b": (6 * d,), "qkv_w": (3 * d, d), "qkv_b": (3 * d,),
            "out_w": (d, d), "out_b": (d,), "mlp1_w": (f, d), "mlp1_b": (f,),
            "mlp2_w": (d, f), "mlp2_b": (d,)}


def block_weights(cfg: Shape, layer: int = 0, seed: int = MASTER_SEED) -> dict:
    """{stream: {tensor: storage array}} for one MMDiT block; weights [out][in]."""
    out = {}
    for s in STREAMS:
        out[s] = {}
        for t, shp in block_weight_shapes(cfg).items():
            out[s][t] = stored(normal(f"{cfg.name}/L{layer}/{s}/{t}", shp, 0.02, seed), cfg.dtype)
    return out


def block_inputs(cfg: Shape, seed: int = MASTER_SEED) -> dict:
    """Inputs of one block call: weights, temb [B][D] fp32, x_img [B][N_i][D], x_txt [B][N_t][D]."""
    b, d = cfg.batch, cfg.hidden
    return {
        "weights": block_weights(cfg, 0, seed),
        "temb": normal(f"{cfg.name}/temb", (b, d), 1.0, seed),
        "x_img": stored(normal(f"{cfg.name}/x_img", (b, cfg.n_img, d), 1.0, seed), cfg.dtype),
        "x_txt": stored(normal(f"{cfg.name}/x_txt", (b, cfg.n_txt, d), 1.0, seed), cfg.dtype),
    }


def step_weight_shapes(cfg: Shape) -> dict:
    d, c = cfg.hidden, cfg.latent_dim
    return {"t1_w": (d, 256), "t1_b": (d,), "t2_w": (d, d), "t2_b": (d,),
            "in_w": (d, c), "in_b": (d,), "fmod_w": (2 * d, d), "fmod_b": (2 * d,),
            "fout_w": (c, d), "fout_b": (c,)}


def step_inputs(cfg: Shape, seed: int = MASTER_SEED) -> dict:
    """Inputs of one full denoise step (timestep MLP, patch embedding, blocks, final layer,
    flow update, reward statistics)."""
    b = cfg.batch
    extra = {t: stored(normal(f"{cfg.name}/{t}", shp, 0.02, seed), cfg.dtype)
             for t, shp in step_weight_shapes(cfg).items()}
    t = float(uniform(f"{cfg.name}/t", (1,), seed=seed)[0])
    t = min(max(t, 0.06), 0.94)   # keep t - dt inside (0, 1) for the SDE domain
    latent = np.stack([sample_noise(k, (cfg.n_img, cfg.latent_dim), seed) for k in range(b)])
    text = normal(f"{cfg.name}/text", (1, cfg.n_txt, cfg.hidden), 1.0, seed)
    text = np.ascontiguousarray(np.broadcast_to(text, (b, cfg.n_txt, cfg.hidden)))
    out = {
        "step_weights": extra,
        "blocks": [block_weights(cfg, i, seed) for i in range(cfg.blocks)],
        "t": t,
        "t_next": max(t - cfg.dt, 0.0),
        "latent": latent.astype(np.float32),
        "x_txt": stored(text, cfg.dtype),
        "eps": normal(f"{cfg.name}/eps", (b, cfg.n_img, cfg.latent_dim), 1.0, seed),
    }
    if cfg.reward_groups:
        out["rewards"] = uniform(f"{cfg.name}/rewards", (cfg.reward_groups, cfg.reward_n), seed=seed)
    return out
