"""Helpers for the GPU parity tests: move seeded storage arrays to the device,
read results back as float64, and the error metric the tests gate on."""
import numpy as np
import torch

import seeded_inputs as si


def dev(a: np.ndarray, dtype: str = "f32") -> torch.Tensor:
    """Storage array (uint16 bf16 bits or float32) -> device tensor of that type."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def host64(t: torch.Tensor) -> np.ndarray:
    """Device tensor (bf16 or fp32) -> exact float64 values on the host."""
    if t.dtype == torch.bfloat16:
        return si.bf16_bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    return t.float().cpu().numpy().astype(np.float64)


def upload_block(w: dict, dtype: str) -> dict:
    return {s: {t: dev(a, dtype) for t, a in ws.items()} for s, ws in w.items()}


def rel_err(got, ref) -> float:
    """Normwise max relative error max|got - ref| / max|ref|."""
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-300))


def block_cfg(ditstep, cfg: si.Shape):
    return ditstep.block_config(cfg.hidden, cfg.heads, cfg.head_dim, cfg.mlp_hidden, cfg.n_img, cfg.n_txt,
                                cfg.grid_h, cfg.grid_w, rope=cfg.rope, dtype=cfg.dtype)
