"""Child process of test_gpu_debug_build: runs a block forward (two tile paths), the MLP-only entry
and a two-block denoise step on seeded inputs with whichever library DITSTEP_LIB selects, and saves
the outputs to the .npz named by argv[1]. Prints "ok <library>" at the end."""
import os
import sys

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import seeded_inputs as si  # noqa: E402
from tests.gpu_util import block_cfg, dev, upload_block  # noqa: E402


def main():
    from paper_2606_19004_amd import ditstep as d
    out = {}
    for name in ("small_bf16", "mlp_short_k128"):
        cfg = si.CONFIGS[name]
        inp = si.block_inputs(cfg)
        c = block_cfg(d, cfg)
        w = upload_block(inp["weights"], cfg.dtype)
        bw = d.block_weights(w["img"], w["txt"])
        ws = d.workspace(d.dit_block_workspace_bytes(c, cfg.batch))
        for entry in ("forward", "mlp"):
            xi, xt = dev(inp["x_img"], cfg.dtype), dev(inp["x_txt"], cfg.dtype)
            fn = d.dit_block_forward if entry == "forward" else d.dit_block_mlp
            fn(c, bw, dev(inp["temb"]), xi, xt, ws)
            torch.cuda.synchronize()
            out[f"{name}_{entry}_img"] = xi.view(torch.int16).cpu().numpy()
            out[f"{name}_{entry}_txt"] = xt.view(torch.int16).cpu().numpy()
    cfg = si.CONFIGS["small_step_bf16"]
    inp = si.step_inputs(cfg)
    c = block_cfg(d, cfg)
    swd = {k: dev(v, cfg.dtype) for k, v in inp["step_weights"].items()}
    blocks = [d.block_weights(b["img"], b["txt"]) for b in (upload_block(x, cfg.dtype) for x in inp["blocks"])]
    lat, v = dev(inp["latent"]), torch.zeros_like(dev(inp["latent"]))
    ws = d.workspace(d.dit_denoise_workspace_bytes(c, cfg.batch, cfg.latent_dim))
    a = cfg.noise_level
    d.dit_denoise_step(c, d.step_weights(swd), blocks, inp["t"], inp["t_next"], a, lat,
                       dev(inp["x_txt"], cfg.dtype), dev(inp["eps"]) if a > 0 else None, v, ws)
    torch.cuda.synchronize()
    out["step_latent"] = lat.cpu().numpy()
    out["step_v"] = v.cpu().numpy()
    np.savez(sys.argv[1], **out)
    print("ok", os.path.basename(d.LIB_PATH), flush=True)


if __name__ == "__main__":
    main()
