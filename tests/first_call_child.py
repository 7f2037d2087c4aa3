"""Child process of test_gpu_first_call_threads: the library's first GEMM calls of a process are
made from four host threads at once (two on the 256 x 256 tile path, two on the 128 x 128 path,
each with its own stream, inputs and workspace); every result must equal, bit for bit, the same
call repeated afterwards one at a time. Prints one line "ok" or raises."""
import os
import sys
import threading

import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import seeded_inputs as si  # noqa: E402
from tests.gpu_util import block_cfg, dev, upload_block  # noqa: E402


def main():
    from paper_2606_19004_amd import ditstep as d
    cases = [(si.CONFIGS["mlp_short_k128"], si.MASTER_SEED + 1), (si.CONFIGS["mlp_short_k128"], si.MASTER_SEED + 2),
             (si.CONFIGS["small_bf16"], si.MASTER_SEED + 3), (si.CONFIGS["small_bf16"], si.MASTER_SEED + 4)]

    def prepare(cfg, seed):
        inp = si.block_inputs(cfg, seed=seed)
        c = block_cfg(d, cfg)
        w = upload_block(inp["weights"], cfg.dtype)
        return (c, d.block_weights(w["img"], w["txt"]), dev(inp["temb"]), dev(inp["x_img"], cfg.dtype),
                dev(inp["x_txt"], cfg.dtype), d.workspace(d.dit_block_workspace_bytes(c, cfg.batch)), w)

    par = [prepare(c, s) for c, s in cases]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in cases]
    gate = threading.Barrier(len(cases))
    errs = []

    def worker(a, st):
        try:
            c, bw, temb, xi, xt, ws, _ = a
            gate.wait()
            d.dit_block_forward(c, bw, temb, xi, xt, ws, stream=st)
            st.synchronize()
        except Exception as e:  # reported after the join
            errs.append(repr(e))

    threads = [threading.Thread(target=worker, args=(a, st)) for a, st in zip(par, streams)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    if errs:
        raise RuntimeError(errs)
    for (cfg, seed), a in zip(cases, par):
        b = prepare(cfg, seed)
        c, bw, temb, xi, xt, ws, _ = b
        d.dit_block_forward(c, bw, temb, xi, xt, ws)
        torch.cuda.synchronize()
        if not (torch.equal(a[3], b[3]) and torch.equal(a[4], b[4])):
            raise AssertionError(f"threaded first call differs from the sequential call ({cfg.name}, seed {seed})")
    print("ok", flush=True)


if __name__ == "__main__":
    main()
