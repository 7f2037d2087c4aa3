#!/usr/bin/env python3
"""Benchmark: milliseconds per K-seed DiT denoise step on one MI355X.

One step = the whole hot path over one batch: timestep embedding, patch
embedding, 8 dual-stream MMDiT blocks (hidden 3072, 24 heads x 128, 1024 image
+ 256 text tokens, K = 16 seeds), velocity head, SDE flow update (a = 0.7),
then per-group reward statistics with argsort over 64 prompt groups x 16
seeds. Inputs are synthetic and seeded (weights N(0, 0.02) in bf16, hidden
states N(0, 1), rewards U(0, 1)), resident in HBM before timing starts.

Prints ONE JSON line: the step time, the dominant kernel's roofline fraction
(its algorithmic FLOPs per launch over its average launch time, timed with
HIP events on its stream), a per-kernel-class breakdown, and the CPU oracle
timed on a bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--config NAME] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import seeded_inputs as si  # noqa: E402

PEAK_BF16_TFLOPS = 2516.6      # MI355X dense bf16 MFMA (256 CUs x 2.4 GHz x 4096 flop/clk)
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
TRAFFIC_JSON = "profiles/gemm_step_512_k16_traffic.json"
KERNEL_MD = "profiles/step_512_k16_kernel_stats.md"
MFMA_MD = "profiles/mfma_step_512_k16_counters.md"
STALL_MD = "profiles/stalls_step_512_k16_counters.md"
STALL_COUNTERS = ("SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_WAIT_INST_LDS", "SQ_ACTIVE_INST_ANY",
                  "SQ_ACTIVE_INST_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_INST_CYCLES_VMEM_RD", "GRBM_GUI_ACTIVE")
# source file whose kernels each counted class runs (a summary is stale once that file changes)
CLASS_SOURCE = {"gemm_qkv_rope": "k_gemm.hip", "gemm_out_gate": "k_gemm.hip", "gemm_mlp_up_gelu": "k_gemm.hip",
                "gemm_mlp_down_gate": "k_gemm.hip", "attention": "k_attn.hip", "ln_modulate": "k_elementwise.hip",
                "mod_gemv": "k_elementwise.hip"}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--config", default="step_512_k16", choices=[k for k, v in si.CONFIGS.items() if v.blocks >= 1])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--headline-only", action="store_true",
                   help="time only the denoise step (no next-row or other-configuration measurements), so that "
                        "a profiler run sees only the step's kernels")
    p.add_argument("--cpu-sample-seeds", type=int, default=16)
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="only run 5 plain device copies of MIB MiB (torch copy kernel); used to scale the "
                        "FETCH_SIZE / WRITE_SIZE counters to bytes")
    p.add_argument("--traffic-summary", metavar="DIR", default=None,
                   help="no GPU: turn the four rocprofv3 --pmc runs under DIR (calib_FETCH_SIZE, "
                        "calib_WRITE_SIZE, bench_FETCH_SIZE, bench_WRITE_SIZE) into " + TRAFFIC_JSON)
    p.add_argument("--mfma-summary", metavar="DIR", default=None,
                   help="no GPU: turn a rocprofv3 --pmc run of SQ_VALU_MFMA_BUSY_CYCLES, SQ_INSTS_VALU_MFMA_MOPS_BF16 "
                        "and GRBM_GUI_ACTIVE under DIR into " + "profiles/mfma_step_512_k16_counters.md")
    p.add_argument("--stall-summary", metavar="DIR", default=None,
                   help="no GPU: turn a rocprofv3 --pmc run of the wave-state counters (SQ_WAVE_CYCLES, SQ_WAIT_ANY, "
                        "SQ_WAIT_INST_ANY, SQ_WAIT_INST_LDS, SQ_ACTIVE_INST_ANY, SQ_ACTIVE_INST_LDS, SQ_LDS_BANK_CONFLICT, "
                        "SQ_INST_CYCLES_VMEM_RD, GRBM_GUI_ACTIVE) under DIR into " + "profiles/stalls_step_512_k16_counters.md")
    p.add_argument("--kernel-summary", metavar="DIR", default=None,
                   help="no GPU: turn rocprofv3 --kernel-trace --stats output under DIR (bench_kernel_stats.csv, "
                        "bench_kernel_trace.csv) plus the bench JSON line in DIR/../bench.json into " + KERNEL_MD)
    return p.parse_args()


def copy_calibration(torch, mib):
    n = mib * (1 << 20) // 4
    src = torch.randn(n, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_per_launch": n * 4, "launches": 5}), flush=True)


def source_sha(name):
    import hashlib
    with open(os.path.join(ROOT, "paper_2606_19004_amd", "csrc", name), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def traffic_from_profile(kernel_class):
    """Measured HBM bytes per launch of one kernel class from the committed counter summary, or
    None when there is none or it was taken on another version of that kernel's source."""
    try:
        rec = json.load(open(os.path.join(ROOT, TRAFFIC_JSON)))
        c = rec["per_kernel_class"][kernel_class]
        if c["source_sha"] != source_sha(CLASS_SOURCE[kernel_class]):
            return None
        return c["hbm_bytes_per_launch"]
    except (OSError, ValueError, KeyError):
        return None


def classify_dispatches(rows):
    """Kernel class of every dispatch of one denoise-step run, in dispatch order. The two gated
    residual GEMMs of a block share one kernel; the out-projection always precedes the MLP down.
    A GEMM call may be two launches (image rows on 256 x 256 tiles, then text rows on 256 x 192
    tiles): the second launch takes the class of the first."""
    import re
    resid_seen = 0
    out = []
    prev = None   # (EPI, class) of the previous dispatch when it was a 256 x 256 GEMM
    for r in rows:
        n = r["Kernel_Name"]
        m = re.search(r"gemm_bf16_kernel<(\d+), (\d+), (\d+), (\d+), (\d+)", n)
        cls = None
        cur = None
        if m and int(m.group(1)) == 256:
            epi, bn = int(m.group(5)), int(m.group(2))
            if bn != 256 and prev is not None and prev[0] == epi:
                cls = prev[1]
            elif epi == 3:
                cls = "gemm_qkv_rope"
            elif epi == 1:
                cls = "gemm_mlp_up_gelu"
            elif epi == 2:
                cls = "gemm_out_gate" if resid_seen % 2 == 0 else "gemm_mlp_down_gate"
                resid_seen += 1
            if bn == 256:
                cur = (epi, cls)
        elif "attn_fwd" in n:
            cls = "attention"
        elif "ln_modulate_kernel" in n:
            cls = "ln_modulate"
        elif "gemv_mfma_kernel<8" in n:   # only the batched modulation GEMV is large enough for 8 row blocks
            cls = "mod_gemv"
        prev = cur
        out.append(cls)
    return out


def group_calls(classes, values):
    """Dispatches grouped into library calls: consecutive GEMM dispatches of one class are the image and
    text launches of one call (no GEMM class follows itself otherwise). Returns (class, [values])."""
    out = []
    for cls, v in zip(classes, values):
        if out and cls is not None and cls.startswith("gemm_") and out[-1][0] == cls:
            out[-1][1].append(v)
        else:
            out.append((cls, [v]))
    return out


def kernel_summary(run_dir, bench_json):
    """Writes the kernel-time summary: rocprofv3's per-kernel stats, per-class averages from the
    per-dispatch trace, and bench.py's own event timing of the same classes for comparison."""
    import csv
    with open(os.path.join(run_dir, "bench_kernel_stats.csv")) as f:
        stats = [r for r in csv.DictReader(f) if "dit::" in r["Name"]]
    with open(os.path.join(run_dir, "bench_kernel_trace.csv")) as f:
        trace = sorted(csv.DictReader(f), key=lambda r: int(r["Start_Timestamp"]))
    per = {}
    durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3 for r in trace]
    for cls, v in group_calls(classify_dispatches(trace), durs):
        if cls:
            per.setdefault(cls, []).append(sum(v))
    with open(bench_json) as f:
        b = json.loads([ln for ln in f if ln.startswith("{")][-1])
    lines = ["# Kernel time summary: full K=16 denoise step (step_512_k16)", "",
             "Workload: 8 dual-stream MMDiT blocks, hidden 3072, 24x128 heads, 1024 image + 256 text tokens, "
             "K=16 seeds,", "SDE flow update, reward statistics 64x16 (bf16 weights and activations, fp32 "
             "accumulation).", "", "Commands (repo root, on one MI355X):", "",
             f"    rocprofv3 --kernel-trace --stats --output-format csv -d {run_dir} -o bench -- python3 bench.py "
             "--steps 5 --warmup 2 --no-cpu-baseline --headline-only",
             f"    python3 bench.py --kernel-summary {run_dir}", "",
             "The trace covers the bench's setup (torch kernels that draw the synthetic weights) plus 5 + 2 "
             "timed/warm-up steps", "and one event-instrumented step (8 steps in all). Library kernels, sorted "
             "by total time:", "", "| kernel | calls | avg us | total ms |", "|---|---|---|---|"]
    for r in stats:
        name = r["Name"].split("(")[0]
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) * 1e-3:.2f} | "
                     f"{float(r['TotalDurationNs']) * 1e-6:.3f} |")
    lines += ["", "Per kernel class (classified per dispatch from the trace; `gemm_bf16_kernel<..., 2, ...>` runs "
              "both the output projection and the MLP down, in that order within a block; a call's image and text "
              "launches, where the text rows run on 256 x 192 tiles, are summed into one call), against bench.py's "
              "HIP-event average of the same class in a run without the profiler:", "",
              "| class | calls | rocprofv3 avg us per call | bench.py events avg us |", "|---|---|---|---|"]
    for cls, v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        ev = b.get("kernels", {}).get(cls, {}).get("avg_us")
        lines.append(f"| {cls} | {len(v)} | {sum(v) / len(v):.2f} | {ev if ev is not None else '-'} |")
    r = b["roofline"]
    lines += ["", f"bench.py (no profiler): {b['value']} ms per step; dominant kernel `{r['kernel']}` averaged "
              f"{r['avg_launch_us']} us per launch with HIP events ({r['achieved']} TFLOP/s, "
              f"{100 * r['frac']:.1f}% of {r['peak']}).",
              "EPI codes in `gemm_bf16_kernel<BM, BN, WM, WN, EPI, OUTF32, MS, TRI>`: 0 plain store, 1 GELU (MLP up), "
              "2 gated residual (output projection, MLP down), 3 QKV with 2D RoPE; MS is the MFMA block size; TRI marks three LDS stages for the activation operand (long K)."]
    with open(os.path.join(ROOT, KERNEL_MD), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def mfma_summary(run_dir, cfg):
    """Per kernel class of the denoise step, from one rocprofv3 --pmc pass: MFMA busy cycles per SIMD
    over the GPU-active clocks (rocprof's MfmaUtil), the clock those active cycles imply over the
    dispatch's duration, and the bf16 MFMA flops the hardware counted (SQ_INSTS_VALU_MFMA_MOPS_BF16
    is in units of 512) against the algorithmic count."""
    import csv
    import glob
    files = glob.glob(os.path.join(run_dir, "*counter_collection.csv"))
    if not files:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    disp = {}
    with open(files[0]) as f:
        for r in csv.DictReader(f):
            d = disp.setdefault(int(r["Dispatch_Id"]), {"row": r})
            d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    order = [disp[k] for k in sorted(disp)]
    simds, xcds = 1024, 8
    M, D, F = cfg.batch * cfg.seq, cfg.hidden, cfg.mlp_hidden
    S = cfg.seq
    algo = {"gemm_qkv_rope": 2.0 * M * D * 3 * D, "gemm_out_gate": 2.0 * M * D * D,
            "gemm_mlp_up_gelu": 2.0 * M * D * F, "gemm_mlp_down_gate": 2.0 * M * F * D,
            "attention": 4.0 * cfg.batch * S * S * D}
    per = {}
    for cls, ds in group_calls(classify_dispatches([d["row"] for d in order]), order):
        if cls not in algo:
            continue
        ns = sum(float(d["row"]["End_Timestamp"]) - float(d["row"]["Start_Timestamp"]) for d in ds)
        active = sum(d["GRBM_GUI_ACTIVE"] for d in ds) / xcds   # per-XCD value, summed over the 8 XCDs by rocprofv3
        per.setdefault(cls, []).append((ns, active, sum(d["SQ_VALU_MFMA_BUSY_CYCLES"] for d in ds),
                                        sum(d["SQ_INSTS_VALU_MFMA_MOPS_BF16"] for d in ds) * 512))
    lines = ["# MFMA counters per kernel class: full K=16 denoise step (step_512_k16)", "",
             "Command (repo root, one MI355X):", "",
             f"    rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 GRBM_GUI_ACTIVE --output-format csv "
             f"-d {run_dir} -o b -- python3 bench.py --steps 1 --warmup 1 --no-cpu-baseline --headline-only",
             f"    python3 bench.py --mfma-summary {run_dir}", "",
             "Per call (a GEMM call's image and text launches summed): MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / "
             "(GRBM_GUI_ACTIVE per XCD x 1024 SIMDs) (rocprof's MfmaUtil); clock = GRBM_GUI_ACTIVE per XCD / dispatch "
             "duration; counted flops = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512. Dispatch durations here are under counter "
             "collection.", "",
             "| class | calls | avg us | clock GHz | MFMA busy | TFLOP/s | % of 2516.6 | counted / algorithmic flops |",
             "|---|---|---|---|---|---|---|---|"]
    out = {}
    for cls in ("gemm_qkv_rope", "gemm_out_gate", "gemm_mlp_up_gelu", "gemm_mlp_down_gate", "attention"):
        v = per.get(cls)
        if not v:
            continue
        n = len(v)
        ns = sum(x[0] for x in v) / n
        ghz = sum(x[1] / x[0] for x in v) / n
        busy = sum(x[2] / (x[1] * simds) for x in v) / n
        counted = sum(x[3] for x in v) / n
        tf = algo[cls] / ns / 1e3
        out[cls] = {"clock_ghz": round(ghz, 3), "mfma_busy": round(busy, 4), "counted_over_algorithmic": round(counted / algo[cls], 4)}
        lines.append(f"| {cls} | {n} | {ns / 1e3:.1f} | {ghz:.2f} | {100 * busy:.1f}% | {tf:.0f} | "
                     f"{100 * tf / PEAK_BF16_TFLOPS:.1f}% | {counted / algo[cls]:.4f} |")
    lines += ["", "MFMA busy is measured against the clock the kernel actually ran at; the % column is against the "
              "published peak, which assumes 2.4 GHz."]
    with open(os.path.join(ROOT, MFMA_MD), "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps(out))


def _dispatch_counters(run_dir):
    """Counter rows of one rocprofv3 --pmc run grouped per dispatch, in dispatch order, with the class of each."""
    import csv
    import glob
    files = glob.glob(os.path.join(run_dir, "*counter_collection.csv"))
    if not files:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    disp = {}
    with open(files[0]) as f:
        for r in csv.DictReader(f):
            d = disp.setdefault(int(r["Dispatch_Id"]), {"row": r})
            d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    order = [disp[k] for k in sorted(disp)]
    return list(zip(order, classify_dispatches([d["row"] for d in order])))


def stall_summary(run_dir):
    """Where the waves of each kernel class spend their cycles, from one rocprofv3 --pmc pass of the SQ
    wave-state counters. SQ_WAVE_CYCLES, SQ_WAIT_*, SQ_ACTIVE_INST_* and SQ_INST_CYCLES_VMEM_RD are
    wave-cycles in units of 4 cycles, summed over waves; ratios to SQ_WAVE_CYCLES are fractions of the
    waves' resident time. SQ_LDS_BANK_CONFLICT is in cycles (per CU, summed); it is shown per CU per
    GPU-active cycle (GRBM_GUI_ACTIVE is summed over the 8 XCDs)."""
    per = {}
    for d, cls in _dispatch_counters(run_dir):
        if cls:
            per.setdefault(cls, []).append(d)
    names = ["gemm_qkv_rope", "gemm_out_gate", "gemm_mlp_up_gelu", "gemm_mlp_down_gate", "attention", "ln_modulate"]
    lines = ["# Wave-state counters per kernel class: full K=16 denoise step (step_512_k16)", "",
             "Command (repo root, one MI355X):", "",
             "    rocprofv3 --pmc " + " ".join(STALL_COUNTERS) + f" --output-format csv -d {run_dir} -o b -- "
             "python3 bench.py --steps 1 --warmup 1 --no-cpu-baseline --headline-only",
             f"    python3 bench.py --stall-summary {run_dir}", "",
             "Fractions of the waves' resident cycles (SQ_WAVE_CYCLES): waiting for anything (SQ_WAIT_ANY), waiting "
             "for an instruction to issue (SQ_WAIT_INST_ANY, of which LDS: SQ_WAIT_INST_LDS), executing any "
             "instruction (SQ_ACTIVE_INST_ANY), executing LDS instructions (SQ_ACTIVE_INST_LDS), sending VMEM read "
             "addresses (SQ_INST_CYCLES_VMEM_RD). LDS bank-conflict cycles are per CU per GPU-active cycle.", "",
             "| class | dispatches | wait any | wait issue | wait LDS issue | active any | active LDS | VMEM rd issue | "
             "LDS conflict / cycle |", "|---|---|---|---|---|---|---|---|---|"]
    out = {}
    for cls in names:
        v = per.get(cls)
        if not v:
            continue
        tot = {c: sum(d.get(c, 0.0) for d in v) for c in STALL_COUNTERS}
        wc = tot["SQ_WAVE_CYCLES"] or 1.0
        fr = {c: tot[c] / wc for c in ("SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_WAIT_INST_LDS", "SQ_ACTIVE_INST_ANY",
                                        "SQ_ACTIVE_INST_LDS", "SQ_INST_CYCLES_VMEM_RD")}
        conf = tot["SQ_LDS_BANK_CONFLICT"] / 256.0 / max(tot["GRBM_GUI_ACTIVE"] / 8.0, 1.0)
        out[cls] = {k: round(x, 4) for k, x in fr.items()}
        out[cls]["lds_conflict_per_cycle"] = round(conf, 4)
        lines.append(f"| {cls} | {len(v)} | " + " | ".join(f"{100 * fr[c]:.1f}%" for c in fr) + f" | {conf:.4f} |")
    with open(os.path.join(ROOT, STALL_MD), "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps(out))


def traffic_summary(run_dir, cfg):
    """Writes the per-class HBM traffic summary from four rocprofv3 --pmc runs: FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch) of a 1 GiB device copy, then of bench.py --steps 1 --warmup 1.
    Each counter is scaled by bytes copied / counter read for the copy kernel."""
    import csv
    import glob

    def rows(sub):
        files = glob.glob(os.path.join(run_dir, sub, "*counter_collection.csv"))
        if not files:
            raise SystemExit(f"no counter_collection.csv under {os.path.join(run_dir, sub)}")
        with open(files[0]) as f:
            return [r for r in csv.DictReader(f)]

    copy_bytes = 1024 * (1 << 20)
    scale, calib = {}, {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        vals = [float(r["Counter_Value"]) for r in rows("calib_" + c) if "copyBuffer" in r["Kernel_Name"]]
        kib = sorted(vals)[len(vals) // 2]
        calib[c + "_kib_per_launch"] = kib
        scale[c] = copy_bytes / (kib * 1024.0)
    per = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        rr = rows("bench_" + c)
        for cls, v in group_calls(classify_dispatches(rr), [float(r["Counter_Value"]) for r in rr]):
            if cls:
                per.setdefault(cls, {}).setdefault(c, []).append(sum(v))
    M, D, F = cfg.batch * cfg.seq, cfg.hidden, cfg.mlp_hidden
    algo = {"gemm_qkv_rope": 2 * (M * D + 3 * D * D + 3 * M * D),
            "gemm_out_gate": 2 * (M * D + D * D + 2 * M * D),
            "gemm_mlp_up_gelu": 2 * (M * D + F * D + M * F),
            "gemm_mlp_down_gate": 2 * (M * F + D * F + 2 * M * D),
            "attention": 2 * 4 * M * D,
            "ln_modulate": 2 * 2 * M * D,
            # modulation of up to 8 blocks x 2 streams: [6D][D] bf16 weights read, [B][6D] fp32 written
            "mod_gemv": 2 * min(8, cfg.blocks) * (6 * D * D * 2 + cfg.batch * 6 * D * 4)}
    classes = {}
    for cls, v in per.items():
        fk = sum(v["FETCH_SIZE"]) / len(v["FETCH_SIZE"])
        wk = sum(v["WRITE_SIZE"]) / len(v["WRITE_SIZE"])
        fb, wb = fk * 1024 * scale["FETCH_SIZE"], wk * 1024 * scale["WRITE_SIZE"]
        classes[cls] = {"launches_counted": len(v["FETCH_SIZE"]), "fetch_kib_per_launch": round(fk, 1),
                        "write_kib_per_launch": round(wk, 1), "fetch_bytes_per_launch": round(fb),
                        "write_bytes_per_launch": round(wb), "hbm_bytes_per_launch": round(fb + wb),
                        "algorithmic_bytes_per_launch": algo[cls],
                        "measured_over_algorithmic": round((fb + wb) / algo[cls], 3),
                        "source": CLASS_SOURCE[cls], "source_sha": source_sha(CLASS_SOURCE[cls])}
    rec = {"workload": f"{cfg.name} (M={M} rows of image+text tokens over K={cfg.batch} seeds, hidden {D}, "
                       f"MLP {F})",
           "calibration": dict(calib, kernel="__amd_rocclr_copyBuffer, 1 GiB device copy",
                               bytes_per_launch=copy_bytes, fetch_scale=round(scale["FETCH_SIZE"], 5),
                               write_scale=round(scale["WRITE_SIZE"], 5)),
           "commands": [f"rocprofv3 --pmc {c} --output-format csv -d {run_dir}/{k}_{c} -o {k[0]} -- python3 bench.py "
                        + ("--copy-calibration 1024" if k == "calib"
                           else "--steps 1 --warmup 1 --no-cpu-baseline --headline-only")
                        for k in ("calib", "bench") for c in ("FETCH_SIZE", "WRITE_SIZE")]
                       + [f"python3 bench.py --traffic-summary {run_dir}"],
           "per_kernel_class": classes}
    with open(os.path.join(ROOT, TRAFFIC_JSON), "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps({k: v["measured_over_algorithmic"] for k, v in classes.items()}))


class DeviceInputs:
    """Seeded synthetic inputs generated on the GPU with the recipe of seeded_inputs."""

    def __init__(self, torch, d, cfg, seed=si.MASTER_SEED):
        self.torch = torch
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        act = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32

        def w(shape, std=0.02):
            return (torch.randn(shape, generator=g, device="cuda", dtype=torch.float32) * std).to(act)

        self.blocks_t = []
        for _ in range(cfg.blocks):
            self.blocks_t.append({s: {t: w(shp) for t, shp in si.block_weight_shapes(cfg).items()}
                                  for s in si.STREAMS})
        self.blocks = [d.block_weights(b["img"], b["txt"]) for b in self.blocks_t]
        self.sw_t = {t: w(shp) for t, shp in si.step_weight_shapes(cfg).items()}
        self.sw = d.step_weights(self.sw_t)
        B = cfg.batch
        self.latent = torch.randn((B, cfg.n_img, cfg.latent_dim), generator=g, device="cuda")
        text = torch.randn((1, cfg.n_txt, cfg.hidden), generator=g, device="cuda").to(act)
        self.x_txt = text.expand(B, -1, -1).contiguous()
        self.eps = torch.randn((B, cfg.n_img, cfg.latent_dim), generator=g, device="cuda")
        self.v = torch.empty_like(self.latent)
        t = float(torch.rand((1,), generator=g, device="cuda").item())
        self.t = min(max(t, 0.06), 0.94)
        self.t_next = self.t - cfg.dt
        G = max(cfg.reward_groups, 1)
        n = max(cfg.reward_n, 1)
        self.k = cfg.reward_k
        self.rewards = torch.rand((G, n), generator=g, device="cuda")
        self.mean = torch.empty(G, device="cuda")
        self.std = torch.empty(G, device="cuda")
        self.adv = torch.empty((G, n), device="cuda")
        self.order = torch.empty((G, n), dtype=torch.int32, device="cuda")
        self.selected = torch.empty((G, max(self.k, 1)), dtype=torch.int32, device="cuda")
        self.reward_status = torch.zeros((1,), dtype=torch.int32, device="cuda")
        self.cfg = d.block_config(cfg.hidden, cfg.heads, cfg.head_dim, cfg.mlp_hidden, cfg.n_img, cfg.n_txt,
                                  cfg.grid_h, cfg.grid_w, rope=cfg.rope, dtype=cfg.dtype)
        self.ws = d.workspace(d.dit_denoise_workspace_bytes(self.cfg, B, cfg.latent_dim))


def make_step(d, cfg, x):
    a = cfg.noise_level

    def step():
        d.dit_denoise_step(x.cfg, x.sw, x.blocks, x.t, x.t_next, a, x.latent, x.x_txt,
                           x.eps if a > 0 else None, x.v, x.ws)
        if cfg.reward_groups:   # finiteness checked on the device: the step never waits for the host
            d.group_reward_stats_async(x.rewards, x.reward_status, 1e-4, x.k, x.mean, x.std, x.adv, x.order,
                                       x.selected)
    return step


def graph_replay(torch, step, steps, warmup):
    """The same step (denoise step and reward statistics) captured once into a HIP graph and
    replayed: wall clock per replay over `steps` replays. The step records only kernels and one
    device-to-device copy, so the graph replays it as launched."""
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step()
    for _ in range(max(warmup, 1)):
        g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        g.replay()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    del g
    return {"ms_per_step": round(ms, 4), "steps": steps}


def next_rows(torch, d, cfg, x):
    """Rows past the denoise step: the SDE step's log-density on this workload's latents (GPU,
    timed with HIP events over 20 launches), and one planner iteration plus the seed-bank update
    for this workload's reward groups (native host code, wall clock over 2000 iterations)."""
    from paper_2606_19004_amd import planner as pn
    out = {}
    if cfg.noise_level > 0:
        B = cfg.batch
        logp = torch.empty(B, dtype=torch.float64, device="cuda")
        d.flow_logprob(x.latent, x.v, x.latent, x.t, x.t_next, cfg.noise_level, logp)
        torch.cuda.synchronize()
        d.dit_profile_begin()
        for _ in range(20):
            d.flow_logprob(x.latent, x.v, x.latent, x.t, x.t_next, cfg.noise_level, logp)
        st = [k for k in d.dit_profile_end() if k["name"] == "flow_logprob"][0]
        avg = st["total_ms"] / st["launches"]
        out["flow_logprob"] = {"avg_us": round(avg * 1e3, 2), "elements": x.latent.numel(),
                               "gbs": round(st["bytes"] / (st["total_ms"] * 1e-3) / 1e9, 1),
                               "frac_hbm": round(st["bytes"] / (st["total_ms"] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
    # TeaCache: a step that reuses the cached residual, and the gate's overhead on a computed step
    if cfg.blocks >= 1:
        a = cfg.noise_level
        cache = d.workspace(d.dit_teacache_cache_bytes(x.cfg, cfg.batch))
        lat = x.latent.clone()
        st = d.teacache_state(1e9)
        d.dit_denoise_step_teacache(x.cfg, x.sw, x.blocks, x.t, x.t_next, a, lat, x.x_txt, x.eps if a > 0 else None,
                                    x.v, st, cache, x.ws)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(10):
            ran, _ = d.dit_denoise_step_teacache(x.cfg, x.sw, x.blocks, x.t, x.t_next, a, lat, x.x_txt,
                                                 x.eps if a > 0 else None, x.v, st, cache, x.ws)
            assert not ran
        torch.cuda.synchronize()
        skip_ms = (time.perf_counter() - t0) / 10 * 1e3
        st0 = d.teacache_state(0.0)
        t0 = time.perf_counter()
        for _ in range(3):
            d.dit_denoise_step_teacache(x.cfg, x.sw, x.blocks, x.t, x.t_next, a, lat, x.x_txt,
                                        x.eps if a > 0 else None, x.v, st0, cache, x.ws)
        torch.cuda.synchronize()
        run_ms = (time.perf_counter() - t0) / 3 * 1e3
        out["teacache"] = {"skipped_step_ms": round(skip_ms, 3), "computed_step_ms": round(run_ms, 3),
                           "note": "wall clock per gated step (one host sync each); the computed step also runs "
                                   "block 0's modulation and LN once more for the distance"}
    pl = pn.Planner([4, 8, 16, 24, 32], [12, 14, 16, 18, 20], beta=0.5, window=10, prompts=32)
    rng = np.random.default_rng(0)
    fb = rng.uniform(0.8, 2.0, 2000).tolist()
    spot = rng.integers(0, 12, 2000).tolist()
    t0 = time.perf_counter()
    for i in range(2000):
        a, _, _ = pl.select(60.0, spot[i], 0.04)
        pl.update(a, fb[i])
    plan_us = (time.perf_counter() - t0) / 2000 * 1e6
    G, n, k = max(cfg.reward_groups, 1), max(cfg.reward_n, 1), max(cfg.reward_k, 1)
    bank = pn.SeedBank(k)
    seeds = rng.integers(0, 2**40, (G, n)).tolist()
    sel = x.selected.cpu().tolist() if cfg.reward_groups else [list(range(k))] * G
    t0 = time.perf_counter()
    for _ in range(200):
        bank.put_selected(list(range(G)), seeds, sel)
    bank_us = (time.perf_counter() - t0) / 200 * 1e6
    out["planner"] = {"select_update_us": round(plan_us, 2), "actions": pl.num_actions,
                      "seed_bank_put_us": round(bank_us, 2), "groups": G, "seeds_per_group": n, "k": k,
                      "note": "host code, wall clock including the Python binding"}
    return out


def other_configs(torch, d):
    """The single-block configurations at their launch shapes, measured after the headline step:
    512^2 block (K=8), 1280^2 block (K=4, joint attention over 6912 tokens), and one sequence-
    parallel rank's share at 1280^2 (6 of 24 heads over 6912 tokens, K=8; MLP on a 1600 + 128 token
    slice, K=8). Per configuration: ms per call (HIP events, median of 5 after 2 warm-ups) and the
    GEMM / attention throughput of one instrumented call."""
    out = {}
    g = torch.Generator(device="cuda")
    g.manual_seed(si.MASTER_SEED)

    def w(shape, std=0.02):
        return (torch.randn(shape, generator=g, device="cuda", dtype=torch.float32) * std).to(torch.bfloat16)

    def timed(fn):
        for _ in range(2):
            fn()
        ts = []
        for _ in range(5):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            b.synchronize()
            ts.append(a.elapsed_time(b))
        d.dit_profile_begin()
        fn()
        st = {k["name"]: k for k in d.dit_profile_end()}
        return sorted(ts)[2], st

    def frac(st, names):
        ks = [st[n] for n in names if n in st]
        fl, ms = sum(k["flops"] for k in ks), sum(k["total_ms"] for k in ks)
        tf = fl / (ms * 1e-3) / 1e12 if ms else 0.0
        return {"tflops": round(tf, 1), "frac": round(tf / PEAK_BF16_TFLOPS, 4), "ms": round(ms, 3)}

    gemms = ["gemm_qkv_rope", "gemm_out_gate", "gemm_mlp_up_gelu", "gemm_mlp_down_gate"]
    for name in ("block_512", "block_1280"):
        cfg = si.CONFIGS[name]
        bw = {s: {t: w(shp) for t, shp in si.block_weight_shapes(cfg).items()} for s in si.STREAMS}
        blk = d.block_weights(bw["img"], bw["txt"])
        c = d.block_config(cfg.hidden, cfg.heads, cfg.head_dim, cfg.mlp_hidden, cfg.n_img, cfg.n_txt, cfg.grid_h,
                           cfg.grid_w, rope=cfg.rope, dtype=cfg.dtype)
        B = cfg.batch
        temb = torch.randn((B, cfg.hidden), generator=g, device="cuda")
        xi = torch.randn((B, cfg.n_img, cfg.hidden), generator=g, device="cuda").to(torch.bfloat16)
        xt = torch.randn((B, cfg.n_txt, cfg.hidden), generator=g, device="cuda").to(torch.bfloat16)
        ws = d.workspace(d.dit_block_workspace_bytes(c, B))
        ms, st = timed(lambda: d.dit_block_forward(c, blk, temb, xi, xt, ws))
        out[name] = {"ms_per_block": round(ms, 3), "K": B, "tokens": cfg.seq, "gemm": frac(st, gemms),
                     "attention": frac(st, ["attention"])}
        del bw, blk, xi, xt, ws
    # one sequence-parallel rank's share at 1280^2: attention over all 6912 tokens for 6 heads ...
    cfg = si.CONFIGS["headslice_1280"]
    B, S, H, hd = cfg.batch, cfg.seq, cfg.heads, cfg.head_dim
    qkv = torch.randn((B, S, 3, H, hd), generator=g, device="cuda").to(torch.bfloat16)
    o = torch.empty((B, S, H * hd), device="cuda", dtype=torch.bfloat16)
    D = H * hd
    flat = qkv.view(-1)
    ms_a, st = timed(lambda: d.joint_attention(flat[0:], flat[D:], flat[2 * D:], o, B, H, S, hd,
                                               (S * 3 * D, 3 * D, hd), (S * D, D, hd)))
    # ... and the full-width MLP on its 1600 + 128 token slice
    cm = si.CONFIGS["mlp_slice_1280"]
    bw = {s: {t: w(shp) for t, shp in si.block_weight_shapes(cm).items()} for s in si.STREAMS}
    blk = d.block_weights(bw["img"], bw["txt"])
    c = d.block_config(cm.hidden, cm.heads, cm.head_dim, cm.mlp_hidden, cm.n_img, cm.n_txt, cm.grid_h, cm.grid_w,
                       rope=cm.rope, dtype=cm.dtype)
    temb = torch.randn((cm.batch, cm.hidden), generator=g, device="cuda")
    xi = torch.randn((cm.batch, cm.n_img, cm.hidden), generator=g, device="cuda").to(torch.bfloat16)
    xt = torch.randn((cm.batch, cm.n_txt, cm.hidden), generator=g, device="cuda").to(torch.bfloat16)
    ws = d.workspace(d.dit_block_workspace_bytes(c, cm.batch))
    ms_m, st_m = timed(lambda: d.dit_block_mlp(c, blk, temb, xi, xt, ws))
    out["sp_rank_1280"] = {"attention_ms": round(ms_a, 3), "attention": frac(st, ["attention"]),
                           "mlp_ms": round(ms_m, 3), "mlp_gemm": frac(st_m, ["gemm_mlp_up_gelu", "gemm_mlp_down_gate"]),
                           "K": B, "heads": H, "tokens": S, "mlp_tokens": cm.seq}
    return out


def cpu_baseline(cfg, n_seeds):
    """Time the oracle on a bounded sample: one block for `n_seeds` seeds (all rows),
    scaled to a full step (blocks x K seeds). Block work dominates the step."""
    from oracle import dit_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # noqa: BLE001
        threads = os.cpu_count() or 1
    import dataclasses
    c1 = dataclasses.replace(cfg, blocks=1, batch=n_seeds)
    inp = si.block_inputs(c1)
    w64 = {s: {t: si.as_f64(a, c1.dtype) for t, a in ws.items()} for s, ws in inp["weights"].items()}
    xi, xt = si.as_f64(inp["x_img"], c1.dtype), si.as_f64(inp["x_txt"], c1.dtype)
    temb = inp["temb"].astype(np.float64)
    t0 = time.perf_counter()
    for b in range(n_seeds):
        O.block_forward_sample(c1, w64, temb[b], xi[b], xt[b])
    sec = time.perf_counter() - t0
    per_seed_block = sec / n_seeds
    ms_step = per_seed_block * cfg.blocks * cfg.batch * 1e3
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    return {"value": round(ms_step, 1), "unit": "ms per K-seed denoise step", "cores": int(threads), "kind": "oracle",
            "cpu_model": model,
            "sample": f"fp64 numpy oracle, one MMDiT block for {n_seeds} seed(s) at the step's shape "
                      f"({cfg.seq} tokens, hidden {cfg.hidden}), {sec:.1f} s measured, scaled x{cfg.blocks} blocks "
                      f"x{cfg.batch} seeds"}


RIDGE_FLOP_PER_BYTE = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)   # ~315 flop/B


def kernel_entry(k: dict) -> dict:
    """One kernel class of the profiled step, classified by its bound: a class whose algorithmic
    flops per algorithmic HBM byte is below the ridge point (peak MFMA / peak HBM) is HBM-bound and
    reports GB/s against the HBM peak; otherwise (or without a byte count) it reports TFLOP/s against
    the bf16 MFMA peak. HBM-bound classes with flops (the GEMVs) report both."""
    avg = k["total_ms"] / k["launches"]
    sec = k["total_ms"] * 1e-3
    e = {"launches": k["launches"], "avg_us": round(avg * 1e3, 2), "total_ms": round(k["total_ms"], 4)}
    hbm = k["bytes"] > 0 and (k["flops"] == 0 or k["flops"] / k["bytes"] < RIDGE_FLOP_PER_BYTE)
    e["bound"] = "hbm" if hbm else "mfma"
    if k["flops"] > 0:
        e["tflops"] = round(k["flops"] / sec / 1e12, 1)
        e["frac_mfma"] = round(e["tflops"] / PEAK_BF16_TFLOPS, 4)
    if hbm:
        e["gbs"] = round(k["bytes"] / sec / 1e9, 1)
        e["frac_hbm"] = round(e["gbs"] / PEAK_HBM_GBS, 4)
    return e


def main():
    args = parse()
    if args.stall_summary:
        stall_summary(args.stall_summary)
        return
    if args.mfma_summary:
        mfma_summary(args.mfma_summary, si.CONFIGS[args.config])
        return
    if args.traffic_summary:
        traffic_summary(args.traffic_summary, si.CONFIGS[args.config])
        return
    if args.kernel_summary:
        kernel_summary(args.kernel_summary, os.path.join(args.kernel_summary, "..", "bench.json"))
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library runs the denoise step on a single MI355X "
              "(no collectives); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import torch
    torch.cuda.set_device(0)
    if args.copy_calibration:
        copy_calibration(torch, args.copy_calibration)
        return
    from paper_2606_19004_amd import ditstep as d
    cfg = si.CONFIGS[args.config]
    x = DeviceInputs(torch, d, cfg)
    step = make_step(d, cfg, x)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms = elapsed * 1e3 / args.steps
    print(f"timed {args.steps} steps: {ms:.3f} ms/step", file=sys.stderr, flush=True)

    # per-kernel-class timing: one more step with HIP events around every launch
    d.dit_profile_begin()
    step()
    stats = d.dit_profile_end()
    kernels = {k["name"]: kernel_entry(k) for k in stats}
    dom = max(stats, key=lambda k: k["total_ms"])
    avg_s = dom["total_ms"] / dom["launches"] * 1e-3
    per_launch = dom["flops"] / dom["launches"]
    achieved = per_launch / avg_s / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic_from_profile(dom["name"]),
                "kernel": dom["name"],
                "flops_per_launch": per_launch, "avg_launch_us": round(avg_s * 1e6, 2)}
    gemm_ms = sum(k["total_ms"] for k in stats if k["name"].startswith("gemm"))
    gemm_fl = sum(k["flops"] for k in stats if k["name"].startswith("gemm"))
    attn = [k for k in stats if k["name"] == "attention"]
    summary = {"gemm_tflops": round(gemm_fl / (gemm_ms * 1e-3) / 1e12, 1) if gemm_ms else None,
               "attention_tflops": round(attn[0]["flops"] / (attn[0]["total_ms"] * 1e-3) / 1e12, 1) if attn else None}
    summary["gemm_frac"] = round(summary["gemm_tflops"] / PEAK_BF16_TFLOPS, 4) if summary["gemm_tflops"] else None
    summary["attention_frac"] = (round(summary["attention_tflops"] / PEAK_BF16_TFLOPS, 4)
                                 if summary["attention_tflops"] else None)

    extra = blocks = graph = None
    if not args.headline_only:
        graph = graph_replay(torch, step, args.steps, args.warmup)
        extra = next_rows(torch, d, cfg, x)
        del x, step
        torch.cuda.empty_cache()
        blocks = other_configs(torch, d) if args.config == "step_512_k16" else None

    cpu = None
    if not args.no_cpu_baseline:
        print("timing the CPU oracle on a bounded sample ...", file=sys.stderr, flush=True)
        cpu = cpu_baseline(cfg, args.cpu_sample_seeds)

    out = {
        "metric": "ms per K-seed denoise step", "value": round(ms, 4), "unit": "ms", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": (f"{cfg.name}: {cfg.blocks} dual-stream MMDiT blocks, hidden {cfg.hidden}, "
                                f"{cfg.heads}x{cfg.head_dim} heads, {cfg.n_img} image + {cfg.n_txt} text tokens, "
                                f"K={cfg.batch} seeds, flow update a={cfg.noise_level}, reward stats "
                                f"{cfg.reward_groups}x{cfg.reward_n}"),
                   "batch": cfg.batch, "seq_len": cfg.seq, "blocks": cfg.blocks, "parallelism": "single GPU"},
        "roofline": roofline,
        "mfma_summary": summary,
        "graph_replay": graph,
        "kernels": kernels,
        "next_rows": extra,
        "other_configs": blocks,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
