"""Host-side logic of bench.py: classification of profiled dispatches into kernel classes and
the staleness check of the committed traffic summary, and the MFMA counter summary (no GPU)."""
import json

import bench


def _row(name):
    return {"Kernel_Name": name}


def test_classify_dispatches_block_order():
    g = "void dit::gemm_bf16_kernel<256, 256, 4, 2, {}, false, 16>(dit::GemmPair, int, int)"
    block = [_row("void dit::ln_modulate_kernel<unsigned short, 6>(dit::LnArgs)"), _row(g.format(3)),
             _row("void dit::attn_fwd_bf16<128>(dit::AttnArgs)"), _row(g.format(2)),
             _row("void dit::ln_modulate_kernel<unsigned short, 6>(dit::LnArgs)"), _row(g.format(1)),
             _row(g.format(2)), _row("dit::gemv_mfma_kernel(dit::GemvArgs, unsigned short const*, int, int)")]
    got = bench.classify_dispatches(block * 2)
    want = ["ln_modulate", "gemm_qkv_rope", "attention", "gemm_out_gate", "ln_modulate", "gemm_mlp_up_gelu",
            "gemm_mlp_down_gate", None]
    assert got == want * 2
    # small-tile GEMMs (patch embedding, velocity head) are not counted as block GEMMs
    assert bench.classify_dispatches([_row("void dit::gemm_bf16_kernel<64, 64, 2, 2, 0, true, 32>(x)")]) == [None]


def test_classify_dispatches_split_text_launch():
    """A GEMM call whose text rows run as a second launch on 256 x 192 tiles: the second launch takes
    the first one's class, the out-projection / MLP-down alternation still counts calls, and
    group_calls sums the two launches into one call."""
    g = "void dit::gemm_bf16_kernel<256, {}, 4, 2, {}, false, 16, true>(dit::GemmPair, int, int)"
    ln = _row("void dit::ln_modulate_kernel<unsigned short, 6>(dit::LnArgs)")
    block = [ln, _row(g.format(256, 3)), _row(g.format(192, 3)), _row("void dit::attn_fwd_bf16<128>(dit::AttnArgs)"),
             _row(g.format(256, 2)), _row(g.format(192, 2)), ln, _row(g.format(256, 1)),
             _row(g.format(256, 2)), _row(g.format(192, 2))]
    got = bench.classify_dispatches(block * 2)
    want = ["ln_modulate", "gemm_qkv_rope", "gemm_qkv_rope", "attention", "gemm_out_gate", "gemm_out_gate",
            "ln_modulate", "gemm_mlp_up_gelu", "gemm_mlp_down_gate", "gemm_mlp_down_gate"]
    assert got == want * 2
    calls = bench.group_calls(got, list(range(len(got))))
    assert [c for c, _ in calls] == ["ln_modulate", "gemm_qkv_rope", "attention", "gemm_out_gate", "ln_modulate",
                                     "gemm_mlp_up_gelu", "gemm_mlp_down_gate"] * 2
    assert calls[1][1] == [1, 2] and calls[6][1] == [8, 9] and calls[7][1] == [10]
    # a 256 x 192 launch with no 256 x 256 launch of its epilogue before it starts a call of its own
    assert bench.classify_dispatches([_row(g.format(192, 1))]) == ["gemm_mlp_up_gelu"]


def test_traffic_lookup_rejects_stale_source(tmp_path, monkeypatch):
    rec = {"per_kernel_class": {"gemm_mlp_down_gate": {"hbm_bytes_per_launch": 123, "source_sha": "0" * 16}}}
    p = tmp_path / "t.json"
    p.write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "TRAFFIC_JSON", str(p))
    assert bench.traffic_from_profile("gemm_mlp_down_gate") is None
    rec["per_kernel_class"]["gemm_mlp_down_gate"]["source_sha"] = bench.source_sha("k_gemm.hip")
    p.write_text(json.dumps(rec))
    assert bench.traffic_from_profile("gemm_mlp_down_gate") == 123
    assert bench.traffic_from_profile("attention") is None


def test_mfma_summary_groups_counter_rows_by_dispatch(tmp_path, monkeypatch):
    """Three counter rows per dispatch must classify as one dispatch (the out-projection / MLP-down
    alternation counts dispatches), and the derived clock, MFMA-busy fraction and counted-flop ratio
    follow from the counter definitions."""
    import csv

    import seeded_inputs as si
    cfg = si.CONFIGS["step_512_k16"]
    M, D, F = cfg.batch * cfg.seq, cfg.hidden, cfg.mlp_hidden
    g = "void dit::gemm_bf16_kernel<256, 256, 4, 2, {}, false, 16, true>(dit::GemmPair, int, int)"
    block = [(g.format(3), 2.0 * M * D * 3 * D), (g.format(2), 2.0 * M * D * D), (g.format(1), 2.0 * M * D * F),
             (g.format(2), 2.0 * M * F * D)]
    fields = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
    rows, did = [], 0
    for name, flops in block * 2:
        did += 1
        ns = 1.0e6                                   # 1 ms per dispatch
        active = 2.0e6 * 8                           # 2 GHz on each of 8 XCDs
        busy = 0.5 * 2.0e6 * 1024                    # half of the SIMD cycles
        for c, v in (("GRBM_GUI_ACTIVE", active), ("SQ_VALU_MFMA_BUSY_CYCLES", busy),
                     ("SQ_INSTS_VALU_MFMA_MOPS_BF16", flops / 512)):
            rows.append({"Dispatch_Id": did, "Kernel_Name": name, "Counter_Name": c, "Counter_Value": v,
                         "Start_Timestamp": 1000, "End_Timestamp": 1000 + ns})
    with open(tmp_path / "b_counter_collection.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=fields)
        w.writeheader()
        w.writerows(rows)
    monkeypatch.setattr(bench, "MFMA_MD", str(tmp_path / "out.md"))
    bench.mfma_summary(str(tmp_path), cfg)
    text = (tmp_path / "out.md").read_text()
    for cls in ("gemm_qkv_rope", "gemm_out_gate", "gemm_mlp_up_gelu", "gemm_mlp_down_gate"):
        line = next(l for l in text.splitlines() if l.startswith(f"| {cls} |"))
        cells = [c.strip() for c in line.strip("|").split("|")]
        assert cells[1] == "2" and cells[3] == "2.00" and cells[4] == "50.0%" and cells[7] == "1.0000", line


def test_stall_summary_fractions_and_conflict_normalisation(tmp_path, monkeypatch):
    """Wave-state counters are summed per kernel class and divided by SQ_WAVE_CYCLES; the LDS
    bank-conflict count is normalised per CU (256) and per XCD-summed active cycle (8 XCDs)."""
    import csv
    g = "void dit::gemm_bf16_kernel<256, 256, 4, 2, {}, false, 16, true>(dit::GemmPair, int, int)"
    ln = "void dit::ln_modulate_kernel<unsigned short, 6>(dit::LnArgs)"
    block = [ln, g.format(3), "void dit::attn_fwd_bf16<128>(dit::AttnArgs)", g.format(2), ln, g.format(1), g.format(2)]
    vals = {"SQ_WAVE_CYCLES": 1000.0, "SQ_WAIT_ANY": 300.0, "SQ_WAIT_INST_ANY": 400.0, "SQ_WAIT_INST_LDS": 25.0,
            "SQ_ACTIVE_INST_ANY": 250.0, "SQ_ACTIVE_INST_LDS": 30.0, "SQ_INST_CYCLES_VMEM_RD": 20.0,
            "SQ_LDS_BANK_CONFLICT": 256.0 * 100.0, "GRBM_GUI_ACTIVE": 8.0 * 1000.0}
    assert set(vals) == set(bench.STALL_COUNTERS)
    fields = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
    rows, did = [], 0
    for name in block * 2:
        did += 1
        for c, v in vals.items():
            # the MLP-up class reads its wave cycles split over two rows of one dispatch
            if name == g.format(1) and c == "SQ_WAVE_CYCLES":
                rows += [{"Dispatch_Id": did, "Kernel_Name": name, "Counter_Name": c, "Counter_Value": v / 2,
                          "Start_Timestamp": 0, "End_Timestamp": 1}] * 2
                continue
            rows.append({"Dispatch_Id": did, "Kernel_Name": name, "Counter_Name": c, "Counter_Value": v,
                         "Start_Timestamp": 0, "End_Timestamp": 1})
    with open(tmp_path / "b_counter_collection.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=fields)
        w.writeheader()
        w.writerows(rows)
    monkeypatch.setattr(bench, "STALL_MD", str(tmp_path / "out.md"))
    bench.stall_summary(str(tmp_path))
    text = (tmp_path / "out.md").read_text()
    for cls, n in (("gemm_qkv_rope", 2), ("gemm_out_gate", 2), ("gemm_mlp_up_gelu", 2), ("gemm_mlp_down_gate", 2),
                   ("attention", 2), ("ln_modulate", 4)):
        line = next(l for l in text.splitlines() if l.startswith(f"| {cls} |"))
        cells = [c.strip() for c in line.strip("|").split("|")]
        assert cells[1] == str(n), line
        assert cells[2:8] == ["30.0%", "40.0%", "2.5%", "25.0%", "3.0%", "2.0%"], line
        assert cells[8] == "0.1000", line


def test_kernel_entry_classifies_by_arithmetic_intensity():
    import bench
    # modulation GEMV of the step: 16 samples -> 16 flop per weight byte, far below the ridge point
    gemv = bench.kernel_entry({"name": "mod_gemv", "launches": 1, "total_ms": 0.5,
                               "flops": 2.0 * 16 * 16 * 18432 * 3072, "bytes": 16 * 18432 * 3072 * 2.0})
    assert gemv["bound"] == "hbm"
    assert gemv["gbs"] == round(16 * 18432 * 3072 * 2.0 / 0.5e-3 / 1e9, 1)
    assert gemv["frac_hbm"] == round(gemv["gbs"] / bench.PEAK_HBM_GBS, 4)
    assert "frac_mfma" in gemv   # flops are still reported
    # a GEMM class carries no byte count: MFMA-bound
    gemm = bench.kernel_entry({"name": "gemm_mlp_up_gelu", "launches": 8, "total_ms": 9.5,
                               "flops": 8 * 1.546e12, "bytes": 0})
    assert gemm["bound"] == "mfma" and "gbs" not in gemm
    assert gemm["frac_mfma"] == round(round(8 * 1.546e12 / 9.5e-3 / 1e12, 1) / bench.PEAK_BF16_TFLOPS, 4)
    # byte-only classes (LayerNorm, flow update) are HBM-bound
    ln = bench.kernel_entry({"name": "ln_modulate", "launches": 2, "total_ms": 0.12, "flops": 0, "bytes": 5.0e8})
    assert ln["bound"] == "hbm" and "tflops" not in ln
    # above the ridge point a class with bytes is MFMA-bound
    dense = bench.kernel_entry({"name": "x", "launches": 1, "total_ms": 1.0, "flops": 1e12, "bytes": 1e9})
    assert dense["bound"] == "mfma" and "gbs" not in dense
