"""Host-side logic of bench.py: classification of profiled dispatches into kernel classes and
the staleness check of the committed traffic summary (no GPU)."""
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
