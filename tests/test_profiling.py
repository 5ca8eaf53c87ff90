"""Host logic of the rocprofv3 summaries and of bench.py's traffic lookup (CPU only)."""
import csv
import json

from paper_2602_12529_amd import profiling as P

FIELDS = ["Correlation_Id", "Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]


def _write_counters(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for i, (name, counter, value) in enumerate(rows):
            w.writerow({"Correlation_Id": i + 1, "Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter,
                        "Counter_Value": value})


def test_short_name_drops_arguments_and_namespaces():
    n = "void ff::(anonymous namespace)::gemm_bf16_pp<2, 3>(ff::(anonymous namespace)::GemmBatch)"
    assert P.short_name(n) == "gemm_bf16_pp<2, 3>"
    assert P.short_name("ff::(anonymous namespace)::qk_rope_vec_kernel(ff::QkvArgs)") == "qk_rope_vec_kernel"


def test_traffic_scaling_and_lookup(tmp_path, monkeypatch):
    copy_bytes = 1 << 20
    # the copy's counters read half the bytes fetched and all the bytes written (KiB)
    _write_counters(tmp_path / "cf.csv", [("fill_kernel", "FETCH_SIZE", 1.0)] +
                    [("__amd_rocclr_copyBuffer", "FETCH_SIZE", 512.0)] * 3)
    _write_counters(tmp_path / "cw.csv", [("fill_kernel", "WRITE_SIZE", 1024.5)] +
                    [("__amd_rocclr_copyBuffer", "WRITE_SIZE", 1024.0)] * 3)
    k = "void ff::(anonymous namespace)::gemm_bf16_pp<2, 3>(ff::(anonymous namespace)::GemmBatch)"
    _write_counters(tmp_path / "f.csv", [(k, "FETCH_SIZE", 100.0), (k, "FETCH_SIZE", 300.0), ("other", "FETCH_SIZE", 7.0)])
    _write_counters(tmp_path / "w.csv", [(k, "WRITE_SIZE", 50.0), (k, "WRITE_SIZE", 50.0), ("other", "WRITE_SIZE", 7.0)])
    out = tmp_path / "prof.md"
    res = P.traffic_md(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), str(tmp_path / "cf.csv"),
                       str(tmp_path / "cw.csv"), copy_bytes, {"gemm_bf16_gated": "gemm_bf16_pp<2, 3>"}, str(out),
                       "title", ["cmd"], "qwen-60dual")
    rec = res["records"][0]
    assert rec["copy_factor_fetch"] == 2048.0 and rec["copy_factor_write"] == 1024.0
    assert rec["fetch_bytes_per_launch"] == 200.0 * 2048 and rec["write_bytes_per_launch"] == 50.0 * 1024
    assert rec["traffic_bytes_per_launch"] == 200.0 * 2048 + 50.0 * 1024
    assert rec["sources_sha256"] == P.sources_sha256("gemm_bf16_gated")
    # bench.py's lookup finds the record while the sources hash the same, and not otherwise
    monkeypatch.setattr(P, "PROFILES", str(tmp_path))
    got = P.lookup_traffic("gemm_bf16_gated", "qwen-60dual")
    assert got is not None and got["traffic_bytes_per_launch"] == rec["traffic_bytes_per_launch"]
    assert P.lookup_traffic("attn_bf16_d128", "qwen-60dual") is None
    assert P.lookup_traffic("gemm_bf16_gated", "flux-block") is None      # another workload's shapes
    stale = out.read_text().replace(rec["sources_sha256"], "0" * 64)
    out.write_text(stale)
    assert P.lookup_traffic("gemm_bf16_gated", "qwen-60dual") is None


def test_sources_hash_follows_kernel_family():
    assert any(s.endswith("gemm.hip") for s in P.sources_of("gemm_bf16_gelu"))
    assert any(s.endswith("attention.hip") for s in P.sources_of("attn_bf16_d128"))
    assert any(s.endswith("sde.hip") for s in P.sources_of("sde_step"))
    assert P.sources_sha256("gemm_bf16") != P.sources_sha256("attn_bf16_d128")


def test_committed_traffic_summary_parses():
    import os
    import re

    path = os.path.join(P.PROFILES, "flux_dual_block_bf16_B8_hbm_traffic.md")
    text = open(path).read()
    blocks = re.findall(r"```json\n(.*?)```", text, flags=re.S)
    recs = json.loads(blocks[0])
    names = {r["kernel"] for r in recs}
    assert {"gemm_bf16_gated", "sde_step", "attn_bf16_d128"} <= names
    for r in recs:
        assert r["traffic_bytes_per_launch"] > 0 and len(r["sources_sha256"]) == 64


def test_counter_summary_per_kernel(tmp_path):
    k = "void ff::(anonymous namespace)::attn_bf16_d128<8, 4>(ff::(anonymous namespace)::AttnParams)"
    _write_counters(tmp_path / "m.csv", [(k, "MfmaUtil", 40.0), (k, "MfmaUtil", 50.0), ("copy", "MfmaUtil", 0.0),
                                         (k, "GRBM_GUI_ACTIVE", 9.0)])
    out = tmp_path / "m.md"
    P.counter_md(str(tmp_path / "m.csv"), ["MfmaUtil"], str(out), "title", ["cmd"], note="a note")
    text = out.read_text()
    assert "| `attn_bf16_d128<8, 4>` | 2 | 45.0 | 40.0 | 50.0 |" in text
    assert "| `copy` | 1 | 0.0 | 0.0 | 0.0 |" in text and "a note" in text and "GRBM" not in text
    P.counter_md(str(tmp_path / "m.csv"), ["MfmaUtil", "GRBM_GUI_ACTIVE"], str(out), "title", ["cmd"])
    assert "| `attn_bf16_d128<8, 4>` | 2 | 45.0 | 40.0 | 50.0 | 9.0 |" in out.read_text()
