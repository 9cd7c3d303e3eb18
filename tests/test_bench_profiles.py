"""bench.py's rocprofv3 summaries and the hash gate on recorded HBM traffic
(CPU only: synthetic counter files)."""
import csv
import json
import os
import re
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]


def _write(path, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(FIELDS, r)))


def test_kernel_names():
    n = bench.bench_kernel_name
    assert n("void augtree::(anonymous namespace)::attn_dkv_kernel<128>(augtree::DkvParams)") == "attn_dkv_kernel"
    assert n("void augtree::(anonymous namespace)::attn_fwd_kernel<64, false>(augtree::FwdParams)") == \
        "attn_fwd_kernel<bf16 out>"
    assert n("void augtree::(anonymous namespace)::attn_dq_kernel<128>(augtree::DqParams)") == "attn_dq_kernel"
    assert n("__amd_rocclr_copyBuffer") is None


def test_pmc_summary_scales_by_copy_calibration(tmp_path):
    d = str(tmp_path)
    k = "void augtree::(anonymous namespace)::attn_dkv_kernel<128>(augtree::DkvParams)"
    # copy of 1 GiB reads 2^19 KiB of FETCH_SIZE (factor 2) and 2^20 KiB of WRITE_SIZE (factor 1)
    _write(f"{d}/cfetch/run_counter_collection.csv", [(1, "copy", "FETCH_SIZE", 1 << 19)])
    _write(f"{d}/cwrite/run_counter_collection.csv", [(1, "copy", "WRITE_SIZE", 1 << 20)])
    _write(f"{d}/fetch/run_counter_collection.csv", [(1, k, "FETCH_SIZE", 1000.0), (2, k, "FETCH_SIZE", 3000.0),
                                                     (3, "copy", "FETCH_SIZE", 5.0)])
    _write(f"{d}/write/run_counter_collection.csv", [(1, k, "WRITE_SIZE", 10.0), (2, k, "WRITE_SIZE", 30.0)])
    md = bench.summarize_pmc(d, "prompt")
    data = json.loads(re.search(r"<!-- traffic-json (\{.*\}) -->", md).group(1))
    e = data["kernels"]["attn_dkv_kernel"]
    assert e["launches"] == 2
    assert e["fetch_bytes_per_launch"] == round(2000.0 * 1024 * 2)
    assert e["write_bytes_per_launch"] == round(20.0 * 1024)
    assert data["source_hash"] == bench.kernel_source_hash()


def test_recorded_traffic_requires_matching_sources(tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    data = {"workload": "prompt", "source_hash": bench.kernel_source_hash(), "path": "tree",
            "kernels": {"attn_dq_kernel": {"bytes_per_launch": 1234}}}
    (prof / "hbm_traffic_prompt_P32768_G8.md").write_text("x\n<!-- traffic-json " + json.dumps(data) + " -->\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    # kernel_source_hash now sees no sources under tmp_path: a different hash
    assert bench.recorded_traffic("prompt", "attn_dq_kernel") is None
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: data["source_hash"])
    assert bench.recorded_traffic("prompt", "attn_dq_kernel") == 1234
    assert bench.recorded_traffic("prompt", "attn_fwd_kernel<bf16 out>") is None
    assert bench.recorded_traffic("balanced", "attn_dq_kernel") is None
    assert bench.recorded_traffic("prompt", "attn_dq_kernel", "calls") is None   # counters of the other path


def test_source_hash_covers_compile_flags(monkeypatch):
    """Recorded counters describe one build: a change of the attention
    sources' compile flags changes the hash, so their traffic is no longer
    reported."""
    from paper_2609_33133_amd import build
    h0 = bench.kernel_source_hash()
    assert "-amdgpu-sched-strategy=max-ilp" in " ".join(build.hip_flags("attn_bwd.hip"))
    assert "-amdgpu-sched-strategy=max-ilp" not in " ".join(build.hip_flags("elementwise.hip"))
    monkeypatch.setattr(build, "ATTN_FLAGS", [])
    assert bench.kernel_source_hash() != h0


def test_trace_summary(tmp_path):
    p = tmp_path / "stats.csv"
    with open(p, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs", "StdDev"])
        w.writerow(["void augtree::(anonymous namespace)::attn_dq_kernel<128>(augtree::DqParams)", 4, 4000000,
                    1000000.0, 100.0, 1, 2, 0])
    md = bench.summarize_trace(str(p))
    assert "| attn_dq_kernel<128> | 4 | 4.00 | 1.0000 | 100.00 |" in md


def test_counter_summary_busy_and_bandwidth(tmp_path):
    d = str(tmp_path)
    fields = FIELDS + ["Start_Timestamp", "End_Timestamp"]
    k = "void augtree::(anonymous namespace)::lse_merge_kernel(augtree::MergeParams)"

    def wr(sub, rows):
        os.makedirs(f"{d}/{sub}", exist_ok=True)
        with open(f"{d}/{sub}/run_counter_collection.csv", "w", newline="") as f:
            w = csv.DictWriter(f, fieldnames=fields)
            w.writeheader()
            for r in rows:
                w.writerow(dict(zip(fields, r)))

    wr("cfetch", [(1, "copy", "FETCH_SIZE", 1 << 19, 0, 1)])
    wr("cwrite", [(1, "copy", "WRITE_SIZE", 1 << 20, 0, 1)])
    # one launch of 1 us: 1000 KiB fetch counter -> 2 * 1000 KiB read; 500 KiB written
    wr("fetch", [(1, k, "FETCH_SIZE", 1000.0, 0, 1000)])
    wr("write", [(1, k, "WRITE_SIZE", 500.0, 0, 1000)])
    # 8 XCDs x 100 cycles -> 100 cycles x 1024 SIMDs; 25600 busy SIMD-cycles = 25 %
    wr("sq", [(1, k, "SQ_VALU_MFMA_BUSY_CYCLES", 25600.0, 0, 1000), (1, k, "GRBM_GUI_ACTIVE", 800.0, 0, 1000)])
    md = bench.summarize_counters(d)
    assert "| lse_merge_kernel | 1 | 0.001 | 25.0 | 2048 | 512 |" in md


def test_pmc_summary_per_role(tmp_path):
    """Library dispatches are attributed to the logged launch roles in order;
    other kernels (runtime copies) are skipped; a count mismatch is an error."""
    d = str(tmp_path)
    fw = "void augtree::(anonymous namespace)::attn_fwd_kernel<128, false>(augtree::FwdParams)"
    dq = "void augtree::(anonymous namespace)::attn_dq_kernel<128>(augtree::DqParams)"
    _write(f"{d}/cfetch/run_counter_collection.csv", [(1, "copy", "FETCH_SIZE", 1 << 19)])
    _write(f"{d}/cwrite/run_counter_collection.csv", [(1, "copy", "WRITE_SIZE", 1 << 20)])
    rows_f = [(1, fw, "FETCH_SIZE", 100.0), (2, "copy", "FETCH_SIZE", 7.0), (3, fw, "FETCH_SIZE", 300.0),
              (4, dq, "FETCH_SIZE", 50.0), (5, fw, "FETCH_SIZE", 900.0)]
    rows_w = [(1, fw, "WRITE_SIZE", 10.0), (3, fw, "WRITE_SIZE", 30.0), (4, dq, "WRITE_SIZE", 5.0),
              (5, fw, "WRITE_SIZE", 90.0)]
    _write(f"{d}/fetch/run_counter_collection.csv", rows_f)
    _write(f"{d}/write/run_counter_collection.csv", rows_w)
    roles = tmp_path / "roles.json"
    roles.write_text(json.dumps({"launches": ["shared:fwd_prefill", "shared:fwd_replay", "shared:dq_replay",
                                              "flattened:fwd_prefill"], "flattened_rows": 100}))
    md = bench.summarize_pmc(d, "tiny", str(roles))
    data = json.loads(re.search(r"<!-- traffic-json (\{.*\}) -->", md).group(1))
    r = data["roles"]
    assert r["shared:fwd_replay"]["fetch_bytes_per_launch"] == round(300.0 * 1024 * 2)
    assert r["flattened:fwd_prefill"]["write_bytes_per_launch"] == round(90.0 * 1024)
    assert "shared:dq_replay" in md
    # the per-kernel figures hold the shared step's dispatches only
    k = data["kernels"]["attn_fwd_kernel<bf16 out>"]
    assert k["launches"] == 2 and k["fetch_bytes_per_launch"] == round(200.0 * 1024 * 2)
    roles.write_text(json.dumps({"launches": ["shared:fwd_prefill"]}))
    try:
        bench.summarize_pmc(d, "tiny", str(roles))
        raise AssertionError("count mismatch not detected")
    except ValueError:
        pass


def test_algorithmic_bytes_count_prompt_kv_once():
    """The replay forward's minimum reads hold the prompt KV once; the
    flattened forward's hold its private copies (G per group)."""
    from paper_2609_33133_amd import inputs as I
    s = I.config_shape("prompt")
    rd, wr = bench.algorithmic_bytes("shared:fwd_replay", s)
    kvp = 2 * s.total_prompt * s.num_kv_heads * s.head_dim * 2
    q = s.total_resp * s.num_q_heads * s.head_dim * 2
    assert rd == q + kvp + 2 * s.total_resp * s.num_kv_heads * s.head_dim * 2
    assert wr == q + s.total_resp * s.num_q_heads * 4
    flat_rows = 8 * 32768 + s.total_resp
    rd_f, _ = bench.algorithmic_bytes("flattened:fwd_prefill", s, flat_rows)
    assert rd_f > 7 * kvp
