"""Host-side pieces of bench.py: the --gpus guard, the rocprofv3 summary and the
rule that measured traffic is reported only for the kernels it was taken on."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]


def _write_csv(path, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0].keys()))
        w.writeheader()
        w.writerows(rows)


def test_profile_summary_scales_counters_by_the_calibration_kernel(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILE_DIR", str(tmp_path / "profiles"))
    upd = "void ssmq::k_update_slab<1, 2, 256, 2>(ssmq::UpdateArgs)"
    neg = "void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel_cuda>"
    cal_kib = bench.CAL_BYTES / 1024.0
    trace = tmp_path / "trace"
    _write_csv(str(trace / "run_kernel_stats.csv"),
               [{"Name": upd, "Calls": 2, "TotalDurationNs": 340000, "AverageNs": 170000,
                 "MinNs": 169000, "MaxNs": 171000}])
    # two launches on the hybrid stack's grid, one of the same kernel on a smaller
    # workload's grid (the configs block), which must not enter the average
    g = {"Grid_Size_X": 1 << 20, "Grid_Size_Y": 1, "Grid_Size_Z": 1}
    _write_csv(str(trace / "run_kernel_trace.csv"),
               [{"Kernel_Name": upd, "Start_Timestamp": 0, "End_Timestamp": 170000, **g},
                {"Kernel_Name": upd, "Start_Timestamp": 500000, "End_Timestamp": 670000, **g},
                {"Kernel_Name": upd, "Start_Timestamp": 900000, "End_Timestamp": 906000,
                 "Grid_Size_X": 1 << 14, "Grid_Size_Y": 1, "Grid_Size_Z": 1}])
    from paper_2609_39185_amd import workloads as wl
    algo = wl.WORKLOADS["hybrid_m2_stack"].entries_per_layer * 4
    for name, counter, cal_read, upd_read in (("fetch", "FETCH_SIZE", cal_kib / 2, algo / 2048.0),
                                              ("write", "WRITE_SIZE", cal_kib, algo / 2048.0)):
        _write_csv(str(tmp_path / name / "run_counter_collection.csv"),
                   [{"Kernel_Name": neg, "Grid_Size": 1 << 26, "Counter_Name": counter,
                     "Counter_Value": cal_read},
                    {"Kernel_Name": upd, "Grid_Size": 1 << 20, "Counter_Name": counter,
                     "Counter_Value": upd_read}])
    assert bench.summarize_profiles("hybrid_m2_stack", str(trace), str(tmp_path / "fetch"),
                                    str(tmp_path / "write")) == 0
    rec = json.load(open(tmp_path / "profiles" / "k_update_slab.hybrid_m2_stack.traffic.json"))
    v = rec["variants"]["bf16:weyl"]
    assert rec["calibration"]["fetch_scale"] == pytest.approx(2.0)
    assert rec["calibration"]["write_scale"] == pytest.approx(1.0)
    # fetch read half the true bytes (scaled x2), write read them all: 1.5x the algorithmic bytes
    assert v["traffic_bytes"] == pytest.approx(1.5 * algo)
    assert v["trace_avg_us"] == pytest.approx(170.0)
    assert v["kernel"] == "k_update_slab<1, 2, 256, 2>"
    # the counters describe the kernels as they are: reported while the digest matches ...
    assert bench.load_traffic("hybrid_m2_stack")["bf16:weyl"]["traffic_bytes"] == v["traffic_bytes"]
    # ... and not once the sources differ
    rec["kernel_sources_sha256"] = "0" * 64
    json.dump(rec, open(tmp_path / "profiles" / "k_update_slab.hybrid_m2_stack.traffic.json", "w"))
    assert bench.load_traffic("hybrid_m2_stack") is None


def test_replay_trace_summary_rates(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILE_DIR", str(tmp_path / "profiles"))
    name = "void ssmq::k_replay<4, 2>(ssmq::ReplayArgs)"
    _write_csv(str(tmp_path / "trace" / "run_kernel_stats.csv"),
               [{"Name": name, "Calls": 1, "TotalDurationNs": 10_000_000, "AverageNs": 10_000_000,
                 "MinNs": 10_000_000, "MaxNs": 10_000_000},
                {"Name": "void other_kernel()", "Calls": 5, "TotalDurationNs": 5, "AverageNs": 1,
                 "MinNs": 1, "MaxNs": 1}])
    assert bench.summarize_replay_trace(str(tmp_path / "trace"), "k_replay.test") == 0
    text = open(tmp_path / "profiles" / "k_replay.test.kernel_trace.md").read()
    row = [ln for ln in text.splitlines() if "k_replay<4, 2>" in ln][0]
    # 8 B x 1,310,720 entries x 4096 steps in 10 ms
    assert "int8:weyl" in row and row.rstrip(" |").endswith(f"{8 * 1310720 * 4096 / 1e7:.0f}")
    assert "other_kernel" not in text


def test_variant_specs_and_their_algorithmic_bytes():
    from paper_2609_39185_amd import workloads as wl
    w = wl.WORKLOADS["hybrid_m2_stack"]
    n = w.entries_per_layer
    v = bench.parse_variant("e4m3:weyl", w)
    assert (v["fmt"], v["rule"], v["group"]) == ("e4m3", "weyl", wl.scale_group_of(w, "e4m3"))
    # one scale per 64x128 head: codes 1 B each way, scale 4 B each way per head
    assert bench.state_bytes_per_launch(w, "e4m3", 0) == 2 * n + 8 * (n // 8192)
    v = bench.parse_variant("e4m3/128:sr", w)
    assert (v["key"], v["fmt"], v["rule"], v["group"]) == ("e4m3/128:sr", "e4m3", "sr", 128)
    assert bench.state_bytes_per_launch(w, "e4m3", 128) == 2 * n + 8 * (n // 128)
    assert bench.state_bytes_per_launch(w, "int4", 16) == n + 8 * (n // 16)
    assert bench.state_bytes_per_launch(w, "bf16") == 4 * n
    with pytest.raises(SystemExit):
        bench.parse_variant("bf16/128:weyl", w)


def test_targets_summary_marks_each_format_against_80_percent():
    import bench
    res = {"bf16:weyl": {"pct_of_peak": 80.9}, "bf16:sr": {"pct_of_peak": 81.0},
           "e4m3:weyl": {"pct_of_peak": 63.9}, "int8/128:weyl": {"pct_of_peak": 58.5}}
    t = bench.targets_summary(res)
    assert set(t) == {"bf16:weyl", "e4m3:weyl", "int8/128:weyl"}
    assert t["bf16:weyl"]["meets_target"] and t["bf16:weyl"]["bound"] == "hbm"
    assert not t["e4m3:weyl"]["meets_target"] and t["e4m3:weyl"]["bound"] == "vector issue"
    assert t["int8/128:weyl"]["target_pct"] == 80.0


def test_instruction_mix_summary_per_wave(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILE_DIR", str(tmp_path / "profiles"))
    upd = "void ssmq::k_update_slab<2, 2, 128, 4, true>(ssmq::UpdateArgs)"
    other = "void at::native::elementwise_kernel<128, 4>"
    a = {"SQ_WAVES": 10, "SQ_INSTS_VALU": 7450, "SQ_INSTS_VALU_FMA_F32": 1295,
         "SQ_INSTS_VALU_MUL_F32": 1437, "SQ_INSTS_VALU_ADD_F32": 161, "SQ_INSTS_VALU_CVT": 977,
         "SQ_INSTS_VALU_INT32": 1101, "SQ_INSTS_VALU_INT64": 85}
    b = {"SQ_WAVES": 20, "SQ_INSTS_VALU_FMA_F64": 130, "SQ_INSTS_VALU_ADD_F64": 0,
         "SQ_INSTS_VALU_MUL_F64": 10, "SQ_INSTS_VALU_TRANS_F32": 10, "SQ_INSTS_SALU": 3184,
         "SQ_INSTS_LDS": 490, "SQ_INSTS_BRANCH": 566}
    for d, cs in (("a", a), ("b", b)):
        rows = [{"Kernel_Name": upd, "Grid_Size": 1 << 22, "Counter_Name": n, "Counter_Value": v}
                for n, v in cs.items()]
        rows.append({"Kernel_Name": other, "Grid_Size": 64, "Counter_Name": "SQ_WAVES",
                     "Counter_Value": 1})
        _write_csv(str(tmp_path / d / "run_counter_collection.csv"), rows)
    assert bench.summarize_mix("hybrid_m2_stack", str(tmp_path / "a"), str(tmp_path / "b")) == 0
    text = open(tmp_path / "profiles" / "k_update_slab.hybrid_m2_stack.valu_mix.md").read()
    row = [ln for ln in text.splitlines() if ln.startswith("| e4m3:weyl")][0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    # per wave of each pass: 745 VALU, of which 129.5 + 143.7 + 16.1 + 97.7 + 110.1 + 8.5
    # + 7.0 (f64) + 0.5 (trans) are counted by kind and 231.9 are the rest
    assert cells[2:] == ["129.5", "143.7", "16.1", "97.7", "110.1", "8.5", "7.0", "0.5", "231.9",
                         "745.0", "159.2", "24.5", "28.3"]
    assert "elementwise_kernel" not in text and "--summarize-mix" in text
