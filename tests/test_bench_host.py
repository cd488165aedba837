"""Host-side checks of bench.py (no GPU): the command line, the sweep table,
the multi-GPU refusal and the rocprofv3 summary writer."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2509_24745_amd.synth import WORKLOADS  # noqa: E402


def test_sweeps_are_well_formed_and_selectable():
    old = sys.argv
    try:
        for name in bench.SWEEPS:
            sys.argv = ["bench.py", "--sweep", name]
            assert bench.parse().sweep == name
    finally:
        sys.argv = old
    for name, points in bench.SWEEPS.items():
        assert points, name
        for wname, kw, variant in points:
            wl = WORKLOADS[wname].replace(**kw) if kw else WORKLOADS[wname]
            assert wl.num_q_heads % wl.num_proxy_groups == 0
            assert variant.replace("+overlap", "") in ("dynamic", "row_ratio", "static_match")
    for fn in ("measure", "run_sweep", "run_stack", "_stack_layer", "_layer_stream", "run_decoder", "run_shard",
               "DecoderPrefill",
               "overlap_stats", "cpu_baseline", "profile_summary"):
        assert callable(getattr(bench, fn)), fn


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stdout


def _write_counters(path, rows):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "run_counter_collection.csv"), "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writerows(rows)


def test_profile_summary_scales_counters_by_the_copy_calibration(tmp_path, monkeypatch):
    d = str(tmp_path / "prof")
    sparse = "_ZN2pa11attn_kernelIDF16bLi128ELi128ELb0EEEvNS_5ShapeE"
    _write_counters(os.path.join(d, "pmc_FETCH_SIZE"), [[sparse, "FETCH_SIZE", 1000.0],
                                                        [sparse, "FETCH_SIZE", 3000.0]])
    _write_counters(os.path.join(d, "pmc_WRITE_SIZE"), [[sparse, "WRITE_SIZE", 500.0]])
    _write_counters(os.path.join(d, "cal_FETCH_SIZE"), [["__amd_rocclr_copyBuffer", "FETCH_SIZE",
                                                         float(1 << 19)]])
    _write_counters(os.path.join(d, "cal_WRITE_SIZE"), [["__amd_rocclr_copyBuffer", "WRITE_SIZE",
                                                         float(1 << 20)]])
    os.makedirs(os.path.join(d, "trace"))
    with open(os.path.join(d, "trace", "run_kernel_stats.csv"), "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs"])
        w.writerow([sparse, 2, 2e6, 1e6, 100.0, 1e6, 1e6])
    out_json = str(tmp_path / "traffic.json")
    monkeypatch.setattr(bench, "TRAFFIC_JSON", out_json)
    md = bench.profile_summary(d, "llama3_8b_n131072")
    rec = json.load(open(out_json))
    # FETCH reads half of a copy's bytes here: scale 2; WRITE scale 1
    assert rec["fetch_bytes"] == pytest.approx(2000.0 * 1024 * 2)
    assert rec["write_bytes"] == pytest.approx(500.0 * 1024)
    assert rec["kernel_sources_sha256"] == bench.kernel_sources_sha256()
    assert "attn_kernel<bf16,d128,b128,sparse>" in md and "rocprofv3" in md


def test_sweep_points_sharing_inputs_have_the_same_input_shapes():
    """Sweep points reuse uploaded inputs only when their input key matches;
    a key that ignored the sequence length once fed 8K tensors to a 16K
    problem.  Equal keys must mean identical input shapes and draws."""
    for name, points in bench.SWEEPS.items():
        seen = {}
        for wname, kw, _ in points:
            wl = WORKLOADS[wname].replace(**kw) if kw else WORKLOADS[wname]
            key = bench.input_key(wname, wl)
            sig = (wl.seq_len, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.dtype,
                   wl.structure, wl.seed)
            assert seen.setdefault(key, sig) == sig, (name, key)
    keys = {bench.input_key(w, WORKLOADS[w].replace(**kw)) for w, kw, _ in bench.SWEEPS["seq_len_llama"]}
    assert len(keys) == len(bench.SWEEPS["seq_len_llama"])
