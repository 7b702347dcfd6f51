"""The measurement pipeline's arithmetic (CPU): the HBM-traffic figure that
bench.py reports is the decode kernel's FETCH_SIZE and WRITE_SIZE counters,
each scaled by what the same counter reads for a copy of known size.  These
tests feed synthetic counter files through the summary and check the
calibration pick and the scaling against hand-computed values, and do the
same for the compute-side counter summary (busy fractions, per-step counts),
the roofline object (bytes per launch over the kernel's average time) and the
per-workload rates, and the rule that a counter summary is used only on the
kernel sources it was taken on."""
import csv
import json
import os

import numpy as np
import pytest

import bench
import workloads as wl


def _write(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Grid_Size",
                                          "Counter_Value"])
        w.writeheader()
        for r in rows:
            w.writerow(r)


def _row(kernel, counter, value, grid=1024):
    return {"Kernel_Name": kernel, "Counter_Name": counter, "Grid_Size": grid,
            "Counter_Value": value}


@pytest.fixture
def counters(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path / "profiles"))
    copy, dec, comb = bench.CALIBRATION_KERNEL, "void dora::decode_kernel<128>", \
        "dora::combine_kernel(dora::CombineParams)"
    gib = bench.CALIBRATION_BYTES // 1024          # KiB moved by the calibration copy
    # FETCH counts the 2 GiB copy twice (factor 0.5); a small copy (a pack set)
    # shares the kernel name and must not enter the calibration.
    _write(tmp_path / "f", [_row(copy, "FETCH_SIZE", 2 * gib), _row(copy, "FETCH_SIZE", 2 * gib),
                            _row(copy, "FETCH_SIZE", 1000.0),
                            _row(dec, "FETCH_SIZE", 400000.0), _row(dec, "FETCH_SIZE", 420000.0)])
    # WRITE counts it exactly (factor 1)
    _write(tmp_path / "w", [_row(copy, "WRITE_SIZE", gib), _row(copy, "WRITE_SIZE", 10.0),
                            _row(dec, "WRITE_SIZE", 5000.0)])
    _write(tmp_path / "l2", [_row(dec, "TCC_HIT_sum", 30.0), _row(dec, "TCC_MISS_sum", 970.0),
                             _row(comb, "TCC_HIT_sum", 1.0), _row(comb, "TCC_MISS_sum", 3.0)])
    return tmp_path


def test_traffic_is_scaled_by_the_largest_copy(counters):
    t = counters
    bench.summarize_pmc(str(t / "f"), str(t / "w"), str(t / "l2"), "rollout7b")
    s = json.load(open(bench.pmc_path("rollout7b")))
    cal = s["calibration"]
    assert cal["dispatches"] == [2, 1]              # the small copies are left out
    assert cal["fetch_factor"] == pytest.approx(0.5)
    assert cal["write_factor"] == pytest.approx(1.0)
    assert s["fetch_kib_per_dispatch"] == pytest.approx(410000.0)
    assert s["write_kib_per_dispatch"] == pytest.approx(5000.0)
    want = 410000.0 * 1024 * 0.5 + 5000.0 * 1024 * 1.0
    assert s["traffic_bytes_per_launch"] == pytest.approx(want)
    w = wl.BY_NAME["rollout7b"]
    ab = wl.algorithmic_bytes(w, wl.sample_lengths(w, wl.seeds(wl.WORKLOADS.index(w))[0]))
    assert s["algorithmic_bytes_per_launch"] == ab["total"]
    assert s["traffic_over_algorithmic"] == pytest.approx(want / ab["total"])
    assert s["l2"]["decode_kernel"]["hit_rate"] == pytest.approx(0.03)
    assert s["kernel_source_hash"] == bench.kernel_source_hash()


def test_missing_decode_dispatches_are_an_error(counters):
    t = counters
    _write(t / "w", [_row(bench.CALIBRATION_KERNEL, "WRITE_SIZE", 1.0)])
    with pytest.raises(ValueError):
        bench.summarize_pmc(str(t / "f"), str(t / "w"), str(t / "l2"), "rollout7b")


def _write_compute(d, rows, gpu=("8", "256", "1024", "2400")):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_agent_info.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Agent_Type", "Num_Xcc", "Cu_Count", "Simd_Count",
                                          "Max_Engine_Clk_Fcompute"])
        w.writeheader()
        w.writerow({"Agent_Type": "CPU", "Num_Xcc": "0", "Cu_Count": "0", "Simd_Count": "0",
                    "Max_Engine_Clk_Fcompute": "0"})
        w.writerow(dict(zip(["Agent_Type", "Num_Xcc", "Cu_Count", "Simd_Count",
                             "Max_Engine_Clk_Fcompute"], ("GPU",) + gpu)))
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value",
                                          "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        for r in rows:
            w.writerow(r)


def _crow(kernel, counter, value, t0=0, t1=100000):
    return {"Kernel_Name": kernel, "Counter_Name": counter, "Counter_Value": value,
            "Start_Timestamp": t0, "End_Timestamp": t1}


def test_compute_counters_give_busy_fractions_and_per_step_counts(tmp_path, monkeypatch):
    """Busy fractions are counter cycles over (GRBM cycles per XCC x SIMDs),
    quad-cycle counters are scaled by 4, and per-step figures divide by the
    workload's (page, KV head) steps; other libraries' kernels are left out."""
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path / "profiles"))
    dec = "void dora::decode_kernel<128, 16, false, 3, false>(dora::DecodeParams)"
    gui = 8 * 200000.0                         # 200,000 cycles per XCC, two dispatches
    _write_compute(tmp_path / "c1", [
        _crow(dec, "GRBM_GUI_ACTIVE", gui, 0, 100000), _crow(dec, "GRBM_GUI_ACTIVE", gui, 0, 100000),
        _crow(dec, "SQ_INSTS_MFMA", 1200.0), _crow(dec, "SQ_INSTS_MFMA", 1200.0),
        _crow(dec, "SQ_VALU_MFMA_BUSY_CYCLES", 0.1 * 200000 * 1024),
        _crow(dec, "SQ_WAVE_CYCLES", 1000.0),
        _crow("void at::native::elementwise_kernel<4>", "SQ_INSTS_MFMA", 5.0)])
    _write_compute(tmp_path / "c2", [
        _crow(dec, "GRBM_GUI_ACTIVE", gui), _crow(dec, "SQ_ACTIVE_INST_VALU", 0.05 * 200000 * 1024),
        _crow(dec, "SQ_WAIT_ANY", 600.0), _crow(dec, "SQ_LDS_BANK_CONFLICT", 0.0)])
    _write_compute(tmp_path / "c3", [_crow(dec, "VmemLatency", 2000.0)])
    bench.summarize_compute([str(tmp_path / c) for c in ("c1", "c2", "c3")], "rollout7b")
    s = json.load(open(bench.compute_path("rollout7b")))
    assert list(s["kernels"]) == [dec]
    k = s["kernels"][dec]
    assert k["dispatches"] == 2 and k["avg_duration_us"] == pytest.approx(100.0)
    d = k["derived"]
    assert d["engine_clock_ghz"] == pytest.approx(2.0)         # 200,000 cycles in 100 us
    assert d["mfma_busy_frac"] == pytest.approx(0.1)
    assert d["valu_busy_frac"] == pytest.approx(0.2)           # quad cycles x 4
    assert d["wave_wait_any_frac"] == pytest.approx(0.6)
    assert d["vmem_latency_cycles"] == pytest.approx(2000.0)
    w = wl.BY_NAME["rollout7b"]
    L = wl.sample_lengths(w, wl.seeds(wl.WORKLOADS.index(w))[0])
    steps = int(wl.pages_needed(L, w.page_size).sum()) * w.num_kv_heads
    assert d["steps_per_launch"] == steps
    assert d["mfma_per_step"] == pytest.approx(1200.0 / steps)
    assert s["device"] == {"cus": 256, "simds": 1024, "xcc": 8, "max_engine_clock_mhz": 2400}
    assert s["kernel_source_hash"] == bench.kernel_source_hash()


def test_bench_trace_sets_trace_beside_events(tmp_path, monkeypatch):
    """The default-run trace summary pairs each decode-kernel instance with the
    workloads that launch it and, for an instance of one workload only, gives
    the ratio of that workload's event average to the trace average."""
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path / "profiles"))
    d = tmp_path / "t"
    os.makedirs(d)
    with open(d / "run_kernel_stats.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Name", "Calls", "AverageNs", "MinNs", "MaxNs"])
        w.writeheader()
        w.writerow({"Name": "void dora::decode_kernel<128, 32, true, 2, false>(dora::DecodeParams)",
                    "Calls": 65, "AverageNs": 2000000.0, "MinNs": 1, "MaxNs": 2})
        w.writerow({"Name": "void dora::decode_kernel<128, 16, false, 3, false>(dora::DecodeParams)",
                    "Calls": 260, "AverageNs": 100000.0, "MinNs": 1, "MaxNs": 2})
    rl = lambda ms: {"roofline": {"avg_launch_ms": ms}}
    line = {"value": 1.0, "unit": "tokens/s", "ms_per_step": 2.1,
            "roofline": {"achieved": 1.0, "frac": 0.5, "algorithmic_bytes_per_launch": 7},
            "workloads": {"moe_fp8": rl(2.02), "rollout7b": rl(0.1), "tail_only": rl(0.17)}}
    (tmp_path / "line.json").write_text("[bench] noise\n" + json.dumps(line) + "\n")
    bench.summarize_bench_trace(str(d), str(tmp_path / "line.json"))
    text = open(os.path.join(bench.PROFILES, f"decode_kernel_{bench.MAIN_WORKLOAD}_bench_trace.md")).read()
    assert "| `decode_kernel<128, 32, true, 2, false>` | moe_fp8 | 65 | 2000.00 | 2020.00 | 1.010 |" in text
    assert "rollout7b, tail_only" in text and "(shared instance)" in text
    assert bench.BENCH_TRACE_CMD in text


def test_pattern_tiles_follow_the_decode_work_order():
    """The exact-pattern reference reads, for every (sequence, KV head, page)
    page-head in that order, the K tile then the V tile at the byte offsets the
    pools' layout gives them (page * Hkv + head tiles into the pool; the V
    pool after the K pool)."""
    w = wl.Workload("t", 3, 4, 2, 64, 16, 0, 64, "lognormal", 40, 1.0, 1, 100)
    lengths = np.array([33, 0, 16], np.int32)
    table = np.array([[5, 9, 2], [0, 0, 0], [7, 0, 0]], np.int32)
    ids = bench.pattern_tiles(w, lengths, table)
    want = []
    for b, L in enumerate(lengths):
        for g in range(w.num_kv_heads):
            for j in range(-(-int(L) // w.page_size)):
                pid = int(table[b, j])
                want += [pid * 2 + g, w.num_pages * 2 + pid * 2 + g]
    assert ids.tolist() == want
    assert ids.dtype == np.int32 and ids.max() < 2 * w.num_pages * w.num_kv_heads


def test_source_hash_ignores_comments_only():
    code = "int f(int x) { // add one\n  return x + 1; /* done */ }\n"
    assert bench._code_only(code) == bench._code_only("int f(int x) {\n return x + 1;  }")
    assert bench._code_only(code) != bench._code_only("int f(int x) { return x + 2; }")


def test_roofline_object_is_bytes_over_the_kernel_average():
    """roofline.frac is the workload's algorithmic bytes per launch over the
    decode kernel's average event time, over the 8 TB/s peak; the two
    reference fractions divide the same rate by the references."""
    rec = {"algorithmic_bytes": {"total": 18_000_000_000}, "split_kernel_ms": 2.5,
           "split_kernel_traffic_bytes": 18_300_000_000, "split_kernel_l2_hit_rate": 0.3,
           "pattern_reference": {"best_gbps": 6_000.0}}
    r = bench.roofline_of(rec, achievable_gbps=6_500.0)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert r["achieved"] == pytest.approx(7_200.0)             # 18 GB / 2.5 ms
    assert r["frac"] == pytest.approx(0.9)
    assert r["frac_of_achievable"] == pytest.approx(7_200.0 / 6_500.0)
    assert r["frac_of_pattern"] == pytest.approx(1.2)
    assert r["traffic"] == 18_300_000_000 and r["avg_launch_ms"] == 2.5
    rec.pop("pattern_reference")
    assert bench.roofline_of(rec, 6_500.0)["frac_of_pattern"] is None


def test_decode_record_rates_follow_the_step_times():
    w = wl.BY_NAME["tiny"]
    lengths = wl.sample_lengths(w, wl.seeds(0)[0])
    ab = wl.algorithmic_bytes(w, lengths)["total"]
    t = {"step_ms": np.array([0.010, 0.012, 0.014]), "split_ms": np.array([0.008, 0.008]),
         "combine_ms": np.array([0.002, 0.004])}
    r = bench.decode_record(w, lengths, t)
    assert r["ms_per_step"] == pytest.approx(0.012)
    assert r["decode_tokens_per_s"] == pytest.approx(w.num_seqs / 12e-6)
    assert r["hbm_gbps"] == pytest.approx(ab / 12e-6 / 1e9)
    assert r["hbm_frac_of_peak"] == pytest.approx(ab / 12e-6 / 1e9 / 8000.0)
    assert r["split_kernel_gbps"] == pytest.approx(ab / 8e-6 / 1e9)
    assert r["combine_ms"] == pytest.approx(0.003)
    assert r["ms_p10_p50_p90"][1] == pytest.approx(0.012)


def test_counter_summaries_are_used_only_on_matching_sources(tmp_path, monkeypatch):
    """A committed counter summary feeds `traffic` only while the kernel
    sources hash to the value it records, and only for its own workload."""
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    w = wl.BY_NAME["rollout7b"]
    path = bench.pmc_path(w.name)
    json.dump({"workload": w.name, "kernel_source_hash": bench.kernel_source_hash()},
              open(path, "w"))
    assert bench.load_pmc(w) is not None
    json.dump({"workload": w.name, "kernel_source_hash": "0" * 16}, open(path, "w"))
    assert bench.load_pmc(w) is None
    json.dump({"workload": "tail_only", "kernel_source_hash": bench.kernel_source_hash()},
              open(path, "w"))
    assert bench.load_pmc(w) is None
    os.remove(path)
    assert bench.load_pmc(w) is None
