"""The measurement pipeline's arithmetic (CPU): the HBM-traffic figure that
bench.py reports is the decode kernel's FETCH_SIZE and WRITE_SIZE counters,
each scaled by what the same counter reads for a copy of known size.  These
tests feed synthetic counter files through the summary and check the
calibration pick and the scaling against hand-computed values."""
import csv
import json
import os

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
