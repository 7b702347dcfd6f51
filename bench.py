"""Benchmark of the decode-attention hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--only-main]
                    [--no-cpu-baseline] [--no-flush] [--gpus 1]

One step = one dora_decode_attn call (stream-K decode kernel + combine) over
one synthetic long-tailed decode batch whose inputs are already resident in
HBM.  Caches (256 MB Infinity Cache, 8 x 4 MB L2) are evicted by a 1 GiB read
before every step, outside the timed events.  The main line is the largest
batch, the MoE-scale one (1024 sequences, fp8 E4M3 KV with per-page scales,
32-token pages, lognormal lengths with median 4096); the other workloads and
the pack/unpack copy are reported under "workloads", each with its own
roofline object.

Prints one JSON line.  value = decode tokens/s = sequences / step time (every
sequence advances one token per step).  roofline: the decode kernel's
algorithmic bytes (K and V of valid tokens, page scales, Q, output, block
table and lengths) over its average duration, measured with HIP events that
the library records around each kernel on the launch stream
(dora_decode_attn_timed).  Two achievable-bandwidth references stand beside
the 8 TB/s peak, both read by the library's own streaming-read kernel
(dora_stream_read, 16-byte non-temporal loads): random 4 KiB tiles of a
16 GiB buffer (achievable_gbps), and each batch's own tile sequence in its
decode work order (pattern_gbps).  traffic: HBM bytes per launch from the
committed rocprofv3 counter summary, while it matches the kernel sources.
The rocprofv3 summaries under profiles/ are made from this script's runs
with the --summarize-* options.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as wl  # noqa: E402

METRIC = "decode-attn tokens/s and HBM GB/s (% of peak) on long-tail length mixes"
HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
MAIN_WORKLOAD = "moe_fp8"
SINGLE_CORE_WORKLOADS = ("tiny", "rollout7b")   # the oracle on one core as well
PROFILES = os.path.join(ROOT, "profiles")
DECODE_KERNEL = "dora::decode_kernel"
CALIBRATION_KERNEL = "__amd_rocclr_copyBuffer"   # the 2 GiB device copy in copy_bandwidth()
CALIBRATION_BYTES = 2 << 30                        # read and written per dispatch
TRACE_CMD = ("cd /tmp && rocprofv3 --kernel-trace --stats --output-format csv "
             "-d $REPO/gpurun_out/prof_trace_{w} -o run -- python $REPO/bench.py --only-main "
             "--workload {w} --no-cpu-baseline --steps 30")
BENCH_TRACE_CMD = ("cd /tmp && rocprofv3 --kernel-trace --stats --output-format csv "
                   "-d $REPO/gpurun_out/prof_trace_bench -o run -- python $REPO/bench.py "
                   "> $REPO/gpurun_out/prof_trace_bench.json")
GRPO_TRACE_CMD = ("cd /tmp && rocprofv3 --kernel-trace --stats --output-format csv "
                  "-d $REPO/gpurun_out/prof_trace_grpo7b -o run -- python $REPO/bench.py "
                  "--grpo-only --steps 30")
PMC_CMD = ("cd /tmp && timeout -s KILL 300 rocprofv3 --pmc {c} --output-format csv "
           "-d $REPO/gpurun_out/pmc_{d}_{w} -o run -- python $REPO/bench.py --only-main "
           "--workload {w} --no-cpu-baseline --steps 5 --warmup 1")
L2_COUNTERS = "TCC_HIT_sum TCC_MISS_sum"
# Compute-side counters, three rocprofv3 --pmc passes (at most 8 SQ counters
# and 2 GRBM counters per pass; VmemLatency and MemUnitStalled are rocprofv3's
# derived metrics).
COMPUTE_PASSES = {
    "C1": ("SQ_INSTS_VALU SQ_INSTS_MFMA SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CU_CYCLES SQ_WAVES "
           "SQ_WAVE_CYCLES SQ_WAIT_INST_ANY SQ_INSTS_VALU_CVT GRBM_GUI_ACTIVE"),
    "C2": ("SQ_ACTIVE_INST_VALU SQ_INSTS_VMEM_RD SQ_INSTS_SALU SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT "
           "SQ_ACTIVE_INST_ANY SQ_WAIT_ANY SQ_BUSY_CYCLES GRBM_GUI_ACTIVE"),
    "C3": "VmemLatency MemUnitStalled",
}
COMPUTE_CMD = ("cd /tmp && timeout -s KILL 300 rocprofv3 --pmc {c} --output-format csv "
               "-d $REPO/gpurun_out/pmc_{p}_{w} -o run -- python $REPO/bench.py {args}")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2604_26256_amd", "csrc", f)
                  for f in ("decode.hip", "decode_core.h", "dora_internal.h", "api.cpp")]


def _code_only(text: str) -> str:
    """C/C++ source with comments removed and whitespace collapsed, so that a
    comment edit does not count as a change of the kernels (string literals
    in these sources hold no comment markers)."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash() -> str:
    """Hash of the code (not the comments) of the sources the decode kernel's
    launches are built from; stored with every counter summary."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=MAIN_WORKLOAD, choices=[w.name for w in wl.WORKLOADS])
    ap.add_argument("--only-main", action="store_true", help="skip the other workloads")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-flush", action="store_true")
    ap.add_argument("--flush-mode", choices=["read", "write"], default="read",
                    help="evict caches by reading (clean lines) or writing 1 GiB")
    ap.add_argument("--event-flags", type=lambda x: int(x, 0), default=EVENT_FLAGS,
                    help="hipEventCreateWithFlags flags of the timing events")
    ap.add_argument("--num-waves", type=int, default=0,
                    help="decode wavefronts (0 = one per resident slot)")
    ap.add_argument("--grpo-only", action="store_true",
                    help="time only the GRPO batch (plain against grouped decode)")
    ap.add_argument("--summarize-grpo-trace", metavar="DIR",
                    help="write the kernel-trace summary of a --grpo-only rocprofv3 run")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="write the kernel-trace summary of a rocprofv3 run under profiles/")
    ap.add_argument("--summarize-bench-trace", nargs=2, metavar=("DIR", "JSON"),
                    help="write the kernel-trace summary of a default bench run under "
                         "rocprofv3, beside the bench line that run printed")
    ap.add_argument("--summarize-pmc", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "L2_DIR"),
                    help="write the HBM-traffic and L2 hit-rate summary of three "
                         "rocprofv3 --pmc runs")
    ap.add_argument("--summarize-compute", nargs=4, metavar=("WORKLOAD", "C1", "C2", "C3"),
                    help="write the compute-side counter summary of three rocprofv3 --pmc "
                         "runs (WORKLOAD: a workload name or grpo7b)")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# rocprofv3 summaries (CPU only: they read the CSV files a GPU run wrote)
# ---------------------------------------------------------------------------

def _find_csv(d, suffix):
    for root, _, files in os.walk(d):
        for f in files:
            if f.endswith(suffix):
                return os.path.join(root, f)
    raise FileNotFoundError(f"no *{suffix} under {d}")


def pmc_path(workload):
    return os.path.join(PROFILES, f"decode_kernel_{workload}_pmc.json")


def summarize_trace(d, workload, grpo=False):
    import csv
    rows = list(csv.DictReader(open(_find_csv(d, "kernel_stats.csv"))))
    if grpo:
        out = os.path.join(PROFILES, "grouped_decode_grpo7b_trace.md")
        head = ["# rocprofv3 kernel trace: GRPO batch, plain and grouped decode", "",
                "Command (repo root as $REPO):", "", "    " + GRPO_TRACE_CMD, "",
                "`decode_kernel<..., false>` is the plain path; the grouped call runs",
                "`prefix_kernel`, `decode_kernel<..., true>` (the suffix) and",
                "`combine_grouped_kernel`.  Per-kernel durations from",
                "`run_kernel_stats.csv` (all dispatches: warm-up and timed calls).", ""]
    else:
        out = os.path.join(PROFILES, f"decode_kernel_{workload}_trace.md")
        head = [f"# rocprofv3 kernel trace: {workload}", "",
                "Command (repo root as $REPO):", "", "    " + TRACE_CMD.format(w=workload), "",
                "Per-kernel durations from `run_kernel_stats.csv` (all dispatches of the run:",
                "warm-up, timed steps and the per-kernel event pass).", ""]
    lines = head + ["| kernel | calls | avg us | min us | max us |", "|---|---|---|---|---|"]
    for r in rows:
        name = r.get("Name") or r.get("KernelName") or ""
        if not any(k in name for k in ("dora::", "reduce_kernel", CALIBRATION_KERNEL)):
            continue
        avg = float(r.get("AverageNs") or r.get("AvgNs")) / 1e3
        lines.append(f"| `{name[:70]}` | {r['Calls']} | {avg:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} |")
    lines += ["", f"Kernel source hash: `{kernel_source_hash()}`", ""]
    os.makedirs(PROFILES, exist_ok=True)
    open(out, "w").write("\n".join(lines))
    print(out)


def _kernel_instance(w):
    """Pattern of the decode kernel's template instance that workload w
    launches (head dim, page size, fp8 or not, the page-buffer count the
    library picks for that geometry, plain rather than suffix decode)."""
    return (rf"decode_kernel<{w.head_dim}, {w.page_size}, "
            rf"{'true' if w.kv_dtype == 1 else 'false'}, \d+, false>")


def summarize_bench_trace(d, line_path):
    """Kernel-trace summary of the default bench command run under rocprofv3,
    set beside the event timings of the bench line that same run printed.
    A decode-kernel instance launched by one workload only (the headline's fp8
    instance) gives a trace average directly comparable with that workload's
    event average; an instance shared by several workloads averages over all
    of their dispatches."""
    import csv
    line = json.loads([ln for ln in open(line_path) if ln.strip().startswith("{")][-1])
    rows = list(csv.DictReader(open(_find_csv(d, "kernel_stats.csv"))))
    stats = {}
    for r in rows:
        name = r.get("Name") or r.get("KernelName") or ""
        stats[name] = (int(r["Calls"]), float(r.get("AverageNs") or r.get("AvgNs")) / 1e3)
    by_inst = {}
    for w in wl.WORKLOADS:
        if w.name in line.get("workloads", {}):
            by_inst.setdefault(_kernel_instance(w), []).append(w.name)
    shared_with_grpo = set()
    if "shared_prefix" in line:       # the GRPO batch's plain decode, timed as a whole call
        shared_with_grpo.add(_kernel_instance(wl.GRPO_WORKLOAD))
    out = os.path.join(PROFILES, f"decode_kernel_{MAIN_WORKLOAD}_bench_trace.md")
    lines = [f"# rocprofv3 kernel trace of the default bench run (headline: {MAIN_WORKLOAD})",
             "", "Command (repo root as $REPO):", "", "    " + BENCH_TRACE_CMD, "",
             "Decode-kernel instances in `run_kernel_stats.csv` (all dispatches of the run),",
             "beside the event average (`roofline.avg_launch_ms`) that the bench line of",
             "the same run reports for each workload launching that instance.", "",
             "| kernel instance | workloads | calls | trace avg us | event avg us | events / trace |",
             "|---|---|---|---|---|---|"]
    for pat, names in by_inst.items():
        hit = [(m.group(0), v) for k, v in stats.items() for m in [re.search(pat, k)] if m]
        if not hit:
            continue
        inst, (calls, tavg) = hit[0]
        ev = [line["workloads"][n]["roofline"]["avg_launch_ms"] * 1e3 for n in names]
        shown = names + (["grpo7b (plain path)"] if pat in shared_with_grpo else [])
        if len(shown) == 1:
            ratio = f"{ev[0] / tavg:.3f}"
        else:
            ratio = "(shared instance)"
        lines.append(f"| `{inst}` | {', '.join(shown)} | {calls} | {tavg:.2f} | "
                     f"{', '.join(f'{e:.2f}' for e in ev)} | {ratio} |")
    rl = line["roofline"]
    lines += ["", f"Bench line of the run: value {line['value']:.0f} {line['unit']}, "
              f"{line['ms_per_step'] * 1e3:.1f} us per step; roofline achieved "
              f"{rl['achieved']:.0f} GB/s, frac {rl['frac']:.3f} "
              f"({rl['algorithmic_bytes_per_launch']} B per launch).", "",
              f"Kernel source hash: `{kernel_source_hash()}`", ""]
    os.makedirs(PROFILES, exist_ok=True)
    open(out, "w").write("\n".join(lines))
    print(out)


def summarize_pmc(fetch_dir, write_dir, l2_dir, workload):
    import csv

    def per_kernel(d, counter):
        acc = {}
        for r in csv.DictReader(open(_find_csv(d, "counter_collection.csv"))):
            if r["Counter_Name"] != counter:
                continue
            acc.setdefault(r["Kernel_Name"], []).append((int(r["Grid_Size"]),
                                                         float(r["Counter_Value"])))
        return acc

    fetch = per_kernel(fetch_dir, "FETCH_SIZE")
    write = per_kernel(write_dir, "WRITE_SIZE")
    hit = per_kernel(l2_dir, "TCC_HIT_sum")
    miss = per_kernel(l2_dir, "TCC_MISS_sum")

    def pick(acc, key, calibration=False):
        vals = [v for k, lst in acc.items() if key in k for v in lst]
        if not vals:
            raise ValueError(f"no dispatches of {key} in the counter data")
        if calibration:
            # the 2 GiB copy: the largest copy of the run (other copies, such as
            # the pack set's, share its grid but move less)
            top = max(v[1] for v in vals)
            vals = [v for v in vals if v[1] >= 0.5 * top]
        return sum(v[1] for v in vals) / len(vals), len(vals)

    cf, ncf = pick(fetch, CALIBRATION_KERNEL, calibration=True)
    cw, ncw = pick(write, CALIBRATION_KERNEL, calibration=True)
    ff = CALIBRATION_BYTES / (cf * 1024)
    fw = CALIBRATION_BYTES / (cw * 1024)
    df, ndf = pick(fetch, DECODE_KERNEL)
    dw, ndw = pick(write, DECODE_KERNEL)
    w = wl.BY_NAME[workload]
    lengths = wl.sample_lengths(w, wl.seeds(wl.WORKLOADS.index(w))[0])
    ab = wl.algorithmic_bytes(w, lengths)["total"]
    traffic = df * 1024 * ff + dw * 1024 * fw
    dh, _ = pick(hit, DECODE_KERNEL)
    dm, _ = pick(miss, DECODE_KERNEL)
    ch, _ = pick(hit, "dora::combine_kernel")
    cm, _ = pick(miss, "dora::combine_kernel")
    summary = {
        "workload": workload, "kernel": "decode_kernel",
        "kernel_source_hash": kernel_source_hash(),
        "commands": [PMC_CMD.format(c="FETCH_SIZE", d="FETCH_SIZE", w=workload),
                     PMC_CMD.format(c="WRITE_SIZE", d="WRITE_SIZE", w=workload),
                     PMC_CMD.format(c=f'"{L2_COUNTERS}"', d="L2", w=workload)],
        "fetch_kib_per_dispatch": df, "write_kib_per_dispatch": dw,
        "dispatches": {"fetch": ndf, "write": ndw},
        "calibration": {"kernel": CALIBRATION_KERNEL, "bytes_read_and_written": CALIBRATION_BYTES,
                        "fetch_kib": cf, "write_kib": cw, "dispatches": [ncf, ncw],
                        "fetch_factor": ff, "write_factor": fw},
        "traffic_bytes_per_launch": traffic,
        "algorithmic_bytes_per_launch": ab,
        "traffic_over_algorithmic": traffic / ab,
        "l2": {"decode_kernel": {"hits_per_dispatch": dh, "misses_per_dispatch": dm,
                                 "hit_rate": dh / (dh + dm)},
               "combine_kernel": {"hits_per_dispatch": ch, "misses_per_dispatch": cm,
                                  "hit_rate": ch / (ch + cm)}},
    }
    os.makedirs(PROFILES, exist_ok=True)
    out = pmc_path(workload)
    json.dump(summary, open(out, "w"), indent=1)
    print(out)


def compute_bench_args(workload):
    return ("--grpo-only --steps 5" if workload == "grpo7b" else
            f"--only-main --workload {workload} --no-cpu-baseline --steps 5 --warmup 1")


def compute_path(workload):
    return os.path.join(PROFILES, f"compute_counters_{workload}.json")


def _work_units(workload):
    """Work per launch of the decode-attention kernels of a bench run, in
    (page, KV head) steps of 16 query columns: {kernel name fragment: units}."""
    if workload == "grpo7b":
        w, M = wl.GRPO_WORKLOAD, wl.GRPO_GROUP
        lengths, shared = wl.grpo_lengths()
        n = wl.pages_needed(lengths, w.page_size)
        tiles = -(-(M * w.group) // 16)            # column tiles of a group's prefix
        lead = shared[::M].astype(np.int64)
        return {"decode_kernel<128, 16, false, 3, false>": int(n.sum()) * w.num_kv_heads,
                "decode_kernel<128, 16, false, 3, true>": int((n - shared).sum()) *
                w.num_kv_heads,
                "prefix_kernel": int(lead.sum()) * w.num_kv_heads * tiles}
    w = wl.BY_NAME[workload]
    lengths = wl.sample_lengths(w, wl.seeds(wl.WORKLOADS.index(w))[0])
    return {"decode_kernel": int(wl.pages_needed(lengths, w.page_size).sum()) * w.num_kv_heads}


def summarize_compute(dirs, workload):
    """Per-dispatch averages of the compute-side counters of every library
    kernel in three --pmc runs, with derived figures: MFMA and VALU busy
    fractions of the SIMDs, the share of wave time spent waiting, mean
    resident waves per CU, the engine clock over the dispatch, and, for the
    decode-attention kernels, instructions per (page, KV head, 16-column)
    step."""
    import csv

    agent = None
    per = {}
    for d in dirs:
        for r in csv.DictReader(open(_find_csv(d, "agent_info.csv"))):
            if r["Agent_Type"] == "GPU":
                agent = r
        for r in csv.DictReader(open(_find_csv(d, "counter_collection.csv"))):
            k = r["Kernel_Name"]
            if not k.startswith(("dora::", "void dora::")):
                continue
            e = per.setdefault(k, {"counters": {}, "durations_ns": []})
            e["counters"].setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
            if r["Counter_Name"] == "GRBM_GUI_ACTIVE" and d == dirs[0]:
                e["durations_ns"].append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    xcc, cus, simds = int(agent["Num_Xcc"]), int(agent["Cu_Count"]), int(agent["Simd_Count"])
    units = _work_units(workload)
    kernels = {}
    for k, e in per.items():
        c = {n: sum(v) / len(v) for n, v in e["counters"].items()}
        dur = sum(e["durations_ns"]) / max(1, len(e["durations_ns"]))
        gui = c.get("GRBM_GUI_ACTIVE", 0.0) / xcc          # cycles of one XCC
        der = {}
        if gui > 0:
            der["engine_clock_ghz"] = gui / dur if dur else None
            der["mfma_busy_frac"] = c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (gui * simds)
            der["valu_busy_frac"] = 4 * c.get("SQ_ACTIVE_INST_VALU", 0.0) / (gui * simds)
            der["mean_waves_per_cu"] = 4 * c.get("SQ_WAVE_CYCLES", 0.0) / (gui * cus)
            der["lds_bank_conflict_frac_of_cu_time"] = \
                c.get("SQ_LDS_BANK_CONFLICT", 0.0) / (gui * cus)
        if c.get("SQ_WAVE_CYCLES"):
            der["wave_wait_any_frac"] = c.get("SQ_WAIT_ANY", 0.0) / c["SQ_WAVE_CYCLES"]
            der["wave_wait_inst_frac"] = c.get("SQ_WAIT_INST_ANY", 0.0) / c["SQ_WAVE_CYCLES"]
        der["vmem_latency_cycles"] = c.get("VmemLatency")
        u = next((v for frag, v in units.items() if frag in k), None)
        if u:
            der["steps_per_launch"] = u
            for n in ("SQ_INSTS_MFMA", "SQ_INSTS_VALU", "SQ_INSTS_VALU_CVT", "SQ_INSTS_SALU",
                      "SQ_INSTS_VMEM_RD", "SQ_INSTS_LDS"):
                if n in c:
                    der[n.lower().replace("sq_insts_", "") + "_per_step"] = c[n] / u
            if "SQ_VALU_MFMA_BUSY_CYCLES" in c:
                der["mfma_busy_cycles_per_step"] = c["SQ_VALU_MFMA_BUSY_CYCLES"] / u
        kernels[k] = {"dispatches": len(e["durations_ns"]), "avg_duration_us": dur / 1e3,
                      "counters_per_dispatch": c, "derived": der}
    out = {
        "workload": workload,
        "kernel_source_hash": kernel_source_hash(),
        "commands": [COMPUTE_CMD.format(c=f'"{v}"', p=p, w=workload,
                                        args=compute_bench_args(workload))
                     for p, v in COMPUTE_PASSES.items()],
        "device": {"cus": cus, "simds": simds, "xcc": xcc,
                   "max_engine_clock_mhz": int(agent["Max_Engine_Clk_Fcompute"])},
        "notes": ["Counters are summed over all XCCs, shader engines and SIMDs by rocprofv3;",
                  "GRBM_GUI_ACTIVE / xcc is the dispatch's length in engine cycles.",
                  "SQ_ACTIVE_INST_VALU, SQ_WAVE_CYCLES, SQ_WAIT_ANY and SQ_WAIT_INST_ANY are",
                  "quad-cycle counts (x4 to cycles); SQ_VALU_MFMA_BUSY_CYCLES is in cycles.",
                  "A step is one (page, KV head) for 16 query columns (a prefix step covers",
                  "one column tile of a group's shared page)."],
        "kernels": kernels,
    }
    os.makedirs(PROFILES, exist_ok=True)
    json.dump(out, open(compute_path(workload), "w"), indent=1)
    print(compute_path(workload))


# Timing events.  HIP events made with hipEventDisableSystemFence skip the
# system-scope fence (an L2 write-back and invalidate) that a default event
# performs when it is recorded: that fence is not part of the timed kernels,
# and the HIP documentation names this flag for timing-only events.
EVENT_FLAGS = 0x20000000  # hipEventDisableSystemFence


class HipEvent:
    hip = None

    def __init__(self, torch, flags):
        if HipEvent.hip is None:
            import ctypes
            h = ctypes.CDLL("libamdhip64.so.7")  # the runtime torch has loaded
            h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                              ctypes.c_void_p]
            h.hipEventDestroy.argtypes = [ctypes.c_void_p]
            HipEvent.hip = h
        import ctypes
        self._ct = ctypes
        self.torch = torch
        self.ev = ctypes.c_void_p()
        if HipEvent.hip.hipEventCreateWithFlags(ctypes.byref(self.ev), flags) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    @property
    def cuda_event(self):
        return self.ev.value

    def record(self):
        stream = self._ct.c_void_p(self.torch.cuda.current_stream().cuda_stream)
        if HipEvent.hip.hipEventRecord(self.ev, stream) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_time(self, end):
        ms = self._ct.c_float()
        if HipEvent.hip.hipEventElapsedTime(self._ct.byref(ms), self.ev, end.ev) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def __del__(self):
        if HipEvent.hip is not None and self.ev:
            HipEvent.hip.hipEventDestroy(self.ev)


def make_events(torch, n):
    evs = [HipEvent(torch, EVENT_FLAGS) for _ in range(n)]
    for e in evs:
        e.record()
    torch.cuda.synchronize()
    return evs


def time_calls(torch, fn, steps, warmup, flush):
    """Per-call GPU time (ms) of fn, the cache evicted before each call.  The
    events are made up front, so nothing in the loop waits for the GPU and the
    flush hides the host's time to enqueue the call."""
    for _ in range(warmup):
        flush()
        fn()
    torch.cuda.synchronize()
    starts, ends = make_events(torch, steps), make_events(torch, steps)
    for i in range(steps):
        flush()
        starts[i].record()
        fn()
        ends[i].record()
    torch.cuda.synchronize()
    return [s.elapsed_time(e) for s, e in zip(starts, ends)]


def time_decode(torch, dora, b, steps, warmup, flush, num_waves=0):
    """Returns dict of per-step and per-kernel timings (ms)."""
    w = b.w
    out = torch.empty_like(b.q)
    kw = dict(num_kv_heads=w.num_kv_heads, page_size=w.page_size, kv_dtype=w.kv_dtype,
              k_scales=b.k_scales, v_scales=b.v_scales, num_waves=num_waves)

    def call(prof=None):
        dora.dora_decode_attn(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                              b.version_ids, out, events=prof, **kw)

    for _ in range(warmup):
        flush()
        call()
    torch.cuda.synchronize()
    # (a) whole steps: events bracket the call only; the flush sits outside them
    starts = make_events(torch, steps)
    ends = make_events(torch, steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        flush()
        starts[i].record()
        call()
        ends[i].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = np.array([s.elapsed_time(e) for s, e in zip(starts, ends)])
    # (b) per kernel: the library records events before the decode kernel,
    # between it and the combine kernel, and after the combine kernel
    ev = make_events(torch, 3)
    handles = [e.cuda_event for e in ev]
    split, comb = [], []
    for i in range(steps):
        flush()
        call(prof=handles)
        torch.cuda.synchronize()
        split.append(ev[0].elapsed_time(ev[1]))
        comb.append(ev[1].elapsed_time(ev[2]))
    return {"step_ms": step_ms, "wall_s": wall, "split_ms": np.array(split),
            "combine_ms": np.array(comb), "out": out}


def decode_record(w, lengths, t):
    ab = wl.algorithmic_bytes(w, lengths)
    st = wl.skew_stats(lengths)
    ms = float(np.mean(t["step_ms"]))
    split_ms = float(np.mean(t["split_ms"]))
    return {
        "ms_per_step": ms,
        "ms_p10_p50_p90": [float(np.percentile(t["step_ms"], q)) for q in (10, 50, 90)],
        "decode_tokens_per_s": w.num_seqs / (ms * 1e-3),
        "context_tokens_per_s": st["sum"] / (ms * 1e-3),
        "hbm_gbps": ab["total"] / (ms * 1e-3) / 1e9,
        "hbm_frac_of_peak": ab["total"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "split_kernel_ms": split_ms,
        "split_kernel_gbps": ab["total"] / (split_ms * 1e-3) / 1e9,
        "combine_ms": float(np.mean(t["combine_ms"])),
        "algorithmic_bytes": ab,
        "lengths": {k: (round(v, 3) if isinstance(v, float) else v) for k, v in st.items()},
    }


def time_grpo(torch, dora, steps, flush):
    """The GRPO-shaped batch (16 responses per prompt sharing the prompt's full
    pages): dora_decode_attn, which reads the shared pages once per member,
    against dora_decode_attn_grouped, which reads them once per group."""
    b, shared = wl.make_grpo_batch(device="cuda")
    w, M = b.w, wl.GRPO_GROUP
    plain = time_decode(torch, dora, b, steps, 2, flush)
    out = torch.empty_like(b.q)
    kw = dict(group_size=M,
              num_kv_heads=w.num_kv_heads, page_size=w.page_size, kv_dtype=w.kv_dtype,
              k_scales=b.k_scales, v_scales=b.v_scales)

    def call():
        dora.dora_decode_attn_grouped(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                                      b.version_ids, out, **kw)

    ts = time_calls(torch, call, steps, 2, flush)
    diff = (out.float() - plain["out"].float()).abs().max().item()
    ab = wl.shared_prefix_algorithmic_bytes(w, b.lengths, shared, M)
    rec = {"config": {"num_seqs": w.num_seqs, "group_size": M,
                      "prompt_tokens": list(wl.GRPO_PROMPT),
                      "heads": [w.num_q_heads, w.num_kv_heads], "head_dim": w.head_dim,
                      "page_size": w.page_size, "kv_dtype": "bf16"},
           "algorithmic_bytes": ab, "max_abs_diff_grouped_vs_plain": diff}
    for name, ms in (("plain", float(np.median(plain["step_ms"]))),
                     ("grouped", float(np.median(ts)))):
        rec[name] = {"ms_per_step": ms,
                     "decode_tokens_per_s": w.num_seqs / (ms * 1e-3),
                     "gbps": ab["total"] / (ms * 1e-3) / 1e9,
                     "frac_of_peak": ab["total"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS}
    rec["speedup"] = rec["plain"]["ms_per_step"] / rec["grouped"]["ms_per_step"]
    del b
    return rec


def time_append(torch, dora, b, steps, flush):
    """KV append of one token per sequence (each sequence rewrites its last
    token, so every page it writes exists), cache evicted before each call."""
    w = b.w
    g = torch.Generator(device="cuda").manual_seed(77)
    kn = torch.randn(w.num_seqs, w.num_kv_heads, w.head_dim, generator=g, device="cuda").to(
        torch.bfloat16)
    vn = torch.randn(w.num_seqs, w.num_kv_heads, w.head_dim, generator=g, device="cuda").to(
        torch.bfloat16)
    kw = dict(num_kv_heads=w.num_kv_heads, page_size=w.page_size, kv_dtype=w.kv_dtype,
              k_scales=b.k_scales, v_scales=b.v_scales)
    ts = time_calls(torch, lambda: dora.dora_kv_append(
        kn, vn, b.block_table, b.seq_lens, b.k_pages, b.v_pages, **kw), steps, 2, flush)
    ab = wl.append_algorithmic_bytes(w, b.lengths)
    ms = float(np.median(ts))
    return {"ms": ms, "algorithmic_bytes": ab, "gbps": ab / (ms * 1e-3) / 1e9}


def time_pack(torch, dora, b, steps, flush):
    """Pack + unpack of the 32-sequence same-version migration set."""
    w = b.w
    rng = np.random.default_rng(5)
    cand = np.nonzero(b.versions_h == 0)[0]
    seqs = np.sort(rng.choice(cand, size=min(w.pack_seqs or 32, len(cand)), replace=False))
    n = wl.pages_needed(b.lengths, w.page_size)
    src = np.concatenate([b.block_table_h[s, :n[s]] for s in seqs]).astype(np.int32)
    npg = len(src)
    free = np.setdiff1d(np.arange(w.num_pages), b.used_pages)[:npg].astype(np.int32)
    src_t = torch.from_numpy(src).cuda()
    dst_t = torch.from_numpy(free).cuda()
    desc = dora.make_pack_desc(kv_dtype=w.kv_dtype, page_size=w.page_size,
                               num_kv_heads=w.num_kv_heads, head_dim=w.head_dim,
                               num_pages=w.num_pages, policy_version=0)
    packed = torch.empty(dora.dora_kv_packed_bytes(desc, npg), dtype=torch.uint8, device="cuda")
    geo = dict(num_kv_heads=w.num_kv_heads, page_size=w.page_size, head_dim=w.head_dim,
               kv_dtype=w.kv_dtype)
    pk = time_calls(torch, lambda: dora.dora_kv_page_pack(
        b.k_pages, b.v_pages, src_t, packed, policy_version=0, n_seqs=len(seqs), **geo),
        steps, 2, flush)
    up = time_calls(torch, lambda: dora.dora_kv_page_unpack(
        packed, dst_t, b.k_pages, b.v_pages, src_version=0, policy_version=0, **geo),
        steps, 2, flush)
    moved = 2 * npg * w.page_bytes          # K and V pages, one way
    rec = {"seqs": int(len(seqs)), "pages": int(npg), "bytes_one_way": int(moved),
           "pack_ms": float(np.mean(pk)), "unpack_ms": float(np.mean(up)),
           "pack_gbps_rw": 2 * moved / (np.mean(pk) * 1e-3) / 1e9,
           "unpack_gbps_rw": 2 * moved / (np.mean(up) * 1e-3) / 1e9}
    rec["offload"] = time_offload(torch, dora, b, src_t, dst_t, packed, geo, len(seqs), moved,
                                  max(3, steps // 2), flush)
    return rec


def time_offload(torch, dora, b, src_t, dst_t, packed, geo, n_seqs, moved, steps, flush):
    """The same set packed straight into pinned host memory and unpacked from
    it (offload and restore), beside plain device<->host copies of the packed
    buffer, which bound what the host link carries."""
    host = torch.empty(packed.numel(), dtype=torch.uint8, pin_memory=True)
    runs = {"pack_to_host": lambda: dora.dora_kv_page_pack(
                b.k_pages, b.v_pages, src_t, host, policy_version=0, n_seqs=n_seqs, **geo),
            "unpack_from_host": lambda: dora.dora_kv_page_unpack(
                host, dst_t, b.k_pages, b.v_pages, src_version=0, policy_version=0, **geo),
            "d2h_copy": lambda: host.copy_(packed, non_blocking=True),
            "h2d_copy": lambda: packed.copy_(host, non_blocking=True)}
    out = {}
    for name, fn in runs.items():
        ts = time_calls(torch, fn, steps, 1, flush)
        ms = float(np.median(ts))
        out[name + "_ms"] = ms
        out[name + "_gbps"] = moved / (ms * 1e-3) / 1e9
    return out


def copy_bandwidth(torch, nbytes=2 << 30):
    """A 2 GiB device-to-device copy (the runtime's copy kernel): the rate is
    context, and its dispatches calibrate the FETCH_SIZE / WRITE_SIZE counters
    (it reads and writes exactly 2 GiB)."""
    a = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1)
    c = torch.empty_like(a)
    for _ in range(3):
        c.copy_(a)
    s, e = make_events(torch, 2)
    s.record()
    for _ in range(10):
        c.copy_(a)
    e.record()
    torch.cuda.synchronize()
    rate = 2 * nbytes / (s.elapsed_time(e) / 10 * 1e-3) / 1e9
    del a, c
    return rate


def stream_read_reference(torch, dora, flush, steps=6, buf_bytes=16 << 30, read_bytes=4 << 30,
                          tile=4096):
    """Achievable read bandwidth with the decode kernel's access pattern: the
    library's streaming-read kernel (dora_stream_read) over 4 GiB of 4 KiB
    tiles of a 16 GiB buffer (long enough that launch and ramp-down cost under
    1%), in random or in sequential order, swept over the wavefronts per CU
    (5, as the decode launches for bf16 pages; 8, every resident slot, as for
    fp8 pages; 12 and 16) and the tiles each wavefront keeps per batch (1, 2
    or 4, two batches in flight).  Median of `steps` calls per variant, caches
    evicted before each; achievable_gbps is the best random variant."""
    props = torch.cuda.get_device_properties(0)
    cus = props.multi_processor_count
    buf = torch.empty(buf_bytes, dtype=torch.uint8, device="cuda")
    n_all = buf_bytes // tile
    n = read_bytes // tile
    rng = np.random.default_rng(4096)
    orders = {"random": rng.permutation(n_all)[:n].astype(np.int32),
              "sequential": np.arange(n, dtype=np.int32)}
    out = {"tile_bytes": tile, "read_bytes": n * tile, "buffer_bytes": buf_bytes,
           "gbps": {}}
    for name, ids in orders.items():
        tiles = torch.from_numpy(ids).cuda()
        for per_cu in (5, 8, 12, 16):
            sink = torch.zeros(cus * per_cu, dtype=torch.int32, device="cuda")
            for tpb in (1, 2, 4):
                ts = time_calls(torch, lambda: dora.dora_stream_read(
                    buf, tiles, sink, tile_bytes=tile, tiles_per_batch=tpb), steps, 2, flush)
                ms = float(np.median(ts))
                out["gbps"][f"{name}_{per_cu}_per_cu_{tpb}_tiles"] = n * tile / (ms * 1e-3) / 1e9
        del tiles
    best = max((v, k) for k, v in out["gbps"].items() if k.startswith("random_"))
    out["achievable_gbps"], out["achievable_variant"] = best
    del buf
    torch.cuda.empty_cache()
    return out


def pattern_tiles(w, lengths, block_table_h):
    """The K and V tiles a decode of this batch reads, in the order of its work
    list ((sequence, KV head, page) page-heads, each one's K tile then its V
    tile), as tile indices into one buffer laid out [K pool][V pool] with the
    pools' own layout: tile (page, head) at page * Hkv + head."""
    H = w.num_kv_heads
    n = wl.pages_needed(lengths, w.page_size)
    parts = []
    for b, nb in enumerate(n):
        pids = block_table_h[b, :nb].astype(np.int64)
        for g in range(H):
            k = pids * H + g
            parts.append(np.stack([k, k + w.num_pages * H], 1).reshape(-1))
    ids = np.concatenate(parts) if parts else np.zeros(0, np.int64)
    return ids.astype(np.int32)


def pattern_reference(torch, dora, w, lengths, block_table_h, decode_waves, flush, steps=6):
    """Achievable read rate for this batch's exact access pattern: the
    streaming-read kernel over the tiles the decode reads, in its order,
    split in equal contiguous ranges over the decode's own wavefront count
    and over 8 per CU, with 2 or 4 tiles per batch.  The buffer holds a K pool
    and a V pool of the batch's geometry (contents irrelevant)."""
    tile = w.page_size * w.head_dim * (1 if w.kv_dtype == 1 else 2)
    ids = pattern_tiles(w, lengths, block_table_h)
    buf = torch.empty(2 * w.num_pages * w.num_kv_heads * tile, dtype=torch.uint8, device="cuda")
    tiles = torch.from_numpy(ids).cuda()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    out = {"tile_bytes": tile, "tiles": int(len(ids)), "gbps": {}}
    for waves in sorted({int(decode_waves), 8 * cus}):
        sink = torch.zeros(waves, dtype=torch.int32, device="cuda")
        for tpb in (2, 4):
            ts = time_calls(torch, lambda: dora.dora_stream_read(
                buf, tiles, sink, tile_bytes=tile, tiles_per_batch=tpb), steps, 2, flush)
            ms = float(np.median(ts))
            out["gbps"][f"{waves}_waves_{tpb}_tiles"] = len(ids) * tile / (ms * 1e-3) / 1e9
    best = max((v, k) for k, v in out["gbps"].items())
    out["best_gbps"], out["best_variant"] = best
    del buf, tiles
    torch.cuda.empty_cache()
    return out


def cpu_baseline(b, budget_s=20.0, min_s=10.0, threads=None):
    """The fp64 oracle on the host cores over the same batch (or a prefix of
    its sequences that fits the time budget), repeated until min_s of work is
    timed, scaled to decode tokens/s.  Threads: `threads` when given, else
    OMP_NUM_THREADS when set (the host's CPU share for this GPU), else every
    core in the affinity mask."""
    import oracle

    mask = len(os.sched_getaffinity(0))
    env = os.environ.get("OMP_NUM_THREADS", "")
    if threads:
        cores = threads
    else:
        cores = min(mask, int(env)) if env.isdigit() and int(env) > 0 else mask
    order = list(range(b.w.num_seqs))
    # calibrate on one sequence, then take as many sequences as the budget allows
    probe = wl.subset_for_oracle(b, order[:1])
    t0 = time.perf_counter()
    oracle.decode(probe["q"], probe["k_pages"], probe["v_pages"], probe["block_table"],
                  probe["seq_lens"], num_kv_heads=b.w.num_kv_heads, page_size=b.w.page_size,
                  kv_dtype=b.w.kv_dtype, k_scales=probe["k_scales"],
                  v_scales=probe["v_scales"], num_pages=probe["num_pages"], nthreads=cores)
    # the probe is one sequence, so at most Hkv of the threads had work: its
    # wall time times that count is its CPU time
    busy = min(cores, b.w.num_kv_heads)
    per_tok = (time.perf_counter() - t0) * busy / max(1, int(b.lengths[0]))
    take, acc = [], 0.0
    for s in order:
        take.append(s)
        acc += per_tok * int(b.lengths[s]) / cores
        if acc >= budget_s:
            break
    sub = wl.subset_for_oracle(b, take)
    # repeat the sample until at least min_s of CPU time is measured
    reps, total = 0, 0.0
    while reps == 0 or total < min_s:
        t0 = time.perf_counter()
        oracle.decode(sub["q"], sub["k_pages"], sub["v_pages"], sub["block_table"],
                      sub["seq_lens"], num_kv_heads=b.w.num_kv_heads, page_size=b.w.page_size,
                      kv_dtype=b.w.kv_dtype, k_scales=sub["k_scales"], v_scales=sub["v_scales"],
                      num_pages=sub["num_pages"], nthreads=cores)
        total += time.perf_counter() - t0
        reps += 1
    dt = total / reps
    ctx = int(b.lengths[take].sum())
    # one decode step of the whole batch costs sum(L) context tokens of work
    step_s = dt * float(b.lengths.sum()) / ctx
    # threads that ran: the oracle's parallel loop is over (sequence, KV head)
    # units, with at most the requested (and OpenMP-available) threads
    used = min(cores, oracle.max_threads(), len(take) * b.w.num_kv_heads)
    return {"value": b.w.num_seqs / step_s, "unit": "tokens/s", "cores": used,
            "threads_requested": cores, "kind": "oracle",
            "sample": f"{len(take)} of {b.w.num_seqs} sequences ({ctx} context tokens), "
                      f"run {reps} times ({total:.1f} s, {dt:.3f} s each), scaled by "
                      f"total/sampled context tokens",
            "affinity_mask_cores": mask,
            "threads_source": ("fixed" if threads else
                               "OMP_NUM_THREADS" if cores != mask or env else "affinity mask"),
            "cpu_model": _cpu_model()}


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def load_pmc(w):
    """The committed rocprofv3 counter summary of this workload's decode
    kernel, or None if absent or taken on a different kernel source."""
    try:
        with open(pmc_path(w.name)) as f:
            pmc = json.load(f)
    except (OSError, ValueError):
        return None
    if pmc.get("kernel_source_hash") != kernel_source_hash() or pmc.get("workload") != w.name:
        return None
    return pmc


def roofline_of(rec, achievable_gbps):
    """Roofline object of one workload's decode kernel: algorithmic bytes per
    launch over the kernel's average duration by events; traffic from the
    committed counter summary when it matches the kernel sources; the
    fraction of the generic streaming-read reference and of the reference on
    this batch's own access pattern."""
    ab = rec["algorithmic_bytes"]["total"]
    ms = rec["split_kernel_ms"]
    gbps = ab / (ms * 1e-3) / 1e9
    pat = rec.get("pattern_reference")
    return {
        "bound": "hbm",
        "kernel": "decode_kernel",
        "achieved": gbps,
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": gbps / HBM_PEAK_GBPS,
        "traffic": rec["split_kernel_traffic_bytes"],
        "l2_hit_rate": rec["split_kernel_l2_hit_rate"],
        "algorithmic_bytes_per_launch": ab,
        "avg_launch_ms": ms,
        "achievable_gbps": achievable_gbps,
        "frac_of_achievable": gbps / achievable_gbps,
        "pattern_gbps": pat["best_gbps"] if pat else None,
        "frac_of_pattern": gbps / pat["best_gbps"] if pat else None,
    }


def main():
    global EVENT_FLAGS
    args = parse()
    EVENT_FLAGS = args.event_flags
    if args.summarize_compute:
        summarize_compute(args.summarize_compute[1:], args.summarize_compute[0])
        return
    if args.summarize_bench_trace:
        summarize_bench_trace(*args.summarize_bench_trace)
        return
    if args.summarize_trace or args.summarize_pmc or args.summarize_grpo_trace:
        if args.summarize_grpo_trace:
            summarize_trace(args.summarize_grpo_trace, None, grpo=True)
        if args.summarize_trace:
            summarize_trace(args.summarize_trace, args.workload)
        if args.summarize_pmc:
            summarize_pmc(*args.summarize_pmc, args.workload)
        return
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(one GPU's share is measured; the decode path would shard by sequence with "
              "no exchange between GPUs)",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2604_26256_amd import dora

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    flush_buf = None if args.no_flush else torch.ones(1 << 28, dtype=torch.float32,
                                                     device="cuda")
    flush_out = torch.empty((), dtype=torch.float32, device="cuda")
    if flush_buf is None:
        flush = lambda: None  # noqa: E731
    elif args.flush_mode == "read":
        # a 1 GiB read leaves only clean lines behind, so no write-back lands
        # inside the next timed step
        flush = lambda: torch.sum(flush_buf, dim=0, out=flush_out)  # noqa: E731
    else:
        flush = lambda: flush_buf.fill_(1.0)  # noqa: E731

    if args.grpo_only:
        print(json.dumps(time_grpo(torch, dora, args.steps, flush), indent=1))
        return
    names = [args.workload] + ([] if args.only_main else
                               [w.name for w in wl.WORKLOADS if w.name != args.workload])
    results, main_rec, main_w = {}, None, None
    cpu = None
    for name in names:
        w = wl.BY_NAME[name]
        idx = wl.WORKLOADS.index(w)
        log(f"workload {name}: generating")
        b = wl.make_batch(w, device="cuda", seed_index=idx)
        torch.cuda.synchronize()
        steps = args.steps if name == args.workload else max(5, args.steps // 3)
        log(f"workload {name}: timing {steps} steps")
        t = time_decode(torch, dora, b, steps, args.warmup if name == args.workload else 2,
                        flush, args.num_waves)
        rec = decode_record(w, b.lengths, t)
        rec["kv_dtype"] = "bf16" if w.kv_dtype == 0 else "fp8_e4m3"
        pmc = load_pmc(w)
        rec["split_kernel_traffic_bytes"] = pmc["traffic_bytes_per_launch"] if pmc else None
        rec["split_kernel_l2_hit_rate"] = pmc["l2"]["decode_kernel"]["hit_rate"] if pmc else None
        rec["append"] = time_append(torch, dora, b, max(5, steps // 2), flush)
        if name in SINGLE_CORE_WORKLOADS and not args.no_cpu_baseline:
            log(f"workload {name}: single-core oracle")
            rec["cpu_baseline_1core"] = cpu_baseline(b, budget_s=6.0, min_s=3.0, threads=1)
        if w.pack_seqs:
            log(f"workload {name}: pack/unpack")
            rec["pack_unpack"] = time_pack(torch, dora, b, max(5, steps // 2), flush)
        results[name] = rec
        log(f"workload {name}: {rec['ms_per_step']:.4f} ms/step, "
            f"{rec['hbm_gbps']:.0f} GB/s, split kernel {rec['split_kernel_gbps']:.0f} GB/s")
        lengths, table_h = b.lengths, b.block_table_h
        waves = dora.dora_decode_num_waves(dora.make_decode_desc(
            num_seqs=w.num_seqs, num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads,
            head_dim=w.head_dim, page_size=w.page_size, block_table_stride=b.stride,
            num_pages=w.num_pages, kv_dtype=w.kv_dtype, num_waves=args.num_waves))
        if name == args.workload:
            main_rec, main_w = rec, w
            main_rec["steps_wall_s"] = t["wall_s"]
            if not args.no_cpu_baseline:
                log("cpu baseline (oracle)")
                cpu = cpu_baseline(b)
        del b, t
        torch.cuda.empty_cache()
        if name != "tiny":
            log(f"workload {name}: reference read of its access pattern")
            rec["pattern_reference"] = pattern_reference(torch, dora, w, lengths, table_h,
                                                         waves, flush)

    grpo = None
    if not args.only_main:
        log("workload grpo7b (responses sharing prompt pages): timing")
        grpo = time_grpo(torch, dora, max(5, args.steps // 3), flush)
        log(f"workload grpo7b: {grpo['plain']['ms_per_step']:.4f} ms/step plain, "
            f"{grpo['grouped']['ms_per_step']:.4f} grouped ({grpo['speedup']:.2f}x)")
        torch.cuda.empty_cache()
    log("streaming-read reference")
    reference = stream_read_reference(torch, dora, flush)
    for rec in results.values():
        rec["roofline"] = roofline_of(rec, reference["achievable_gbps"])
    copy_gbps = copy_bandwidth(torch)
    w = main_w
    line = {
        "metric": METRIC,
        "value": main_rec["decode_tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_rec["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # the arithmetic: bf16 MFMA operands, fp32 accumulation and softmax
        # (fp8 pages are widened to bf16 in registers, exactly)
        "dtype": "bf16" if w.kv_dtype == 0 else "bf16 (KV stored fp8_e4m3)",
        "data": "synthetic",
        "config": {
            "workload": w.name, "num_seqs": w.num_seqs, "num_q_heads": w.num_q_heads,
            "num_kv_heads": w.num_kv_heads, "head_dim": w.head_dim, "page_size": w.page_size,
            "kv_dtype": main_rec["kv_dtype"], "pool_pages": w.num_pages,
            "lengths": f"{w.length_law}(median {w.median}, sigma {w.sigma}) clipped "
                       f"[{w.lo}, {w.hi}]" if w.length_law == "lognormal"
                       else f"uniform [{w.lo}, {w.hi}]",
            "parallelism": "single GPU",
        },
        "hbm_gbps": main_rec["hbm_gbps"],
        "hbm_frac_of_peak": main_rec["hbm_frac_of_peak"],
        "context_tokens_per_s": main_rec["context_tokens_per_s"],
        "roofline": main_rec["roofline"],
        "stream_read_reference": reference,
        "copy_gbps_measured": copy_gbps,
        "cpu_baseline": cpu,
        "flush_between_steps": None if args.no_flush else args.flush_mode,
        "timing_event_flags": hex(EVENT_FLAGS),
        "workloads": results,
        "shared_prefix": grpo,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
