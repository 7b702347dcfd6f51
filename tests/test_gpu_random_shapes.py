"""Seeded random geometries against the fp64 oracle: head dim, page size, KV
dtype, KV heads, group size, batch size, length mix (short, lognormal,
page-boundary values, long) and wavefront count all drawn per case, so that
combinations the hand-picked cases miss are covered.  Each case's decode is
compared with the oracle (max-abs 2e-2 bf16, 5e-2 fp8); where the batch
forms groups of two, the grouped call is compared with the plain one.  A
second sweep also draws the softmax scale and the minimum range, and runs
each case through a prepared call as well (bitwise equal to the plain one);
a third draws GRPO batches whose groups share prompt pages and compares the
grouped call with the oracle."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from gpu_util import TOL, gpu_batch, lib, max_abs_err, oracle_for, run_decode

pytestmark = pytest.mark.gpu

CASES = 120


def _case(rng):
    d = int(rng.choice([64, 128]))
    P = int(rng.choice([16, 32]))
    dt = int(rng.integers(0, 2))
    Hkv = int(rng.integers(1, 9))
    G = int(rng.integers(1, 17))
    B = int(rng.integers(1, 41))
    kind = int(rng.integers(0, 4))
    if kind == 0:
        lens = rng.integers(0, 300, B)
    elif kind == 1:
        lens = np.clip(np.rint(np.exp(rng.normal(np.log(400), 1.3, B))), 0, 9000)
    elif kind == 2:
        lens = rng.choice([0, 1, P - 1, P, P + 1, 2 * P, 3 * P + 1, 1000], B)
    else:
        lens = rng.integers(2000, 6000, B)
    waves = int(rng.choice([0, 0, 1, 3, 17, 100, 700]))
    return d, P, dt, Hkv, G, B, lens.astype(np.int32), waves


def test_random_geometries_match_the_oracle():
    rng = np.random.default_rng(20260426)
    d_ = lib()
    for case in range(CASES):
        d, P, dt, Hkv, G, B, lens, waves = _case(rng)
        print(f"[case {case}] d={d} P={P} dt={dt} Hkv={Hkv} G={G} B={B} waves={waves} "
              f"max len={lens.max()}", flush=True)
        pages = max(64, int(wl.pages_needed(lens, P).sum()) * 2 + 8)
        w = wl.Workload("r", B, G * Hkv, Hkv, d, P, dt, pages, "uniform", lo=1, hi=1)
        b = gpu_batch(w, lengths=lens, seed_index=2000 + case)
        out = run_decode(b, num_waves=waves)
        err = max_abs_err(out, oracle_for(b))
        assert err <= TOL[dt], (case, err)
        if B % 2 == 0 and 2 * G <= 128:
            og = torch.empty_like(b.q)
            d_.dora_decode_attn_grouped(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                                        b.version_ids, og, group_size=2, num_kv_heads=Hkv,
                                        page_size=P, kv_dtype=dt, k_scales=b.k_scales,
                                        v_scales=b.v_scales)
            torch.cuda.synchronize()
            assert (og.float() - out.float()).abs().max().item() <= TOL[dt], case


def test_random_scales_ranges_and_prepared_calls():
    rng = np.random.default_rng(20261202)
    d_ = lib()
    for case in range(100):
        d = int(rng.choice([64, 128]))
        P = int(rng.choice([16, 32]))
        dt = int(rng.integers(0, 2))
        Hkv, G, B = int(rng.integers(1, 9)), int(rng.integers(1, 17)), int(rng.integers(1, 49))
        lens = np.clip(np.rint(np.exp(rng.normal(np.log(500), 1.4, B))), 0, 12000)
        lens = lens.astype(np.int32)
        if rng.random() < 0.3:
            lens[rng.integers(0, B)] = 0
        scale = float(rng.choice([0.0, 0.05, 0.3, 1.0]))
        waves = int(rng.choice([0, 0, 5, 50, 333, 2500]))
        min_range = int(rng.choice([0, 1, 2, 31]))
        print(f"[case {case}] d={d} P={P} dt={dt} Hkv={Hkv} G={G} B={B} scale={scale} "
              f"waves={waves} min_range={min_range} max len={lens.max()}", flush=True)
        pages = max(64, int(wl.pages_needed(lens, P).sum()) * 2 + 8)
        w = wl.Workload("r", B, G * Hkv, Hkv, d, P, dt, pages, "uniform", lo=1, hi=1)
        b = gpu_batch(w, lengths=lens, seed_index=4000 + case)
        kw = dict(num_waves=waves, min_range_pages=min_range, sm_scale=scale)
        out = run_decode(b, **kw)
        s = wl.subset_for_oracle(b, list(range(B)))
        ref = oracle.decode(s["q"], s["k_pages"], s["v_pages"], s["block_table"],
                            s["seq_lens"], num_kv_heads=Hkv, page_size=P, kv_dtype=dt,
                            scale=scale, k_scales=s["k_scales"], v_scales=s["v_scales"],
                            version_ids=s["versions"], page_owner=s["page_owner"],
                            num_pages=s["num_pages"])
        err = max_abs_err(out, ref)
        assert err <= TOL[dt], (case, err)
        prep = d_.PreparedDecode(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                                 b.version_ids, torch.empty_like(b.q), num_kv_heads=Hkv,
                                 page_size=P, kv_dtype=dt, k_scales=b.k_scales,
                                 v_scales=b.v_scales, **kw)
        again = prep()
        torch.cuda.synchronize()
        assert torch.equal(again, out), case


def test_random_grpo_batches_grouped_match_the_oracle():
    rng = np.random.default_rng(20261203)
    d_ = lib()
    for case in range(40):
        d = int(rng.choice([64, 128]))
        P = int(rng.choice([16, 32]))
        dt = int(rng.integers(0, 2))
        Hkv, G = int(rng.integers(1, 9)), int(rng.integers(1, 17))
        M = int(rng.choice([m for m in (2, 3, 4, 8, 16) if m * G <= 128]))
        B = M * int(rng.integers(1, 5))
        lo = int(rng.integers(1, 400))
        hi = lo + int(rng.integers(1, 1500))
        print(f"[case {case}] grpo d={d} P={P} dt={dt} Hkv={Hkv} G={G} M={M} B={B} "
              f"prompts [{lo}, {hi}]", flush=True)
        w = wl.Workload("g", B, G * Hkv, Hkv, d, P, dt, B * ((hi + 2000) // P + 2) + 64,
                        "lognormal", 300, 1.0, 1, 2000)
        b, _ = wl.make_grpo_batch(w, group_size=M, prompt_range=(lo, hi), device="cuda",
                                  seed_index=5000 + case)
        og = torch.empty_like(b.q)
        d_.dora_decode_attn_grouped(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                                    b.version_ids, og, group_size=M, num_kv_heads=Hkv,
                                    page_size=P, kv_dtype=dt, k_scales=b.k_scales,
                                    v_scales=b.v_scales)
        torch.cuda.synchronize()
        err = max_abs_err(og, oracle_for(b))
        assert err <= TOL[dt], (case, err)
