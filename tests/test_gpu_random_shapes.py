"""Seeded random geometries against the fp64 oracle: head dim, page size, KV
dtype, KV heads, group size, batch size, length mix (short, lognormal,
page-boundary values, long) and wavefront count all drawn per case, so that
combinations the hand-picked cases miss are covered.  Each case's decode is
compared with the oracle (max-abs 2e-2 bf16, 5e-2 fp8); where the batch
forms groups of two, the grouped call is compared with the plain one."""
import numpy as np
import pytest
import torch

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
