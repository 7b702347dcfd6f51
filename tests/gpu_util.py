"""Shared helpers of the GPU parity tests: run the library through its C ABI
binding and the fp64 oracle on the same seeded inputs, then compare."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import workloads as wl

TOL = {0: 2e-2, 1: 5e-2}   # max-abs error bound on bf16 outputs: bf16 KV, fp8 KV


def lib():
    from paper_2604_26256_amd import dora
    return dora


def gpu_batch(w: wl.Workload, lengths=None, seed_index=0, poison=True):
    """Inputs generated on the GPU (torch's device generator)."""
    return wl.make_batch(w, device="cuda", seed_index=seed_index, lengths=lengths,
                         poison=poison)


def run_decode(b: wl.Batch, out=None, **kw):
    d = lib()
    if out is None:
        out = torch.empty_like(b.q)
    d.dora_decode_attn(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.version_ids, out,
                       num_kv_heads=b.w.num_kv_heads, page_size=b.w.page_size,
                       kv_dtype=b.w.kv_dtype, k_scales=b.k_scales, v_scales=b.v_scales, **kw)
    torch.cuda.synchronize()
    return out


def oracle_for(b: wl.Batch, seqs=None, nthreads=0):
    """fp64 oracle output [len(seqs)][Hq][d] on host copies of the inputs."""
    if seqs is None:
        seqs = list(range(b.w.num_seqs))
    s = wl.subset_for_oracle(b, seqs)
    return oracle.decode(s["q"], s["k_pages"], s["v_pages"], s["block_table"], s["seq_lens"],
                         num_kv_heads=b.w.num_kv_heads, page_size=b.w.page_size,
                         kv_dtype=b.w.kv_dtype, k_scales=s["k_scales"], v_scales=s["v_scales"],
                         version_ids=s["versions"], page_owner=s["page_owner"],
                         num_pages=s["num_pages"], nthreads=nthreads)


def max_abs_err(out: torch.Tensor, ref: np.ndarray, seqs=None) -> float:
    o = out.float().cpu().double().numpy()
    if seqs is not None:
        o = o[list(seqs)]
    assert np.isfinite(o).all(), "non-finite output"
    return float(np.abs(o - ref).max()) if ref.size else 0.0


def sample_seqs(lengths: np.ndarray, k: int, seed: int):
    """The longest, the shortest, the median and k random other sequences."""
    order = np.argsort(lengths, kind="stable")
    pick = {int(order[-1]), int(order[0]), int(order[len(order) // 2])}
    rng = np.random.default_rng(seed)
    rest = [i for i in range(len(lengths)) if i not in pick]
    if rest:
        pick.update(int(x) for x in rng.choice(rest, size=min(k, len(rest)), replace=False))
    return sorted(pick)
