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


def decode_waves(b: wl.Batch, **kw) -> int:
    """Wavefronts the library launches for b's decode (dora_decode_num_waves)."""
    d = lib()
    desc = d.make_decode_desc(num_seqs=b.w.num_seqs, num_q_heads=b.w.num_q_heads,
                              num_kv_heads=b.w.num_kv_heads, head_dim=b.w.head_dim,
                              page_size=b.w.page_size, block_table_stride=b.stride,
                              num_pages=b.w.num_pages, kv_dtype=b.w.kv_dtype, **kw)
    return d.dora_decode_num_waves(desc)


def cut_segments(lengths, page_size, stride, num_kv_heads, waves, min_range=8):
    """The (sequence, KV head) segments a launch cuts across wavefronts, from
    the work split the header documents: T = Hkv x (pages of the batch)
    page-heads in (sequence, head, page) order, W = min(waves, ceil(T /
    min_range)) equal ranges, the first T mod W one longer.  Returns a sorted
    list of (b, g)."""
    n = np.minimum(wl.pages_needed(lengths, page_size), stride).astype(np.int64)
    Hkv = int(num_kv_heads)
    T = Hkv * int(n.sum())
    if T == 0:
        return []
    W = min(int(waves), -(-T // min_range))
    q, rem = divmod(T, W)
    bounds = np.array([w * q + min(w, rem) for w in range(1, W)], np.int64)
    # segment starts in flattened order
    seq_start = Hkv * np.concatenate([[0], np.cumsum(n)[:-1]])
    starts = (seq_start[:, None] + np.arange(Hkv)[None, :] * n[:, None]).reshape(-1)
    lens = np.repeat(n, Hkv)
    keep = lens > 0
    starts, lens = starts[keep], lens[keep]
    ids = np.nonzero(keep)[0]
    k = np.searchsorted(starts, bounds, side="right") - 1
    inside = (k >= 0) & (bounds > starts[np.maximum(k, 0)]) & \
        (bounds < starts[np.maximum(k, 0)] + lens[np.maximum(k, 0)])
    segs = sorted({(int(ids[i] // Hkv), int(ids[i] % Hkv)) for i in k[inside]})
    return segs


def page_chunks(lengths, page_size, max_pages):
    """Consecutive runs of sequence indices holding at most max_pages pages
    each (one sequence per run at least), to bound host copies."""
    n = wl.pages_needed(lengths, page_size)
    runs, cur, acc = [], [], 0
    for i, nb in enumerate(n):
        if cur and acc + nb > max_pages:
            runs.append(cur)
            cur, acc = [], 0
        cur.append(i)
        acc += int(nb)
    if cur:
        runs.append(cur)
    return runs
