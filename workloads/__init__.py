"""Seeded synthetic inputs for the decode-attention hot path.

This module serves both the GPU library's tests/benchmark and the oracle's: it
draws lengths, page placements, version tags and values, and lays values out in
the documented page formats.  It holds none of the attention arithmetic.

Workloads stand in for the paper's rollout batches (DAPO-Math-17k responses and
production traces, whose length histograms are only plotted): lengths are
lognormal with the stated medians and spreads, clipped, so that p99 exceeds ten
times the median as the paper reports for reasoning workloads (Sec. 1 and
Sec. 2.2, "Workload skewness"); the tail-only phase holds only a few very long
survivors; the multi-version batch tags sequences with three coexisting policy
versions sharing one pool (Sec. 3.2).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np

BASE_SEED = 26042625
FP8_MAX = 448.0  # largest finite OCP E4M3FN value


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    num_seqs: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    kv_dtype: int            # 0 bf16, 1 fp8 e4m3 with one fp32 scale per page
    num_pages: int           # pool capacity
    length_law: str          # "lognormal" or "uniform"
    median: float = 0.0
    sigma: float = 0.0
    lo: int = 1
    hi: int = 1
    version_probs: tuple = (1.0,)
    pack_seqs: int = 0       # sequences moved by the pack/unpack measurement
    min_p99_over_median: float = 0.0  # skew the drawn lengths must exceed (0: none)

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def elem_bytes(self) -> int:
        return 2 if self.kv_dtype == 0 else 1

    @property
    def page_bytes(self) -> int:
        """Bytes of one K page (all KV heads); a V page has the same size."""
        return self.num_kv_heads * self.page_size * self.head_dim * self.elem_bytes

    def scaled(self, num_seqs: int, num_pages: Optional[int] = None) -> "Workload":
        return dataclasses.replace(self, num_seqs=num_seqs,
                                   num_pages=num_pages if num_pages else self.num_pages)


# The five workloads.  Pool sizes where the workload leaves them open: the
# smallest power of two >= 1.25x the worst page demand; the multi-version pool
# is the stated 2^20 pages with page size 16 like the other bf16 workloads.
# The long-tailed workloads must show the skew the paper reports (p99 above
# ten times the median): their lengths are redrawn until they do.
WORKLOADS = [
    Workload("tiny", 8, 8, 2, 64, 16, 0, 1024, "lognormal", 256, 1.0, 1, 2048),
    Workload("rollout7b", 64, 28, 4, 128, 16, 0, 32768, "lognormal", 2048, 1.2, 64, 32768,
             min_p99_over_median=10.0),
    Workload("tail_only", 4, 32, 8, 128, 16, 0, 32768, "uniform", lo=32768, hi=98304),
    Workload("multi_version", 512, 64, 8, 128, 16, 0, 1 << 20, "lognormal", 1024, 1.3, 16,
             65536, version_probs=(0.5, 0.3, 0.2), pack_seqs=32, min_p99_over_median=10.0),
    Workload("moe_fp8", 1024, 64, 8, 128, 32, 1, 1 << 19, "lognormal", 4096, 1.2, 128, 131072,
             min_p99_over_median=10.0),
]
BY_NAME = {w.name: w for w in WORKLOADS}


def seeds(index: int, n: int = 8) -> list:
    """Independent integer seeds for one workload's sub-streams."""
    ss = np.random.SeedSequence(BASE_SEED + index)
    return [int(c.generate_state(1, np.uint64)[0] & 0x7FFFFFFFFFFFFFFF) for c in ss.spawn(n)]


def p99_over_median(lengths) -> float:
    a = np.asarray(lengths, dtype=np.float64)
    med = float(np.median(a))
    return float(np.percentile(a, 99) / med) if med > 0 else 0.0


def sample_lengths(w: Workload, seed: int, max_draws: int = 1000) -> np.ndarray:
    """Lengths of w's batch.  Lognormal: clip(rint(exp(N(ln median, sigma))),
    lo, hi).  If w states a minimum p99/median, whole batches are drawn from the
    same generator until one exceeds it (the first draw that does is kept)."""
    rng = np.random.default_rng(seed)
    if w.length_law == "uniform":
        return rng.integers(w.lo, w.hi + 1, size=w.num_seqs).astype(np.int32)
    for _ in range(max_draws):
        x = np.exp(rng.normal(math.log(w.median), w.sigma, size=w.num_seqs))
        lengths = np.clip(np.rint(x), w.lo, w.hi).astype(np.int32)
        if p99_over_median(lengths) > w.min_p99_over_median:
            return lengths
    raise ValueError(f"{w.name}: no draw in {max_draws} reaches p99/median > "
                     f"{w.min_p99_over_median}")


def sample_versions(w: Workload, seed: int) -> np.ndarray:
    """Exact per-version counts (rounded shares, remainder to version 0), shuffled."""
    probs = np.asarray(w.version_probs, dtype=np.float64)
    counts = np.floor(probs * w.num_seqs + 0.5).astype(np.int64)
    counts[0] += w.num_seqs - counts.sum()
    v = np.repeat(np.arange(len(counts), dtype=np.int32), counts)
    np.random.default_rng(seed).shuffle(v)
    return v


def bubble(lengths: Sequence[int]) -> float:
    """Inter-node bubble of a batch: (max L - mean L) / max L (App. C.3)."""
    a = np.asarray(lengths, dtype=np.float64)
    if a.size == 0 or a.max() <= 0:
        return 0.0
    return float((a.max() - a.mean()) / a.max())


def skew_stats(lengths: Sequence[int]) -> dict:
    a = np.asarray(lengths, dtype=np.float64)
    med = float(np.median(a))
    return {"sum": int(a.sum()), "mean": float(a.mean()), "median": med,
            "p99": float(np.percentile(a, 99)), "max": int(a.max()),
            "p99_over_median": p99_over_median(a), "bubble": bubble(a)}


def pages_needed(lengths: np.ndarray, page_size: int) -> np.ndarray:
    return (np.asarray(lengths, np.int64) + page_size - 1) // page_size


def place_pages(lengths: np.ndarray, page_size: int, num_pages: int, seed: int,
                stride: Optional[int] = None):
    """Give each sequence its pages, in logical order, from one seeded random
    permutation of the whole pool (so consecutive logical pages are scattered).
    Returns (block_table int32 [B][stride], used page ids int64 in table order)."""
    n = pages_needed(lengths, page_size)
    total = int(n.sum())
    if total > num_pages:
        raise ValueError(f"pool of {num_pages} pages cannot hold {total}")
    perm = np.random.default_rng(seed).permutation(num_pages)[:total].astype(np.int64)
    if stride is None:
        stride = max(1, int(n.max()) if n.size else 1)
    bt = np.zeros((len(lengths), stride), dtype=np.int32)
    off = 0
    for b, nb in enumerate(n):
        bt[b, :nb] = perm[off:off + nb]
        off += nb
    return bt, perm


def page_owner_map(block_table: np.ndarray, lengths: np.ndarray, versions: np.ndarray,
                   page_size: int, num_pages: int) -> np.ndarray:
    own = np.full(num_pages, -1, dtype=np.int16)
    n = pages_needed(lengths, page_size)
    for b in range(len(lengths)):
        own[block_table[b, :n[b]]] = versions[b]
    return own


# ---------------------------------------------------------------------------
# Page layouts (documented in the library header):
#   K page [Hkv][d / X][P][X] with X = 16 bytes / element size
#   V page [Hkv][d][P]
# ---------------------------------------------------------------------------

def chunk_elems(kv_dtype: int) -> int:
    return 16 // (2 if kv_dtype == 0 else 1)


def k_tokens_to_pages(k: np.ndarray, page_size: int, kv_dtype: int) -> np.ndarray:
    """Contiguous keys [n*P][Hkv][d] -> n K pages [n][Hkv][d/X][P][X]."""
    T, H, d = k.shape
    X = chunk_elems(kv_dtype)
    n = T // page_size
    assert n * page_size == T and d % X == 0
    return np.ascontiguousarray(
        k.reshape(n, page_size, H, d // X, X).transpose(0, 2, 3, 1, 4))


def v_tokens_to_pages(v: np.ndarray, page_size: int) -> np.ndarray:
    """Contiguous values [n*P][Hkv][d] -> n V pages [n][Hkv][d][P]."""
    T, H, d = v.shape
    n = T // page_size
    assert n * page_size == T
    return np.ascontiguousarray(v.reshape(n, page_size, H, d).transpose(0, 2, 3, 1))


def k_pages_to_tokens(kp: np.ndarray) -> np.ndarray:
    """Inverse of k_tokens_to_pages: [n][Hkv][d/X][P][X] -> [n*P][Hkv][d]."""
    n, H, C, P, X = kp.shape
    return np.ascontiguousarray(kp.transpose(0, 3, 1, 2, 4).reshape(n * P, H, C * X))


def v_pages_to_tokens(vp: np.ndarray) -> np.ndarray:
    n, H, d, P = vp.shape
    return np.ascontiguousarray(vp.transpose(0, 3, 1, 2).reshape(n * P, H, d))


def page_shapes(w: Workload):
    X = chunk_elems(w.kv_dtype)
    kshape = (w.num_kv_heads, w.head_dim // X, w.page_size, X)
    vshape = (w.num_kv_heads, w.head_dim, w.page_size)
    return kshape, vshape


# ---------------------------------------------------------------------------
# Batch generation (torch; runs on the CPU or on the device that will hold it)
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Batch:
    w: Workload
    lengths: np.ndarray          # host int32 [B]
    block_table_h: np.ndarray    # host int32 [B][stride]
    versions_h: np.ndarray       # host int32 [B]
    used_pages: np.ndarray       # host int64, pages in table order
    q: "object"                  # torch bf16 [B][Hq][d]
    k_pages: "object"            # torch bf16 / uint8 [num_pages][...K page]
    v_pages: "object"
    k_scales: "object"           # torch fp32 [num_pages] or None
    v_scales: "object"
    block_table: "object"        # torch int32 on device
    seq_lens: "object"
    version_ids: "object"
    page_owner: "object"         # torch int16 [num_pages]

    @property
    def stride(self) -> int:
        return int(self.block_table_h.shape[1])


def _nan_code(kv_dtype: int) -> int:
    return 0x7FC0 if kv_dtype == 0 else 0x7F


def _fill_pages(torch, pool, pages: np.ndarray, shape, kv_dtype, gen, device, scales,
                chunk: int):
    """Fill pool[pages] with N(0,1) values (bf16 RNE, or fp8 codes with one
    scale per page: scale = max(amax, 2^-126) / 448, codes = RNE(x / scale)
    clamped to +-448)."""
    n = len(pages)
    for s in range(0, n, chunk):
        idx_np = pages[s:s + chunk]
        idx = torch.from_numpy(idx_np).to(device)
        x = torch.randn((len(idx_np),) + tuple(shape), generator=gen, device=device,
                        dtype=torch.float32)
        if kv_dtype == 0:
            pool.index_copy_(0, idx, x.to(torch.bfloat16))
        else:
            amax = x.abs().reshape(len(idx_np), -1).amax(dim=1)
            sc = torch.clamp(amax, min=2.0 ** -126) / FP8_MAX
            y = torch.clamp(x / sc.view(-1, *([1] * len(shape))), -FP8_MAX, FP8_MAX)
            codes = y.to(torch.float8_e4m3fn).view(torch.uint8)
            pool.index_copy_(0, idx, codes)
            scales.index_copy_(0, idx, sc)
        del x


def _poison_tails(torch, k_pages, v_pages, bt: np.ndarray, lengths: np.ndarray, P: int,
                  kv_dtype: int, device):
    """Write NaN codes into the unused slots of every sequence's last page."""
    nan = _nan_code(kv_dtype)
    for b, L in enumerate(lengths):
        r = int(L) % P
        if L == 0 or r == 0:
            continue
        p = int(bt[b, (int(L) - 1) // P])
        if kv_dtype == 0:
            kv = k_pages[p].view(torch.int16)
            vv = v_pages[p].view(torch.int16)
            val = nan - 65536 if nan >= 32768 else nan
        else:
            kv, vv, val = k_pages[p], v_pages[p], nan
        kv[:, :, r:, :] = val
        vv[:, :, r:] = val


def make_batch(w: Workload, device="cpu", seed_index: Optional[int] = None,
               lengths: Optional[np.ndarray] = None, poison: bool = True,
               stride: Optional[int] = None, chunk_pages: int = 8192) -> Batch:
    """Seeded batch of workload `w` on `device`.  Values are drawn with torch's
    generator on that device; lengths, placement and versions with numpy."""
    import torch

    idx = seed_index if seed_index is not None else (
        WORKLOADS.index(BY_NAME[w.name]) if w.name in BY_NAME else 0)
    sd = seeds(idx)
    if lengths is None:
        lengths = sample_lengths(w, sd[0])
    lengths = np.asarray(lengths, dtype=np.int32)
    if w.num_seqs != len(lengths):
        w = w.scaled(len(lengths))
    bt, used = place_pages(lengths, w.page_size, w.num_pages, sd[1], stride)
    versions = (sample_versions(w, sd[2]) if len(w.version_probs) > 1
                else np.zeros(w.num_seqs, np.int32))
    owner = page_owner_map(bt, lengths, versions, w.page_size, w.num_pages)

    kshape, vshape = page_shapes(w)
    kvdt = torch.bfloat16 if w.kv_dtype == 0 else torch.uint8
    k_pages = torch.zeros((w.num_pages,) + kshape, dtype=kvdt, device=device) \
        if w.num_pages * w.page_bytes <= (1 << 28) else \
        torch.empty((w.num_pages,) + kshape, dtype=kvdt, device=device)
    v_pages = torch.zeros((w.num_pages,) + vshape, dtype=kvdt, device=device) \
        if w.num_pages * w.page_bytes <= (1 << 28) else \
        torch.empty((w.num_pages,) + vshape, dtype=kvdt, device=device)
    k_scales = v_scales = None
    if w.kv_dtype == 1:
        k_scales = torch.ones(w.num_pages, dtype=torch.float32, device=device)
        v_scales = torch.ones(w.num_pages, dtype=torch.float32, device=device)

    gq = torch.Generator(device=device).manual_seed(sd[3])
    gk = torch.Generator(device=device).manual_seed(sd[4])
    gv = torch.Generator(device=device).manual_seed(sd[5])
    q = torch.randn((w.num_seqs, w.num_q_heads, w.head_dim), generator=gq, device=device,
                    dtype=torch.float32).to(torch.bfloat16)
    _fill_pages(torch, k_pages, used, kshape, w.kv_dtype, gk, device, k_scales, chunk_pages)
    _fill_pages(torch, v_pages, used, vshape, w.kv_dtype, gv, device, v_scales, chunk_pages)
    if poison:
        _poison_tails(torch, k_pages, v_pages, bt, lengths, w.page_size, w.kv_dtype, device)

    return Batch(
        w=w, lengths=lengths, block_table_h=bt, versions_h=versions, used_pages=used, q=q,
        k_pages=k_pages, v_pages=v_pages, k_scales=k_scales, v_scales=v_scales,
        block_table=torch.from_numpy(bt).to(device),
        seq_lens=torch.from_numpy(lengths).to(device),
        version_ids=torch.from_numpy(versions.astype(np.int32)).to(device),
        page_owner=torch.from_numpy(owner).to(device))


# A GRPO-shaped rollout batch: responses of one prompt share the prompt's full
# pages (16 responses per prompt as in the paper's setup, App. B); response
# lengths follow the 7B-class long-tail law; prompts are 1-4k tokens.
GRPO_WORKLOAD = Workload("grpo7b", 64, 28, 4, 128, 16, 0, 32768, "lognormal", 2048, 1.2, 64,
                         32768)
GRPO_GROUP = 16
GRPO_PROMPT = (1024, 4096)


def grpo_lengths(w: Workload = GRPO_WORKLOAD, group_size: int = GRPO_GROUP,
                 prompt_range=GRPO_PROMPT, seed_index: int = 5):
    """Lengths of a GRPO-shaped batch (prompt plus response per member) and
    each member's shared full prompt pages: (lengths int32 [B], shared int32
    [B])."""
    sd = seeds(seed_index)
    rng = np.random.default_rng(sd[6])
    n_groups = w.num_seqs // group_size
    assert n_groups * group_size == w.num_seqs
    prompt = rng.integers(prompt_range[0], prompt_range[1] + 1, n_groups)
    lengths = (np.repeat(prompt, group_size) + sample_lengths(w, sd[0])).astype(np.int32)
    shared = np.repeat(prompt // w.page_size, group_size).astype(np.int32)
    return lengths, shared


def make_grpo_batch(w: Workload = GRPO_WORKLOAD, group_size: int = GRPO_GROUP,
                    prompt_range=GRPO_PROMPT, device="cpu", seed_index: int = 5,
                    poison: bool = True):
    """Batch whose sequences come in groups of `group_size` responses to one
    prompt: every member's block table starts with the same page ids for the
    prompt's full pages (the partial last prompt page is private, as in a
    copy-on-write pool).  Returns (batch, shared_pages int32 [B])."""
    import torch

    lengths, shared = grpo_lengths(w, group_size, prompt_range, seed_index)
    n_groups = w.num_seqs // group_size
    b = make_batch(w, device=device, seed_index=seed_index, lengths=lengths, poison=poison)
    bt = b.block_table_h.copy()
    for g in range(n_groups):
        lead = g * group_size
        for m in range(lead + 1, lead + group_size):
            bt[m, :shared[m]] = bt[lead, :shared[m]]
    n = pages_needed(lengths, w.page_size)
    b.block_table_h = bt
    b.block_table = torch.from_numpy(bt).to(device)
    b.used_pages = np.unique(np.concatenate([bt[i, :n[i]] for i in range(w.num_seqs)]))
    return b, shared


def shared_prefix_algorithmic_bytes(w: Workload, lengths: np.ndarray, shared: np.ndarray,
                                    group_size: int) -> dict:
    """algorithmic_bytes with each shared page's K and V counted once per group
    (block-table entries are still read per sequence)."""
    ab = algorithmic_bytes(w, lengths)
    shared = np.asarray(shared, np.int64)
    members = np.arange(len(shared)) % group_size != 0          # all but the group leader
    dup = int(shared[members].sum()) * w.page_size * w.num_kv_heads * w.head_dim * 2 * \
        w.elem_bytes
    ab = dict(ab)
    ab["kv"] -= dup
    ab["total"] -= dup
    ab["duplicate_kv_not_counted"] = dup  # members' re-reads of shared pages
    return ab


def subset_for_oracle(batch: Batch, seqs: Sequence[int]) -> dict:
    """Host copies of the inputs of a few sequences, with their pages renumbered
    into a compact pool, for the oracle (which cannot hold the full pool)."""
    import torch

    w = batch.w
    seqs = [int(s) for s in seqs]
    lens = batch.lengths[seqs]
    n = pages_needed(lens, w.page_size)
    stride = max(1, int(n.max()) if len(n) else 1)
    pages = [batch.block_table_h[s, :nb] for s, nb in zip(seqs, n)]
    flat = np.concatenate(pages) if pages else np.zeros(0, np.int64)
    uniq, inv = np.unique(flat, return_inverse=True)
    bt = np.zeros((len(seqs), stride), np.int32)
    off = 0
    for i, nb in enumerate(n):
        bt[i, :nb] = inv[off:off + nb]
        off += nb
    idx = torch.from_numpy(uniq.astype(np.int64)).to(batch.k_pages.device)

    def host(t):
        t = t.index_select(0, idx).cpu()
        return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 \
            else t.numpy()

    out = {
        "q": batch.q[seqs].cpu().view(torch.int16).numpy().view(np.uint16),
        "k_pages": host(batch.k_pages), "v_pages": host(batch.v_pages),
        "block_table": bt, "seq_lens": lens.astype(np.int32),
        "versions": batch.versions_h[seqs].astype(np.int32),
        "num_pages": int(len(uniq)),
        "k_scales": None, "v_scales": None,
    }
    if w.kv_dtype == 1:
        out["k_scales"] = batch.k_scales.index_select(0, idx).cpu().numpy()
        out["v_scales"] = batch.v_scales.index_select(0, idx).cpu().numpy()
    own = np.full(len(uniq), -1, np.int16)
    for i, s in enumerate(seqs):
        own[bt[i, :n[i]]] = batch.versions_h[s]
    out["page_owner"] = own
    return out


def append_algorithmic_bytes(w: Workload, lengths: np.ndarray) -> int:
    """Bytes one KV append must move: the new token's bf16 K and V read, their
    stored form written, its length and block-table entry, and for fp8 the two
    page scales read and written.  Requantisation of a page whose scale grows
    depends on the values and is not counted."""
    active = int((np.asarray(lengths) > 0).sum())
    n = w.num_kv_heads * w.head_dim
    per = 2 * n * 2 + 2 * n * w.elem_bytes + 4 + 4 + (16 if w.kv_dtype == 1 else 0)
    return active * per


def algorithmic_bytes(w: Workload, lengths: np.ndarray) -> dict:
    """Bytes the decode step must move at least once: K and V of valid tokens,
    page scales (fp8), Q, the output, block-table entries and lengths."""
    lengths = np.asarray(lengths, np.int64)
    n = pages_needed(lengths, w.page_size)
    kv = int(lengths.sum()) * w.num_kv_heads * w.head_dim * 2 * w.elem_bytes
    scales = int(n.sum()) * 2 * 4 if w.kv_dtype == 1 else 0
    qo = 2 * w.num_seqs * w.num_q_heads * w.head_dim * 2
    meta = int(n.sum()) * 4 + w.num_seqs * 4
    return {"kv": kv, "scales": scales, "q_out": qo, "meta": meta,
            "total": kv + scales + qo + meta}
