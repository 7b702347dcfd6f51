"""CPU checks of the synthetic inputs and of the tests' own host logic.

* The long-tailed workloads show the skew the paper reports for rollout
  batches (p99 above ten times the median, Sec. 1 and Sec. 2.2): the drawn
  lengths satisfy each workload's stated bound, stay inside its clip range,
  and a first draw that already satisfies it is kept unchanged.
* The set of (sequence, KV head) segments a decode launch cuts across
  wavefronts, which the full-size parity tests use, equals a brute-force
  enumeration of the documented equal-range split.
* The helpers that lay token-major keys and values out as pages follow the
  C header's page layouts element by element.
"""
import math

import numpy as np
import pytest

import workloads as wl
from gpu_util import cut_segments, page_chunks


@pytest.mark.parametrize("idx", range(len(wl.WORKLOADS)))
def test_workload_lengths_meet_the_stated_skew(idx):
    w = wl.WORKLOADS[idx]
    L = wl.sample_lengths(w, wl.seeds(idx)[0])
    assert len(L) == w.num_seqs and L.min() >= w.lo and L.max() <= w.hi
    if w.min_p99_over_median:
        assert wl.p99_over_median(L) > w.min_p99_over_median
        st = wl.skew_stats(L)
        assert st["bubble"] > 0.8      # the batch is dominated by its longest sequence


def test_first_satisfying_draw_is_kept():
    w = wl.BY_NAME["moe_fp8"]
    seed = wl.seeds(wl.WORKLOADS.index(w))[0]
    rng = np.random.default_rng(seed)
    x = np.exp(rng.normal(math.log(w.median), w.sigma, size=w.num_seqs))
    first = np.clip(np.rint(x), w.lo, w.hi).astype(np.int32)
    assert wl.p99_over_median(first) > 10
    assert np.array_equal(wl.sample_lengths(w, seed), first)


def test_redraw_is_deterministic_and_raises_when_impossible():
    w = wl.BY_NAME["rollout7b"]
    seed = wl.seeds(1)[0]
    assert np.array_equal(wl.sample_lengths(w, seed), wl.sample_lengths(w, seed))
    impossible = wl.Workload("x", 64, 8, 2, 64, 16, 0, 1024, "lognormal", 100, 0.1, 1, 200,
                             min_p99_over_median=10.0)
    with pytest.raises(ValueError):
        wl.sample_lengths(impossible, 1, max_draws=20)


def _cut_brute(lengths, P, stride, Hkv, waves, min_range):
    n = [min(-(-int(L) // P), stride) if L > 0 else 0 for L in lengths]
    owner = []                       # page-head index -> (b, g)
    for b, nb in enumerate(n):
        for g in range(Hkv):
            owner += [(b, g)] * nb
    T = len(owner)
    if T == 0:
        return []
    W = min(waves, -(-T // min_range))
    q, rem = divmod(T, W)
    rng_of = []
    for w in range(W):
        rng_of += [w] * (q + (1 if w < rem else 0))
    seen = {}
    for x, seg in enumerate(owner):
        seen.setdefault(seg, set()).add(rng_of[x])
    return sorted(s for s, r in seen.items() if len(r) > 1)


@pytest.mark.parametrize("seed", range(12))
def test_cut_segments_match_brute_force(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 12))
    P = int(rng.choice([16, 32]))
    lengths = rng.integers(0, 400, size=B)
    lengths[rng.random(B) < 0.2] = 0
    stride = max(1, int(rng.integers(1, 30)))
    Hkv = int(rng.integers(1, 5))
    waves = int(rng.integers(1, 40))
    mr = int(rng.choice([1, 3, 8]))
    assert cut_segments(lengths, P, stride, Hkv, waves, mr) == \
        _cut_brute(lengths, P, stride, Hkv, waves, mr)


def test_page_chunks_cover_every_sequence_once():
    L = np.array([10, 500, 3, 3000, 16, 17, 900], np.int32)
    runs = page_chunks(L, 16, 64)
    assert sorted(i for r in runs for i in r) == list(range(len(L)))
    n = wl.pages_needed(L, 16)
    for r in runs:
        assert len(r) == 1 or n[r].sum() <= 64


@pytest.mark.parametrize("kv_dtype,P,H,d", [(0, 16, 2, 64), (1, 32, 3, 128), (0, 32, 1, 128)])
def test_page_layout_helpers_follow_the_documented_layout(kv_dtype, P, H, d):
    """The helpers that build pages from token-major keys and values (used by
    the oracle pins) place every element where the C header's layouts say:
    key (t, h, i) at k_pages[t / P][h][i / X][t % P][i % X], X = 16 bytes of
    elements; value (t, h, i) at v_pages[t / P][h][i][t % P]; and the inverse
    helpers undo them."""
    n = 3
    rng = np.random.default_rng(P + H + d)
    k = rng.integers(0, 1 << 15, size=(n * P, H, d)).astype(np.int32)
    v = rng.integers(0, 1 << 15, size=(n * P, H, d)).astype(np.int32)
    X = wl.chunk_elems(kv_dtype)
    kp = wl.k_tokens_to_pages(k, P, kv_dtype)
    vp = wl.v_tokens_to_pages(v, P)
    assert kp.shape == (n, H, d // X, P, X) and vp.shape == (n, H, d, P)
    for t in range(n * P):
        for h in range(H):
            for i in range(d):
                assert kp[t // P, h, i // X, t % P, i % X] == k[t, h, i]
                assert vp[t // P, h, i, t % P] == v[t, h, i]
    assert np.array_equal(wl.k_pages_to_tokens(kp), k)
    assert np.array_equal(wl.v_pages_to_tokens(vp), v)


def test_algorithmic_bytes_by_hand():
    """The roofline numerator on a case computed by hand: K and V of valid
    tokens only (no tail slots), fp8 page scales, Q and the output, one
    block-table entry per page and one length per sequence."""
    w = wl.Workload("h", 3, 8, 2, 64, 16, 0, 64, "uniform", lo=1, hi=1)
    ab = wl.algorithmic_bytes(w, np.array([17, 0, 32], np.int32))
    assert ab["kv"] == (17 + 0 + 32) * 2 * 64 * 2 * 2      # tokens x Hkv x d x (K, V) x 2 B
    assert ab["scales"] == 0
    assert ab["q_out"] == 2 * 3 * 8 * 64 * 2              # Q and out, bf16
    assert ab["meta"] == (2 + 0 + 2) * 4 + 3 * 4          # table entries, lengths
    assert ab["total"] == ab["kv"] + ab["q_out"] + ab["meta"]
    w8 = wl.Workload("h8", 3, 8, 2, 64, 32, 1, 64, "uniform", lo=1, hi=1)
    ab8 = wl.algorithmic_bytes(w8, np.array([17, 0, 33], np.int32))
    assert ab8["kv"] == (17 + 33) * 2 * 64 * 2 * 1          # fp8: one byte per element
    assert ab8["scales"] == (1 + 0 + 2) * 2 * 4             # fp32 K and V scale per page
    assert ab8["meta"] == (1 + 0 + 2) * 4 + 3 * 4


def test_shared_prefix_bytes_count_shared_pages_once_per_group():
    """Grouped accounting: every member but the group's first has its shared
    pages' K and V subtracted once; table entries are still read per member."""
    w = wl.Workload("g", 4, 8, 2, 64, 16, 0, 64, "uniform", lo=1, hi=1)
    lengths = np.array([100, 90, 50, 60], np.int32)
    shared = np.array([5, 5, 3, 3], np.int32)          # groups of two
    plain = wl.algorithmic_bytes(w, lengths)
    g = wl.shared_prefix_algorithmic_bytes(w, lengths, shared, 2)
    dup = (5 + 3) * 16 * 2 * 64 * 2 * 2                 # members 1 and 3: pages x P x Hkv x d x (K, V) x 2 B
    assert g["duplicate_kv_not_counted"] == dup
    assert g["kv"] == plain["kv"] - dup and g["total"] == plain["total"] - dup
    assert g["meta"] == plain["meta"]
