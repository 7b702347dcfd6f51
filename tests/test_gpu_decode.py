"""GPU parity of dora_decode_attn (through the C ABI) against the fp64 oracle.

Bar: max-abs error <= 2e-2 on bf16-KV outputs and <= 5e-2 on fp8-KV outputs;
bitwise equality where the result is unique (length-1 sequences, page
permutation, migration, repeated runs).
"""
import numpy as np
import pytest
import torch

import workloads as wl
from gpu_util import (TOL, cut_segments, decode_waves, gpu_batch, lib, max_abs_err, oracle_for,
                      page_chunks, run_decode)

pytestmark = pytest.mark.gpu


def _w(name="t", B=8, Hq=8, Hkv=2, d=64, P=16, dt=0, pages=None, lens=None):
    pages = pages or max(64, int(wl.pages_needed(np.asarray(lens), P).sum()) * 2 + 8)
    return wl.Workload(name, B, Hq, Hkv, d, P, dt, pages, "uniform", lo=1, hi=1)


RAGGED = [0, 1, 2, 15, 16, 17, 31, 32, 33, 100, 257, 1000, 4097]


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("P", [16, 32])
@pytest.mark.parametrize("dt", [0, 1])
@pytest.mark.parametrize("G", [1, 4, 7, 16])
def test_shapes_ragged_lengths(d, P, dt, G):
    print(f"[case] shapes d={d} P={P} dt={dt} G={G}", flush=True)
    Hkv = 2
    lens = np.array(RAGGED, np.int32)
    w = _w(B=len(lens), Hq=G * Hkv, Hkv=Hkv, d=d, P=P, dt=dt, lens=lens)
    b = gpu_batch(w, lengths=lens, seed_index=100 + d + P + dt + G)
    out = run_decode(b)
    ref = oracle_for(b)
    err = max_abs_err(out, ref)
    assert err <= TOL[dt], err
    assert torch.all(out[0] == 0), "empty sequence must give zeros"


def test_tiny_workload_full_parity():
    w = wl.WORKLOADS[0]
    print(f"[case] {w.name}", flush=True)
    b = gpu_batch(w, seed_index=0)
    out = run_decode(b)
    err = max_abs_err(out, oracle_for(b))
    assert err <= TOL[0], err


@pytest.mark.parametrize("waves", [1, 2, 7, 64, 1000, 0])
def test_wave_count_invariance(waves):
    """Cutting the work among 1 ... 1000 wavefronts (ranges as small as one
    page-head, so segments are cut into many partials) agrees with the oracle
    and with the default cut."""
    print(f"[case] waves={waves}", flush=True)
    lens = np.array([5, 700, 1300, 33, 2048, 16, 0, 1], np.int32)
    w = _w(B=len(lens), Hq=16, Hkv=2, d=128, P=16, dt=0, lens=lens)
    b = gpu_batch(w, lengths=lens, seed_index=7)
    out = run_decode(b, num_waves=waves, min_range_pages=1)
    ref = oracle_for(b)
    assert max_abs_err(out, ref) <= TOL[0]
    base = run_decode(b)
    diff = (out.float() - base.float()).abs().max().item()
    assert diff <= TOL[0]


def test_wave_count_invariance_fp8_page32():
    lens = np.array([2000, 64, 4500, 1], np.int32)
    w = _w(B=len(lens), Hq=16, Hkv=2, d=128, P=32, dt=1, lens=lens)
    b = gpu_batch(w, lengths=lens, seed_index=8)
    ref = oracle_for(b)
    for waves in (1, 5, 300):
        out = run_decode(b, num_waves=waves, min_range_pages=1)
        assert max_abs_err(out, ref) <= TOL[1]


def test_deterministic_bitwise():
    lens = np.array([3000, 17, 900, 4000, 1], np.int32)
    w = _w(B=len(lens), Hq=28, Hkv=4, d=128, P=16, dt=0, lens=lens)
    b = gpu_batch(w, lengths=lens, seed_index=9)
    a = run_decode(b).clone()
    for _ in range(3):
        assert torch.equal(run_decode(b), a)


def test_length_one_is_value_row_bitwise():
    lens = np.ones(6, np.int32)
    w = _w(B=6, Hq=8, Hkv=2, d=128, P=16, dt=0, lens=lens)
    b = gpu_batch(w, lengths=lens, seed_index=10)
    out = run_decode(b)
    for s in range(6):
        pg = int(b.block_table_h[s, 0])
        for h in range(8):
            v = b.v_pages[pg, h // 4, :, 0]          # token slot 0, all head dims
            assert torch.equal(out[s, h], v)


def test_physical_page_permutation_bitwise():
    lens = np.array([300, 1, 77, 1024], np.int32)
    w = _w(B=4, Hq=8, Hkv=2, d=128, P=16, dt=0, lens=lens)
    b = gpu_batch(w, lengths=lens, seed_index=11)
    ref = run_decode(b).clone()
    perm = torch.randperm(w.num_pages, generator=torch.Generator().manual_seed(3)).cuda()
    k2 = torch.empty_like(b.k_pages)
    v2 = torch.empty_like(b.v_pages)
    k2[perm] = b.k_pages
    v2[perm] = b.v_pages
    bt2 = perm[b.block_table.long()].to(torch.int32)
    b.k_pages, b.v_pages, b.block_table = k2, v2, bt2.contiguous()
    assert torch.equal(run_decode(b), ref)


def test_batch_permutation():
    """Permuting the batch permutes the outputs.  The work cut moves with the
    order, so the match is to tolerance, not bitwise."""
    lens = np.array([300, 1, 77, 1024, 5000, 0], np.int32)
    w = _w(B=6, Hq=8, Hkv=2, d=128, P=16, dt=0, lens=lens)
    b = gpu_batch(w, lengths=lens, seed_index=12)
    ref = run_decode(b).clone()
    perm = torch.tensor([3, 5, 0, 4, 1, 2])
    b.q = b.q[perm.cuda()].contiguous()
    b.block_table = b.block_table[perm.cuda()].contiguous()
    b.seq_lens = b.seq_lens[perm.cuda()].contiguous()
    b.version_ids = b.version_ids[perm.cuda()].contiguous()
    diff = (run_decode(b).float() - ref[perm.cuda()].float()).abs().max().item()
    assert diff <= TOL[0]


def test_workspace_contents_ignored():
    lens = np.array([800, 2000, 3], np.int32)
    w = _w(B=3, Hq=8, Hkv=2, d=128, P=16, dt=0, lens=lens)
    b = gpu_batch(w, lengths=lens, seed_index=13)
    d = lib()
    ref = run_decode(b, num_waves=40, min_range_pages=1).clone()
    desc = d.make_decode_desc(num_seqs=3, num_q_heads=8, num_kv_heads=2, head_dim=128,
                              page_size=16, block_table_stride=b.stride,
                              num_pages=w.num_pages, num_waves=40, min_range_pages=1)
    ws = torch.full((d.dora_decode_workspace_bytes(desc) // 4,), float("nan"),
                    device="cuda").view(torch.uint8)
    out = torch.full_like(b.q, float("nan"))
    run_decode(b, out=out, num_waves=40, min_range_pages=1, workspace=ws)
    assert torch.equal(out, ref)


def test_batch_larger_than_one_launch():
    """More sequences than one decode launch takes (8192): the call is cut into
    launches; outputs of sequences in both launches match the oracle."""
    rng = np.random.default_rng(3)
    lens = rng.integers(0, 40, 9000).astype(np.int32)
    w = _w(B=len(lens), Hq=8, Hkv=2, d=64, P=16, dt=0, lens=lens)
    b = gpu_batch(w, lengths=lens, seed_index=14)
    out = run_decode(b)
    seqs = [0, 1, 8190, 8191, 8192, 8193, 8999] + [int(i) for i in rng.choice(9000, 20)]
    seqs = sorted(set(seqs))
    assert max_abs_err(out, oracle_for(b, seqs), seqs) <= TOL[0]


def test_validate_flag_accepts_good_and_rejects_bad_pages():
    w = wl.WORKLOADS[3].scaled(48, num_pages=8192)   # three versions in one pool
    b = gpu_batch(w, seed_index=3, lengths=np.random.default_rng(1).integers(1, 1500, 48)
                  .astype(np.int32))
    d = lib()
    run_decode(b, flags=d.DORA_FLAG_VALIDATE, page_owner=b.page_owner)
    # a page of another version in sequence 0's table
    other = int(np.nonzero(b.versions_h != b.versions_h[0])[0][0])
    bt = b.block_table.clone()
    bt[0, 0] = b.block_table[other, 0]
    b2 = b
    b2.block_table = bt
    with pytest.raises(d.DoraError) as e:
        run_decode(b2, flags=d.DORA_FLAG_VALIDATE, page_owner=b.page_owner)
    assert e.value.status == d.DORA_ERR_DEVICE_CHECK
    bt = bt.clone()
    bt[0, 0] = w.num_pages + 5
    b2.block_table = bt
    with pytest.raises(d.DoraError) as e:
        run_decode(b2, flags=d.DORA_FLAG_VALIDATE)
    assert e.value.status == d.DORA_ERR_DEVICE_CHECK



@pytest.mark.parametrize("bad", ["len_past_table", "len_negative", "page_negative"])
def test_validate_flag_rejects_bad_lengths_and_ids(bad):
    """DORA_FLAG_VALIDATE also rejects a length the block table cannot hold,
    a negative length and a negative page id, before any decode launch (the
    output keeps its sentinel), and a good call right after passes (the
    check's flag is cleared on every call)."""
    print(f"[case] validate {bad}", flush=True)
    lens = np.array([40, 300, 17, 129], np.int32)
    w = _w(B=len(lens), Hq=8, Hkv=2, d=64, P=16, dt=0, lens=lens)
    b = gpu_batch(w, lengths=lens, seed_index=9)
    d = lib()
    good_bt, good_lens = b.block_table.clone(), b.seq_lens.clone()
    stride = b.block_table.shape[1]
    if bad == "len_past_table":
        b.seq_lens[1] = stride * w.page_size + 1
    elif bad == "len_negative":
        b.seq_lens[2] = -1
    else:
        b.block_table[3, 2] = -3
    sentinel = torch.full_like(b.q, 7.0)
    out = sentinel.clone()
    with pytest.raises(d.DoraError) as e:
        run_decode(b, out=out, flags=d.DORA_FLAG_VALIDATE)
    assert e.value.status == d.DORA_ERR_DEVICE_CHECK
    assert torch.equal(out, sentinel)
    b.block_table, b.seq_lens = good_bt, good_lens
    out = run_decode(b, flags=d.DORA_FLAG_VALIDATE)
    assert max_abs_err(out, oracle_for(b)) <= TOL[0]

def test_empty_batch_is_a_no_op():
    d = lib()
    q = torch.empty((0, 8, 64), dtype=torch.bfloat16, device="cuda")
    kp = torch.zeros((4, 2, 8, 16, 8), dtype=torch.bfloat16, device="cuda")
    vp = torch.zeros((4, 2, 64, 16), dtype=torch.bfloat16, device="cuda")
    bt = torch.zeros((0, 1), dtype=torch.int32, device="cuda")
    z = torch.zeros(0, dtype=torch.int32, device="cuda")
    d.dora_decode_attn(q, kp, vp, bt, z, z, q.clone(), num_kv_heads=2, page_size=16)


# ---------------------------------------------------------------------------
# the long-tail workloads at full size, in the launch configuration the
# benchmark times: every output element of every sequence against the oracle
# (in runs of sequences, to bound the host copies).
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("idx", [1, 2, 3, 4])
def test_full_size_workloads_every_sequence(idx):
    w = wl.WORKLOADS[idx]
    print(f"[case] full-size {w.name}", flush=True)
    b = gpu_batch(w, seed_index=idx)
    out = run_decode(b)
    assert torch.isfinite(out.float()).all()
    waves = decode_waves(b)
    cuts = cut_segments(b.lengths, w.page_size, b.stride, w.num_kv_heads, waves)
    # the default launch splits segments across wavefronts, so the combine runs
    assert cuts, "no segment is cut: the combine path would go untested"
    err, runs = 0.0, page_chunks(b.lengths, w.page_size, 24576)
    for seqs in runs:
        ref = oracle_for(b, seqs)
        err = max(err, max_abs_err(out, ref, seqs))
    print(f"[case] {w.name}: {w.num_seqs} seqs in {len(runs)} runs, {waves} waves, "
          f"{len(cuts)} cut segments in {len({c[0] for c in cuts})} seqs, "
          f"max-abs err {err:.3e}", flush=True)
    assert err <= TOL[w.kv_dtype], err
    del b, out
    torch.cuda.empty_cache()


def test_profiling_events_bracket_each_kernel():
    """The three events bracket the decode and the combine kernel: positive
    durations, and the call's result is unchanged."""
    lens = np.array([3000, 17, 900, 4000, 1], np.int32)
    w = _w(B=len(lens), Hq=28, Hkv=4, d=128, P=16, dt=0, lens=lens)
    b = gpu_batch(w, lengths=lens, seed_index=15)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    for e in evs:
        e.record()
    torch.cuda.synchronize()
    ref = run_decode(b).clone()
    out = run_decode(b, events=[e.cuda_event for e in evs])
    assert torch.equal(out, ref)
    dec, comb = (evs[i].elapsed_time(evs[i + 1]) for i in range(2))
    assert 0 < dec < 1000 and 0 < comb < 1000, (dec, comb)
