"""Grouped decode (response groups sharing a prompt's pages), through the C
ABI: dora_decode_attn_grouped reads each group's shared pages once and must
give what the oracle gives reading them through every member's block table,
and what dora_decode_attn gives, within the decode tolerance."""
import numpy as np
import pytest
import torch

import workloads as wl
from gpu_util import TOL, lib, max_abs_err, oracle_for, run_decode, sample_seqs

pytestmark = pytest.mark.gpu


def _grouped(b, M, **kw):
    out = torch.empty_like(b.q)
    det = torch.full((b.w.num_seqs // M,), -1, dtype=torch.int32, device="cuda")
    lib().dora_decode_attn_grouped(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                                   b.version_ids, out, group_size=M,
                                   num_kv_heads=b.w.num_kv_heads, page_size=b.w.page_size,
                                   kv_dtype=b.w.kv_dtype, k_scales=b.k_scales,
                                   v_scales=b.v_scales, shared_pages_out=det, **kw)
    torch.cuda.synchronize()
    return out, det.cpu().numpy()


def _set_tables(b, bt, lens=None):
    b.block_table_h = bt
    b.block_table = torch.from_numpy(bt).cuda()
    if lens is not None:
        b.lengths = lens
        b.seq_lens = torch.from_numpy(lens).cuda()


@pytest.mark.parametrize("dt,P,d,G,M", [
    (0, 16, 128, 7, 4),      # the 7B-class group of 7 query heads
    (1, 32, 128, 8, 4),      # fp8 pages of 32 tokens
    (0, 16, 64, 4, 8),
    (0, 32, 64, 1, 16),      # one query head per KV head, 16 members
    (1, 16, 128, 16, 2),     # 16 query heads per KV head: 32 columns
    (0, 16, 128, 8, 16),     # 128 columns: the widest group
    (1, 32, 128, 8, 16),     # the widest group over fp8 pages of 32 tokens
    (1, 16, 64, 4, 8),       # fp8, d 64
])
def test_grouped_matches_oracle_and_plain_decode(dt, P, d, G, M):
    print(f"[case] grouped dt={dt} P={P} d={d} G={G} M={M}", flush=True)
    Hkv = 2
    w = wl.Workload("g", 2 * M, G * Hkv, Hkv, d, P, dt, 8192, "lognormal", 200, 1.0, 1, 2500)
    b, shared = wl.make_grpo_batch(w, group_size=M, prompt_range=(P + 3, 900), device="cuda",
                                   seed_index=30 + dt + P + G + M)
    out, det = _grouped(b, M)
    assert det.tolist() == shared[::M].tolist()          # the prompt's full pages
    assert max_abs_err(out, oracle_for(b)) <= TOL[dt]
    assert (out.float() - run_decode(b).float()).abs().max().item() <= TOL[dt]


def test_grouped_edge_cases():
    """Groups of three: a member that is all prompt (empty suffix), a group
    whose members share nothing, a member that leaves the prompt's pages early
    (the group shares only what all members share), a member of length 0; then
    groups of one (nothing shared) and a batch without any sharing."""
    w = wl.Workload("e", 12, 14, 2, 128, 16, 0, 4096, "lognormal", 300, 1.0, 1, 2000)
    b, shared = wl.make_grpo_batch(w, group_size=3, prompt_range=(100, 600), device="cuda",
                                   seed_index=40)
    bt, lens = b.block_table_h.copy(), b.lengths.copy()
    lens[1] = shared[1] * 16                          # group 0: member 1 is its prompt only
    for m in (4, 5):
        bt[m, 0] = bt[3, 1]                           # group 1: first pages differ (full pages)
    bt[8, 2] = bt[6, 3]                               # group 2: member 8 diverges at page 2
    lens[10] = 0                                      # group 3: an empty member
    _set_tables(b, bt, lens)
    ref = oracle_for(b)
    out, det = _grouped(b, 3)
    assert det.tolist() == [shared[0], 0, 2, 0]
    assert max_abs_err(out, ref) <= TOL[0]
    assert not out[10].float().abs().any()
    out, det = _grouped(b, 1)
    assert not det.any()
    assert max_abs_err(out, ref) <= TOL[0]
    plain = wl.make_batch(wl.Workload("n", 8, 28, 4, 128, 16, 0, 4096, "lognormal", 300, 1.0, 1,
                                      2000), device="cuda", seed_index=42)
    out, det = _grouped(plain, 4)
    assert not det.any()
    assert max_abs_err(out, oracle_for(plain)) <= TOL[0]


def test_grouped_is_deterministic():
    b, shared = wl.make_grpo_batch(wl.Workload("d", 8, 28, 4, 128, 16, 0, 8192, "lognormal",
                                               500, 1.0, 1, 3000),
                                   group_size=4, prompt_range=(200, 1500), device="cuda",
                                   seed_index=41)
    a = _grouped(b, 4)[0].clone()
    for _ in range(2):
        assert torch.equal(_grouped(b, 4)[0], a)


@pytest.mark.parametrize("fill", [0x00, 0xFF, 0x7F])
def test_grouped_workspace_contents_ignored(fill):
    """Every per-call value the grouped kernels read back (the prefix lengths,
    partials, suffix rows and the whole-or-cut flag of each segment) is written
    earlier in the same call: a workspace filled with zeros (every segment
    'whole'), all-ones bytes (every flag set, NaN partials) or 0x7F bytes
    gives the bit-identical output of a fresh workspace, with segments both
    whole and cut (a range of 8 page-heads cuts most of them)."""
    print(f"[case] grouped workspace fill {fill:#x}", flush=True)
    w = wl.Workload("ws", 12, 28, 4, 128, 16, 0, 8192, "lognormal", 300, 1.0, 1, 2500)
    b, shared = wl.make_grpo_batch(w, group_size=4, prompt_range=(100, 900), device="cuda",
                                   seed_index=45)
    d = lib()
    desc = d.make_decode_desc(num_seqs=w.num_seqs, num_q_heads=w.num_q_heads,
                              num_kv_heads=w.num_kv_heads, head_dim=w.head_dim,
                              page_size=w.page_size, block_table_stride=b.block_table.shape[1],
                              num_pages=w.num_pages, kv_dtype=0)
    need = d.dora_decode_grouped_workspace_bytes(desc, 4)
    ref, _ = _grouped(b, 4, workspace=torch.zeros(need, dtype=torch.uint8, device="cuda"))
    ws = torch.full((need,), fill, dtype=torch.uint8, device="cuda")
    out, det = _grouped(b, 4, workspace=ws)
    assert det.tolist() == shared[::4].tolist()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    assert max_abs_err(out, oracle_for(b)) <= TOL[0]


def test_grouped_full_size_grpo_batch_every_sequence():
    """The GRPO batch the benchmark times: every sequence against the oracle
    (each member read through its own block table) and the plain path."""
    print("[case] grouped full-size grpo7b", flush=True)
    b, shared = wl.make_grpo_batch(device="cuda")
    out, det = _grouped(b, wl.GRPO_GROUP)
    assert det.tolist() == shared[::wl.GRPO_GROUP].tolist()
    assert torch.isfinite(out.float()).all()
    assert (out.float() - run_decode(b).float()).abs().max().item() <= TOL[0]
    assert max_abs_err(out, oracle_for(b)) <= TOL[0]


def test_grouped_batch_larger_than_one_launch():
    """9,000 sequences in groups of 8: the suffix decode is cut into launches of
    8,192 sequences, and a group (1,024) straddles the cut; sequences on both
    sides match the oracle and the plain path."""
    w = wl.Workload("big", 9000, 8, 2, 64, 16, 0, 131072, "lognormal", 20, 1.0, 1, 60)
    b, shared = wl.make_grpo_batch(w, group_size=8, prompt_range=(16, 100), device="cuda",
                                   seed_index=43)
    out, det = _grouped(b, 8)
    assert det.tolist() == shared[::8].tolist()
    assert (out.float() - run_decode(b).float()).abs().max().item() <= TOL[0]
    seqs = sorted(set([0, 7, 8184, 8191, 8192, 8199, 8999] + sample_seqs(b.lengths, 6, seed=7)))
    assert max_abs_err(out, oracle_for(b, seqs), seqs) <= TOL[0]


def test_grouped_validate_flag():
    w = wl.Workload("v", 8, 14, 2, 128, 16, 0, 4096, "lognormal", 300, 1.0, 1, 2000)
    b, shared = wl.make_grpo_batch(w, group_size=4, prompt_range=(100, 600), device="cuda",
                                   seed_index=44)
    d = lib()
    good, _ = _grouped(b, 4, flags=d.DORA_FLAG_VALIDATE, page_owner=b.page_owner)
    assert max_abs_err(good, oracle_for(b)) <= TOL[0]
    bt = b.block_table.clone()
    bt[5, 0] = w.num_pages + 3                       # out of the pool
    b.block_table = bt
    with pytest.raises(d.DoraError) as e:
        _grouped(b, 4, flags=d.DORA_FLAG_VALIDATE, page_owner=b.page_owner)
    assert e.value.status == d.DORA_ERR_DEVICE_CHECK


def test_grouped_random_geometries():
    """16 seeded random GRPO-shaped batches (dtype, page size, head dim, 1-4
    KV heads, group size M and query group G with M x G <= 128, 1-3 groups,
    prompt lengths and response mixes drawn per case): the detected shared
    prefix equals the prompt's full pages, and the grouped output matches
    the oracle and the plain decode within the decode tolerance."""
    rng = np.random.default_rng(5150)
    for case in range(16):
        dt = int(rng.integers(0, 2))
        P = int(rng.choice([16, 32]))
        d = int(rng.choice([64, 128]))
        Hkv = int(rng.integers(1, 5))
        M = int(rng.choice([2, 3, 4, 8, 16]))
        G = int(rng.integers(1, 128 // M + 1)) if M > 8 else int(rng.integers(1, 17))
        G = min(G, 16, 128 // M)
        groups = int(rng.integers(1, 4))
        lo = int(rng.integers(P + 1, 600))
        hi = lo + int(rng.integers(1, 1500))
        print(f"[case {case}] grouped dt={dt} P={P} d={d} Hkv={Hkv} G={G} M={M} "
              f"groups={groups} prompts=({lo},{hi})", flush=True)
        w = wl.Workload("gr", groups * M, G * Hkv, Hkv, d, P, dt, 8192, "lognormal", 200, 1.0,
                        1, 2500)
        b, shared = wl.make_grpo_batch(w, group_size=M, prompt_range=(lo, hi), device="cuda",
                                       seed_index=4000 + case)
        out, det = _grouped(b, M)
        assert det.tolist() == shared[::M].tolist(), case
        assert max_abs_err(out, oracle_for(b)) <= TOL[dt], case
        assert (out.float() - run_decode(b).float()).abs().max().item() <= TOL[dt], case
