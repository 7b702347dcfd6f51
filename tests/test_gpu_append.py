"""GPU parity of dora_kv_append (through the C ABI) against the oracle.

Bar: pages and per-page scales bit-exact after every sequence of appends (the
append is byte work; its fp8 decisions are taken in fp32 on both sides), then
decode over the appended pool within the decode tolerance.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from gpu_util import TOL, lib, max_abs_err

pytestmark = pytest.mark.gpu


def _finite_codes(shape, dt, g):
    """Random page contents: bf16 bit patterns, or fp8 codes without NaN."""
    if dt == 0:
        return torch.randint(0, 65536, shape, generator=g, dtype=torch.int32).to(
            torch.int16).view(torch.bfloat16)
    c = torch.randint(0, 256, shape, generator=g, dtype=torch.int32).to(torch.uint8)
    c[(c & 0x7F) == 0x7F] = 0x7E
    return c


def _setup(B, Hkv, d, P, dt, steps, seed, num_pages=None, spread=0.8):
    """Pool, block table and `steps` tokens per sequence; token magnitudes vary
    by exp(N(0, spread)) so that fp8 page scales grow and hold."""
    g = torch.Generator().manual_seed(seed)
    start = torch.randint(0, 2 * P, (B,), generator=g).numpy().astype(np.int32)
    start[0] = 0                                   # a fresh sequence: first token at slot 0
    final = start + steps
    num_pages = num_pages or int(wl.pages_needed(final, P).sum()) + 7
    bt, _ = wl.place_pages(final, P, num_pages, seed=seed + 1)
    X = wl.chunk_elems(dt)
    k = _finite_codes((num_pages, Hkv, d // X, P, X), dt, g)
    v = _finite_codes((num_pages, Hkv, d, P), dt, g)
    ks = vs = None
    if dt == 1:
        ks = torch.rand(num_pages, generator=g) * 0.05 + 1e-3
        vs = torch.rand(num_pages, generator=g) * 0.05 + 1e-3
    mags = torch.exp(torch.randn(steps, B, 1, 1, generator=g) * spread)
    kn = (torch.randn(steps, B, Hkv, d, generator=g) * mags).to(torch.bfloat16)
    vn = (torch.randn(steps, B, Hkv, d, generator=g) * mags).to(torch.bfloat16)
    return start, bt, k, v, ks, vs, kn, vn


def _np_codes(t, dt):
    return t.contiguous().view(torch.int16).numpy().view(np.uint16) if dt == 0 else \
        t.contiguous().numpy()


@pytest.mark.parametrize("dt", [0, 1])
@pytest.mark.parametrize("P", [16, 32])
@pytest.mark.parametrize("Hkv,d", [(1, 64), (4, 128), (8, 128)])
def test_append_bit_exact_vs_oracle(dt, P, Hkv, d):
    print(f"[case] append dt={dt} P={P} Hkv={Hkv} d={d}", flush=True)
    B, steps = 6, 2 * P + 3
    start, bt, k, v, ks, vs, kn, vn = _setup(B, Hkv, d, P, dt, steps, seed=20 + P + d + Hkv + dt)
    # host (oracle) copies
    hk, hv = _np_codes(k, dt).copy(), _np_codes(v, dt).copy()
    hks = None if ks is None else ks.numpy().copy()
    hvs = None if vs is None else vs.numpy().copy()
    # device pool
    d_k, d_v = k.cuda(), v.cuda()
    d_ks = None if ks is None else ks.cuda()
    d_vs = None if vs is None else vs.cuda()
    d_bt = torch.from_numpy(bt).cuda()
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    D = lib()
    for s in range(steps):
        lens = (start + s + 1).astype(np.int32)
        lens[B - 1] = 0                            # one sequence never appends
        kb = _np_codes(kn[s], 0)
        vb = _np_codes(vn[s], 0)
        assert oracle.kv_append(kb, vb, bt, lens, hk, hv, kv_dtype=dt, page_size=P,
                                k_scales=hks, v_scales=hvs) == 0
        D.dora_kv_append(kn[s].cuda(), vn[s].cuda(), d_bt, torch.from_numpy(lens).cuda(),
                         d_k, d_v, num_kv_heads=Hkv, page_size=P, kv_dtype=dt, k_scales=d_ks,
                         v_scales=d_vs, dev_status=status)
        assert int(status.item()) == 0
    torch.cuda.synchronize()
    assert np.array_equal(_np_codes(d_k.cpu(), dt), hk)
    assert np.array_equal(_np_codes(d_v.cpu(), dt), hv)
    if dt == 1:
        assert np.array_equal(d_ks.cpu().numpy().view(np.uint32), hks.view(np.uint32))
        assert np.array_equal(d_vs.cpu().numpy().view(np.uint32), hvs.view(np.uint32))


@pytest.mark.parametrize("dt", [0, 1])
def test_append_then_decode_matches_oracle(dt):
    """The decode loop's two calls: append the token, then attend over it.
    Values N(0,1), as the decode tolerance assumes; the per-token maxima still
    vary, so fp8 page scales grow along the way."""
    B, Hkv, Hq, d, P, steps = 5, 2, 14, 128, 16, 20
    start, bt, k, v, ks, vs, kn, vn = _setup(B, Hkv, d, P, dt, steps, seed=40 + dt, spread=0.0)
    # a clean prefix (no garbage among attended tokens): append it too
    start[:] = 0
    d_k, d_v = k.cuda(), v.cuda()
    d_ks = None if ks is None else ks.cuda()
    d_vs = None if vs is None else vs.cuda()
    d_bt = torch.from_numpy(bt).cuda()
    D = lib()
    g = torch.Generator().manual_seed(41)
    q = (torch.randn(B, Hq, d, generator=g)).to(torch.bfloat16).cuda()
    for s in range(steps):
        lens = torch.full((B,), s + 1, dtype=torch.int32)
        D.dora_kv_append(kn[s].cuda(), vn[s].cuda(), d_bt, lens.cuda(), d_k, d_v,
                         num_kv_heads=Hkv, page_size=P, kv_dtype=dt, k_scales=d_ks,
                         v_scales=d_vs)
        out = torch.empty_like(q)
        D.dora_decode_attn(q, d_k, d_v, d_bt, lens.cuda(), None, out, num_kv_heads=Hkv,
                           page_size=P, kv_dtype=dt, k_scales=d_ks, v_scales=d_vs)
        ref = oracle.decode(_np_codes(q.cpu(), 0), _np_codes(d_k.cpu(), dt),
                            _np_codes(d_v.cpu(), dt), bt, lens.numpy(), num_kv_heads=Hkv,
                            page_size=P, kv_dtype=dt,
                            k_scales=None if d_ks is None else d_ks.cpu().numpy(),
                            v_scales=None if d_vs is None else d_vs.cpu().numpy())
        assert max_abs_err(out, ref) <= TOL[dt]


def test_append_skips_bad_pages_and_reports():
    B, Hkv, d, P = 4, 2, 64, 16
    start, bt, k, v, ks, vs, kn, vn = _setup(B, Hkv, d, P, 1, 1, seed=50)
    lens = (start + 1).astype(np.int32)
    bad = bt.copy()
    bad[1, (lens[1] - 1) // P] = 10 ** 6           # out of the pool
    hk, hv = _np_codes(k, 1).copy(), _np_codes(v, 1).copy()
    hks, hvs = ks.numpy().copy(), vs.numpy().copy()
    good = lens.copy()
    good[1] = 0                                    # the oracle's view: sequence 1 skipped
    assert oracle.kv_append(_np_codes(kn[0], 0), _np_codes(vn[0], 0), bt, good, hk, hv,
                            kv_dtype=1, page_size=P, k_scales=hks, v_scales=hvs) == 0
    d_k, d_v, d_ks, d_vs = k.cuda(), v.cuda(), ks.cuda(), vs.cuda()
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    D = lib()
    D.dora_kv_append(kn[0].cuda(), vn[0].cuda(), torch.from_numpy(bad).cuda(),
                     torch.from_numpy(lens).cuda(), d_k, d_v, num_kv_heads=Hkv, page_size=P,
                     kv_dtype=1, k_scales=d_ks, v_scales=d_vs, dev_status=status)
    assert int(status.item()) == D.DORA_ERR_DEVICE_CHECK
    assert np.array_equal(_np_codes(d_k.cpu(), 1), hk)
    assert np.array_equal(_np_codes(d_v.cpu(), 1), hv)
    assert np.array_equal(d_ks.cpu().numpy(), hks) and np.array_equal(d_vs.cpu().numpy(), hvs)
    # under VALIDATE, a page of another version is skipped too
    owner = torch.zeros(k.shape[0], dtype=torch.int16)
    owner[int(bt[2, (lens[2] - 1) // P])] = 1
    vid = torch.zeros(B, dtype=torch.int32)
    before = d_k.clone()
    status.fill_(0)
    D.dora_kv_append(kn[0].cuda(), vn[0].cuda(), torch.from_numpy(bt).cuda(),
                     torch.from_numpy(np.where(np.arange(B) == 2, lens, 0).astype(np.int32))
                     .cuda(), d_k, d_v, num_kv_heads=Hkv, page_size=P, kv_dtype=1,
                     k_scales=d_ks, v_scales=d_vs, version_ids=vid.cuda(),
                     page_owner=owner.cuda(), flags=D.DORA_FLAG_VALIDATE, dev_status=status)
    assert int(status.item()) == D.DORA_ERR_DEVICE_CHECK
    assert torch.equal(d_k, before)


@pytest.mark.parametrize("idx", [1, 4])
def test_append_full_size_workload_sampled(idx):
    """The 64-sequence bf16 and the 1024-sequence fp8 batches: every sequence
    rewrites its last token (same seq_lens, so the page exists); a sample of
    pages is checked against the oracle."""
    w = wl.WORKLOADS[idx]
    print(f"[case] append full-size {w.name}", flush=True)
    b = wl.make_batch(w, device="cuda", seed_index=idx)
    g = torch.Generator().manual_seed(60 + idx)
    kn = (torch.randn(w.num_seqs, w.num_kv_heads, w.head_dim, generator=g) * 1.7).to(
        torch.bfloat16)
    vn = (torch.randn(w.num_seqs, w.num_kv_heads, w.head_dim, generator=g) * 1.7).to(
        torch.bfloat16)
    rng = np.random.default_rng(idx)
    seqs = sorted(set([0, w.num_seqs - 1] + [int(i) for i in rng.choice(w.num_seqs, 6)]))
    seqs = [s for s in seqs if b.lengths[s] > 0]
    pages = [int(b.block_table_h[s, (b.lengths[s] - 1) // w.page_size]) for s in seqs]
    idx_t = torch.tensor(pages, dtype=torch.long, device="cuda")
    hk = _np_codes(b.k_pages[idx_t].cpu(), w.kv_dtype).copy()
    hv = _np_codes(b.v_pages[idx_t].cpu(), w.kv_dtype).copy()
    hks = None if b.k_scales is None else b.k_scales[idx_t].cpu().numpy().copy()
    hvs = None if b.v_scales is None else b.v_scales[idx_t].cpu().numpy().copy()
    D = lib()
    D.dora_kv_append(kn.cuda(), vn.cuda(), b.block_table, b.seq_lens, b.k_pages, b.v_pages,
                     num_kv_heads=w.num_kv_heads, page_size=w.page_size, kv_dtype=w.kv_dtype,
                     k_scales=b.k_scales, v_scales=b.v_scales)
    torch.cuda.synchronize()
    # the oracle on a mini-pool of the sampled sequences' pages
    last = (b.lengths[seqs] - 1) // w.page_size
    mini_bt = np.zeros((len(seqs), int(last.max()) + 1), np.int32)
    mini_bt[np.arange(len(seqs)), last] = np.arange(len(seqs))
    assert oracle.kv_append(_np_codes(kn[seqs], 0), _np_codes(vn[seqs], 0), mini_bt,
                            b.lengths[seqs].astype(np.int32), hk, hv, kv_dtype=w.kv_dtype,
                            page_size=w.page_size, k_scales=hks, v_scales=hvs) == 0
    assert np.array_equal(_np_codes(b.k_pages[idx_t].cpu(), w.kv_dtype), hk)
    assert np.array_equal(_np_codes(b.v_pages[idx_t].cpu(), w.kv_dtype), hv)
    if w.kv_dtype == 1:
        assert np.array_equal(b.k_scales[idx_t].cpu().numpy(), hks)
        assert np.array_equal(b.v_scales[idx_t].cpu().numpy(), hvs)
    del b
    torch.cuda.empty_cache()


def test_append_random_geometries_bit_exact():
    """24 seeded random geometries (dtype, page size, 1-8 KV heads, head dim,
    1-12 sequences, 1 to 2P+3 appends, three spreads of token magnitude):
    pages and fp8 scales bit-exact against the oracle after every run."""
    rng = np.random.default_rng(424242)
    D = lib()
    for case in range(24):
        dt = int(rng.integers(0, 2))
        P = int(rng.choice([16, 32]))
        Hkv = int(rng.integers(1, 9))
        d = int(rng.choice([64, 128]))
        B = int(rng.integers(1, 13))
        steps = int(rng.integers(1, 2 * P + 4))
        spread = float(rng.choice([0.3, 0.8, 2.0]))
        print(f"[case {case}] append dt={dt} P={P} Hkv={Hkv} d={d} B={B} steps={steps} "
              f"spread={spread}", flush=True)
        start, bt, k, v, ks, vs, kn, vn = _setup(B, Hkv, d, P, dt, steps, seed=500 + case,
                                                 spread=spread)
        hk, hv = _np_codes(k, dt).copy(), _np_codes(v, dt).copy()
        hks = None if ks is None else ks.numpy().copy()
        hvs = None if vs is None else vs.numpy().copy()
        d_k, d_v = k.cuda(), v.cuda()
        d_ks = None if ks is None else ks.cuda()
        d_vs = None if vs is None else vs.cuda()
        d_bt = torch.from_numpy(bt).cuda()
        status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        for s in range(steps):
            lens = (start + s + 1).astype(np.int32)
            assert oracle.kv_append(_np_codes(kn[s], 0), _np_codes(vn[s], 0), bt, lens, hk, hv,
                                    kv_dtype=dt, page_size=P, k_scales=hks, v_scales=hvs) == 0
            D.dora_kv_append(kn[s].cuda(), vn[s].cuda(), d_bt, torch.from_numpy(lens).cuda(),
                             d_k, d_v, num_kv_heads=Hkv, page_size=P, kv_dtype=dt,
                             k_scales=d_ks, v_scales=d_vs, dev_status=status)
            assert int(status.item()) == 0, (case, s)
        torch.cuda.synchronize()
        assert np.array_equal(_np_codes(d_k.cpu(), dt), hk), case
        assert np.array_equal(_np_codes(d_v.cpu(), dt), hv), case
        if dt == 1:
            assert np.array_equal(d_ks.cpu().numpy().view(np.uint32), hks.view(np.uint32)), case
            assert np.array_equal(d_vs.cpu().numpy().view(np.uint32), hvs.view(np.uint32)), case
