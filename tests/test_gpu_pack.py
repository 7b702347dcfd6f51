"""GPU pack/unpack (through the C ABI): bit-exact against the oracle's
whole-page gather, and migration that preserves decode bitwise (KV states are
equal on every instance of a version, Sec. 3.4)."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from gpu_util import gpu_batch, lib, run_decode

pytestmark = pytest.mark.gpu


def _host_codes(t: torch.Tensor) -> np.ndarray:
    t = t.cpu()
    return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()


def _pack(b, pages_np, version):
    d = lib()
    w = b.w
    n = len(pages_np)
    desc = d.make_pack_desc(kv_dtype=w.kv_dtype, page_size=w.page_size,
                            num_kv_heads=w.num_kv_heads, head_dim=w.head_dim,
                            num_pages=w.num_pages, policy_version=version)
    packed = torch.empty(d.dora_kv_packed_bytes(desc, n), dtype=torch.uint8, device="cuda")
    src = torch.from_numpy(np.asarray(pages_np, np.int32)).cuda()
    d.dora_kv_page_pack(b.k_pages, b.v_pages, src, packed, num_kv_heads=w.num_kv_heads,
                        page_size=w.page_size, head_dim=w.head_dim, kv_dtype=w.kv_dtype,
                        policy_version=version, n_seqs=3, k_scales=b.k_scales,
                        v_scales=b.v_scales)
    torch.cuda.synchronize()
    return packed


@pytest.mark.parametrize("dt", [0, 1])
def test_pack_bit_exact_vs_oracle(dt):
    P = 16 if dt == 0 else 32
    lens = np.array([100, 33, 1, 700], np.int32)
    w = wl.Workload("p", 4, 16, 4, 128, P, dt, 512, "uniform", lo=1, hi=1)
    b = gpu_batch(w, lengths=lens, seed_index=20 + dt)
    n = wl.pages_needed(lens, P)
    src = np.concatenate([b.block_table_h[i, :n[i]] for i in range(4)]).astype(np.int32)
    packed = _pack(b, src, version=2)
    ref = oracle.pack(_host_codes(b.k_pages), _host_codes(b.v_pages), src, kv_dtype=dt,
                      page_size=P, num_kv_heads=4, head_dim=128, policy_version=2, n_seqs=3,
                      k_scales=None if dt == 0 else b.k_scales.cpu().numpy(),
                      v_scales=None if dt == 0 else b.v_scales.cpu().numpy())
    got = packed.cpu().numpy()
    assert got.size == ref.size
    assert np.array_equal(got, ref)


def _host_pool(t: torch.Tensor) -> np.ndarray:
    """Host copy of a page pool (or scale array) as raw bytes, any dtype."""
    t = t.detach().contiguous().cpu()
    return t.view(torch.uint8).numpy().copy() if t.dtype != torch.uint8 else t.numpy().copy()


def _oracle_unpack_expected(packed_host, dst_pages, k_before, v_before, ks_before, vs_before,
                            *, dt, P, Hkv, d, version):
    """oracle.unpack of the same packed bytes into host copies of the
    destination pool as it was before the GPU unpack."""
    kp, vp = k_before.copy(), v_before.copy()
    ks = None if ks_before is None else ks_before.view(np.float32).copy()
    vs = None if vs_before is None else vs_before.view(np.float32).copy()
    rc = oracle.unpack(packed_host, np.asarray(dst_pages, np.int32), kp, vp, kv_dtype=dt,
                       page_size=P, num_kv_heads=Hkv, head_dim=d, policy_version=version,
                       k_scales=ks, v_scales=vs)
    assert rc == 0, rc
    return kp, vp, ks, vs


def _assert_pools_equal_oracle(dst_k, dst_v, dst_ks, dst_vs, expected):
    kp, vp, ks, vs = expected
    assert np.array_equal(_host_pool(dst_k), kp), "K pool differs from oracle.unpack"
    assert np.array_equal(_host_pool(dst_v), vp), "V pool differs from oracle.unpack"
    if ks is not None:
        assert np.array_equal(_host_pool(dst_ks), ks.view(np.uint8)), "k scales differ"
        assert np.array_equal(_host_pool(dst_vs), vs.view(np.uint8)), "v scales differ"


@pytest.mark.parametrize("where", ["device", "pinned_host"])
@pytest.mark.parametrize("dt", [0, 1])
def test_unpack_bit_exact_vs_oracle(dt, where):
    """GPU unpack (from a device buffer, or from pinned host memory) equals
    oracle.unpack of the same packed bytes, byte for byte over the whole
    destination pool: the written pages with their tail slots (NaN-poisoned
    at the source), the pages left alone, and the fp8 page scales."""
    print(f"[case] unpack vs oracle dt={dt} {where}", flush=True)
    d = lib()
    P = 16 if dt == 0 else 32
    lens = np.array([700, 33, 1, 130, 64], np.int32)
    Hkv, D = 4, 128
    w = wl.Workload("up", len(lens), 16, Hkv, D, P, dt, 512, "uniform", lo=1, hi=1)
    b = gpu_batch(w, lengths=lens, seed_index=24 + dt)
    n = wl.pages_needed(lens, P)
    src = np.concatenate([b.block_table_h[i, :n[i]] for i in range(len(lens))]).astype(np.int32)
    version = 1
    packed = _pack(b, src, version)
    if where == "pinned_host":
        host = torch.empty(packed.numel(), dtype=torch.uint8, pin_memory=True)
        host.copy_(packed.cpu())
        packed = host
    # destination pool: another geometry-equal pool filled with random bytes
    g = torch.Generator(device="cuda").manual_seed(1234 + dt)
    nb = w.num_pages
    dst_k = torch.randint(0, 256, (b.k_pages.numel() * b.k_pages.element_size(),),
                          generator=g, device="cuda", dtype=torch.uint8)
    dst_v = torch.randint(0, 256, (b.v_pages.numel() * b.v_pages.element_size(),),
                          generator=g, device="cuda", dtype=torch.uint8)
    dst_k = dst_k.view(b.k_pages.dtype).view(b.k_pages.shape)
    dst_v = dst_v.view(b.v_pages.dtype).view(b.v_pages.shape)
    dst_ks = dst_vs = None
    if dt:
        dst_ks = torch.rand(nb, generator=g, device="cuda", dtype=torch.float32)
        dst_vs = torch.rand(nb, generator=g, device="cuda", dtype=torch.float32)
    dst_pages = np.random.default_rng(7 + dt).permutation(nb)[:len(src)].astype(np.int32)
    expected = _oracle_unpack_expected(
        _host_pool(packed), dst_pages, _host_pool(dst_k), _host_pool(dst_v),
        None if dst_ks is None else _host_pool(dst_ks),
        None if dst_vs is None else _host_pool(dst_vs), dt=dt, P=P, Hkv=Hkv, d=D,
        version=version)
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    d.dora_kv_page_unpack(packed, torch.from_numpy(dst_pages).cuda(), dst_k, dst_v,
                          src_version=version, num_kv_heads=Hkv, page_size=P, head_dim=D,
                          kv_dtype=dt, policy_version=version, k_scales=dst_ks,
                          v_scales=dst_vs, dev_status=status)
    torch.cuda.synchronize()
    assert status.item() == d.DORA_OK
    _assert_pools_equal_oracle(dst_k, dst_v, dst_ks, dst_vs, expected)


@pytest.mark.parametrize("dt", [0, 1])
def test_migration_preserves_decode_bitwise(dt):
    """Two same-version instances (two host pools over two device pools):
    migrate sequences with pack -> unpack; decode on the destination equals
    decode on the source bit for bit."""
    d = lib()
    P = 16 if dt == 0 else 32
    lens = np.array([1500, 40, 3, 2222], np.int32)
    w = wl.Workload("m", 4, 16, 4, 128, P, dt, 1024, "uniform", lo=1, hi=1)
    src_pool = d.Pool(w.num_pages, P, 3, seed=11)
    dst_pool = d.Pool(w.num_pages, P, 3, seed=99)
    version = 1
    ids = [src_pool.add_seq(version, int(L)) for L in lens]
    bt, lens_h, vers = src_pool.block_table(ids)
    b = gpu_batch(w, lengths=lens, seed_index=30 + dt)
    # re-home the generated pages at the host pool's placement
    old = b.block_table_h
    k2 = torch.zeros_like(b.k_pages)
    v2 = torch.zeros_like(b.v_pages)
    n = wl.pages_needed(lens, P)
    for i in range(4):
        k2[torch.from_numpy(bt[i, :n[i]].astype(np.int64)).cuda()] = \
            b.k_pages[torch.from_numpy(old[i, :n[i]].astype(np.int64)).cuda()]
        v2[torch.from_numpy(bt[i, :n[i]].astype(np.int64)).cuda()] = \
            b.v_pages[torch.from_numpy(old[i, :n[i]].astype(np.int64)).cuda()]
    if dt:
        ks2 = torch.ones_like(b.k_scales)
        vs2 = torch.ones_like(b.v_scales)
        for i in range(4):
            ks2[torch.from_numpy(bt[i, :n[i]].astype(np.int64)).cuda()] = \
                b.k_scales[torch.from_numpy(old[i, :n[i]].astype(np.int64)).cuda()]
            vs2[torch.from_numpy(bt[i, :n[i]].astype(np.int64)).cuda()] = \
                b.v_scales[torch.from_numpy(old[i, :n[i]].astype(np.int64)).cuda()]
        b.k_scales, b.v_scales = ks2, vs2
    b.k_pages, b.v_pages = k2, v2
    b.block_table = torch.from_numpy(bt).cuda()
    b.version_ids = torch.from_numpy(vers).cuda()
    before = run_decode(b).clone()

    # migrate every sequence to the destination instance
    dst_k = torch.zeros_like(b.k_pages)
    dst_v = torch.zeros_like(b.v_pages)
    dst_ks = torch.zeros_like(b.k_scales) if dt else None
    dst_vs = torch.zeros_like(b.v_scales) if dt else None
    new_ids = []
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    for sid in ids:
        nid, sp, dp = src_pool.migrate_seq(sid, dst_pool, version)
        packed = _pack(b, sp, version)
        # what the oracle's unpack makes of the same bytes and the same pool
        expected = _oracle_unpack_expected(
            _host_pool(packed), dp, _host_pool(dst_k), _host_pool(dst_v),
            None if dst_ks is None else _host_pool(dst_ks),
            None if dst_vs is None else _host_pool(dst_vs), dt=dt, P=P, Hkv=4, d=128,
            version=version)
        d.dora_kv_page_unpack(packed, torch.from_numpy(dp).cuda(), dst_k, dst_v,
                              src_version=version, num_kv_heads=4, page_size=P, head_dim=128,
                              kv_dtype=dt, policy_version=version, k_scales=dst_ks,
                              v_scales=dst_vs, dev_status=status)
        torch.cuda.synchronize()
        assert status.item() == d.DORA_OK
        _assert_pools_equal_oracle(dst_k, dst_v, dst_ks, dst_vs, expected)
        src_pool.free_seq(sid)
        new_ids.append(nid)
    bt2, lens2, vers2 = dst_pool.block_table(new_ids, stride=bt.shape[1])
    assert np.array_equal(lens2, lens_h) and np.array_equal(vers2, vers)
    b.k_pages, b.v_pages = dst_k, dst_v
    if dt:
        b.k_scales, b.v_scales = dst_ks, dst_vs
    b.block_table = torch.from_numpy(bt2).cuda()
    after = run_decode(b)
    assert torch.equal(after, before)
    assert src_pool.stats(version)[0] == 0


def test_unpack_rejects_other_version_and_bad_header():
    d = lib()
    lens = np.array([64, 20], np.int32)
    w = wl.Workload("u", 2, 8, 2, 64, 16, 0, 64, "uniform", lo=1, hi=1)
    b = gpu_batch(w, lengths=lens, seed_index=40)
    src = np.concatenate([b.block_table_h[0, :4], b.block_table_h[1, :2]]).astype(np.int32)
    packed = _pack(b, src, version=0)
    dst = torch.arange(6, dtype=torch.int32, device="cuda") + 50
    k = torch.zeros_like(b.k_pages)
    v = torch.zeros_like(b.v_pages)
    # host-side: the request's version differs from the destination's
    with pytest.raises(d.DoraError) as e:
        d.dora_kv_page_unpack(packed, dst, k, v, src_version=0, num_kv_heads=2, page_size=16,
                              head_dim=64, policy_version=1)
    assert e.value.status == d.DORA_ERR_VERSION_MISMATCH
    # device-side: the buffer's header says version 0, the caller claims 1 -> nothing written
    st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    d.dora_kv_page_unpack(packed, dst, k, v, src_version=1, num_kv_heads=2, page_size=16,
                          head_dim=64, policy_version=1, dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == d.DORA_ERR_VERSION_MISMATCH
    assert not k.any() and not v.any()
    # corrupted magic -> invalid argument, nothing written
    bad = packed.clone()
    bad[0] ^= 0xFF
    d.dora_kv_page_unpack(bad, dst, k, v, src_version=0, num_kv_heads=2, page_size=16,
                          head_dim=64, policy_version=0, dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == d.DORA_ERR_INVALID_ARG
    assert not k.any() and not v.any()


def test_pack_multi_version_workload_32_seqs():
    """The multi-version workload's 32-sequence pack, bit-exact vs the oracle."""
    w = wl.WORKLOADS[3]
    print(f"[case] pack {w.name}", flush=True)
    b = gpu_batch(w, seed_index=3)
    rng = np.random.default_rng(5)
    version = 0
    cand = np.nonzero(b.versions_h == version)[0]
    seqs = np.sort(rng.choice(cand, size=32, replace=False))
    n = wl.pages_needed(b.lengths, w.page_size)
    src = np.concatenate([b.block_table_h[s, :n[s]] for s in seqs]).astype(np.int32)
    packed = _pack(b, src, version)
    idx = torch.from_numpy(src.astype(np.int64)).cuda()
    kc = _host_codes(b.k_pages.index_select(0, idx))
    vc = _host_codes(b.v_pages.index_select(0, idx))
    ref = oracle.pack(kc, vc, np.arange(len(src), dtype=np.int32), kv_dtype=0, page_size=16,
                      num_kv_heads=8, head_dim=128, policy_version=version, n_seqs=3)
    got = packed.cpu().numpy()
    # the oracle saw a compacted pool holding the same pages; the buffers match whole
    assert np.array_equal(got, ref)
    # unpack the set into a fresh destination pool of its own (the full pool is
    # 64 GiB, too large to compare on the host), at scattered pages, against
    # oracle.unpack of the same bytes
    nd = len(src) + 1024
    dst_k = torch.full((nd,) + tuple(b.k_pages.shape[1:]), 3.0, dtype=b.k_pages.dtype,
                       device="cuda")
    dst_v = torch.full((nd,) + tuple(b.v_pages.shape[1:]), -5.0, dtype=b.v_pages.dtype,
                       device="cuda")
    dst_pages = np.random.default_rng(8).permutation(nd)[:len(src)].astype(np.int32)
    expected = _oracle_unpack_expected(ref, dst_pages, _host_pool(dst_k), _host_pool(dst_v),
                                       None, None, dt=0, P=16, Hkv=8, d=128, version=version)
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    lib().dora_kv_page_unpack(packed, torch.from_numpy(dst_pages).cuda(), dst_k, dst_v,
                              src_version=version, num_kv_heads=8, page_size=16, head_dim=128,
                              policy_version=version, dev_status=status)
    torch.cuda.synchronize()
    assert status.item() == 0
    _assert_pools_equal_oracle(dst_k, dst_v, None, None, expected)
    del b, dst_k, dst_v
    torch.cuda.empty_cache()


def test_pack_unpack_random_geometries_bit_exact():
    """20 seeded random geometries (dtype, page size, 1-8 KV heads, head dim,
    1-12 sequences of random lengths, the page list in a random order, pages
    unpacked to random distinct ids of a pool of random bytes): the packed
    buffer equals oracle.pack byte for byte, and the destination pool after
    the unpack equals oracle.unpack's."""
    d = lib()
    rng = np.random.default_rng(9090)
    for case in range(20):
        dt = int(rng.integers(0, 2))
        P = int(rng.choice([16, 32]))
        Hkv = int(rng.integers(1, 9))
        D = int(rng.choice([64, 128]))
        B = int(rng.integers(1, 13))
        lens = rng.integers(1, 1500, B).astype(np.int32)
        n = wl.pages_needed(lens, P)
        nb = int(n.sum()) * 2 + 16
        print(f"[case {case}] pack/unpack dt={dt} P={P} Hkv={Hkv} d={D} B={B} pages={n.sum()}",
              flush=True)
        w = wl.Workload("pr", B, Hkv, Hkv, D, P, dt, nb, "uniform", lo=1, hi=1)
        b = gpu_batch(w, lengths=lens, seed_index=3000 + case)
        src = np.concatenate([b.block_table_h[i, :n[i]] for i in range(B)]).astype(np.int32)
        src = src[rng.permutation(len(src))]
        version = int(rng.integers(0, 3))
        packed = _pack(b, src, version)
        ks_h = None if dt == 0 else b.k_scales.cpu().numpy()
        vs_h = None if dt == 0 else b.v_scales.cpu().numpy()
        ref = oracle.pack(_host_codes(b.k_pages), _host_codes(b.v_pages), src, kv_dtype=dt,
                          page_size=P, num_kv_heads=Hkv, head_dim=D, policy_version=version,
                          n_seqs=3, k_scales=ks_h, v_scales=vs_h)
        assert np.array_equal(packed.cpu().numpy(), ref), case
        g = torch.Generator(device="cuda").manual_seed(7000 + case)
        dst_k = torch.randint(0, 256, (b.k_pages.numel() * b.k_pages.element_size(),),
                              generator=g, device="cuda", dtype=torch.uint8)
        dst_v = torch.randint(0, 256, (b.v_pages.numel() * b.v_pages.element_size(),),
                              generator=g, device="cuda", dtype=torch.uint8)
        dst_k = dst_k.view(b.k_pages.dtype).view(b.k_pages.shape)
        dst_v = dst_v.view(b.v_pages.dtype).view(b.v_pages.shape)
        dst_ks = dst_vs = None
        if dt:
            dst_ks = torch.rand(nb, generator=g, device="cuda", dtype=torch.float32)
            dst_vs = torch.rand(nb, generator=g, device="cuda", dtype=torch.float32)
        dst_pages = rng.permutation(nb)[:len(src)].astype(np.int32)
        expected = _oracle_unpack_expected(
            _host_pool(packed), dst_pages, _host_pool(dst_k), _host_pool(dst_v),
            None if dst_ks is None else _host_pool(dst_ks),
            None if dst_vs is None else _host_pool(dst_vs), dt=dt, P=P, Hkv=Hkv, d=D,
            version=version)
        status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        d.dora_kv_page_unpack(packed, torch.from_numpy(dst_pages).cuda(), dst_k, dst_v,
                              src_version=version, num_kv_heads=Hkv, page_size=P, head_dim=D,
                              kv_dtype=dt, policy_version=version, k_scales=dst_ks,
                              v_scales=dst_vs, dev_status=status)
        torch.cuda.synchronize()
        assert status.item() == d.DORA_OK, case
        _assert_pools_equal_oracle(dst_k, dst_v, dst_ks, dst_vs, expected)
