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
        d.dora_kv_page_unpack(packed, torch.from_numpy(dp).cuda(), dst_k, dst_v,
                              src_version=version, num_kv_heads=4, page_size=P, head_dim=128,
                              kv_dtype=dt, policy_version=version, k_scales=dst_ks,
                              v_scales=dst_vs, dev_status=status)
        torch.cuda.synchronize()
        assert status.item() == d.DORA_OK
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
    del b
    torch.cuda.empty_cache()
