"""CPU checks of the C ABI: the library loads, exports every symbol the header
declares, and rejects bad arguments before any launch (no GPU is touched:
every call here returns during host-side validation)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", f) for f in sorted(os.listdir(os.path.join(ROOT,
                                                                                "include")))
           if f.endswith(".h")]


@pytest.fixture(scope="module")
def d():
    from paper_2604_26256_amd import build as B
    if not os.path.exists(B.LIB):
        B.build()
    from paper_2604_26256_amd import dora
    return dora


def _declared_functions():
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names.update(re.findall(r"\b(dora_[a-z0-9_]+)\s*\(", src))
    return sorted(names)


def test_exports_every_declared_symbol(d):
    assert len(HEADERS) >= 2, HEADERS
    names = _declared_functions()
    assert len(names) >= 20, names
    for n in ("dora_decode_num_waves", "dora_decode_attn_timed", "dora_stream_read"):
        assert n in names
    lib = d.library()
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings(d):
    for code in range(9):
        s = d.status_string(code)
        assert s and s != "unknown status"
    assert d.status_string(99) == "unknown status"


def _desc(d, **kw):
    base = dict(num_seqs=4, num_q_heads=8, num_kv_heads=2, head_dim=128, page_size=16,
                block_table_stride=64, num_pages=1024)
    base.update(kw)
    return d.make_decode_desc(**base)


def test_workspace_bytes(d):
    ok = d.dora_decode_workspace_bytes(_desc(d))
    assert ok > 0 and ok % 256 == 0
    # the workspace scales with the decode wavefronts: no more than the batch
    # can use (B * Hkv * stride page-heads, 8 each), and no more than the
    # device's share once the batch is large
    big = d.dora_decode_workspace_bytes(_desc(d, num_seqs=400))
    assert ok < big == d.dora_decode_workspace_bytes(_desc(d, num_seqs=4000))
    assert d.dora_decode_workspace_bytes(_desc(d, num_q_heads=36, num_kv_heads=2)) == 0  # G=18
    assert d.dora_decode_workspace_bytes(_desc(d, head_dim=96)) == 0
    assert d.dora_decode_workspace_bytes(_desc(d, page_size=8)) == 0
    assert d.dora_decode_workspace_bytes(_desc(d, num_q_heads=7)) == 0       # not a multiple
    assert d.dora_decode_workspace_bytes(_desc(d, kv_dtype=5)) == 0
    # two partial slots per decode wavefront
    few = d.dora_decode_workspace_bytes(_desc(d, num_waves=10))
    many = d.dora_decode_workspace_bytes(_desc(d, num_waves=1000))
    assert many - few >= 990 * 2 * 4 * 128 * 4
    assert d.dora_decode_workspace_bytes(_desc(d, num_kv_heads=128, num_q_heads=128)) == 0
    assert d.dora_decode_workspace_bytes(_desc(d, block_table_stride=1 << 19)) == 0


FAKE = 0x10000  # aligned non-null stand-in; never dereferenced (calls fail validation)


def _call(d, desc, q=FAKE, k=FAKE, v=FAKE, bt=FAKE, lens=FAKE, vid=FAKE, out=FAKE, ws=FAKE,
          wsb=1 << 30):
    P = ctypes.c_void_p
    return d.library().dora_decode_attn(ctypes.byref(desc), P(q), P(k), P(v), P(bt), P(lens),
                                        P(vid), P(out), P(ws), wsb, None)


def test_decode_host_validation(d):
    assert _call(d, _desc(d, num_q_heads=7)) == d.DORA_ERR_INVALID_ARG
    assert _call(d, _desc(d, num_seqs=-1)) == d.DORA_ERR_INVALID_ARG
    assert _call(d, _desc(d, block_table_stride=0)) == d.DORA_ERR_INVALID_ARG
    assert _call(d, _desc(d, head_dim=96)) == d.DORA_ERR_UNSUPPORTED
    assert _call(d, _desc(d, num_q_heads=34, num_kv_heads=2)) == d.DORA_ERR_UNSUPPORTED
    assert _call(d, _desc(d, flags=0x80)) == d.DORA_ERR_INVALID_ARG
    assert _call(d, _desc(d, num_waves=-1)) == d.DORA_ERR_INVALID_ARG
    assert _call(d, _desc(d, min_range_pages=-2)) == d.DORA_ERR_INVALID_ARG
    assert _call(d, _desc(d, sm_scale=-1.0)) == d.DORA_ERR_INVALID_ARG
    assert _call(d, _desc(d), q=0) == d.DORA_ERR_INVALID_ARG
    assert _call(d, _desc(d), ws=0) == d.DORA_ERR_INVALID_ARG
    assert _call(d, _desc(d), out=FAKE + 2) == d.DORA_ERR_INVALID_ARG          # misaligned
    assert _call(d, _desc(d, kv_dtype=1)) == d.DORA_ERR_INVALID_ARG            # no fp8 scales
    need = d.dora_decode_workspace_bytes(_desc(d))
    assert _call(d, _desc(d), wsb=need - 1) == d.DORA_ERR_WORKSPACE_TOO_SMALL
    assert _call(d, _desc(d, num_seqs=0)) == d.DORA_OK                         # nothing to do
    assert d.library().dora_decode_attn(None, None, None, None, None, None, None, None, None, 0,
                                        None) == d.DORA_ERR_INVALID_ARG


def test_grouped_host_validation_and_workspace(d):
    lib = d.library()
    P = ctypes.c_void_p
    desc = _desc(d, num_seqs=8, num_q_heads=28, num_kv_heads=4)          # G = 7
    base = lib.dora_decode_grouped_workspace_bytes(ctypes.byref(desc), 4)
    assert base > d.dora_decode_workspace_bytes(desc)
    assert d.dora_decode_grouped_workspace_bytes(desc, 4) == base
    assert lib.dora_decode_grouped_workspace_bytes(ctypes.byref(desc), 3) == 0     # 8 % 3
    assert lib.dora_decode_grouped_workspace_bytes(ctypes.byref(desc), 0) == 0
    big = _desc(d, num_seqs=32, num_q_heads=28, num_kv_heads=4)
    assert lib.dora_decode_grouped_workspace_bytes(ctypes.byref(big), 32) == 0     # 32*7 cols

    def call(desc, M, **kw):
        a = dict(q=FAKE, k=FAKE, v=FAKE, bt=FAKE, lens=FAKE, out=FAKE, ws=FAKE)
        a.update(kw)
        return lib.dora_decode_attn_grouped(ctypes.byref(desc), P(a["q"]), P(a["k"]), P(a["v"]),
                                            P(a["bt"]), P(a["lens"]), None, P(a["out"]), M,
                                            None, P(a["ws"]), a.get("ws_bytes", 1 << 40), None)

    assert call(desc, 0) == d.DORA_ERR_INVALID_ARG
    assert call(desc, 3) == d.DORA_ERR_INVALID_ARG
    assert call(big, 32) == d.DORA_ERR_UNSUPPORTED
    assert call(desc, 4, q=0) == d.DORA_ERR_INVALID_ARG
    assert call(desc, 4, out=FAKE + 2) == d.DORA_ERR_INVALID_ARG
    assert call(desc, 4, ws_bytes=base - 1) == d.DORA_ERR_WORKSPACE_TOO_SMALL
    assert call(_desc(d, num_seqs=0), 4) == d.DORA_OK


def test_append_host_validation(d):
    P = ctypes.c_void_p
    lib = d.library()

    def call(desc, kn=FAKE, vn=FAKE, bt=FAKE, lens=FAKE, kp=FAKE, vp=FAKE, ks=FAKE, vs=FAKE):
        return lib.dora_kv_append(ctypes.byref(desc), P(kn), P(vn), P(bt), P(lens), None,
                                  P(kp), P(vp), P(ks), P(vs), None, None)

    assert call(_desc(d, head_dim=96)) == d.DORA_ERR_UNSUPPORTED
    assert call(_desc(d, page_size=8)) == d.DORA_ERR_UNSUPPORTED
    assert call(_desc(d, num_seqs=-1)) == d.DORA_ERR_INVALID_ARG
    assert call(_desc(d), kn=0) == d.DORA_ERR_INVALID_ARG
    assert call(_desc(d), kp=FAKE + 4) == d.DORA_ERR_INVALID_ARG              # misaligned
    assert call(_desc(d, kv_dtype=1), ks=0) == d.DORA_ERR_INVALID_ARG          # fp8, no scales
    assert call(_desc(d, num_seqs=0)) == d.DORA_OK                             # nothing to do
    assert lib.dora_kv_append(None, None, None, None, None, None, None, None, None, None, None,
                              None) == d.DORA_ERR_INVALID_ARG


def test_pack_host_validation_and_size(d):
    lib = d.library()
    for dt in (0, 1):
        desc = d.make_pack_desc(kv_dtype=dt, page_size=16, num_kv_heads=8, head_dim=128,
                                num_pages=100, policy_version=1)
        for n in (0, 1, 37):
            assert d.dora_kv_packed_bytes(desc, n) == oracle.packed_bytes(dt, 16, 8, 128, n)
    desc = d.make_pack_desc(kv_dtype=0, page_size=16, num_kv_heads=8, head_dim=128,
                            num_pages=100, policy_version=1)
    P = ctypes.c_void_p
    need = d.dora_kv_packed_bytes(desc, 3)
    assert lib.dora_kv_page_pack(ctypes.byref(desc), P(FAKE), P(FAKE), None, None, P(FAKE), 3,
                                 P(FAKE), need - 1, None) == d.DORA_ERR_WORKSPACE_TOO_SMALL
    assert lib.dora_kv_page_pack(ctypes.byref(desc), P(FAKE), P(FAKE), None, None, None, 3,
                                 P(FAKE), need, None) == d.DORA_ERR_INVALID_ARG
    assert lib.dora_kv_page_unpack(ctypes.byref(desc), 2, P(FAKE), need, P(FAKE), 3, P(FAKE),
                                   P(FAKE), None, None, None, None) == \
        d.DORA_ERR_VERSION_MISMATCH
    bad = d.make_pack_desc(kv_dtype=3, page_size=16, num_kv_heads=8, head_dim=128,
                           num_pages=100, policy_version=1)
    assert d.dora_kv_packed_bytes(bad, 1) == 0


# ---------------------------------------------------------------------------
# host page pool
# ---------------------------------------------------------------------------

def test_pool_alloc_free_and_ownership(d):
    pool = d.Pool(64, 16, 3, seed=0)
    a = pool.add_seq(0, 40)          # 3 pages
    b = pool.add_seq(2, 16)          # 1 page
    assert list(pool.seq_pages(a)) == [0, 1, 2] and list(pool.seq_pages(b)) == [3]
    assert pool.stats(0) == (3, 60) and pool.stats(2) == (1, 60) and pool.stats(-1) == (4, 60)
    own = pool.page_owner()
    assert list(own[:4]) == [0, 0, 0, 2] and (own[4:] == -1).all()
    pool.extend_seq(a, 49)           # 4 pages
    assert pool.seq_info(a) == (49, 0, 4)
    pool.free_seq(a)
    assert pool.stats(0) == (0, 63)
    assert (pool.page_owner() == np.array([-1, -1, -1, 2] + [-1] * 60)).all()
    with pytest.raises(d.DoraError) as e:
        pool.free_seq(a)
    assert e.value.status == d.DORA_ERR_NOT_FOUND


def test_pool_exhaustion_leaves_state_unchanged(d):
    pool = d.Pool(10, 16, 1, seed=5)
    a = pool.add_seq(0, 16 * 8)
    before = (pool.stats(0), pool.page_owner().copy())
    with pytest.raises(d.DoraError) as e:
        pool.add_seq(0, 16 * 3)
    assert e.value.status == d.DORA_ERR_POOL_EXHAUSTED
    with pytest.raises(d.DoraError):
        pool.extend_seq(a, 16 * 11)
    assert pool.stats(0) == before[0] and (pool.page_owner() == before[1]).all()
    assert pool.seq_info(a) == (128, 0, 8)


def test_pool_seeded_scatter_and_block_table(d):
    pool = d.Pool(4096, 16, 2, seed=1234)
    ids = [pool.add_seq(i % 2, L) for i, L in enumerate([1, 100, 2000, 17])]
    pages = np.concatenate([pool.seq_pages(i) for i in ids])
    assert len(np.unique(pages)) == len(pages)
    assert not np.array_equal(pages, np.arange(len(pages)))    # scattered
    table, lens, vers = pool.block_table(ids)
    assert table.shape == (4, 125) and list(lens) == [1, 100, 2000, 17]
    assert list(vers) == [0, 1, 0, 1]
    assert list(table[1, :7]) == list(pool.seq_pages(ids[1])) and not table[1, 7:].any()
    with pytest.raises(d.DoraError):
        pool.block_table(ids, stride=10)                        # sequence too long
    again = d.Pool(4096, 16, 2, seed=1234)
    ids2 = [again.add_seq(i % 2, L) for i, L in enumerate([1, 100, 2000, 17])]
    assert np.array_equal(np.concatenate([again.seq_pages(i) for i in ids2]), pages)


def test_pool_migration_rules(d):
    src = d.Pool(256, 16, 3, seed=3)
    dst = d.Pool(256, 16, 3, seed=4)
    s = src.add_seq(1, 300)
    with pytest.raises(d.DoraError) as e:
        src.migrate_seq(s, dst, 2)                          # other version
    assert e.value.status == d.DORA_ERR_VERSION_MISMATCH
    same, sp, dp = src.migrate_seq(s, src, 1)               # locality: nothing moves
    assert same == s and len(sp) == 0 and len(dp) == 0
    nid, sp, dp = src.migrate_seq(s, dst, 1)
    assert list(sp) == list(src.seq_pages(s)) and list(dp) == list(dst.seq_pages(nid))
    assert dst.seq_info(nid) == (300, 1, 19) and dst.stats(1)[0] == 19
    assert (dst.page_owner()[dp] == 1).all()


def test_num_waves_query(d):
    """The wave count the workspace is sized for: the caller's num_waves when
    set; otherwise no more than the batch can use (B * Hkv * stride page-heads
    over the 8-page minimum range) and at most 4 per CU for bf16 pages and 7
    for fp8 pages (with no device here the library assumes 256 CUs at 8
    resident waves each)."""
    assert d.dora_decode_num_waves(_desc(d, num_waves=77)) == 77
    small = _desc(d, num_seqs=2, num_kv_heads=2, num_q_heads=4, block_table_stride=8)
    assert d.dora_decode_num_waves(small) == 2 * 2 * 8 // 8
    assert d.dora_decode_num_waves(_desc(d, min_range_pages=1, num_seqs=2, num_kv_heads=2,
                                         num_q_heads=4, block_table_stride=8)) == 32
    big = d.dora_decode_num_waves(_desc(d, num_seqs=4000))
    assert big == 256 * 4
    assert d.dora_decode_num_waves(_desc(d, num_seqs=4000, kv_dtype=1)) == 256 * 7
    assert d.dora_decode_num_waves(_desc(d, head_dim=96)) == 0


def test_measure_entry_points_reject_bad_arguments(d):
    P = ctypes.c_void_p
    lib = d.library()
    desc = _desc(d)
    ev = (P * 3)(FAKE, FAKE, None)
    args = [P(FAKE)] * 7 + [P(FAKE), 1 << 30, None]
    assert lib.dora_decode_attn_timed(ctypes.byref(desc), *args, None) == d.DORA_ERR_INVALID_ARG
    assert lib.dora_decode_attn_timed(ctypes.byref(desc), *args,
                                      ctypes.cast(ev, P)) == d.DORA_ERR_INVALID_ARG
    bad = _desc(d, head_dim=96)
    ev_ok = (P * 3)(FAKE, FAKE, FAKE)
    assert lib.dora_decode_attn_timed(ctypes.byref(bad), *args,
                                      ctypes.cast(ev_ok, P)) == d.DORA_ERR_UNSUPPORTED
    sr = lib.dora_stream_read
    assert sr(None, 1 << 20, P(FAKE), 4, 4096, 4, P(FAKE), 8, None) == d.DORA_ERR_INVALID_ARG
    assert sr(P(FAKE), 1 << 20, P(FAKE), 4, 4096, 4, None, 8, None) == d.DORA_ERR_INVALID_ARG
    assert sr(P(FAKE), 1 << 20, P(FAKE), 4, 4096, 4, P(FAKE), 0, None) == d.DORA_ERR_INVALID_ARG
    assert sr(P(FAKE + 4), 1 << 20, P(FAKE), 4, 4096, 4, P(FAKE), 8, None) == \
        d.DORA_ERR_INVALID_ARG
    assert sr(P(FAKE), 1 << 20, None, 4, 4096, 4, P(FAKE), 8, None) == d.DORA_ERR_INVALID_ARG
    assert sr(P(FAKE), 1 << 20, P(FAKE), -1, 4096, 4, P(FAKE), 8, None) == \
        d.DORA_ERR_INVALID_ARG
    assert sr(P(FAKE), 1 << 20, P(FAKE), 4, 3072, 4, P(FAKE), 8, None) == d.DORA_ERR_UNSUPPORTED
    assert sr(P(FAKE), 1 << 20, P(FAKE), 4, 4096, 8, P(FAKE), 8, None) == d.DORA_ERR_UNSUPPORTED
    assert sr(P(FAKE), 1 << 20, P(FAKE), 4, 4096, 3, P(FAKE), 8, None) == d.DORA_ERR_UNSUPPORTED


def test_noalloc_entry_refuses_before_any_launch(d):
    """dora_decode_attn_noalloc: a workspace beyond its fixed array, the
    VALIDATE flag and invalid descriptors are refused on the host."""
    P = ctypes.c_void_p
    lib = d.library()
    args = [P(FAKE)] * 7 + [None]
    big = _desc(d, num_waves=200000)
    assert d.dora_decode_workspace_bytes(big) > d.NOALLOC_WORKSPACE_BYTES
    assert lib.dora_decode_attn_noalloc(ctypes.byref(big), *args) == \
        d.DORA_ERR_WORKSPACE_TOO_SMALL
    val = _desc(d, flags=d.DORA_FLAG_VALIDATE)
    assert lib.dora_decode_attn_noalloc(ctypes.byref(val), *args) == d.DORA_ERR_INVALID_ARG
    bad = _desc(d, head_dim=96)
    assert lib.dora_decode_attn_noalloc(ctypes.byref(bad), *args) == d.DORA_ERR_UNSUPPORTED
    assert lib.dora_decode_attn_noalloc(None, *args) == d.DORA_ERR_INVALID_ARG
    # every supported geometry fits at the default launch of a 256-CU part
    for hd in (64, 128):
        for dt in (0, 1):
            full = _desc(d, num_seqs=8192, num_q_heads=128, num_kv_heads=8, head_dim=hd,
                         kv_dtype=dt, block_table_stride=4096)
            assert 0 < d.dora_decode_workspace_bytes(full) <= d.NOALLOC_WORKSPACE_BYTES


def test_prepared_decode_checks_arguments_like_the_plain_call(d):
    """The prepared call runs the plain call's checks when it is made: host
    tensors, wrong dtypes and wrong page shapes are refused before anything
    reaches the library; an empty batch is a no-op."""
    import torch
    B, Hq, Hkv, D, P, n = 3, 8, 2, 128, 16, 32
    q = torch.zeros(B, Hq, D, dtype=torch.bfloat16)
    k = torch.zeros(n, Hkv, D // 8, P, 8, dtype=torch.bfloat16)
    v = torch.zeros(n, Hkv, D, P, dtype=torch.bfloat16)
    bt = torch.zeros(B, 4, dtype=torch.int32)
    lens = torch.ones(B, dtype=torch.int32)
    out = torch.empty_like(q)
    kw = dict(num_kv_heads=Hkv, page_size=P)
    for fn in (d.dora_decode_attn, d.PreparedDecode):
        with pytest.raises(ValueError, match="on the GPU"):
            fn(q, k, v, bt, lens, None, out, **kw)
        with pytest.raises(ValueError, match="v_pages must be"):
            fn(q, k, v[:, :, :64], bt, lens, None, out, **kw)
        with pytest.raises(ValueError, match="k_pages must be"):
            fn(q, k, v, bt, lens, None, out, num_kv_heads=Hkv, page_size=32)
    empty = d.PreparedDecode(q[:0], k, v, bt[:0], lens[:0], None, out[:0], **kw)
    assert empty() is not None and empty().numel() == 0
