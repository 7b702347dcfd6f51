"""Offload to host memory and restore (through the C ABI): pack straight into
pinned host memory and unpack from it, the hierarchical memory management of
Sec. 3.4.  Bar: the host buffer is byte-identical to the oracle's pack, and a
sequence offloaded, evicted and restored into other pages decodes bit for bit
as before."""
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


def _raw(t: torch.Tensor) -> np.ndarray:
    """Host copy of a device pool as raw bytes."""
    return t.contiguous().cpu().view(torch.uint8).numpy().copy() if t.dtype != torch.uint8 \
        else t.cpu().numpy().copy()


def _geo(w):
    return dict(num_kv_heads=w.num_kv_heads, page_size=w.page_size, head_dim=w.head_dim,
                kv_dtype=w.kv_dtype)


def _packed_bytes(d, w, n):
    desc = d.make_pack_desc(kv_dtype=w.kv_dtype, page_size=w.page_size,
                            num_kv_heads=w.num_kv_heads, head_dim=w.head_dim,
                            num_pages=w.num_pages, policy_version=0)
    return d.dora_kv_packed_bytes(desc, n)


@pytest.mark.parametrize("dt", [0, 1])
def test_pack_to_pinned_host_matches_oracle(dt):
    d = lib()
    P = 16 if dt == 0 else 32
    lens = np.array([300, 17, 1, 900], np.int32)
    w = wl.Workload("o", 4, 16, 4, 128, P, dt, 512, "uniform", lo=1, hi=1)
    b = gpu_batch(w, lengths=lens, seed_index=70 + dt)
    n = wl.pages_needed(lens, P)
    src = np.concatenate([b.block_table_h[i, :n[i]] for i in range(4)]).astype(np.int32)
    host = torch.empty(_packed_bytes(d, w, len(src)), dtype=torch.uint8, pin_memory=True)
    host.fill_(0xA5)
    d.dora_kv_page_pack(b.k_pages, b.v_pages, torch.from_numpy(src).cuda(), host,
                        policy_version=3, n_seqs=4, k_scales=b.k_scales, v_scales=b.v_scales,
                        **_geo(w))
    torch.cuda.synchronize()
    ref = oracle.pack(_host_codes(b.k_pages), _host_codes(b.v_pages), src, kv_dtype=dt,
                      page_size=P, num_kv_heads=4, head_dim=128, policy_version=3, n_seqs=4,
                      k_scales=None if dt == 0 else b.k_scales.cpu().numpy(),
                      v_scales=None if dt == 0 else b.v_scales.cpu().numpy())
    assert np.array_equal(host.numpy(), ref)


@pytest.mark.parametrize("dt", [0, 1])
def test_offload_evict_restore_decodes_bitwise(dt):
    """Offload two sequences to host memory, overwrite their device pages (the
    pool reuses them), restore into other free pages and rewrite the block
    table: decode is bitwise unchanged."""
    d = lib()
    P = 16 if dt == 0 else 32
    lens = np.array([1200, 5, 640, 77, 2048], np.int32)
    w = wl.Workload("r", 5, 16, 4, 128, P, dt, 1024, "uniform", lo=1, hi=1)
    b = gpu_batch(w, lengths=lens, seed_index=80 + dt)
    before = run_decode(b).clone()
    n = wl.pages_needed(lens, P)
    moved = [0, 2]
    src = np.concatenate([b.block_table_h[i, :n[i]] for i in moved]).astype(np.int32)
    host = torch.empty(_packed_bytes(d, w, len(src)), dtype=torch.uint8, pin_memory=True)
    d.dora_kv_page_pack(b.k_pages, b.v_pages, torch.from_numpy(src).cuda(), host,
                        policy_version=0, n_seqs=len(moved), k_scales=b.k_scales,
                        v_scales=b.v_scales, **_geo(w))
    torch.cuda.synchronize()
    # eviction: the pages are reused by someone else
    idx = torch.from_numpy(src.astype(np.int64)).cuda()
    b.k_pages[idx] = b.k_pages[idx].flip(0)
    b.v_pages[idx] = b.v_pages[idx].flip(0)
    if dt:
        b.k_scales[idx] = 7.0
        b.v_scales[idx] = 7.0
    # restore into free pages
    free = np.setdiff1d(np.arange(w.num_pages), b.used_pages)[:len(src)].astype(np.int32)
    # oracle.unpack of the same host bytes into host copies of the pool as it is now
    kp, vp = _raw(b.k_pages), _raw(b.v_pages)
    ks = b.k_scales.cpu().numpy().copy() if dt else None
    vs = b.v_scales.cpu().numpy().copy() if dt else None
    assert oracle.unpack(host.numpy(), free, kp, vp, kv_dtype=dt, page_size=P,
                         num_kv_heads=4, head_dim=128, policy_version=0, k_scales=ks,
                         v_scales=vs) == 0
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    d.dora_kv_page_unpack(host, torch.from_numpy(free).cuda(), b.k_pages, b.v_pages,
                          src_version=0, policy_version=0, k_scales=b.k_scales,
                          v_scales=b.v_scales, dev_status=status, **_geo(w))
    torch.cuda.synchronize()
    assert status.item() == d.DORA_OK
    # the restored pool equals the oracle's byte for byte (tail slots included)
    assert np.array_equal(_raw(b.k_pages), kp) and np.array_equal(_raw(b.v_pages), vp)
    if dt:
        assert np.array_equal(b.k_scales.cpu().numpy().view(np.uint32), ks.view(np.uint32))
        assert np.array_equal(b.v_scales.cpu().numpy().view(np.uint32), vs.view(np.uint32))
    bt = b.block_table_h.copy()
    off = 0
    for i in moved:
        bt[i, :n[i]] = free[off:off + n[i]]
        off += n[i]
    b.block_table = torch.from_numpy(bt).cuda()
    assert torch.equal(run_decode(b), before)


def test_unpack_from_pinned_host_checks_the_header():
    d = lib()
    lens = np.array([64, 20], np.int32)
    w = wl.Workload("h", 2, 8, 2, 64, 16, 0, 64, "uniform", lo=1, hi=1)
    b = gpu_batch(w, lengths=lens, seed_index=90)
    n = wl.pages_needed(lens, 16)
    src = np.concatenate([b.block_table_h[i, :n[i]] for i in range(2)]).astype(np.int32)
    host = torch.empty(_packed_bytes(d, w, len(src)), dtype=torch.uint8, pin_memory=True)
    d.dora_kv_page_pack(b.k_pages, b.v_pages, torch.from_numpy(src).cuda(), host,
                        policy_version=0, **_geo(w))
    torch.cuda.synchronize()
    host[0] ^= 0xFF                                 # corrupt the magic
    k0 = b.k_pages.clone()
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    d.dora_kv_page_unpack(host, torch.from_numpy(src).cuda(), b.k_pages, b.v_pages,
                          src_version=0, policy_version=0, dev_status=status, **_geo(w))
    torch.cuda.synchronize()
    assert status.item() != d.DORA_OK
    assert torch.equal(b.k_pages.view(torch.int16), k0.view(torch.int16))  # bits: tails are NaN
    with pytest.raises(ValueError):
        d.dora_kv_page_pack(b.k_pages, b.v_pages, torch.from_numpy(src).cuda(),
                            torch.empty(host.numel(), dtype=torch.uint8), policy_version=0,
                            **_geo(w))
