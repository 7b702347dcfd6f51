"""dora_decode_attn_noalloc through the C ABI: the decode call whose workspace
is the library's fixed per-GPU array.  Two calls in a row, the second on a
smaller batch of another geometry, each equal bit for bit to dora_decode_attn
on the same inputs (same launch, same arithmetic) and within the oracle
tolerance; sizes beyond the array and the VALIDATE flag are refused before any
launch; the calls allocate no device memory, and a call captured in a HIP
graph replays equal to the eager call."""
import numpy as np
import pytest
import torch

import workloads as wl
from gpu_util import TOL, gpu_batch, lib, max_abs_err, oracle_for, run_decode

pytestmark = pytest.mark.gpu


def _noalloc(b, out=None, **kw):
    d = lib()
    if out is None:
        out = torch.empty_like(b.q)
    d.dora_decode_attn_noalloc(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                               b.version_ids, out, num_kv_heads=b.w.num_kv_heads,
                               page_size=b.w.page_size, kv_dtype=b.w.kv_dtype,
                               k_scales=b.k_scales, v_scales=b.v_scales, **kw)
    torch.cuda.synchronize()
    return out


def test_noalloc_equals_decode_twice_second_smaller():
    # first: fp8 pages, 64 query / 8 KV heads, 32-token pages, long-tailed lengths
    w1 = wl.Workload("na1", 96, 64, 8, 128, 32, 1, 16384, "lognormal", 1500, 1.2, 16, 20000)
    b1 = gpu_batch(w1, seed_index=91)
    print(f"[case] noalloc call 1: {w1.num_seqs} seqs fp8", flush=True)
    ref1 = run_decode(b1).clone()
    out1 = _noalloc(b1, out=torch.full_like(b1.q, 9.0))
    assert torch.equal(out1.view(torch.int16), ref1.view(torch.int16))
    seqs = [0, int(np.argmax(b1.lengths)), 95]
    assert max_abs_err(out1, oracle_for(b1, seqs), seqs) <= TOL[1]
    # second: a smaller bf16 batch of another geometry, right after
    lens = np.array([1, 0, 33, 700, 16, 4097], np.int32)
    w2 = wl.Workload("na2", len(lens), 8, 2, 64, 16, 0, 1024, "uniform", lo=1, hi=1)
    b2 = gpu_batch(w2, lengths=lens, seed_index=92)
    print(f"[case] noalloc call 2: {w2.num_seqs} seqs bf16", flush=True)
    ref2 = run_decode(b2).clone()
    out2 = _noalloc(b2, out=torch.full_like(b2.q, 9.0))
    assert torch.equal(out2.view(torch.int16), ref2.view(torch.int16))
    assert max_abs_err(out2, oracle_for(b2)) <= TOL[0]


def test_noalloc_refuses_oversized_workspace_and_validate():
    d = lib()
    lens = np.array([300, 40], np.int32)
    w = wl.Workload("na3", 2, 64, 4, 128, 16, 0, 256, "uniform", lo=1, hi=1)
    b = gpu_batch(w, lengths=lens, seed_index=93)
    sentinel = torch.full_like(b.q, 5.0)
    out = sentinel.clone()
    with pytest.raises(d.DoraError) as e:
        _noalloc(b, out=out, num_waves=200000)     # ~3.3 GB of partials
    assert e.value.status == d.DORA_ERR_WORKSPACE_TOO_SMALL
    with pytest.raises(d.DoraError) as e:
        _noalloc(b, out=out, flags=d.DORA_FLAG_VALIDATE)
    assert e.value.status == d.DORA_ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert torch.equal(out, sentinel)


def test_noalloc_allocates_no_device_memory():
    lens = np.array([5000, 3, 900, 129], np.int32)
    w = wl.Workload("na4", len(lens), 28, 4, 128, 16, 0, 2048, "uniform", lo=1, hi=1)
    b = gpu_batch(w, lengths=lens, seed_index=94)
    out = torch.empty_like(b.q)
    _noalloc(b, out=out)                            # first call on the device: address lookup
    free0 = torch.cuda.mem_get_info()[0]
    for _ in range(5):
        _noalloc(b, out=out)
    assert torch.cuda.mem_get_info()[0] == free0
    assert torch.equal(out.view(torch.int16), run_decode(b).view(torch.int16))


def test_noalloc_captures_in_a_graph_and_replays_equal_eager():
    """The callers this entry point is for include code under HIP graph
    capture: one call captured after a first eager call on the device (which
    looks the array's address up), then replayed with new queries copied into
    the captured buffer; every replay equals dora_decode_attn on the same
    inputs bit for bit, with eager work and a synchronisation between
    replays."""
    d = lib()
    lens = np.array([2000, 1, 0, 517, 64, 3000, 16, 95], np.int32)
    w = wl.Workload("na5", len(lens), 32, 4, 128, 16, 0, 2048, "uniform", lo=1, hi=1)
    b = gpu_batch(w, lengths=lens, seed_index=95)
    kw = dict(num_kv_heads=w.num_kv_heads, page_size=w.page_size, kv_dtype=w.kv_dtype,
              k_scales=b.k_scales, v_scales=b.v_scales)
    q_s, out_g = b.q.clone(), torch.empty_like(b.q)
    _noalloc(b, out=out_g)                         # eager first call on the device
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            d.dora_decode_attn_noalloc(q_s, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                                       b.version_ids, out_g, **kw)
    torch.cuda.current_stream().wait_stream(s)
    gen = torch.Generator(device="cuda").manual_seed(96)
    for rep in range(3):
        print(f"[case] noalloc graph replay {rep}", flush=True)
        q_new = torch.randn(b.q.shape, generator=gen, device="cuda").to(torch.bfloat16)
        q_s.copy_(q_new)
        out_g.fill_(7.0)
        g.replay()
        torch.cuda.synchronize()
        out_e = torch.empty_like(b.q)
        d.dora_decode_attn(q_new, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                           b.version_ids, out_e, **kw)
        torch.cuda.synchronize()
        assert torch.equal(out_g.view(torch.int16), out_e.view(torch.int16)), rep
