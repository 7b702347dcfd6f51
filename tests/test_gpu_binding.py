"""GPU checks of the binding's own behaviour and of the measurement entry
points (include/dora_measure.h), through the C ABI:

* calls on two streams at once each get a workspace of their own, so two
  geometry-identical batches decoded concurrently give, bit for bit, what each
  gives alone (the header's no-shared-state contract, kept by the binding);
* the streaming-read reference reads exactly the tiles it is given: its
  per-wavefront checksums equal an XOR fold computed on the host.
"""
import numpy as np
import pytest
import torch

import workloads as wl
from gpu_util import gpu_batch, lib

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("grouped", [False, True])
def test_two_streams_do_not_share_a_workspace(grouped):
    print(f"[case] two streams grouped={grouped}", flush=True)
    d = lib()
    w = wl.Workload("s", 32, 28, 4, 128, 16, 0, 8192, "lognormal", 900, 1.2, 16, 6000)
    if grouped:
        b1, _ = wl.make_grpo_batch(w, group_size=8, prompt_range=(64, 700), device="cuda",
                                   seed_index=61)
        b2, _ = wl.make_grpo_batch(w, group_size=8, prompt_range=(64, 700), device="cuda",
                                   seed_index=62)
    else:
        b1 = gpu_batch(w, seed_index=61)
        b2 = gpu_batch(w, seed_index=62, lengths=b1.lengths[::-1].copy())
    # one block-table stride for both (entries past a sequence's pages are
    # never read): same geometry, so the same workspace size
    stride = max(b1.stride, b2.stride)
    for b in (b1, b2):
        pad = stride - b.stride
        if pad:
            b.block_table_h = np.pad(b.block_table_h, ((0, 0), (0, pad)))
            b.block_table = torch.from_numpy(b.block_table_h).cuda()
    assert b1.stride == b2.stride

    def call(b, out, stream):
        kw = dict(num_kv_heads=w.num_kv_heads, page_size=w.page_size, stream=stream)
        if grouped:
            d.dora_decode_attn_grouped(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                                       b.version_ids, out, group_size=8, **kw)
        else:
            d.dora_decode_attn(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                               b.version_ids, out, **kw)

    ref = []
    for b in (b1, b2):
        o = torch.empty_like(b.q)
        call(b, o, None)
        torch.cuda.synchronize()
        ref.append(o)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for rep in range(6):
        outs = [torch.empty_like(b1.q), torch.empty_like(b2.q)]
        cur = torch.cuda.current_stream()
        s1.wait_stream(cur)
        s2.wait_stream(cur)
        for _ in range(3):   # several calls in flight on each stream
            with torch.cuda.stream(s1):
                call(b1, outs[0], s1)
            with torch.cuda.stream(s2):
                call(b2, outs[1], s2)
        torch.cuda.synchronize()
        for o, r in zip(outs, ref):
            assert torch.equal(o.view(torch.int16), r.view(torch.int16)), rep


@pytest.mark.parametrize("tile,tpb", [(1024, 16), (1024, 1), (4096, 1), (4096, 4), (16384, 1)])
def test_stream_read_checksums(tile, tpb):
    print(f"[case] stream read tile={tile} tiles per batch={tpb}", flush=True)
    d = lib()
    nbytes = 32 << 20
    g = torch.Generator(device="cuda").manual_seed(tile)
    buf = torch.randint(0, 256, (nbytes,), generator=g, dtype=torch.uint8, device="cuda")
    n_all = nbytes // tile
    rng = np.random.default_rng(tile)
    ids = rng.integers(0, n_all, size=777).astype(np.int32)
    ids[5] = n_all          # outside the buffer: skipped
    ids[100] = -2           # negative: skipped
    waves = 37
    sink = torch.full((waves,), 0x5A5A, dtype=torch.int32, device="cuda")
    d.dora_stream_read(buf, torch.from_numpy(ids).cuda(), sink, tile_bytes=tile,
                       tiles_per_batch=tpb)
    torch.cuda.synchronize()
    words = buf.cpu().numpy().view(np.uint32).reshape(n_all, tile // 4)
    q, rem = divmod(len(ids), waves)
    want = []
    for w_ in range(waves):
        t0 = w_ * q + min(w_, rem)
        t1 = t0 + q + (1 if w_ < rem else 0)
        x = np.uint32(0)
        for t in range(t0, t1):
            if 0 <= ids[t] < n_all:
                x ^= np.bitwise_xor.reduce(words[ids[t]])
        want.append(int(x))
    got = sink.cpu().numpy().view(np.uint32).tolist()
    assert got == want


def test_stream_read_empty_list_and_bad_args():
    d = lib()
    buf = torch.zeros(1 << 16, dtype=torch.uint8, device="cuda")
    sink = torch.full((5,), 9, dtype=torch.int32, device="cuda")
    d.dora_stream_read(buf, torch.zeros(0, dtype=torch.int32, device="cuda"), sink)
    torch.cuda.synchronize()
    assert sink.tolist() == [0] * 5
    with pytest.raises(d.DoraError) as e:
        d.dora_stream_read(buf, torch.zeros(4, dtype=torch.int32, device="cuda"), sink,
                           tile_bytes=3000)
    assert e.value.status == d.DORA_ERR_UNSUPPORTED



@pytest.mark.parametrize("kv_dtype", [0, 1])
def test_prepared_decode_follows_in_place_updates(kv_dtype):
    """A prepared call gives, bit for bit, what dora_decode_attn gives on the
    same buffers, also after the queries and lengths are refilled in place
    (lengths anywhere from 0 to their pages' capacity), and matches the
    oracle on the last refill."""
    print(f"[case] prepared decode kv_dtype={kv_dtype}", flush=True)
    from gpu_util import max_abs_err, oracle_for
    d = lib()
    P = 16 if kv_dtype == 0 else 32
    w = wl.Workload("p", 24, 16, 2, 128, P, kv_dtype, 8192, "lognormal", 600, 1.0, 16, 4000)
    b = gpu_batch(w, seed_index=71, poison=False)
    kw = dict(num_kv_heads=w.num_kv_heads, page_size=w.page_size, kv_dtype=w.kv_dtype,
              k_scales=b.k_scales, v_scales=b.v_scales)
    out = torch.empty_like(b.q)
    prep = d.PreparedDecode(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                            b.version_ids, out, **kw)
    capacity = ((b.lengths + P - 1) // P) * P  # tokens the sequences' pages hold
    rng = np.random.default_rng(71)
    gen = torch.Generator(device="cuda").manual_seed(71)
    for step in range(4):
        if step:
            b.q.copy_(torch.randn(b.q.shape, generator=gen, device="cuda").to(torch.bfloat16))
            b.lengths = rng.integers(0, capacity + 1).astype(np.int32)
            b.lengths[0] = 0
            b.seq_lens.copy_(torch.from_numpy(b.lengths).cuda())
        ref = torch.empty_like(b.q)
        d.dora_decode_attn(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                           b.version_ids, ref, **kw)
        assert prep() is out
        torch.cuda.synchronize()
        assert torch.equal(out, ref), step
    err = max_abs_err(out, oracle_for(b))
    print(f"[case] prepared decode: max-abs err {err:.3e}", flush=True)
    assert err <= (2e-2 if kv_dtype == 0 else 5e-2)
    empty = d.PreparedDecode(b.q[:0], b.k_pages, b.v_pages, b.block_table[:0], b.seq_lens[:0],
                             b.version_ids[:0], out[:0], **kw)
    assert empty().numel() == 0
