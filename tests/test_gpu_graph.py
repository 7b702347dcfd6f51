"""The decode loop's calls captured once in a HIP graph and replayed.

A serving loop captures its per-token work and replays it with new inputs
copied into the same buffers.  The library's entry points make no host round
trip, allocate nothing when given a workspace and record no memset, so they
capture as they are.  Each replay must equal, bit for bit, the same calls made
eagerly on a second copy of the state (same kernels, same launch shapes), and
the last step must still agree with the fp64 oracle.  Between replays the
test does eager work of its own and synchronises, so replays after the first
are checked under the conditions a loop creates.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from gpu_util import TOL, lib, max_abs_err, oracle_for

pytestmark = pytest.mark.gpu


def _codes(t, dt):
    t = t.contiguous().cpu()
    return t.view(torch.int16).numpy().view(np.uint16) if dt == 0 else t.numpy()


def _pool(num_pages, Hkv, d, P, dt, g):
    """A pool of N(0,1) keys and values (fp8: codes of N(0, 1/4), unit scales)."""
    X = wl.chunk_elems(dt)
    kshape, vshape = (num_pages, Hkv, d // X, P, X), (num_pages, Hkv, d, P)
    if dt == 0:
        k = torch.randn(kshape, generator=g).to(torch.bfloat16)
        v = torch.randn(vshape, generator=g).to(torch.bfloat16)
        return k.cuda(), v.cuda(), None, None
    k = (torch.randn(kshape, generator=g) * 0.5).to(torch.float8_e4m3fn).view(torch.uint8)
    v = (torch.randn(vshape, generator=g) * 0.5).to(torch.float8_e4m3fn).view(torch.uint8)
    ones = torch.ones(num_pages, dtype=torch.float32)
    return k.cuda(), v.cuda(), ones.cuda(), ones.clone().cuda()


@pytest.mark.parametrize("dt", [0, 1])
def test_append_decode_step_graph_replays_equal_eager(dt):
    """One captured step = append the token's K/V, then decode over it; seven
    replays with new tokens, new queries and lengths grown by one each."""
    print(f"[case] graph append+decode dt={dt}", flush=True)
    B, Hkv, Hq, d, P, steps = 9, 2, 14, 128, 16, 8
    g = torch.Generator().manual_seed(70 + dt)
    L0 = np.array([0, 1, 15, 16, 31, 100, 257, 700, 1500], np.int32)
    final = L0 + steps
    num_pages = int(wl.pages_needed(final, P).sum()) + 5
    bt_h, _ = wl.place_pages(final, P, num_pages, seed=71 + dt)
    bt = torch.from_numpy(bt_h).cuda()
    kg, vg, ksg, vsg = _pool(num_pages, Hkv, d, P, dt, g)
    ke, ve = kg.clone(), vg.clone()
    kse = None if ksg is None else ksg.clone()
    vse = None if vsg is None else vsg.clone()
    qs = torch.randn(steps, B, Hq, d, generator=g).to(torch.bfloat16).cuda()
    kn = torch.randn(steps, B, Hkv, d, generator=g).to(torch.bfloat16).cuda()
    vn = torch.randn(steps, B, Hkv, d, generator=g).to(torch.bfloat16).cuda()
    lens = [torch.from_numpy(L0 + 1 + s).cuda() for s in range(steps)]

    D = lib()
    kw = dict(num_kv_heads=Hkv, page_size=P, kv_dtype=dt)
    desc = D.make_decode_desc(num_seqs=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d,
                              page_size=P, block_table_stride=bt.shape[1], num_pages=num_pages,
                              kv_dtype=dt, k_scales=ksg, v_scales=vsg)
    need = D.dora_decode_workspace_bytes(desc)
    ws_g = torch.empty(need, dtype=torch.uint8, device="cuda")
    ws_e = torch.empty(need, dtype=torch.uint8, device="cuda")

    def step(k, v, ks, vs, q, knew, vnew, ln, out, ws):
        D.dora_kv_append(knew, vnew, bt, ln, k, v, k_scales=ks, v_scales=vs, **kw)
        D.dora_decode_attn(q, k, v, bt, ln, None, out, k_scales=ks, v_scales=vs, workspace=ws,
                           **kw)

    # static inputs of the captured step; step 0 runs eagerly on both copies
    q_s, kn_s, vn_s, len_s = qs[0].clone(), kn[0].clone(), vn[0].clone(), lens[0].clone()
    out_g, out_e = torch.empty_like(q_s), torch.empty_like(q_s)
    step(kg, vg, ksg, vsg, q_s, kn_s, vn_s, len_s, out_g, ws_g)
    step(ke, ve, kse, vse, qs[0], kn[0], vn[0], lens[0], out_e, ws_e)
    torch.cuda.synchronize()
    assert torch.equal(out_g.view(torch.int16), out_e.view(torch.int16))

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(kg, vg, ksg, vsg, q_s, kn_s, vn_s, len_s, out_g, ws_g)
    for s in range(1, steps):
        q_s.copy_(qs[s])
        kn_s.copy_(kn[s])
        vn_s.copy_(vn[s])
        len_s.copy_(lens[s])
        graph.replay()
        step(ke, ve, kse, vse, qs[s], kn[s], vn[s], lens[s], out_e, ws_e)
        torch.cuda.synchronize()
        assert torch.equal(out_g.view(torch.int16), out_e.view(torch.int16)), f"replay {s}"
        assert torch.equal(kg.view(torch.uint8), ke.view(torch.uint8)), f"replay {s}"
        assert torch.equal(vg.view(torch.uint8), ve.view(torch.uint8)), f"replay {s}"
        if dt == 1:
            assert torch.equal(ksg, kse) and torch.equal(vsg, vse), f"replay {s}"
    ref = oracle.decode(_codes(q_s, 0), _codes(kg, dt), _codes(vg, dt), bt_h, L0 + steps,
                        num_kv_heads=Hkv, page_size=P, kv_dtype=dt,
                        k_scales=None if ksg is None else ksg.cpu().numpy(),
                        v_scales=None if vsg is None else vsg.cpu().numpy())
    assert max_abs_err(out_g, ref) <= TOL[dt]
    del graph


def test_grouped_decode_graph_replays_equal_eager():
    """The grouped call captured once; replays with new queries and with the
    responses shortened step by step (the shared prefix is found again on the
    device at every replay)."""
    print("[case] graph grouped", flush=True)
    M, Hkv, G, d, P = 4, 2, 7, 128, 16
    w = wl.Workload("g", 3 * M, G * Hkv, Hkv, d, P, 0, 8192, "lognormal", 300, 1.0, 1, 2500)
    b, shared = wl.make_grpo_batch(w, group_size=M, prompt_range=(P + 3, 700), device="cuda",
                                   seed_index=77)
    D = lib()
    desc = D.make_decode_desc(num_seqs=w.num_seqs, num_q_heads=w.num_q_heads, num_kv_heads=Hkv,
                              head_dim=d, page_size=P, block_table_stride=b.block_table.shape[1],
                              num_pages=w.num_pages, kv_dtype=0)
    need = D.dora_decode_grouped_workspace_bytes(desc, M)
    ws_g = torch.empty(need, dtype=torch.uint8, device="cuda")
    ws_e = torch.empty(need, dtype=torch.uint8, device="cuda")
    kw = dict(group_size=M, num_kv_heads=Hkv, page_size=P, kv_dtype=0)
    g = torch.Generator(device="cuda").manual_seed(78)
    steps = 5
    qs = [torch.randn(b.q.shape, generator=g, device="cuda").to(torch.bfloat16)
          for _ in range(steps)]
    # shorten every response by 37 tokens a step, never into the prompt
    prompt = shared * P
    lens = [np.maximum(b.lengths - 37 * s, np.minimum(b.lengths, prompt + 1)).astype(np.int32)
            for s in range(steps)]
    lens_d = [torch.from_numpy(x).cuda() for x in lens]
    det_g = torch.full((w.num_seqs // M,), -1, dtype=torch.int32, device="cuda")
    det_e = det_g.clone()

    q_s, len_s = qs[0].clone(), lens_d[0].clone()
    out_g, out_e = torch.empty_like(q_s), torch.empty_like(q_s)

    def call(q, ln, out, det, ws):
        D.dora_decode_attn_grouped(q, b.k_pages, b.v_pages, b.block_table, ln, None, out,
                                   shared_pages_out=det, workspace=ws, **kw)

    call(q_s, len_s, out_g, det_g, ws_g)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call(q_s, len_s, out_g, det_g, ws_g)
    for s in range(steps):
        q_s.copy_(qs[s])
        len_s.copy_(lens_d[s])
        det_g.fill_(-1)
        graph.replay()
        call(qs[s], lens_d[s], out_e, det_e, ws_e)
        torch.cuda.synchronize()
        assert torch.equal(out_g.view(torch.int16), out_e.view(torch.int16)), f"replay {s}"
        assert torch.equal(det_g, det_e), f"replay {s}"
    assert det_g.cpu().numpy().tolist() == shared[::M].tolist()
    b.q, b.lengths, b.seq_lens = q_s, lens[-1], lens_d[-1]
    assert max_abs_err(out_g, oracle_for(b)) <= TOL[0]
    del graph
