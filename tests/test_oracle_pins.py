"""Pins of the fp64 oracle to facts outside itself (CPU only).

The oracle is the statement of softmax(q K^T * scale) V over a sequence's
cached tokens, read through the paged, multi-version pool.  These tests tie it
to: exhaustive decoder tables from torch's own dtypes, torch's float64 scaled
dot-product attention (GQA mode) on contiguous tensors laid into pages by an
independent numpy scatter, closed forms (length 1, two tokens, identical keys,
vanishing scale, dominant key), invariants (page permutation, value shift,
tail-slot contents) and a brute-force twin.
"""
import json
import math
import os
import struct

import numpy as np
import pytest
import torch

import oracle
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# helpers: build a paged problem from contiguous per-sequence tensors
# ---------------------------------------------------------------------------

def _bf16_codes(x: torch.Tensor) -> np.ndarray:
    return x.to(torch.bfloat16).contiguous().view(torch.int16).numpy().view(np.uint16)


def _bf16_f64(codes: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(codes.view(np.int16).copy()).view(torch.bfloat16).double()


def _e4m3_f64(codes: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(codes.copy()).view(torch.float8_e4m3fn).double()


class Problem:
    """Contiguous K/V per sequence plus the same data scattered into a pool."""

    def __init__(self, lens, Hq, Hkv, d, P, kv_dtype=0, seed=0, num_pages=None, poison=True,
                 k_fn=None, v_fn=None, q_fn=None):
        g = torch.Generator().manual_seed(seed)
        rng = np.random.default_rng(seed)
        self.lens = np.asarray(lens, np.int32)
        self.B, self.Hq, self.Hkv, self.d, self.P, self.kv_dtype = (
            len(lens), Hq, Hkv, d, P, kv_dtype)
        n = wl.pages_needed(self.lens, P)
        total = int(n.sum())
        self.num_pages = num_pages or max(4, 2 * total + 3)
        perm = rng.permutation(self.num_pages)[:total]
        self.stride = max(1, int(n.max()) if len(n) else 1)
        self.bt = np.zeros((self.B, self.stride), np.int32)
        X = wl.chunk_elems(kv_dtype)
        codes_t = np.uint16 if kv_dtype == 0 else np.uint8
        nan = 0x7FC0 if kv_dtype == 0 else 0x7F
        self.kp = np.zeros((self.num_pages, Hkv, d // X, P, X), codes_t)
        self.vp = np.zeros((self.num_pages, Hkv, d, P), codes_t)
        self.ks = self.vs = None
        if kv_dtype == 1:
            self.ks = (2.0 ** rng.uniform(-6, 2, self.num_pages)).astype(np.float32)
            self.vs = (2.0 ** rng.uniform(-6, 2, self.num_pages)).astype(np.float32)
        q = q_fn(g) if q_fn else torch.randn(self.B, Hq, d, generator=g)
        self.q = _bf16_codes(q)
        self.K, self.V = [], []   # contiguous fp64 [L][Hkv][d] (dequantised)
        off = 0
        for b, L in enumerate(self.lens):
            nb = int(n[b])
            pages = perm[off:off + nb]
            off += nb
            self.bt[b, :nb] = pages
            kc = k_fn(g, b, int(L)) if k_fn else torch.randn(int(L), Hkv, d, generator=g)
            vc = v_fn(g, b, int(L)) if v_fn else torch.randn(int(L), Hkv, d, generator=g)
            if kv_dtype == 0:
                kcode, vcode = _bf16_codes(kc), _bf16_codes(vc)
            else:
                kcode = (kc * 8).clamp(-448, 448).to(torch.float8_e4m3fn).view(
                    torch.uint8).numpy()
                vcode = (vc * 8).clamp(-448, 448).to(torch.float8_e4m3fn).view(
                    torch.uint8).numpy()
            pad = nb * P - int(L)
            fill = nan if poison else 0
            kpad = np.concatenate([kcode, np.full((pad, Hkv, d), fill, codes_t)])
            vpad = np.concatenate([vcode, np.full((pad, Hkv, d), fill, codes_t)])
            if nb:
                self.kp[pages] = wl.k_tokens_to_pages(kpad, P, kv_dtype)
                self.vp[pages] = wl.v_tokens_to_pages(vpad, P)
            if kv_dtype == 0:
                Kf, Vf = _bf16_f64(kcode), _bf16_f64(vcode)
            else:
                tok_page = np.repeat(pages, P)[:int(L)]
                Kf = _e4m3_f64(kcode) * torch.from_numpy(
                    self.ks[tok_page].astype(np.float64)).view(-1, 1, 1)
                Vf = _e4m3_f64(vcode) * torch.from_numpy(
                    self.vs[tok_page].astype(np.float64)).view(-1, 1, 1)
            self.K.append(Kf)
            self.V.append(Vf)

    def oracle(self, scale=0.0, **kw):
        return oracle.decode(self.q, self.kp, self.vp, self.bt, self.lens,
                             num_kv_heads=self.Hkv, page_size=self.P, kv_dtype=self.kv_dtype,
                             scale=scale, k_scales=self.ks, v_scales=self.vs, **kw)

    def brute(self, scale=0.0):
        return oracle.decode_brute(self.q, self.kp, self.vp, self.bt, self.lens,
                                   num_kv_heads=self.Hkv, page_size=self.P,
                                   kv_dtype=self.kv_dtype, scale=scale, k_scales=self.ks,
                                   v_scales=self.vs)

    def sdpa(self, scale=None):
        """torch float64 scaled_dot_product_attention, GQA mode, per sequence."""
        qf = _bf16_f64(self.q)
        out = torch.zeros(self.B, self.Hq, self.d, dtype=torch.float64)
        for b in range(self.B):
            if self.lens[b] == 0:
                continue
            qq = qf[b].view(1, self.Hq, 1, self.d)
            kk = self.K[b].permute(1, 0, 2).unsqueeze(0).contiguous()
            vv = self.V[b].permute(1, 0, 2).unsqueeze(0).contiguous()
            o = torch.nn.functional.scaled_dot_product_attention(
                qq, kk, vv, scale=scale, enable_gqa=True)
            out[b] = o.view(self.Hq, self.d)
        return out.numpy()


# ---------------------------------------------------------------------------
# decoders: exhaustive against torch's dtypes and the format definitions
# ---------------------------------------------------------------------------

def test_bf16_decoder_exhaustive():
    codes = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = _bf16_f64(codes).numpy()
    got = np.array([oracle.bf16_to_f64(c) for c in codes])
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(got))
    assert np.array_equal(ref[~nan], got[~nan])


def test_e4m3_decoder_exhaustive():
    codes = np.arange(256, dtype=np.uint8)
    ref = _e4m3_f64(codes).numpy()
    got = np.array([oracle.e4m3_to_f64(c) for c in codes])
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(got))
    assert nan.sum() == 2  # only S.1111.111
    assert np.array_equal(ref[~nan], got[~nan])
    # format landmarks: 1.0, largest normal, smallest subnormal, smallest normal
    assert oracle.e4m3_to_f64(0x38) == 1.0
    assert oracle.e4m3_to_f64(0x7E) == 448.0
    assert oracle.e4m3_to_f64(0xFE) == -448.0
    assert oracle.e4m3_to_f64(0x01) == 2.0 ** -9
    assert oracle.e4m3_to_f64(0x08) == 2.0 ** -6


# ---------------------------------------------------------------------------
# attention: library routine, closed forms, invariants
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("lens,Hq,Hkv,d,P,dt", [
    ([1, 5, 16, 17, 40], 8, 2, 64, 16, 0),
    ([33, 7, 64], 28, 4, 128, 16, 0),      # group of 7
    ([3, 50], 4, 4, 64, 32, 0),            # MHA, page 32
    ([9, 31, 70], 16, 1, 64, 16, 0),       # one KV head, group of 16
    ([5, 33, 64, 1], 16, 2, 128, 32, 1),   # fp8 keys/values, per-page scales
    ([18, 40], 8, 2, 64, 16, 1),           # fp8, page 16
])
def test_oracle_matches_torch_sdpa_gqa(lens, Hq, Hkv, d, P, dt):
    pb = Problem(lens, Hq, Hkv, d, P, dt, seed=sum(lens) + Hq)
    got = pb.oracle()
    ref = pb.sdpa()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_oracle_explicit_scale_matches_sdpa():
    pb = Problem([12, 29], 4, 2, 64, 16, 0, seed=3)
    np.testing.assert_allclose(pb.oracle(scale=0.37), pb.sdpa(scale=0.37), rtol=0, atol=1e-12)


def test_oracle_agrees_with_brute_force_twin():
    for dt in (0, 1):
        pb = Problem([1, 15, 16, 17, 45], 8, 2, 64, 16 if dt == 0 else 32, dt, seed=11 + dt)
        np.testing.assert_allclose(pb.oracle(), pb.brute(), rtol=0, atol=1e-12)


def test_length_one_returns_its_value_row_exactly():
    pb = Problem([1, 1, 1], 8, 2, 64, 16, 0, seed=5)
    out = pb.oracle()
    for b in range(3):
        for h in range(8):
            assert np.array_equal(out[b, h], pb.V[b][0, h // 4].numpy())


def test_two_tokens_logistic_closed_form():
    pb = Problem([2], 2, 1, 64, 16, 0, seed=7)
    out = pb.oracle()
    qf = _bf16_f64(pb.q)[0].numpy()
    K, V = pb.K[0].numpy(), pb.V[0].numpy()
    for h in range(2):
        a = (qf[h] @ K[0, 0] - qf[h] @ K[1, 0]) / 8.0     # scale 1/sqrt(64)
        w0 = 1.0 / (1.0 + math.exp(-a))                    # logistic
        ref = w0 * V[0, 0] + (1.0 - w0) * V[1, 0]
        np.testing.assert_allclose(out[0, h], ref, rtol=0, atol=1e-13)


def test_identical_keys_give_mean_of_values():
    def k_same(g, b, L):
        row = torch.randn(1, 2, 64, generator=g)
        return row.expand(L, 2, 64).clone()
    pb = Problem([37, 5], 8, 2, 64, 16, 0, seed=9, k_fn=k_same)
    out = pb.oracle()
    for b in range(2):
        mean = pb.V[b].mean(dim=0).numpy()          # [Hkv][d]
        for h in range(8):
            np.testing.assert_allclose(out[b, h], mean[h // 4], rtol=0, atol=1e-12)


def test_vanishing_scale_gives_mean_of_values():
    pb = Problem([23], 4, 2, 64, 16, 0, seed=13)
    out = pb.oracle(scale=1e-30)
    mean = pb.V[0].mean(dim=0).numpy()
    for h in range(4):
        np.testing.assert_allclose(out[0, h], mean[h // 2], rtol=0, atol=1e-12)


def test_dominant_key_selects_its_value():
    # q fixed; key j = 8*q (exact in bf16) outscores N(0,1) keys by far.
    qv = torch.randn(1, 1, 64, generator=torch.Generator().manual_seed(1))

    def k_dom(g, b, L):
        k = torch.randn(L, 1, 64, generator=g) * 0.01
        k[L // 2] = 8 * qv[0]
        return k
    pb = Problem([20], 1, 1, 64, 16, 0, seed=2, k_fn=k_dom, q_fn=lambda g: qv)
    out = pb.oracle()
    np.testing.assert_allclose(out[0, 0], pb.V[0][10, 0].numpy(), rtol=0, atol=1e-9)


def test_value_shift_shifts_output():
    # Small-integer values are exact in bf16, so V + 1 is exact too.
    def v_int(g, b, L):
        return torch.randint(-4, 5, (L, 2, 64), generator=g).float()
    base = Problem([19, 40], 4, 2, 64, 16, 0, seed=21, v_fn=v_int)
    shifted = Problem([19, 40], 4, 2, 64, 16, 0, seed=21,
                      v_fn=lambda g, b, L: v_int(g, b, L) + 1.0)
    np.testing.assert_allclose(shifted.oracle(), base.oracle() + 1.0, rtol=0, atol=1e-12)


def test_physical_page_permutation_is_bitwise_invariant():
    pb = Problem([17, 48, 5], 8, 2, 64, 16, 0, seed=31)
    ref = pb.oracle()
    perm = np.random.default_rng(0).permutation(pb.num_pages)
    kp2, vp2 = np.empty_like(pb.kp), np.empty_like(pb.vp)
    kp2[perm] = pb.kp
    vp2[perm] = pb.vp
    bt2 = perm[pb.bt].astype(np.int32)
    got = oracle.decode(pb.q, kp2, vp2, bt2, pb.lens, num_kv_heads=2, page_size=16)
    assert np.array_equal(got, ref)


def test_pages_shared_between_sequences_equal_private_copies():
    """Block tables of several sequences naming the same leading pages (a shared
    prompt) decode exactly as if each sequence held its own copy."""
    pb = Problem([40, 33, 50, 64], 8, 2, 64, 16, 0, seed=33)
    shared = 2                                      # pages 0 and 1 of sequence 0
    bt = pb.bt.copy()
    for s in (1, 2, 3):
        bt[s, :shared] = pb.bt[0, :shared]          # point at sequence 0's pages
    got_shared = oracle.decode(pb.q, pb.kp, pb.vp, bt, pb.lens, num_kv_heads=2, page_size=16)
    kp2, vp2 = pb.kp.copy(), pb.vp.copy()
    for s in (1, 2, 3):                             # private copies of sequence 0's pages
        kp2[pb.bt[s, :shared]] = pb.kp[pb.bt[0, :shared]]
        vp2[pb.bt[s, :shared]] = pb.vp[pb.bt[0, :shared]]
    got_copies = oracle.decode(pb.q, kp2, vp2, pb.bt, pb.lens, num_kv_heads=2, page_size=16)
    assert np.array_equal(got_shared, got_copies)


def test_tail_slots_never_read():
    a = Problem([17, 3, 31], 8, 2, 64, 16, 0, seed=41, poison=True)
    b = Problem([17, 3, 31], 8, 2, 64, 16, 0, seed=41, poison=False)
    oa, ob = a.oracle(), b.oracle()
    assert np.isfinite(oa).all()
    assert np.array_equal(oa, ob)


def test_empty_sequence_gives_zero_and_empty_batch():
    pb = Problem([0, 4, 0], 4, 2, 64, 16, 0, seed=51)
    out = pb.oracle()
    assert np.all(out[0] == 0) and np.all(out[2] == 0)
    np.testing.assert_allclose(out, pb.sdpa(), rtol=0, atol=1e-12)
    empty = oracle.decode(np.zeros((0, 4, 64), np.uint16), pb.kp, pb.vp,
                          np.zeros((0, 1), np.int32), np.zeros(0, np.int32),
                          num_kv_heads=2, page_size=16)
    assert empty.shape == (0, 4, 64)


def test_version_ownership_and_page_range_are_enforced():
    pb = Problem([20, 9], 4, 2, 64, 16, 0, seed=61)
    owner = np.full(pb.num_pages, -1, np.int16)
    owner[pb.bt[0, :2]] = 0
    owner[pb.bt[1, :1]] = 1
    vid = np.array([0, 1], np.int32)
    pb.oracle(version_ids=vid, page_owner=owner)   # consistent: passes
    bad = owner.copy()
    bad[pb.bt[1, 0]] = 0
    rc = oracle.decode_rc(pb.q, pb.kp, pb.vp, pb.bt, pb.lens, num_kv_heads=2, page_size=16,
                          version_ids=vid, page_owner=bad)
    assert rc == 3
    bt = pb.bt.copy()
    bt[0, 1] = pb.num_pages
    rc = oracle.decode_rc(pb.q, pb.kp, pb.vp, bt, pb.lens, num_kv_heads=2, page_size=16)
    assert rc == 2


# ---------------------------------------------------------------------------
# pack / unpack: documented byte format, round trip, version rule
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dt", [0, 1])
def test_pack_format_and_round_trip(dt):
    P = 16 if dt == 0 else 32
    pb = Problem([20, 70, 5], 8, 2, 64, P, dt, seed=71 + dt)
    n = wl.pages_needed(pb.lens, P)
    src = np.concatenate([pb.bt[b, :n[b]] for b in range(3)]).astype(np.int32)
    buf = oracle.pack(pb.kp, pb.vp, src, kv_dtype=dt, page_size=P, num_kv_heads=2,
                      head_dim=64, policy_version=2, n_seqs=3, k_scales=pb.ks,
                      v_scales=pb.vs)
    page_bytes = 2 * P * 64 * (2 if dt == 0 else 1)
    assert buf.size == 256 + 2 * len(src) * page_bytes + (8 * len(src) if dt else 0)
    assert oracle.packed_bytes(dt, P, 2, 64, len(src)) == buf.size
    hdr = bytes(buf[:256])
    assert hdr[:8] == b"DORAKV01"
    fmt, ver, kdt, ps, hk, hd = struct.unpack_from("<6i", hdr, 8)
    npg, pbytes = struct.unpack_from("<2q", hdr, 32)
    nseq, = struct.unpack_from("<i", hdr, 48)
    assert (fmt, ver, kdt, ps, hk, hd, npg, pbytes, nseq) == (
        1, 2, dt, P, 2, 64, len(src), page_bytes, 3)
    assert not any(hdr[52:])
    body = buf[256:]
    kflat = pb.kp.reshape(pb.num_pages, -1).view(np.uint8)
    vflat = pb.vp.reshape(pb.num_pages, -1).view(np.uint8)
    kb = len(src) * page_bytes
    assert np.array_equal(body[:kb], kflat[src].reshape(-1))
    assert np.array_equal(body[kb:2 * kb], vflat[src].reshape(-1))
    if dt:
        sc = body[2 * kb:].view(np.float32)
        assert np.array_equal(sc[:len(src)], pb.ks[src])
        assert np.array_equal(sc[len(src):], pb.vs[src])
    # unpack into fresh pages of a second pool, then decode must be bitwise equal
    dst = np.random.default_rng(5).permutation(pb.num_pages)[:len(src)].astype(np.int32)
    kp2, vp2 = np.zeros_like(pb.kp), np.zeros_like(pb.vp)
    ks2 = np.zeros_like(pb.ks) if dt else None
    vs2 = np.zeros_like(pb.vs) if dt else None
    rc = oracle.unpack(buf, dst, kp2, vp2, kv_dtype=dt, page_size=P, num_kv_heads=2,
                       head_dim=64, policy_version=2, k_scales=ks2, v_scales=vs2)
    assert rc == 0
    assert np.array_equal(kp2[dst], pb.kp[src]) and np.array_equal(vp2[dst], pb.vp[src])
    remap = dict(zip(src.tolist(), dst.tolist()))
    bt2 = np.vectorize(lambda p: remap.get(int(p), 0))(pb.bt).astype(np.int32)
    for b in range(3):
        bt2[b, n[b]:] = 0
    before = pb.oracle()
    after = oracle.decode(pb.q, kp2, vp2, bt2, pb.lens, num_kv_heads=2, page_size=P,
                          kv_dtype=dt, k_scales=ks2, v_scales=vs2)
    assert np.array_equal(before, after)
    # cross-version unpack is refused and writes nothing
    kp3 = np.zeros_like(pb.kp)
    rc = oracle.unpack(buf, dst, kp3, np.zeros_like(pb.vp), kv_dtype=dt, page_size=P,
                       num_kv_heads=2, head_dim=64, policy_version=1,
                       k_scales=None if not dt else np.zeros_like(pb.ks),
                       v_scales=None if not dt else np.zeros_like(pb.vs))
    assert rc == 4 and not kp3.any()


# ---------------------------------------------------------------------------
# workload statistic printed in the paper
# ---------------------------------------------------------------------------

def test_bubble_statistic_matches_paper_case_study():
    with open(os.path.join(GOLDEN, "bubble_case_study.json")) as f:
        g = json.load(f)
    # A batch with the printed max and mean: one long response, the rest equal.
    n = 1000
    rest = (g["mean_len"] * n - g["max_len"]) / (n - 1)
    lens = np.array([g["max_len"]] + [rest] * (n - 1))
    assert abs(lens.mean() - g["mean_len"]) < 1e-9
    assert abs(100 * wl.bubble(lens) - g["bubble_percent_printed"]) <= g["printed_precision"]
