"""Pins of the oracle's KV append (CPU only).

The append stores each sequence's current-token K/V into its page slot.  For
bf16 pages that is a plain store; it is pinned to an independent numpy scatter
of whole sequences.  For fp8 pages the oracle also keeps one fp32 scale per
page under a grow-only policy; its encoder is pinned to torch's float8_e4m3fn
conversion, and the policy to the cases that reduce to that conversion: the
first token of a page, tokens that fit the current scale, and a scale that
grows by an exact power of two.  Growth by any other ratio is pinned by exact
rational arithmetic in which each fp32 step of the stated policy is rounded
once, on data chosen (by exhaustive search over the E4M3 codes) so that the
other association of the requantisation product gives other codes.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl


def _bf16(x: torch.Tensor) -> np.ndarray:
    return x.to(torch.bfloat16).contiguous().view(torch.int16).numpy().view(np.uint16)


def _bf16_f32(codes: np.ndarray) -> np.ndarray:
    return torch.from_numpy(codes.view(np.int16).copy()).view(torch.bfloat16).float().numpy()


def _torch_e4m3(x: np.ndarray) -> np.ndarray:
    """torch's nearest-even conversion, after clamping to the finite range."""
    x = np.clip(np.asarray(x, np.float32), -448.0, 448.0)
    return torch.from_numpy(x.copy()).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def _e4m3_f32(codes: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.asarray(codes, np.uint8).copy()).view(
        torch.float8_e4m3fn).float().numpy()


def _empty_pool(num_pages, Hkv, d, P, dt):
    X = wl.chunk_elems(dt)
    et = np.uint16 if dt == 0 else np.uint8
    k = np.zeros((num_pages, Hkv, d // X, P, X), et)
    v = np.zeros((num_pages, Hkv, d, P), et)
    ks = np.ones(num_pages, np.float32) if dt == 1 else None
    vs = np.ones(num_pages, np.float32) if dt == 1 else None
    return k, v, ks, vs


# ---------------------------------------------------------------------------
# encoder
# ---------------------------------------------------------------------------

def test_e4m3_encoder_matches_torch_on_grid_midpoints_and_random():
    grid = _e4m3_f32(np.arange(256, dtype=np.uint8))
    grid = np.unique(grid[np.isfinite(grid)])                      # 253 values, -448 .. 448
    mids = (grid[:-1].astype(np.float64) + grid[1:]) / 2            # exact in fp32
    mids = mids.astype(np.float32)
    up = np.nextafter(mids, np.float32(np.inf))
    dn = np.nextafter(mids, np.float32(-np.inf))
    rng = np.random.default_rng(5)
    rnd = (rng.standard_normal(20000) * np.exp(rng.uniform(-14, 7, 20000))).astype(np.float32)
    big = np.array([448.0, 448.5, 463.9, 464.0, 464.1, 480.0, 1e6, 3e38, -1e9], np.float32)
    tiny = np.array([0.0, -0.0, 2.0 ** -10, 2.0 ** -10 * 1.0001, 3 * 2.0 ** -11, 1e-30, -1e-30],
                    np.float32)
    vals = np.concatenate([grid, mids, up, dn, rnd, big, tiny]).astype(np.float32)
    got = oracle.f32_to_e4m3(vals)
    assert np.array_equal(got, _torch_e4m3(vals))


# ---------------------------------------------------------------------------
# bf16: plain store
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("Hkv,d,P", [(2, 64, 16), (4, 128, 32), (1, 128, 16)])
def test_append_bf16_equals_page_scatter_of_the_sequence(Hkv, d, P):
    lens = np.array([1, 15, 16, 17, 40, 64], np.int32)
    S = 9                                   # the last S tokens arrive by append
    num_pages = 64
    bt, _ = wl.place_pages(lens, P, num_pages, seed=3)
    g = torch.Generator().manual_seed(4)
    toks_k = [_bf16(torch.randn(int(L), Hkv, d, generator=g)) for L in lens]
    toks_v = [_bf16(torch.randn(int(L), Hkv, d, generator=g)) for L in lens]
    # reference: whole sequences scattered by the numpy layout helpers
    ref_k, ref_v, _, _ = _empty_pool(num_pages, Hkv, d, P, 0)
    for b, L in enumerate(lens):
        n = -(-int(L) // P)
        kk = np.zeros((n * P, Hkv, d), np.uint16)
        vv = np.zeros((n * P, Hkv, d), np.uint16)
        kk[:L], vv[:L] = toks_k[b], toks_v[b]
        ref_k[bt[b, :n]] = wl.k_tokens_to_pages(kk, P, 0)
        ref_v[bt[b, :n]] = wl.v_tokens_to_pages(vv, P)
    # oracle: the same prefix scattered, then S appends, one token per call
    k, v, _, _ = _empty_pool(num_pages, Hkv, d, P, 0)
    start = np.maximum(lens - S, 0)
    for b, L in enumerate(lens):
        n = -(-int(start[b]) // P)
        if n == 0:
            continue
        kk = np.zeros((n * P, Hkv, d), np.uint16)
        vv = np.zeros((n * P, Hkv, d), np.uint16)
        kk[:start[b]], vv[:start[b]] = toks_k[b][:start[b]], toks_v[b][:start[b]]
        k[bt[b, :n]] = wl.k_tokens_to_pages(kk, P, 0)
        v[bt[b, :n]] = wl.v_tokens_to_pages(vv, P)
    for s in range(S):
        cur = np.minimum(start + s + 1, lens).astype(np.int32)
        cur[start + s >= lens] = 0                 # sequence already complete: nothing
        kn = np.zeros((len(lens), Hkv, d), np.uint16)
        vn = np.zeros((len(lens), Hkv, d), np.uint16)
        for b in range(len(lens)):
            if cur[b] > 0:
                kn[b], vn[b] = toks_k[b][cur[b] - 1], toks_v[b][cur[b] - 1]
        assert oracle.kv_append(kn, vn, bt, cur, k, v, kv_dtype=0, page_size=P) == 0
    assert np.array_equal(k, ref_k) and np.array_equal(v, ref_v)


# ---------------------------------------------------------------------------
# fp8: the page-scale policy, by its cases that reduce to torch's conversion
# ---------------------------------------------------------------------------

def _one_seq(P, Hkv, d, num_pages=4):
    bt = np.array([[2, 0, 3]], np.int32)
    return bt, _empty_pool(num_pages, Hkv, d, P, 1)


def _k_slot(k, page, slot):
    """[Hkv][d] codes of one token slot of a K page (layout [Hkv][d/16][P][16])."""
    kp = k[page]                                   # [Hkv][d/16][P][16]
    return kp[:, :, slot, :].reshape(kp.shape[0], -1)


def _v_slot(v, page, slot):
    return v[page][:, :, slot]


@pytest.mark.parametrize("P,Hkv,d", [(16, 2, 64), (32, 8, 128)])
def test_append_fp8_first_token_of_a_page_is_torch_quantisation(P, Hkv, d):
    bt, (k, v, ks, vs) = _one_seq(P, Hkv, d)
    g = torch.Generator().manual_seed(7)
    kn = _bf16(torch.randn(1, Hkv, d, generator=g) * 3.0)
    vn = _bf16(torch.randn(1, Hkv, d, generator=g) * 1e-3)
    L = np.array([P + 1], np.int32)                # token P: slot 0 of the second page
    assert oracle.kv_append(kn, vn, bt, L, k, v, kv_dtype=1, page_size=P, k_scales=ks,
                            v_scales=vs) == 0
    page = bt[0, 1]
    for new, pool, scales, slot_of in ((kn, k, ks, _k_slot), (vn, v, vs, _v_slot)):
        x = _bf16_f32(new[0])
        s = max(np.float32(np.abs(x).max()) / np.float32(448.0), np.float32(2.0 ** -126))
        assert scales[page] == s
        assert np.array_equal(slot_of(pool, page, 0), _torch_e4m3(x / s))
    others = [i for i in range(len(ks)) if i != page]
    assert (ks[others] == 1).all() and (vs[others] == 1).all()   # other pages untouched


def test_append_fp8_smaller_tokens_keep_scale_and_earlier_codes():
    P, Hkv, d = 16, 2, 64
    bt, (k, v, ks, vs) = _one_seq(P, Hkv, d)
    g = torch.Generator().manual_seed(8)
    base = torch.randn(Hkv, d, generator=g)
    history = []
    for t in range(5):                              # amax shrinks token by token
        kn = _bf16((base * (4.0 / (t + 1)))[None])
        vn = _bf16((torch.randn(Hkv, d, generator=g) * (2.0 / (t + 1)))[None])
        assert oracle.kv_append(kn, vn, bt, np.array([t + 1], np.int32), k, v, kv_dtype=1,
                                page_size=P, k_scales=ks, v_scales=vs) == 0
        history.append((kn, vn))
        page = bt[0, 0]
        if t == 0:
            s_k, s_v = ks[page], vs[page]
        assert ks[page] == s_k and vs[page] == s_v
        for u, (kk, vv) in enumerate(history):      # every stored token, unchanged
            assert np.array_equal(_k_slot(k, page, u), _torch_e4m3(_bf16_f32(kk[0]) / s_k))
            assert np.array_equal(_v_slot(v, page, u), _torch_e4m3(_bf16_f32(vv[0]) / s_v))


def test_append_fp8_doubling_amax_requantises_earlier_tokens_by_half():
    P, Hkv, d = 16, 2, 64
    bt, (k, v, ks, vs) = _one_seq(P, Hkv, d)
    g = torch.Generator().manual_seed(9)
    x0 = torch.randn(Hkv, d, generator=g)
    x0 = x0 / x0.abs().max() * 56.0                 # amax 56 -> scale 56/448 = 1/8 exactly
    x1 = torch.randn(Hkv, d, generator=g)
    x1 = x1 / x1.abs().max() * 112.0                # amax 112 -> scale 1/4 exactly
    for t, x in enumerate((x0, x1)):
        kn = _bf16(x[None])
        assert oracle.kv_append(kn, kn.copy(), bt, np.array([t + 1], np.int32), k, v,
                                kv_dtype=1, page_size=P, k_scales=ks, v_scales=vs) == 0
    page = bt[0, 0]
    assert ks[page] == np.float32(0.25) and vs[page] == np.float32(0.25)
    first = _torch_e4m3(_bf16_f32(_bf16(x0[None])[0]) / np.float32(0.125))   # token 0 at 1/8
    halved = _torch_e4m3(_e4m3_f32(first) / np.float32(2.0))                 # then 1/8 -> 1/4
    assert np.array_equal(_k_slot(k, page, 0), halved)
    assert np.array_equal(_v_slot(v, page, 0), halved)
    assert np.array_equal(_k_slot(k, page, 1),
                          _torch_e4m3(_bf16_f32(_bf16(x1[None])[0]) / np.float32(0.25)))


def test_append_then_decode_tracks_unquantised_attention():
    """Information pin: a page sequence built token by token under the policy
    decodes close to fp64 attention over the unquantised values."""
    P, Hkv, Hq, d, T = 16, 2, 8, 64, 45
    bt = np.array([[5, 1, 7]], np.int32)
    k, v, ks, vs = _empty_pool(8, Hkv, d, P, 1)
    g = torch.Generator().manual_seed(10)
    mags = torch.exp(torch.randn(T, generator=g) * 0.7)
    kt = _bf16(torch.randn(T, Hkv, d, generator=g) * mags[:, None, None])
    vt = _bf16(torch.randn(T, Hkv, d, generator=g) * mags[:, None, None])
    for t in range(T):
        assert oracle.kv_append(kt[t][None], vt[t][None], bt, np.array([t + 1], np.int32), k, v,
                                kv_dtype=1, page_size=P, k_scales=ks, v_scales=vs) == 0
    q = _bf16(torch.randn(1, Hq, d, generator=g))
    out = oracle.decode(q, k, v, bt, np.array([T], np.int32), num_kv_heads=Hkv, page_size=P,
                        kv_dtype=1, k_scales=ks, v_scales=vs)
    qf = torch.from_numpy(_bf16_f32(q)).double()[0]
    kf = torch.from_numpy(_bf16_f32(kt)).double().repeat_interleave(Hq // Hkv, dim=1)
    vf = torch.from_numpy(_bf16_f32(vt)).double().repeat_interleave(Hq // Hkv, dim=1)
    w = torch.softmax(torch.einsum("hd,thd->ht", qf, kf) / d ** 0.5, dim=-1)
    ref = torch.einsum("ht,thd->hd", w, vf).numpy()
    assert np.abs(out[0] - ref).max() < 0.15 * np.abs(ref).max() + 0.05


def test_append_error_codes_and_empty_sequences():
    P, Hkv, d = 16, 2, 64
    bt, (k, v, ks, vs) = _one_seq(P, Hkv, d)
    kn = _bf16(torch.ones(1, Hkv, d))
    before = (k.copy(), v.copy(), ks.copy(), vs.copy())
    args = dict(kv_dtype=1, page_size=P, k_scales=ks, v_scales=vs)
    assert oracle.kv_append(kn, kn, bt, np.array([0], np.int32), k, v, **args) == 0
    assert oracle.kv_append(kn, kn, bt, np.array([3 * P + 1], np.int32), k, v, **args) == 5
    bad = bt.copy()
    bad[0, 0] = 99
    assert oracle.kv_append(kn, kn, bad, np.array([1], np.int32), k, v, **args) == 2
    for a, b in zip(before, (k, v, ks, vs)):
        assert np.array_equal(a, b)


def test_append_fp8_token_with_the_page_maximum_does_not_grow_the_scale():
    """Rewriting the last token with the values that set the page's scale (a
    decode loop that retries a step) changes nothing, including where fp32
    rounding puts amax / s0 just above 448."""
    P, Hkv, d = 16, 8, 128
    bt, (k, v, ks, vs) = _one_seq(P, Hkv, d)
    g = torch.Generator().manual_seed(11)
    toks = [torch.randn(Hkv, d, generator=g) * m for m in (0.1, 0.1, 0.05)]
    # token 1's maximum is 0.51171875 (a bf16 value), for which
    # 0.51171875 / (0.51171875 / 448) rounds above 448 in fp32
    toks[1][0, 0] = 0.51171875
    toks = [_bf16(x[None]) for x in toks]
    for t, x in enumerate(toks):
        assert oracle.kv_append(x, x, bt, np.array([t + 1], np.int32), k, v, kv_dtype=1,
                                page_size=P, k_scales=ks, v_scales=vs) == 0
    page = bt[0, 0]
    snap = (k[page].copy(), v[page].copy(), ks[page], vs[page])
    for _ in range(3):                              # token 1 set the scale; rewrite it
        assert oracle.kv_append(toks[1], toks[1], bt, np.array([2], np.int32), k, v,
                                kv_dtype=1, page_size=P, k_scales=ks, v_scales=vs) == 0
    assert ks[page] == snap[2] and vs[page] == snap[3]
    assert np.array_equal(_k_slot(k, page, 0), _k_slot(snap[0][None], 0, 0))
    assert np.array_equal(k[page], snap[0]) and np.array_equal(v[page], snap[1])


# ---------------------------------------------------------------------------
# fp8: a scale that grows by a ratio that is no power of two, pinned by exact
# rational arithmetic with each fp32 step of the policy rounded explicitly
# ---------------------------------------------------------------------------

from fractions import Fraction  # noqa: E402


def _bf16_exact(code: int) -> Fraction:
    """Value of a bf16 code from its fields (sign, 8-bit exponent, 7-bit
    mantissa); finite codes only."""
    s, e, m = (code >> 15) & 1, (code >> 7) & 0xFF, code & 0x7F
    assert e != 0xFF
    v = Fraction(m, 128) * Fraction(2) ** -126 if e == 0 else \
        (1 + Fraction(m, 128)) * Fraction(2) ** (e - 127)
    return -v if s else v


def _round_even(q: Fraction) -> int:
    n = q.numerator // q.denominator
    r = q - n
    return n + 1 if r > Fraction(1, 2) or (r == Fraction(1, 2) and n % 2) else n


def _fl32(q: Fraction) -> Fraction:
    """Nearest binary32 value (ties to even), normal or subnormal."""
    if q == 0:
        return Fraction(0)
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    ulp = Fraction(2) ** (max(e, -126) - 23)
    r = _round_even(a / ulp) * ulp
    assert r < Fraction(2) ** 128
    return r if q > 0 else -r


def _e4m3_exact(code: int) -> Fraction:
    s, e, m = (code >> 7) & 1, (code >> 3) & 0xF, code & 7
    assert not (e == 15 and m == 7)
    v = Fraction(m, 8) * Fraction(2) ** -6 if e == 0 else \
        (1 + Fraction(m, 8)) * Fraction(2) ** (e - 7)
    return -v if s else v


def _e4m3_enc(x: Fraction) -> int:
    """Nearest OCP E4M3FN code, ties to even mantissa, saturating at 448."""
    sign = 0x80 if x < 0 else 0
    a = abs(x)
    if a >= 448:
        return sign | 0x7E
    e = -6
    while e < 8 and Fraction(2) ** (e + 1) <= a:
        e += 1
    n = _round_even(a / Fraction(2) ** (e - 3))   # units of the grid step at exponent e
    if e == -6 and n < 8:                         # subnormal (n = 8 is the smallest normal)
        return sign | n
    if n == 16:                                   # rounded up to the next binade
        e, n = e + 1, 8
    code = ((e + 7) << 3) | (n - 8)
    return sign | min(code, 0x7E)


def _exact_two_token_page(x0_codes, x1_codes):
    """The stated policy on a page that receives token 0 then token 1 (both as
    bf16 codes), every fp32 operation rounded once: returns (codes of token 0
    after token 1, codes of token 1, final scale)."""
    x0 = [_bf16_exact(int(c)) for c in x0_codes]
    x1 = [_bf16_exact(int(c)) for c in x1_codes]
    fresh = lambda xs: max(_fl32(max(abs(v) for v in xs) / 448), Fraction(2) ** -126)  # noqa
    s0 = fresh(x0)
    c0 = [_e4m3_enc(_fl32(v / s0)) for v in x0]
    f1 = fresh(x1)
    assert not f1 <= s0                                   # the page grows
    s = f1
    re0 = [_e4m3_enc(_fl32(_fl32(_e4m3_exact(c) * s0) / s)) for c in c0]
    c1 = [_e4m3_enc(_fl32(v / s)) for v in x1]
    # the association the policy does not use, to check the data tell them apart
    alt0 = [_e4m3_enc(_fl32(_e4m3_exact(c) * _fl32(s0 / s))) for c in c0]
    return re0, c1, s, alt0


def _bf16_code(q: Fraction) -> int:
    """Nearest bf16 code (ties to even) of a value in the normal range."""
    sign = 0x8000 if q < 0 else 0
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    n = _round_even(a / Fraction(2) ** (e - 7))
    if n == 256:
        e, n = e + 1, 128
    return sign | ((e + 127) << 7) | (n - 128)


def _discriminating_token(amax0: Fraction, amax1: Fraction, width: int):
    """bf16 codes of a token 0 whose maximum is amax0 and whose other values
    requantise differently under the two associations once a token with
    maximum amax1 grows the page (found by exhaustive search over the E4M3
    codes), padded with the first such value."""
    s0 = max(_fl32(amax0 / 448), Fraction(2) ** -126)
    s = max(_fl32(amax1 / 448), Fraction(2) ** -126)
    picks = []
    for c in range(1, 0x7F):
        a = _e4m3_enc(_fl32(_fl32(_e4m3_exact(c) * s0) / s))
        b = _e4m3_enc(_fl32(_e4m3_exact(c) * _fl32(s0 / s)))
        if a == b:
            continue
        x = _bf16_code(_e4m3_exact(c) * s0)      # a bf16 value that encodes to c at s0
        if _e4m3_enc(_fl32(_bf16_exact(x) / s0)) == c and _bf16_exact(x) < amax0:
            picks.append(x)
    codes = [_bf16_code(amax0)] + picks
    codes += [picks[0] if picks else codes[0]] * (width - len(codes))
    return np.array(codes[:width], np.uint16), len(picks)


@pytest.mark.parametrize("amax0,amax1", [(4.3125, 8.25), (2.15625, 5.625), (0.59375, 0.625),
                                         (10.5, 30.0)])
def test_append_fp8_growth_by_any_ratio_matches_exact_rounding(amax0, amax1):
    """Requantisation of the earlier token when the page scale grows by a
    ratio that is no power of two: each code equals enc(fl32(fl32(dec(c) *
    s0) / s)), computed in exact arithmetic with each fp32 step rounded once;
    token 0 holds values for which the other association, enc(fl32(dec(c) *
    fl32(s0 / s))), gives another code, so this pin tells them apart."""
    P, Hkv, d = 16, 2, 64
    bt, (k, v, ks, vs) = _one_seq(P, Hkv, d)
    x0, n_disc = _discriminating_token(Fraction(amax0), Fraction(amax1), Hkv * d)
    assert n_disc > 0, "no E4M3 code separates the two associations for this ratio"
    g = torch.Generator().manual_seed(int(amax1 * 64))
    x1 = _bf16(torch.randn(1, Hkv, d, generator=g)).reshape(-1)
    x1 = np.where(np.arange(x1.size) == 0, np.uint16(_bf16_code(Fraction(amax1))), x1)
    x1 = np.where(np.abs(_bf16_f32(x1)) > amax1, np.uint16(0), x1).astype(np.uint16)
    t0 = x0.reshape(1, Hkv, d)
    t1 = x1.reshape(1, Hkv, d)
    for t, tok in enumerate((t0, t1)):
        assert oracle.kv_append(tok, tok.copy(), bt, np.array([t + 1], np.int32), k, v,
                                kv_dtype=1, page_size=P, k_scales=ks, v_scales=vs) == 0
    page = bt[0, 0]
    re0, c1, s, alt0 = _exact_two_token_page(x0, x1)
    assert re0 != alt0
    for pool, scales, slot_of in ((k, ks, _k_slot), (v, vs, _v_slot)):
        assert Fraction(float(scales[page])) == s
        assert slot_of(pool, page, 0).reshape(-1).tolist() == re0
        assert slot_of(pool, page, 1).reshape(-1).tolist() == c1
