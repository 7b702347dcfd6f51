"""fp64 CPU oracle for DORA's rollout decode-attention hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The GPU library
never loads it and shares no code with it.

``dora_oracle.c`` states the operation from its definition (scaled dot-product
attention of one decode query per head over the sequence's cached keys and
values, gathered from a paged pool; the paper's decode step, Sec. 2.2 Eq. (1),
with per-request version tags, Sec. 3.2) and the whole-page pack/unpack of
same-version KV migration (Sec. 3.4).  This module only marshals numpy arrays
into it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dora_oracle.c")
# DORA_ORACLE_LIBRARY selects another build of the same source (the
# sanitizer build of the CPU checks); default: the in-tree one.
_LIB_PATH = os.environ.get("DORA_ORACLE_LIBRARY") or os.path.join(_HERE, "liboracle.so")
_lib = None

ERR_NAMES = {0: "ok", 1: "invalid argument", 2: "page out of range", 3: "version mismatch",
             4: "version mismatch"}


class OracleError(RuntimeError):
    pass


def build(force: bool = True) -> str:
    """Compile dora_oracle.c into liboracle.so (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        # -ffp-contract=off: the append's fp32 steps must round one by one
        cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
               _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    c_i, c_i64, c_d, c_p = ctypes.c_int, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
    lib.oracle_bf16_to_f64.argtypes = [ctypes.c_uint16]
    lib.oracle_bf16_to_f64.restype = c_d
    lib.oracle_e4m3_to_f64.argtypes = [ctypes.c_uint8]
    lib.oracle_e4m3_to_f64.restype = c_d
    dec_args = [c_i, c_i, c_i, c_i, c_i, c_i64, c_i, c_i, c_d, c_p, c_p, c_p, c_p, c_p, c_p, c_p]
    lib.oracle_decode.argtypes = dec_args + [c_p, c_p, c_p, c_i]
    lib.oracle_decode.restype = c_i
    lib.oracle_decode_brute.argtypes = dec_args + [c_p]
    lib.oracle_decode_brute.restype = c_i
    lib.oracle_packed_bytes.argtypes = [c_i, c_i, c_i, c_i, c_i64]
    lib.oracle_packed_bytes.restype = c_i64
    lib.oracle_pack.argtypes = [c_i, c_i, c_i, c_i, c_i64, c_i, c_i, c_p, c_p, c_p, c_p, c_p,
                                c_i64, c_p]
    lib.oracle_pack.restype = c_i
    lib.oracle_unpack.argtypes = [c_i, c_i, c_i, c_i, c_i64, c_i, c_p, c_p, c_i64, c_p, c_p,
                                  c_p, c_p]
    lib.oracle_unpack.restype = c_i
    lib.oracle_f32_to_e4m3.argtypes = [ctypes.c_float]
    lib.oracle_f32_to_e4m3.restype = ctypes.c_uint8
    lib.oracle_kv_append.argtypes = [c_i, c_i, c_i, c_i, c_i64, c_i, c_i, c_p, c_p, c_p, c_p,
                                     c_p, c_p, c_p, c_p]
    lib.oracle_kv_append.restype = c_i
    lib.oracle_max_threads.argtypes = []
    lib.oracle_max_threads.restype = c_i
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def bf16_to_f64(code: int) -> float:
    return _load().oracle_bf16_to_f64(int(code))


def e4m3_to_f64(code: int) -> float:
    return _load().oracle_e4m3_to_f64(int(code))


def max_threads() -> int:
    return _load().oracle_max_threads()


def _kv_bytes(a, kv_dtype):
    # Pages are passed as raw element codes: uint16 (bf16) or uint8 (fp8).
    want = np.uint16 if kv_dtype == 0 else np.uint8
    a = np.ascontiguousarray(a)
    if a.dtype != want:
        a = a.view(want)
    return a


def _decode_common(q, k_pages, v_pages, block_table, seq_lens, *, num_kv_heads, page_size,
                   kv_dtype, scale, k_scales, v_scales, num_pages):
    q = np.ascontiguousarray(q)
    if q.dtype != np.uint16:
        q = q.view(np.uint16)
    B, Hq, d = q.shape
    k_pages = _kv_bytes(k_pages, kv_dtype)
    v_pages = _kv_bytes(v_pages, kv_dtype)
    bt = _c(block_table, np.int32)
    if bt.ndim != 2 or bt.shape[0] != B:
        raise ValueError("block_table must be [B][stride]")
    lens = _c(seq_lens, np.int32)
    if num_pages is None:
        num_pages = k_pages.size // (num_kv_heads * page_size * d)
    ks = _c(k_scales, np.float32)
    vs = _c(v_scales, np.float32)
    out = np.empty((B, Hq, d), dtype=np.float64)
    args = (B, Hq, num_kv_heads, d, page_size, int(num_pages), max(1, bt.shape[1]), kv_dtype,
            float(scale), _ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(ks), _ptr(vs), _ptr(bt),
            _ptr(lens))
    return args, out, (q, k_pages, v_pages, bt, lens, ks, vs)


def decode(q, k_pages, v_pages, block_table, seq_lens, *, num_kv_heads, page_size,
           kv_dtype=0, scale=0.0, k_scales=None, v_scales=None, version_ids=None,
           page_owner=None, num_pages=None, nthreads=0):
    """Reference decode attention; returns fp64 [B][Hq][d].

    q: bf16 codes (uint16 or a bf16 view) [B][Hq][d]; k_pages / v_pages: element
    codes in the documented page layouts; scale <= 0 means 1/sqrt(d).
    """
    args, out, keep = _decode_common(q, k_pages, v_pages, block_table, seq_lens,
                                     num_kv_heads=num_kv_heads, page_size=page_size,
                                     kv_dtype=kv_dtype, scale=scale, k_scales=k_scales,
                                     v_scales=v_scales, num_pages=num_pages)
    vid = _c(version_ids, np.int32)
    own = _c(page_owner, np.int16)
    rc = _load().oracle_decode(*args, _ptr(vid), _ptr(own), _ptr(out), int(nthreads))
    del keep
    if rc != 0:
        raise OracleError(f"oracle_decode: {ERR_NAMES.get(rc, rc)} ({rc})")
    return out


def decode_rc(*a, **kw):
    """Like decode() but returns the C status code instead of raising."""
    try:
        decode(*a, **kw)
    except OracleError as e:
        return int(str(e).rsplit("(", 1)[1].rstrip(")"))
    return 0


def decode_brute(q, k_pages, v_pages, block_table, seq_lens, *, num_kv_heads, page_size,
                 kv_dtype=0, scale=0.0, k_scales=None, v_scales=None, num_pages=None):
    """Brute-force twin (no gather, long double, two-pass softmax)."""
    args, out, keep = _decode_common(q, k_pages, v_pages, block_table, seq_lens,
                                     num_kv_heads=num_kv_heads, page_size=page_size,
                                     kv_dtype=kv_dtype, scale=scale, k_scales=k_scales,
                                     v_scales=v_scales, num_pages=num_pages)
    rc = _load().oracle_decode_brute(*args, _ptr(out))
    del keep
    if rc != 0:
        raise OracleError(f"oracle_decode_brute: {ERR_NAMES.get(rc, rc)} ({rc})")
    return out


def packed_bytes(kv_dtype, page_size, num_kv_heads, head_dim, n_pages) -> int:
    return int(_load().oracle_packed_bytes(kv_dtype, page_size, num_kv_heads, head_dim,
                                           n_pages))


def pack(k_pages, v_pages, src_pages, *, kv_dtype, page_size, num_kv_heads, head_dim,
         policy_version, n_seqs=1, k_scales=None, v_scales=None):
    """Whole-page gather into the documented packed format; returns uint8 array."""
    kp = np.ascontiguousarray(k_pages).view(np.uint8)
    vp = np.ascontiguousarray(v_pages).view(np.uint8)
    pb = num_kv_heads * page_size * head_dim * (2 if kv_dtype == 0 else 1)
    num_pages = kp.size // pb
    src = _c(src_pages, np.int32)
    n = int(src.size)
    buf = np.zeros(packed_bytes(kv_dtype, page_size, num_kv_heads, head_dim, n), np.uint8)
    ks = _c(k_scales, np.float32)
    vs = _c(v_scales, np.float32)
    rc = _load().oracle_pack(kv_dtype, page_size, num_kv_heads, head_dim, num_pages,
                             policy_version, n_seqs, _ptr(kp), _ptr(vp), _ptr(ks), _ptr(vs),
                             _ptr(src), n, _ptr(buf))
    if rc != 0:
        raise OracleError(f"oracle_pack: {ERR_NAMES.get(rc, rc)} ({rc})")
    return buf


def unpack(packed, dst_pages, k_pages, v_pages, *, kv_dtype, page_size, num_kv_heads,
           head_dim, policy_version, k_scales=None, v_scales=None) -> int:
    """Whole-page scatter, in place into k_pages / v_pages (numpy); returns rc."""
    pb = num_kv_heads * page_size * head_dim * (2 if kv_dtype == 0 else 1)
    kp = k_pages.view(np.uint8).reshape(-1)
    vp = v_pages.view(np.uint8).reshape(-1)
    if not (k_pages.flags.c_contiguous and v_pages.flags.c_contiguous):
        raise ValueError("pages must be C-contiguous")
    num_pages = kp.size // pb
    dst = _c(dst_pages, np.int32)
    pk = np.ascontiguousarray(packed, dtype=np.uint8)
    return int(_load().oracle_unpack(kv_dtype, page_size, num_kv_heads, head_dim, num_pages,
                                     policy_version, _ptr(pk), _ptr(dst), int(dst.size),
                                     _ptr(kp), _ptr(vp), _ptr(k_scales), _ptr(v_scales)))


def f32_to_e4m3(x) -> np.ndarray:
    """Nearest OCP E4M3FN code of each fp32 value (ties to even, saturating)."""
    f = _load().oracle_f32_to_e4m3
    xs = np.asarray(x, dtype=np.float32).reshape(-1)
    return np.array([f(float(v)) for v in xs], dtype=np.uint8).reshape(np.shape(x))


def kv_append(k_new, v_new, block_table, seq_lens, k_pages, v_pages, *, kv_dtype, page_size,
              k_scales=None, v_scales=None) -> int:
    """Store each sequence's token seq_lens[b] - 1 (k_new / v_new: bf16 codes
    [B][Hkv][d]) into its page slot, in place in the numpy page arrays (and, for
    fp8, the per-page scales).  Returns the C status code."""
    kn = np.ascontiguousarray(k_new)
    vn = np.ascontiguousarray(v_new)
    if kn.dtype != np.uint16:
        kn = kn.view(np.uint16)
    if vn.dtype != np.uint16:
        vn = vn.view(np.uint16)
    B, Hkv, d = kn.shape
    for a in (k_pages, v_pages, k_scales, v_scales):
        if a is not None and not a.flags.c_contiguous:
            raise ValueError("pages and scales must be C-contiguous (written in place)")
    kp = k_pages.view(np.uint8).reshape(-1)
    vp = v_pages.view(np.uint8).reshape(-1)
    pb = Hkv * page_size * d * (2 if kv_dtype == 0 else 1)
    bt = _c(block_table, np.int32)
    lens = _c(seq_lens, np.int32)
    if kv_dtype == 1 and (k_scales is None or v_scales is None or
                          k_scales.dtype != np.float32 or v_scales.dtype != np.float32):
        raise ValueError("fp8 pages need float32 k_scales / v_scales arrays")
    return int(_load().oracle_kv_append(B, Hkv, d, page_size, kp.size // pb, max(1, bt.shape[1]),
                                        kv_dtype, _ptr(bt), _ptr(lens), _ptr(kn), _ptr(vn),
                                        _ptr(kp), _ptr(vp), _ptr(k_scales), _ptr(v_scales)))
