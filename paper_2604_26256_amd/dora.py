"""Python binding of the libdora C ABI (include/dora.h): argument marshalling only.

Every step of the decode path and of pack/unpack runs in the library's HIP
kernels; this module checks that torch tensors match the geometry the kernels
assume (dtype, shape, contiguity, alignment, device), converts them to raw
pointers and passes torch's current HIP stream.  There is no fallback: if
libdora.so is missing, importing this module raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# DORA_LIBRARY selects another build of the library (the host-sanitizer build
# of the CPU checks); default: the in-tree gfx950 build.
LIB_PATH = os.environ.get("DORA_LIBRARY") or os.path.join(_PKG, "libdora.so")

DORA_OK = 0
DORA_ERR_INVALID_ARG = 1
DORA_ERR_UNSUPPORTED = 2
DORA_ERR_WORKSPACE_TOO_SMALL = 3
DORA_ERR_VERSION_MISMATCH = 4
DORA_ERR_POOL_EXHAUSTED = 5
DORA_ERR_DEVICE_CHECK = 6
DORA_ERR_HIP = 7
DORA_ERR_NOT_FOUND = 8

DORA_KV_BF16 = 0
DORA_KV_FP8_E4M3 = 1
DORA_FLAG_VALIDATE = 0x1


class DoraError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


class dora_decode_desc(ctypes.Structure):
    _fields_ = [
        ("num_seqs", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32), ("block_table_stride", ctypes.c_int32),
        ("num_pages", ctypes.c_int64), ("kv_dtype", ctypes.c_int32),
        ("sm_scale", ctypes.c_float), ("k_scales", ctypes.c_void_p),
        ("v_scales", ctypes.c_void_p), ("page_owner", ctypes.c_void_p),
        ("flags", ctypes.c_uint32), ("num_waves", ctypes.c_int32),
        ("min_range_pages", ctypes.c_int32),
    ]


class dora_pack_desc(ctypes.Structure):
    _fields_ = [
        ("kv_dtype", ctypes.c_int32), ("page_size", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("num_pages", ctypes.c_int64), ("policy_version", ctypes.c_int32),
        ("n_seqs", ctypes.c_int32),
    ]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2604_26256_amd.build`")
_lib = ctypes.CDLL(LIB_PATH)

_P, _I32, _I64, _SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
_DescP = ctypes.POINTER(dora_decode_desc)
_PackP = ctypes.POINTER(dora_pack_desc)

_lib.dora_status_string.argtypes = [ctypes.c_int]
_lib.dora_status_string.restype = ctypes.c_char_p
_lib.dora_decode_workspace_bytes.argtypes = [_DescP]
_lib.dora_decode_workspace_bytes.restype = _SZ
_lib.dora_decode_num_waves.argtypes = [_DescP]
_lib.dora_decode_num_waves.restype = _I64
_lib.dora_decode_attn_timed.argtypes = [_DescP, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P, _P]
_lib.dora_decode_attn_timed.restype = ctypes.c_int
_lib.dora_stream_read.argtypes = [_P, _I64, _P, _I64, _I32, _I32, _P, _I32, _P]
_lib.dora_stream_read.restype = ctypes.c_int
_lib.dora_decode_attn.argtypes = [_DescP, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]
_lib.dora_decode_attn.restype = ctypes.c_int
_lib.dora_decode_attn_noalloc.argtypes = [_DescP, _P, _P, _P, _P, _P, _P, _P, _P]
_lib.dora_decode_attn_noalloc.restype = ctypes.c_int
_lib.dora_decode_grouped_workspace_bytes.argtypes = [_DescP, _I32]
_lib.dora_decode_grouped_workspace_bytes.restype = _SZ
_lib.dora_decode_attn_grouped.argtypes = [_DescP, _P, _P, _P, _P, _P, _P, _P, _I32, _P, _P,
                                          _SZ, _P]
_lib.dora_decode_attn_grouped.restype = ctypes.c_int
_lib.dora_kv_append.argtypes = [_DescP, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]
_lib.dora_kv_append.restype = ctypes.c_int
_lib.dora_plan_partition.argtypes = [ctypes.POINTER(_I64), _I32, _I32, ctypes.POINTER(_I32)]
_lib.dora_plan_partition.restype = ctypes.c_int
_lib.dora_plan_supplement.argtypes = [ctypes.POINTER(_I32), ctypes.POINTER(_I32), _I32, _I32,
                                      _I64, ctypes.POINTER(_I32)]
_lib.dora_plan_supplement.restype = ctypes.c_int
_lib.dora_kv_packed_bytes.argtypes = [_PackP, _I64]
_lib.dora_kv_packed_bytes.restype = _SZ
_lib.dora_kv_page_pack.argtypes = [_PackP, _P, _P, _P, _P, _P, _I64, _P, _SZ, _P]
_lib.dora_kv_page_pack.restype = ctypes.c_int
_lib.dora_kv_page_unpack.argtypes = [_PackP, _I32, _P, _SZ, _P, _I64, _P, _P, _P, _P, _P, _P]
_lib.dora_kv_page_unpack.restype = ctypes.c_int
_lib.dora_pool_create.argtypes = [_I64, _I32, _I32, ctypes.c_uint64, ctypes.POINTER(_P)]
_lib.dora_pool_create.restype = ctypes.c_int
_lib.dora_pool_destroy.argtypes = [_P]
_lib.dora_pool_destroy.restype = None
_lib.dora_pool_add_seq.argtypes = [_P, _I32, _I32, ctypes.POINTER(_I64)]
_lib.dora_pool_add_seq.restype = ctypes.c_int
_lib.dora_pool_extend_seq.argtypes = [_P, _I64, _I32]
_lib.dora_pool_extend_seq.restype = ctypes.c_int
_lib.dora_pool_free_seq.argtypes = [_P, _I64]
_lib.dora_pool_free_seq.restype = ctypes.c_int
_lib.dora_pool_seq_info.argtypes = [_P, _I64, _P, _P, _P]
_lib.dora_pool_seq_info.restype = ctypes.c_int
_lib.dora_pool_seq_pages.argtypes = [_P, _I64, _P, _I32, ctypes.POINTER(_I32)]
_lib.dora_pool_seq_pages.restype = ctypes.c_int
_lib.dora_pool_block_table.argtypes = [_P, _P, _I32, _I32, _P, _P, _P]
_lib.dora_pool_block_table.restype = ctypes.c_int
_lib.dora_pool_page_owner.argtypes = [_P, _P]
_lib.dora_pool_page_owner.restype = ctypes.c_int
_lib.dora_pool_stats.argtypes = [_P, _I32, ctypes.POINTER(_I64), ctypes.POINTER(_I64)]
_lib.dora_pool_stats.restype = ctypes.c_int
_lib.dora_pool_migrate_seq.argtypes = [_P, _I64, _P, _I32, ctypes.POINTER(_I64), _P, _P, _I32,
                                       ctypes.POINTER(_I32)]
_lib.dora_pool_migrate_seq.restype = ctypes.c_int


def library():
    """The loaded ctypes library (for symbol checks)."""
    return _lib


def status_string(status: int) -> str:
    return _lib.dora_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != DORA_OK:
        raise DoraError(status, where)


# ---------------------------------------------------------------------------
# tensor marshalling helpers
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _dev_ptr(t, name, dtypes, shape=None, numel=None, align=16):
    torch = _torch()
    if t is None:
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU (got {t.device})")
    if t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype} not in {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)} != expected {tuple(shape)}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name}: {t.numel()} elements != expected {numel}")
    if t.data_ptr() % align != 0:
        raise ValueError(f"{name} must be {align}-byte aligned")
    return ctypes.c_void_p(t.data_ptr())


def _buf_ptr(t, name):
    """A uint8 buffer the GPU can address: device memory, or pinned host memory
    (torch's pin_memory allocations are hipHostMalloc'd and mapped, so the same
    pointer works in kernels)."""
    torch = _torch()
    if isinstance(t, torch.Tensor) and t.device.type == "cpu":
        if not t.is_pinned():
            raise ValueError(f"{name}: host buffers must be pinned (pin_memory=True)")
        if t.dtype != torch.uint8 or not t.is_contiguous() or t.data_ptr() % 16:
            raise ValueError(f"{name}: contiguous, 16-byte aligned uint8 required")
        return ctypes.c_void_p(t.data_ptr())
    return _dev_ptr(t, name, (torch.uint8,))


def _opt_ptr(t, name, dtypes, **kw):
    return None if t is None else _dev_ptr(t, name, dtypes, **kw)


def _stream_handle(stream):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _kv_geometry(k_pages, v_pages, num_kv_heads, page_size, head_dim, kv_dtype):
    torch = _torch()
    X = 16 // (2 if kv_dtype == DORA_KV_BF16 else 1)
    if head_dim % X:
        raise ValueError("head_dim must be a multiple of 16 bytes of elements")
    kshape_tail = (num_kv_heads, head_dim // X, page_size, X)
    vshape_tail = (num_kv_heads, head_dim, page_size)
    if tuple(k_pages.shape[1:]) != kshape_tail:
        raise ValueError(f"k_pages must be [num_pages]{list(kshape_tail)}, got "
                         f"{list(k_pages.shape)}")
    if tuple(v_pages.shape[1:]) != vshape_tail or v_pages.shape[0] != k_pages.shape[0]:
        raise ValueError(f"v_pages must be [num_pages]{list(vshape_tail)}, got "
                         f"{list(v_pages.shape)}")
    kv_types = (torch.bfloat16,) if kv_dtype == DORA_KV_BF16 else (torch.uint8,
                                                                   torch.float8_e4m3fn)
    return int(k_pages.shape[0]), kv_types


def make_decode_desc(*, num_seqs, num_q_heads, num_kv_heads, head_dim, page_size,
                     block_table_stride, num_pages, kv_dtype=DORA_KV_BF16, sm_scale=0.0,
                     k_scales=None, v_scales=None, page_owner=None, flags=0, num_waves=0,
                     min_range_pages=0) -> dora_decode_desc:
    d = dora_decode_desc()
    d.num_seqs, d.num_q_heads, d.num_kv_heads = num_seqs, num_q_heads, num_kv_heads
    d.head_dim, d.page_size, d.block_table_stride = head_dim, page_size, block_table_stride
    d.num_pages, d.kv_dtype, d.sm_scale = num_pages, kv_dtype, float(sm_scale)
    d.k_scales = None if k_scales is None else k_scales.data_ptr()
    d.v_scales = None if v_scales is None else v_scales.data_ptr()
    d.page_owner = None if page_owner is None else page_owner.data_ptr()
    d.flags, d.num_waves, d.min_range_pages = flags, num_waves, min_range_pages
    return d


def dora_decode_workspace_bytes(desc: dora_decode_desc) -> int:
    return int(_lib.dora_decode_workspace_bytes(ctypes.byref(desc)))


def dora_decode_grouped_workspace_bytes(desc: dora_decode_desc, group_size) -> int:
    """Workspace of dora_decode_attn_grouped (0 on invalid arguments)."""
    return int(_lib.dora_decode_grouped_workspace_bytes(ctypes.byref(desc), int(group_size)))


def dora_decode_num_waves(desc: dora_decode_desc) -> int:
    """Decode wavefronts per launch for this descriptor on the current device."""
    return int(_lib.dora_decode_num_waves(ctypes.byref(desc)))


# Workspaces the binding allocates when the caller passes none: one per
# (device, stream), allocated on that stream (so the caching allocator orders
# its reuse after the stream's pending work), and replaced when a call needs a
# different size.  Calls on different streams never share one.
_ws_cache = {}


def _cached_workspace(cache, device, stream, need):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream(device)
    key = (device.index, s.cuda_stream)
    ws = cache.get(key)
    if ws is None or ws.numel() != need:
        cache.pop(key, None)
        with torch.cuda.stream(s):
            ws = torch.empty(need, dtype=torch.uint8, device=device)
        cache[key] = ws
    return ws


def _decode_args(q, k_pages, v_pages, block_table, seq_lens, version_ids, out, *, num_kv_heads,
                 page_size, kv_dtype, sm_scale, k_scales, v_scales, page_owner, flags,
                 num_waves, min_range_pages):
    torch = _torch()
    B, Hq, D = (int(x) for x in q.shape)
    num_pages, kv_types = _kv_geometry(k_pages, v_pages, num_kv_heads, page_size, D, kv_dtype)
    if block_table.dim() != 2 or block_table.shape[0] != B:
        raise ValueError("block_table must be [B][stride]")
    stride = int(block_table.shape[1])
    desc = make_decode_desc(num_seqs=B, num_q_heads=Hq, num_kv_heads=num_kv_heads, head_dim=D,
                            page_size=page_size, block_table_stride=max(1, stride),
                            num_pages=num_pages, kv_dtype=kv_dtype, sm_scale=sm_scale,
                            k_scales=k_scales, v_scales=v_scales, page_owner=page_owner,
                            flags=flags, num_waves=num_waves,
                            min_range_pages=min_range_pages)
    if B == 0:
        return desc, None
    args = [
        _dev_ptr(q, "q", (torch.bfloat16,), shape=(B, Hq, D)),
        _dev_ptr(k_pages, "k_pages", kv_types),
        _dev_ptr(v_pages, "v_pages", kv_types),
        _dev_ptr(block_table, "block_table", (torch.int32,), shape=(B, stride), align=4),
        _dev_ptr(seq_lens, "seq_lens", (torch.int32,), shape=(B,), align=4),
        _opt_ptr(version_ids, "version_ids", (torch.int32,), shape=(B,), align=4),
        _dev_ptr(out, "out", (torch.bfloat16,), shape=(B, Hq, D)),
    ]
    if kv_dtype == DORA_KV_FP8_E4M3:
        _dev_ptr(k_scales, "k_scales", (torch.float32,), shape=(num_pages,), align=4)
        _dev_ptr(v_scales, "v_scales", (torch.float32,), shape=(num_pages,), align=4)
    if page_owner is not None:
        _dev_ptr(page_owner, "page_owner", (torch.int16,), shape=(num_pages,), align=2)
    return desc, args


def dora_decode_attn(q, k_pages, v_pages, block_table, seq_lens, version_ids, out, *,
                     num_kv_heads: int, page_size: int, kv_dtype: int = DORA_KV_BF16,
                     sm_scale: float = 0.0, k_scales=None, v_scales=None, page_owner=None,
                     flags: int = 0, num_waves: int = 0, min_range_pages: int = 0,
                     workspace=None, stream=None, events=None):
    """Decode-step attention over the paged pool (see include/dora.h).

    q, out: bf16 [B][Hq][d]; k_pages: [num_pages][Hkv][d/X][P][X]; v_pages:
    [num_pages][Hkv][d][P] (bf16, or uint8 / float8_e4m3fn codes with fp32
    k_scales / v_scales [num_pages]); block_table int32 [B][stride]; seq_lens,
    version_ids int32 [B].  num_waves / min_range_pages override how the
    work is cut (0 = library default).  stream: a torch stream (default: the
    current one).  The workspace is allocated when not given (cached per
    device and stream).  events: three raw hipEvent_t handles, which selects
    dora_decode_attn_timed (include/dora_measure.h).  Returns `out`.
    """
    desc, args = _decode_args(q, k_pages, v_pages, block_table, seq_lens, version_ids, out,
                              num_kv_heads=num_kv_heads, page_size=page_size,
                              kv_dtype=kv_dtype, sm_scale=sm_scale, k_scales=k_scales,
                              v_scales=v_scales, page_owner=page_owner, flags=flags,
                              num_waves=num_waves, min_range_pages=min_range_pages)
    if args is None:
        return out
    need = dora_decode_workspace_bytes(desc)
    if need == 0:
        # invalid or unsupported geometry: let the library name the reason
        _check(_lib.dora_decode_attn(ctypes.byref(desc), *args, None, 0,
                                     _stream_handle(stream)), "dora_decode_attn")
    if workspace is None:
        workspace = _cached_workspace(_ws_cache, q.device, stream, need)
    ws_ptr = _dev_ptr(workspace, "workspace", (_torch().uint8,))
    if events is None:
        st = _lib.dora_decode_attn(ctypes.byref(desc), *args, ws_ptr, workspace.numel(),
                                   _stream_handle(stream))
        _check(st, "dora_decode_attn")
    else:
        if len(events) != 3:
            raise ValueError("events needs 3 hipEvent_t handles")
        arr = (ctypes.c_void_p * 3)(*[ctypes.c_void_p(e) for e in events])
        st = _lib.dora_decode_attn_timed(ctypes.byref(desc), *args, ws_ptr, workspace.numel(),
                                         _stream_handle(stream), ctypes.cast(arr, _P))
        _check(st, "dora_decode_attn_timed")
    return out


class PreparedDecode:
    """dora_decode_attn with its arguments checked and marshalled once, for
    host loops that call the same batch buffers step after step.

    Takes the arguments of dora_decode_attn and checks them as it does; a call
    of the object then runs only the C call, so it costs the C ABI's own host
    time, a fraction of what dora_decode_attn spends checking every tensor on
    every call.  The object keeps references to the tensors and
    their device addresses: refill q, block_table, seq_lens, version_ids (and
    the pages and scales) in place between calls, on the same stream or
    ordered before it; new tensors need a new object.  Geometry, flags and
    the stream (default: the current stream when the object is made) are
    fixed.  It owns a workspace of its own (or uses the one given), so calls
    of different objects never share one; calls of one object are ordered by
    its stream.  Returns `out` from each call."""

    def __init__(self, q, k_pages, v_pages, block_table, seq_lens, version_ids, out, *,
                 num_kv_heads: int, page_size: int, kv_dtype: int = DORA_KV_BF16,
                 sm_scale: float = 0.0, k_scales=None, v_scales=None, page_owner=None,
                 flags: int = 0, num_waves: int = 0, min_range_pages: int = 0,
                 workspace=None, stream=None):
        torch = _torch()
        self.out = out
        self._keep = (q, k_pages, v_pages, block_table, seq_lens, version_ids, out, k_scales,
                      v_scales, page_owner)
        self._desc, args = _decode_args(
            q, k_pages, v_pages, block_table, seq_lens, version_ids, out,
            num_kv_heads=num_kv_heads, page_size=page_size, kv_dtype=kv_dtype,
            sm_scale=sm_scale, k_scales=k_scales, v_scales=v_scales, page_owner=page_owner,
            flags=flags, num_waves=num_waves, min_range_pages=min_range_pages)
        self._args = None
        if args is None:  # empty batch: every call is a no-op
            return
        s = stream if stream is not None else torch.cuda.current_stream(q.device)
        handle = ctypes.c_void_p(s.cuda_stream)
        need = dora_decode_workspace_bytes(self._desc)
        if need == 0:  # invalid or unsupported geometry: let the library name the reason
            _check(_lib.dora_decode_attn(ctypes.byref(self._desc), *args, None, 0, handle),
                   "dora_decode_attn")
        if workspace is None:
            with torch.cuda.stream(s):
                workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
        elif workspace.numel() < need:
            raise ValueError(f"workspace: {workspace.numel()} bytes, {need} needed")
        self.workspace = workspace
        ws_ptr = _dev_ptr(workspace, "workspace", (torch.uint8,))
        self._args = (ctypes.byref(self._desc), *args, ws_ptr, workspace.numel(), handle)

    def __call__(self):
        if self._args is not None:
            st = _lib.dora_decode_attn(*self._args)
            if st != DORA_OK:
                raise DoraError(st, "dora_decode_attn")
        return self.out


NOALLOC_WORKSPACE_BYTES = 48 << 20   # DORA_NOALLOC_WORKSPACE_BYTES


def dora_decode_attn_noalloc(q, k_pages, v_pages, block_table, seq_lens, version_ids, out, *,
                             num_kv_heads: int, page_size: int, kv_dtype: int = DORA_KV_BF16,
                             sm_scale: float = 0.0, k_scales=None, v_scales=None,
                             page_owner=None, flags: int = 0, num_waves: int = 0,
                             min_range_pages: int = 0, stream=None):
    """dora_decode_attn with the library's fixed per-GPU workspace: neither the
    library nor this wrapper allocates device memory.  Calls that overlap on
    one GPU race on that workspace (see include/dora.h).  Returns `out`."""
    desc, args = _decode_args(q, k_pages, v_pages, block_table, seq_lens, version_ids, out,
                              num_kv_heads=num_kv_heads, page_size=page_size,
                              kv_dtype=kv_dtype, sm_scale=sm_scale, k_scales=k_scales,
                              v_scales=v_scales, page_owner=page_owner, flags=flags,
                              num_waves=num_waves, min_range_pages=min_range_pages)
    if args is None:
        return out
    _check(_lib.dora_decode_attn_noalloc(ctypes.byref(desc), *args, _stream_handle(stream)),
           "dora_decode_attn_noalloc")
    return out


def dora_stream_read(base, tiles, sink, *, tile_bytes=4096, tiles_per_batch=4, stream=None):
    """Streaming-read reference (include/dora_measure.h): read the tiles of
    `base` (device uint8) listed in `tiles` (device int32) with non-temporal
    loads, tiles_per_batch tiles per batch and two batches in flight, one
    wavefront per entry of `sink` (device int32/uint32 words)."""
    torch = _torch()
    n = int(tiles.numel())
    st = _lib.dora_stream_read(
        _dev_ptr(base, "base", (torch.uint8,)), base.numel(),
        _dev_ptr(tiles, "tiles", (torch.int32,), numel=n, align=4) if n else None, n,
        int(tile_bytes), int(tiles_per_batch),
        _dev_ptr(sink, "sink", (torch.int32, torch.uint32), align=4),
        int(sink.numel()), _stream_handle(stream))
    _check(st, "dora_stream_read")
    return sink


_gws_cache = {}


def dora_decode_attn_grouped(q, k_pages, v_pages, block_table, seq_lens, version_ids, out, *,
                             group_size, num_kv_heads, page_size, kv_dtype=DORA_KV_BF16,
                             sm_scale=0.0, k_scales=None, v_scales=None, page_owner=None,
                             flags=0, shared_pages_out=None, workspace=None, stream=None):
    """Decode attention for groups of `group_size` consecutive sequences; the
    pages a group's members share (same leading page ids, full pages) are read
    once per group.  shared_pages_out: optional device int32 [B / group_size]
    that receives each group's shared page count.  See include/dora.h."""
    torch = _torch()
    B, Hq, D = (int(x) for x in q.shape)
    num_pages, kv_types = _kv_geometry(k_pages, v_pages, num_kv_heads, page_size, D, kv_dtype)
    if block_table.dim() != 2 or block_table.shape[0] != B:
        raise ValueError("block_table must be [B][stride]")
    stride = int(block_table.shape[1])
    desc = make_decode_desc(num_seqs=B, num_q_heads=Hq, num_kv_heads=num_kv_heads, head_dim=D,
                            page_size=page_size, block_table_stride=max(1, stride),
                            num_pages=num_pages, kv_dtype=kv_dtype, sm_scale=sm_scale,
                            k_scales=k_scales, v_scales=v_scales, page_owner=page_owner,
                            flags=flags)
    if B == 0:
        return out
    M = int(group_size)
    args = [
        _dev_ptr(q, "q", (torch.bfloat16,), shape=(B, Hq, D)),
        _dev_ptr(k_pages, "k_pages", kv_types),
        _dev_ptr(v_pages, "v_pages", kv_types),
        _dev_ptr(block_table, "block_table", (torch.int32,), shape=(B, stride), align=4),
        _dev_ptr(seq_lens, "seq_lens", (torch.int32,), shape=(B,), align=4),
        _opt_ptr(version_ids, "version_ids", (torch.int32,), shape=(B,), align=4),
        _dev_ptr(out, "out", (torch.bfloat16,), shape=(B, Hq, D)),
        M,
        _opt_ptr(shared_pages_out, "shared_pages_out", (torch.int32,),
                 shape=(B // M if M > 0 else 0,), align=4),
    ]
    if kv_dtype == DORA_KV_FP8_E4M3:
        _dev_ptr(k_scales, "k_scales", (torch.float32,), shape=(num_pages,), align=4)
        _dev_ptr(v_scales, "v_scales", (torch.float32,), shape=(num_pages,), align=4)
    need = int(_lib.dora_decode_grouped_workspace_bytes(ctypes.byref(desc), M))
    if need == 0:  # invalid arguments: the call reports which status
        _check(_lib.dora_decode_attn_grouped(ctypes.byref(desc), *args, None, 0,
                                             _stream_handle(stream)),
               "dora_decode_attn_grouped")
    if workspace is None:
        workspace = _cached_workspace(_gws_cache, q.device, stream, need)
    st = _lib.dora_decode_attn_grouped(ctypes.byref(desc), *args,
                                       _dev_ptr(workspace, "workspace", (torch.uint8,)),
                                       workspace.numel(), _stream_handle(stream))
    _check(st, "dora_decode_attn_grouped")
    return out


def dora_kv_append(k_new, v_new, block_table, seq_lens, k_pages, v_pages, *, num_kv_heads,
                   page_size, kv_dtype=DORA_KV_BF16, k_scales=None, v_scales=None,
                   version_ids=None, page_owner=None, flags=0, dev_status=None, stream=None):
    """Store each sequence's current token (k_new / v_new: bf16 [B][Hkv][d],
    token seq_lens[b] - 1) into its page slot, in place (see include/dora.h).
    fp8 pools update their per-page k_scales / v_scales (fp32 [num_pages])."""
    torch = _torch()
    B, Hkv, D = (int(x) for x in k_new.shape)
    if Hkv != num_kv_heads:
        raise ValueError("k_new must be [B][num_kv_heads][head_dim]")
    num_pages, kv_types = _kv_geometry(k_pages, v_pages, num_kv_heads, page_size, D, kv_dtype)
    if block_table.dim() != 2 or block_table.shape[0] != B:
        raise ValueError("block_table must be [B][stride]")
    stride = int(block_table.shape[1])
    desc = make_decode_desc(num_seqs=B, num_q_heads=num_kv_heads, num_kv_heads=num_kv_heads,
                            head_dim=D, page_size=page_size, block_table_stride=max(1, stride),
                            num_pages=num_pages, kv_dtype=kv_dtype, page_owner=page_owner,
                            flags=flags)
    if B == 0:
        return
    fp8 = kv_dtype == DORA_KV_FP8_E4M3
    args = [
        _dev_ptr(k_new, "k_new", (torch.bfloat16,), shape=(B, Hkv, D)),
        _dev_ptr(v_new, "v_new", (torch.bfloat16,), shape=(B, Hkv, D)),
        _dev_ptr(block_table, "block_table", (torch.int32,), shape=(B, stride), align=4),
        _dev_ptr(seq_lens, "seq_lens", (torch.int32,), shape=(B,), align=4),
        _opt_ptr(version_ids, "version_ids", (torch.int32,), shape=(B,), align=4),
        _dev_ptr(k_pages, "k_pages", kv_types),
        _dev_ptr(v_pages, "v_pages", kv_types),
        _dev_ptr(k_scales, "k_scales", (torch.float32,), shape=(num_pages,), align=4)
        if fp8 else None,
        _dev_ptr(v_scales, "v_scales", (torch.float32,), shape=(num_pages,), align=4)
        if fp8 else None,
        _opt_ptr(dev_status, "dev_status", (torch.int32,), numel=1, align=4),
    ]
    if page_owner is not None:
        _dev_ptr(page_owner, "page_owner", (torch.int16,), shape=(num_pages,), align=2)
    _check(_lib.dora_kv_append(ctypes.byref(desc), *args, _stream_handle(stream)),
           "dora_kv_append")


def plan_partition(workload, n_groups):
    """DP groups per policy version (oldest first) in proportion to workload."""
    n = len(workload)
    out = (ctypes.c_int32 * n)()
    _check(_lib.dora_plan_partition((ctypes.c_int64 * n)(*[int(w) for w in workload]), n,
                                    int(n_groups), out), "dora_plan_partition")
    return list(out)


def plan_supplement(groups, active, slots_per_group, latest_quota):
    """Prompts to inject per version: latest first, legacy up to idle slots."""
    n = len(groups)
    out = (ctypes.c_int32 * n)()
    _check(_lib.dora_plan_supplement((ctypes.c_int32 * n)(*[int(g) for g in groups]),
                                     (ctypes.c_int32 * n)(*[int(a) for a in active]), n,
                                     int(slots_per_group), int(latest_quota), out),
           "dora_plan_supplement")
    return list(out)


# ---------------------------------------------------------------------------
# pack / unpack
# ---------------------------------------------------------------------------

def make_pack_desc(*, kv_dtype, page_size, num_kv_heads, head_dim, num_pages, policy_version,
                   n_seqs=1) -> dora_pack_desc:
    d = dora_pack_desc()
    d.kv_dtype, d.page_size, d.num_kv_heads, d.head_dim = kv_dtype, page_size, num_kv_heads, \
        head_dim
    d.num_pages, d.policy_version, d.n_seqs = num_pages, policy_version, n_seqs
    return d


def dora_kv_packed_bytes(desc: dora_pack_desc, n_pages: int) -> int:
    return int(_lib.dora_kv_packed_bytes(ctypes.byref(desc), int(n_pages)))


def dora_kv_page_pack(k_pages, v_pages, src_pages, packed, *, num_kv_heads, page_size, head_dim,
                      kv_dtype=DORA_KV_BF16, policy_version=0, n_seqs=1, k_scales=None,
                      v_scales=None, stream=None):
    """Gather pages src_pages (device int32) into `packed`: a device uint8
    buffer, or a pinned host one (offload to host memory)."""
    torch = _torch()
    num_pages, kv_types = _kv_geometry(k_pages, v_pages, num_kv_heads, page_size, head_dim,
                                       kv_dtype)
    desc = make_pack_desc(kv_dtype=kv_dtype, page_size=page_size, num_kv_heads=num_kv_heads,
                          head_dim=head_dim, num_pages=num_pages,
                          policy_version=policy_version, n_seqs=n_seqs)
    n = int(src_pages.numel())
    fp8 = kv_dtype == DORA_KV_FP8_E4M3
    st = _lib.dora_kv_page_pack(
        ctypes.byref(desc), _dev_ptr(k_pages, "k_pages", kv_types),
        _dev_ptr(v_pages, "v_pages", kv_types),
        _dev_ptr(k_scales, "k_scales", (torch.float32,), shape=(num_pages,), align=4) if fp8
        else None,
        _dev_ptr(v_scales, "v_scales", (torch.float32,), shape=(num_pages,), align=4) if fp8
        else None,
        _dev_ptr(src_pages, "src_pages", (torch.int32,), numel=n, align=4) if n else None, n,
        _buf_ptr(packed, "packed"), packed.numel(), _stream_handle(stream))
    _check(st, "dora_kv_page_pack")
    return packed


def dora_kv_page_unpack(packed, dst_pages, k_pages, v_pages, *, src_version, num_kv_heads,
                        page_size, head_dim, kv_dtype=DORA_KV_BF16, policy_version=0,
                        k_scales=None, v_scales=None, dev_status=None, stream=None):
    """Scatter `packed` (device, or pinned host memory: restore from host) into
    pages dst_pages of a destination pool of version policy_version;
    src_version is the version tag of the migrating request."""
    torch = _torch()
    num_pages, kv_types = _kv_geometry(k_pages, v_pages, num_kv_heads, page_size, head_dim,
                                       kv_dtype)
    desc = make_pack_desc(kv_dtype=kv_dtype, page_size=page_size, num_kv_heads=num_kv_heads,
                          head_dim=head_dim, num_pages=num_pages,
                          policy_version=policy_version)
    n = int(dst_pages.numel())
    fp8 = kv_dtype == DORA_KV_FP8_E4M3
    st = _lib.dora_kv_page_unpack(
        ctypes.byref(desc), int(src_version), _buf_ptr(packed, "packed"),
        packed.numel(),
        _dev_ptr(dst_pages, "dst_pages", (torch.int32,), numel=n, align=4) if n else None, n,
        _dev_ptr(k_pages, "k_pages", kv_types), _dev_ptr(v_pages, "v_pages", kv_types),
        _dev_ptr(k_scales, "k_scales", (torch.float32,), shape=(num_pages,), align=4) if fp8
        else None,
        _dev_ptr(v_scales, "v_scales", (torch.float32,), shape=(num_pages,), align=4) if fp8
        else None,
        _opt_ptr(dev_status, "dev_status", (torch.int32,), numel=1, align=4),
        _stream_handle(stream))
    _check(st, "dora_kv_page_unpack")


# ---------------------------------------------------------------------------
# host page pool
# ---------------------------------------------------------------------------

class Pool:
    """Host page pool (dora_pool_*): pages, owners and per-version sequences."""

    def __init__(self, num_pages: int, page_size: int, num_versions: int, seed: int = 0):
        h = ctypes.c_void_p()
        _check(_lib.dora_pool_create(num_pages, page_size, num_versions, seed,
                                     ctypes.byref(h)), "dora_pool_create")
        self._h = h
        self.num_pages, self.page_size, self.num_versions = num_pages, page_size, num_versions

    def close(self):
        if self._h:
            _lib.dora_pool_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def handle(self):
        return self._h

    def add_seq(self, version: int, num_tokens: int) -> int:
        sid = ctypes.c_int64()
        _check(_lib.dora_pool_add_seq(self._h, version, num_tokens, ctypes.byref(sid)),
               "dora_pool_add_seq")
        return sid.value

    def extend_seq(self, seq_id: int, new_num_tokens: int):
        _check(_lib.dora_pool_extend_seq(self._h, seq_id, new_num_tokens), "dora_pool_extend_seq")

    def free_seq(self, seq_id: int):
        _check(_lib.dora_pool_free_seq(self._h, seq_id), "dora_pool_free_seq")

    def seq_info(self, seq_id: int):
        t, v, n = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(_lib.dora_pool_seq_info(self._h, seq_id, ctypes.byref(t), ctypes.byref(v),
                                       ctypes.byref(n)), "dora_pool_seq_info")
        return t.value, v.value, n.value

    def seq_pages(self, seq_id: int) -> np.ndarray:
        _, _, n = self.seq_info(seq_id)
        out = np.zeros(max(1, n), np.int32)
        got = ctypes.c_int32()
        _check(_lib.dora_pool_seq_pages(self._h, seq_id, out.ctypes.data_as(_P), len(out),
                                        ctypes.byref(got)), "dora_pool_seq_pages")
        return out[:got.value]

    def block_table(self, seq_ids: Sequence[int], stride: Optional[int] = None):
        ids = np.asarray(seq_ids, np.int64)
        if stride is None:
            stride = max([self.seq_info(int(s))[2] for s in ids] + [1])
        table = np.zeros((len(ids), stride), np.int32)
        lens = np.zeros(len(ids), np.int32)
        vers = np.zeros(len(ids), np.int32)
        _check(_lib.dora_pool_block_table(self._h, ids.ctypes.data_as(_P), len(ids), stride,
                                          table.ctypes.data_as(_P), lens.ctypes.data_as(_P),
                                          vers.ctypes.data_as(_P)), "dora_pool_block_table")
        return table, lens, vers

    def page_owner(self) -> np.ndarray:
        out = np.zeros(self.num_pages, np.int16)
        _check(_lib.dora_pool_page_owner(self._h, out.ctypes.data_as(_P)), "dora_pool_page_owner")
        return out

    def stats(self, version: int = -1):
        used, free = ctypes.c_int64(), ctypes.c_int64()
        _check(_lib.dora_pool_stats(self._h, version, ctypes.byref(used), ctypes.byref(free)),
               "dora_pool_stats")
        return used.value, free.value

    def migrate_seq(self, seq_id: int, dst: "Pool", dst_version: int):
        """Returns (dst_seq_id, src_pages, dst_pages) for pack/unpack."""
        _, _, n = self.seq_info(seq_id)
        cap = max(1, n)
        src = np.zeros(cap, np.int32)
        dstp = np.zeros(cap, np.int32)
        new_id, got = ctypes.c_int64(), ctypes.c_int32()
        _check(_lib.dora_pool_migrate_seq(self._h, seq_id, dst._h, dst_version,
                                          ctypes.byref(new_id), src.ctypes.data_as(_P),
                                          dstp.ctypes.data_as(_P), cap, ctypes.byref(got)),
               "dora_pool_migrate_seq")
        return new_id.value, src[:got.value], dstp[:got.value]
