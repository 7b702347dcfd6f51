"""MI355X (gfx950) decode-attention hot path of DORA's rollout stage.

The compute lives in libdora.so (HIP kernels behind the C ABI declared in
include/dora.h); ``paper_2604_26256_amd.dora`` is its thin ctypes binding.
The binding is loaded on first use, so ``paper_2604_26256_amd.build`` can run
before the library exists.
"""
_EXPORTS = (
    "DORA_FLAG_VALIDATE", "DORA_KV_BF16", "DORA_KV_FP8_E4M3", "DoraError", "Pool",
    "PreparedDecode",
    "dora_decode_attn", "dora_decode_attn_grouped", "dora_decode_workspace_bytes",
    "dora_kv_append", "dora_kv_packed_bytes", "dora_kv_page_pack", "dora_kv_page_unpack",
    "make_decode_desc", "make_pack_desc", "plan_partition", "plan_supplement",
    "status_string",
)
__all__ = list(_EXPORTS)


def __getattr__(name):
    if name in _EXPORTS:
        from . import dora
        return getattr(dora, name)
    raise AttributeError(name)
