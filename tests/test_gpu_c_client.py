"""The library driven from C on the GPU: tests/c_gpu_client.c, built by
__graft_entry__.build() into tests/libc_gpu_client.so, allocates its buffers
with hipMalloc, builds a ragged batch in the header's page layouts, checks
dora_decode_attn against the fp64 oracle (2e-2) and a pack/unpack migration
byte for byte; a second entry point runs fp8 rollout steps from C (host pool,
KV append against the oracle's append byte for byte, decode against the
oracle, the no-allocation call, a migration to a second pool).  The entry
points run in this process (no exec)."""
import ctypes
import os

import pytest

pytestmark = pytest.mark.gpu

LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libc_gpu_client.so")


def test_c_client_decodes_and_migrates_on_the_gpu(capfd):
    print("[case] C client", flush=True)
    if not os.path.exists(LIB):
        pytest.fail("tests/libc_gpu_client.so is not built (run __graft_entry__.build())")
    rc = ctypes.CDLL(LIB).dora_c_gpu_client()
    out = capfd.readouterr().out
    assert rc == 0 and out.strip().endswith("ok"), out


def test_c_client_runs_fp8_rollout_steps_on_the_gpu(capfd):
    print("[case] C client step loop", flush=True)
    if not os.path.exists(LIB):
        pytest.fail("tests/libc_gpu_client.so is not built (run __graft_entry__.build())")
    rc = ctypes.CDLL(LIB).dora_c_gpu_step_loop()
    out = capfd.readouterr().out
    assert rc == 0 and out.strip().endswith("ok"), out
