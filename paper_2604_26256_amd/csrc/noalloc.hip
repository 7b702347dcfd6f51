// dora_decode_attn_noalloc: the decode call with its workspace in a fixed
// device array of this library, for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops, harnesses that
// forbid allocation).
//
// The array is a file-scope __device__ variable, so each GPU the library runs
// on holds its own copy, at its own address, from module load until the
// process ends.  In host code its name is only a stand-in for the symbol: the
// device address comes from hipGetSymbolAddress, taken once per device with
// that device current and kept in a per-device table, and only that address
// is ever handed to kernels.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "dora_internal.h"

namespace dora {

// DORA_NOALLOC_WORKSPACE_BYTES: the largest decode workspace of any supported
// geometry at the library's default launch on a 256-CU part (1,792
// wavefronts, group 16, head_dim 128: 29.9 MB), with headroom for parts with
// more compute units or a larger caller-set wavefront count.
constexpr size_t kScratchBytes = DORA_NOALLOC_WORKSPACE_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of the current device's copy of `scratch`.
dora_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return DORA_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return DORA_ERR_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DORA_OK;
}

}  // namespace
}  // namespace dora

using namespace dora;

extern "C" {

dora_status dora_decode_attn_noalloc(const dora_decode_desc* desc, const void* q,
                                     const void* k_pages, const void* v_pages,
                                     const int32_t* block_table, const int32_t* seq_lens,
                                     const int32_t* version_ids, void* out,
                                     dora_stream_t stream) {
  if (desc && (desc->flags & DORA_FLAG_VALIDATE)) return DORA_ERR_INVALID_ARG;
  const size_t need = dora_decode_workspace_bytes(desc);
  if (need == 0)  // invalid or unsupported descriptor: the plain call names the status
    return decode_attn(desc, q, k_pages, v_pages, block_table, seq_lens, version_ids, out,
                       nullptr, 0, (hipStream_t)stream, nullptr);
  if (need > kScratchBytes) return DORA_ERR_WORKSPACE_TOO_SMALL;
  if (desc->num_seqs == 0) return DORA_OK;
  void* ws = nullptr;
  const dora_status st = scratch_address(&ws);
  if (st != DORA_OK) return st;
  return decode_attn(desc, q, k_pages, v_pages, block_table, seq_lens, version_ids, out, ws,
                     kScratchBytes, (hipStream_t)stream, nullptr);
}

}  // extern "C"
