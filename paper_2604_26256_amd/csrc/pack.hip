// Whole-page KV gather (pack) and scatter (unpack) for same-version request
// migration: the KV-data phase of the paper's two-phase state transfer
// (Sec. 3.4).  Pages are moved as raw bytes, so the copy is bit-exact and the
// destination decodes exactly as the source did.
//
// Both kernels are HBM-bound streaming copies: each workgroup moves one
// 16 KiB chunk of one page (K or V) with 16-byte loads, all loads issued before
// the stores, so a wave keeps 4 x 1 KiB in flight.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include "dora_internal.h"

namespace dora {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCopyThreads = 256;
constexpr int kCopyUnroll = 4;
constexpr int64_t kChunkBytes = (int64_t)kCopyThreads * kCopyUnroll * 16;  // 16 KiB

void make_pack_header(const dora_pack_desc& d, int64_t n_pages, PackHeader* h) {
  memset(h, 0, sizeof *h);
  const int e = d.kv_dtype == DORA_KV_BF16 ? 2 : 1;
  const int64_t page_bytes = (int64_t)d.num_kv_heads * d.page_size * d.head_dim * e;
  uint8_t* p = (uint8_t*)h->words;
  memcpy(p + 0, "DORAKV01", 8);
  int32_t v32;
  v32 = 1;                memcpy(p + 8, &v32, 4);
  v32 = d.policy_version; memcpy(p + 12, &v32, 4);
  v32 = d.kv_dtype;       memcpy(p + 16, &v32, 4);
  v32 = d.page_size;      memcpy(p + 20, &v32, 4);
  v32 = d.num_kv_heads;   memcpy(p + 24, &v32, 4);
  v32 = d.head_dim;       memcpy(p + 28, &v32, 4);
  memcpy(p + 32, &n_pages, 8);
  memcpy(p + 40, &page_bytes, 8);
  v32 = d.n_seqs;         memcpy(p + 48, &v32, 4);
}

// Copy `bytes` (multiple of 16) from src to dst, this workgroup's chunk only.
__device__ __forceinline__ void copy_chunk(uint8_t* __restrict__ dst,
                                           const uint8_t* __restrict__ src, int64_t bytes) {
  u32x4 r[kCopyUnroll];
#pragma unroll
  for (int i = 0; i < kCopyUnroll; ++i) {
    const int64_t o = ((int64_t)i * kCopyThreads + threadIdx.x) * 16;
    if (o < bytes) r[i] = *(const u32x4*)(src + o);
  }
#pragma unroll
  for (int i = 0; i < kCopyUnroll; ++i) {
    const int64_t o = ((int64_t)i * kCopyThreads + threadIdx.x) * 16;
    if (o < bytes) *(u32x4*)(dst + o) = r[i];
  }
}

__device__ __forceinline__ void zero_chunk(uint8_t* __restrict__ dst, int64_t bytes) {
#pragma unroll
  for (int i = 0; i < kCopyUnroll; ++i) {
    const int64_t o = ((int64_t)i * kCopyThreads + threadIdx.x) * 16;
    if (o < bytes) *(u32x4*)(dst + o) = u32x4{0u, 0u, 0u, 0u};
  }
}

// grid.x = n_pages * 2 (K, V) * chunks_per_page, plus one trailing workgroup
// that writes the header and (fp8) the page scales.
__global__ __launch_bounds__(kCopyThreads) void pack_kernel(PackParams p) {
  const int64_t cpp = (p.page_bytes + kChunkBytes - 1) / kChunkBytes;
  const int64_t copies = p.n_pages * 2 * cpp;
  const int64_t wg = blockIdx.x;
  uint8_t* body = p.packed + 256;
  if (wg == copies) {
    if (threadIdx.x < 64) ((uint32_t*)p.packed)[threadIdx.x] = p.hdr.words[threadIdx.x];
    if (p.has_scales) {
      float* ks = (float*)(body + 2 * p.n_pages * p.page_bytes);
      float* vs = ks + p.n_pages;
      for (int64_t j = threadIdx.x; j < p.n_pages; j += kCopyThreads) {
        const int32_t pid = p.pages[j];
        const bool ok = pid >= 0 && pid < p.num_pages;
        ks[j] = ok ? p.k_scales[pid] : 0.f;
        vs[j] = ok ? p.v_scales[pid] : 0.f;
      }
    }
    return;
  }
  const int64_t j = wg / (2 * cpp);
  const int64_t rem = wg - j * 2 * cpp;
  const int which = (int)(rem / cpp);  // 0: K, 1: V
  const int64_t c = rem - which * cpp;
  const int64_t off = c * kChunkBytes;
  const int64_t bytes = p.page_bytes - off < kChunkBytes ? p.page_bytes - off : kChunkBytes;
  uint8_t* dst = body + ((int64_t)which * p.n_pages + j) * p.page_bytes + off;
  const int32_t pid = p.pages[j];
  if (pid < 0 || pid >= p.num_pages) {  // out-of-contract id: stay in bounds
    zero_chunk(dst, bytes);
    return;
  }
  const uint8_t* src = (which ? p.v_pages : p.k_pages) + (int64_t)pid * p.page_bytes + off;
  copy_chunk(dst, src, bytes);
}

// Every workgroup checks the header first; on any mismatch nothing is written
// and workgroup 0 reports the status.
__global__ __launch_bounds__(kCopyThreads) void unpack_kernel(PackParams p) {
  __shared__ int bad;
  if (threadIdx.x == 0) bad = 0;
  __syncthreads();
  if (threadIdx.x < 64) {
    const uint32_t w = ((const uint32_t*)p.packed_in)[threadIdx.x];
    // word 12 (n_seqs) is informational; word 3 holds the policy version
    if (threadIdx.x != 12 && w != p.hdr.words[threadIdx.x]) {
      atomicOr(&bad, threadIdx.x == 3 ? 2 : 1);
    }
  }
  __syncthreads();
  const int64_t cpp = (p.page_bytes + kChunkBytes - 1) / kChunkBytes;
  const int64_t copies = p.n_pages * 2 * cpp;
  const int64_t wg = blockIdx.x;
  if (bad) {
    if (wg == 0 && threadIdx.x == 0 && p.dev_status)
      *p.dev_status = (bad & 1) ? (int32_t)DORA_ERR_INVALID_ARG
                                : (int32_t)DORA_ERR_VERSION_MISMATCH;
    return;
  }
  const uint8_t* body = p.packed_in + 256;
  if (wg == copies) {
    if (threadIdx.x == 0 && p.dev_status) *p.dev_status = (int32_t)DORA_OK;
    if (p.has_scales) {
      const float* ks = (const float*)(body + 2 * p.n_pages * p.page_bytes);
      const float* vs = ks + p.n_pages;
      for (int64_t j = threadIdx.x; j < p.n_pages; j += kCopyThreads) {
        const int32_t pid = p.pages[j];
        if (pid >= 0 && pid < p.num_pages) {
          p.ks_out[pid] = ks[j];
          p.vs_out[pid] = vs[j];
        }
      }
    }
    return;
  }
  const int64_t j = wg / (2 * cpp);
  const int64_t rem = wg - j * 2 * cpp;
  const int which = (int)(rem / cpp);
  const int64_t c = rem - which * cpp;
  const int64_t off = c * kChunkBytes;
  const int64_t bytes = p.page_bytes - off < kChunkBytes ? p.page_bytes - off : kChunkBytes;
  const int32_t pid = p.pages[j];
  if (pid < 0 || pid >= p.num_pages) return;  // out-of-contract id: skip
  const uint8_t* src = body + ((int64_t)which * p.n_pages + j) * p.page_bytes + off;
  uint8_t* dst = (which ? p.v_out : p.k_out) + (int64_t)pid * p.page_bytes + off;
  copy_chunk(dst, src, bytes);
}

hipError_t launch_pack(const PackParams& p, hipStream_t s) {
  const int64_t cpp = (p.page_bytes + kChunkBytes - 1) / kChunkBytes;
  const int64_t grid = p.n_pages * 2 * cpp + 1;
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)grid), dim3(kCopyThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_unpack(const PackParams& p, hipStream_t s) {
  const int64_t cpp = (p.page_bytes + kChunkBytes - 1) / kChunkBytes;
  const int64_t grid = p.n_pages * 2 * cpp + 1;
  hipLaunchKernelGGL(unpack_kernel, dim3((unsigned)grid), dim3(kCopyThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace dora
