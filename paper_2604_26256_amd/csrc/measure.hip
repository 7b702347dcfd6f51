// Measurement entry points (include/dora_measure.h): the decode call with
// per-kernel timing events, and a streaming-read reference kernel with the
// decode kernel's access pattern (random tiles, 16-byte non-temporal loads),
// which gives the achievable read bandwidth the decode kernel is compared with.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dora_internal.h"
#include "dora_measure.h"

namespace dora {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// One wavefront per workgroup.  A batch is TPB tiles of CHUNKS KiB (each lane
// loads 16 bytes of every KiB); two batches are in flight: the next batch's
// loads are issued before the current one is folded.  Tile ids come 64 at a
// time, one per lane, and are broadcast with readlane.  A tile past the range
// or outside the buffer is redirected to the buffer's first 16 bytes for
// every lane (a single line request) and folds in as zero, so every batch
// issues the same loads.
template <int CHUNKS, int TPB>
__global__ __launch_bounds__(64) void stream_read_kernel(const uint8_t* base, int64_t base_bytes,
                                                         const int32_t* tiles, int64_t n_tiles,
                                                         uint32_t* sink) {
  constexpr int LOADS = CHUNKS * TPB;
  constexpr int64_t TILE = (int64_t)CHUNKS * 1024;
  static_assert(64 % TPB == 0, "a batch must not straddle a chunk of 64 tile ids");
  const int lane = threadIdx.x;
  const int64_t W = gridDim.x, w = blockIdx.x;
  const int64_t q = n_tiles / W, rem = n_tiles - q * W;
  const int64_t t0 = w * q + (w < rem ? w : rem);
  const int64_t t1 = t0 + q + (w < rem ? 1 : 0);

  int64_t cbase = t0;
  int idx_cur = t0 + lane < t1 ? tiles[t0 + lane] : -1;
  int idx_nxt = t0 + 64 + lane < t1 ? tiles[t0 + 64 + lane] : -1;

  // Issue the loads of the batch starting at tile t; keep[k] says whether
  // tile k of the batch is real.
  auto issue = [&](u32x4 (&r)[LOADS], bool (&keep)[TPB], int64_t t) {
    if (t - cbase >= 64) {
      cbase += 64;
      idx_cur = idx_nxt;
      idx_nxt = cbase + 64 + lane < t1 ? tiles[cbase + 64 + lane] : -1;
    }
#pragma unroll
    for (int k = 0; k < TPB; ++k) {
      const int64_t tt = t + k;
      const int id = tt < t1 ? __builtin_amdgcn_readlane(idx_cur, (int)(tt - cbase)) : -1;
      const bool ok = id >= 0 && (int64_t)id * TILE + TILE <= base_bytes;
      keep[k] = ok;
      const uint8_t* tb = base + (ok ? (int64_t)id * TILE : 0);
#pragma unroll
      for (int c = 0; c < CHUNKS; ++c)
        r[k * CHUNKS + c] = __builtin_nontemporal_load(
            (const u32x4*)(tb + (ok ? c * 1024 + lane * 16 : 0)));
    }
  };
  u32x4 acc = u32x4{0u, 0u, 0u, 0u};
  auto fold = [&](const u32x4 (&r)[LOADS], const bool (&keep)[TPB]) {
#pragma unroll
    for (int k = 0; k < TPB; ++k)
#pragma unroll
      for (int c = 0; c < CHUNKS; ++c)
        if (keep[k]) acc ^= r[k * CHUNKS + c];
  };

  u32x4 a[LOADS], b[LOADS];
  bool ka[TPB], kb[TPB];
  issue(a, ka, t0);
  for (int64_t t = t0; t < t1; t += 2 * TPB) {
    issue(b, kb, t + TPB);
    fold(a, ka);
    issue(a, ka, t + 2 * TPB);
    fold(b, kb);
  }
  uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x ^= (uint32_t)__shfl_xor((int)x, off);
  if (lane == 0) sink[w] = x;
}

// Kernel for (tile KiB, tiles per batch): at most 16 loads per lane per batch.
template <int CHUNKS, int TPB>
static const void* read_kernel_if_fits() {
  if constexpr (CHUNKS * TPB <= 16)
    return (const void*)&stream_read_kernel<CHUNKS, TPB>;
  else
    return nullptr;
}

template <int CHUNKS>
static const void* read_kernel_for(int tpb) {
  switch (tpb) {
    case 1: return read_kernel_if_fits<CHUNKS, 1>();
    case 2: return read_kernel_if_fits<CHUNKS, 2>();
    case 4: return read_kernel_if_fits<CHUNKS, 4>();
    case 8: return read_kernel_if_fits<CHUNKS, 8>();
    case 16: return read_kernel_if_fits<CHUNKS, 16>();
  }
  return nullptr;
}

}  // namespace dora

using namespace dora;

extern "C" {

dora_status dora_decode_attn_timed(const dora_decode_desc* desc, const void* q,
                                   const void* k_pages, const void* v_pages,
                                   const int32_t* block_table, const int32_t* seq_lens,
                                   const int32_t* version_ids, void* out, void* workspace,
                                   size_t workspace_bytes, dora_stream_t stream,
                                   void* const* events) {
  if (!events || !events[0] || !events[1] || !events[2]) return DORA_ERR_INVALID_ARG;
  hipEvent_t ev[3] = {(hipEvent_t)events[0], (hipEvent_t)events[1], (hipEvent_t)events[2]};
  return decode_attn(desc, q, k_pages, v_pages, block_table, seq_lens, version_ids, out,
                     workspace, workspace_bytes, (hipStream_t)stream, ev);
}

dora_status dora_stream_read(const void* base, int64_t base_bytes, const int32_t* tiles,
                             int64_t n_tiles, int32_t tile_bytes, int32_t tiles_per_batch,
                             uint32_t* sink, int32_t waves, dora_stream_t stream) {
  if (!base || !sink || waves < 1 || base_bytes < 16 || n_tiles < 0 ||
      (n_tiles > 0 && !tiles) || ((uintptr_t)base & 15u) != 0)
    return DORA_ERR_INVALID_ARG;
  const void* fn = nullptr;
  switch (tile_bytes) {
    case 1024: fn = read_kernel_for<1>(tiles_per_batch); break;
    case 2048: fn = read_kernel_for<2>(tiles_per_batch); break;
    case 4096: fn = read_kernel_for<4>(tiles_per_batch); break;
    case 8192: fn = read_kernel_for<8>(tiles_per_batch); break;
    case 16384: fn = read_kernel_for<16>(tiles_per_batch); break;
    default: break;
  }
  if (!fn) return DORA_ERR_UNSUPPORTED;
  const uint8_t* b = (const uint8_t*)base;
  void* args[] = {(void*)&b, (void*)&base_bytes, (void*)&tiles, (void*)&n_tiles, (void*)&sink};
  return hipLaunchKernel(fn, dim3((unsigned)waves), dim3(64), args, 0, (hipStream_t)stream) ==
                 hipSuccess
             ? DORA_OK
             : DORA_ERR_HIP;
}

}  // extern "C"
