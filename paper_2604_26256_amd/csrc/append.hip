// KV append: the write that precedes every decode step.  Each sequence's
// current token (counted in seq_lens, the token the next decode step attends
// with; the per-token step of Sec. 2.2) is stored into its page slot.
//
// One workgroup per sequence.  bf16 pages take a plain store.  fp8 pages keep
// one fp32 scale per page for K and one for V; the paper leaves the policy
// open, and the one taken is grow-only:
//   amax = max |x| over the token's Hkv x d values
//   fresh = max(amax / 448, 2^-126)          (always a normal number)
//   slot 0:                          s = fresh
//   slot > 0, not amax / s0 <= 448:  s = fresh, and every earlier code c of
//                                    the page (all heads) becomes
//                                    enc((dec(c) * s0) / s)
//   otherwise:                       s = s0
//   the token's codes are enc(x / s), and the page's scale becomes s.
// All steps round in fp32 (IEEE, one operation at a time); enc is the nearest
// OCP E4M3FN code, ties to even, saturating at +-448.
//
// The work is a few KiB per sequence, so the kernel is launch-bound; it only
// has to keep its writes coalesced where the layout allows (one 16-byte store
// per K chunk) and avoid touching a page more than once.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dora_internal.h"

namespace dora {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kAppendThreads = 256;

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

// Value of an E4M3FN code, exact in fp32.
__device__ __forceinline__ float e4m3_to_f32(uint32_t c) {
  const uint32_t sign = (c & 0x80u) << 24;
  const uint32_t e = (c >> 3) & 0xFu, m = c & 0x7u;
  if (e == 0xFu && m == 0x7u) return __uint_as_float(sign | 0x7FC00000u);
  if (e == 0) {  // subnormal (or zero): m * 2^-9
    const float v = (float)m * 0x1p-9f;
    return sign ? -v : v;
  }
  return __uint_as_float(sign | ((e + 120u) << 23) | (m << 20));
}

// Nearest E4M3FN code of x, ties to the even mantissa, saturating to +-448.
// Works on the fp32 bit pattern: the 20 mantissa bits below the kept 3 decide
// the rounding, and a carry out of the mantissa moves into the exponent.
__device__ __forceinline__ uint32_t f32_to_e4m3(float x) {
  const uint32_t u = __float_as_uint(x);
  const uint32_t sign = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7FFFFFFFu;
  if (a > 0x7F800000u) return sign | 0x7Fu;                 // NaN
  if (a >= 0x43E00000u) return sign | 0x7Eu;                // >= 448 (inf included)
  if (a < 0x3C800000u) {                                    // below 2^-6: steps of 2^-9
    const float m = __builtin_rintf(__uint_as_float(a) * 512.0f);  // exact scaling, RNE
    return sign | (uint32_t)m;                              // 8 -> 0x08 = 2^-6
  }
  const uint32_t keep = (a >> 20) & 0x7u, rest = a & 0xFFFFFu;
  uint32_t code = ((((a >> 23) - 120u) << 3) | keep);
  if (rest > 0x80000u || (rest == 0x80000u && (keep & 1u))) code += 1u;
  return sign | code;
}

__device__ __forceinline__ float block_max(float v, float* sred) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  const int wave = threadIdx.x >> 6;
  __syncthreads();  // sred may still be read from a previous call
  if ((threadIdx.x & 63) == 0) sred[wave] = v;
  __syncthreads();
  float m = sred[0];
  for (int i = 1; i < kAppendThreads / 64; ++i) m = fmaxf(m, sred[i]);
  return m;
}

// Byte offset of element (head h, token slot t, dim i) inside a page.
template <int E>
__device__ __forceinline__ int64_t k_offset(int d, int P, int h, int t, int i) {
  constexpr int X = 16 / E;
  return ((((int64_t)h * (d / X) + i / X) * P + t) * X + i % X) * E;
}
template <int E>
__device__ __forceinline__ int64_t v_offset(int d, int P, int h, int t, int i) {
  return (((int64_t)h * d + i) * P + t) * E;
}

// Store one token (Hkv x d bf16 values x) into slot `slot` of one page of the K
// (IS_K) or V pool.
template <bool FP8, bool IS_K>
__device__ void store_token(const AppendParams& p, const uint16_t* __restrict__ x,
                            uint8_t* __restrict__ page, float* scale, int slot, float* sred,
                            float* sold) {
  const int d = p.head_dim, P = p.page_size, n = p.num_kv_heads * d;
  if constexpr (!FP8) {
    // 4 consecutive dims per thread: one 8-byte load; one 8-byte K store (the
    // 4 values sit in one 16-byte chunk), four 2-byte V stores
    for (int e = 4 * (int)threadIdx.x; e < n; e += 4 * kAppendThreads) {
      const uint2 w = *(const uint2*)(x + e);
      const int h = e / d, i = e - h * d;
      if constexpr (IS_K) {
        *(uint2*)(page + k_offset<2>(d, P, h, slot, i)) = w;
      } else {
        const uint16_t v[4] = {(uint16_t)(w.x & 0xFFFFu), (uint16_t)(w.x >> 16),
                               (uint16_t)(w.y & 0xFFFFu), (uint16_t)(w.y >> 16)};
#pragma unroll
        for (int k = 0; k < 4; ++k)
          *(uint16_t*)(page + v_offset<2>(d, P, h, slot, i + k)) = v[k];
      }
    }
    return;
  }
  // fp8: the token's amax, then the page scale decision (uniform per block).
  // Thread 0 reads the current scale and publishes it in LDS before the
  // reduction's barriers; it alone stores the new scale, at the end.
  if (threadIdx.x == 0) *sold = slot > 0 ? *scale : 0.f;
  float amax = 0.f;
  for (int e = threadIdx.x; e < n; e += kAppendThreads)
    amax = fmaxf(amax, fabsf(bf16_bits_to_f32(x[e])));
  amax = block_max(amax, sred);
  const float s0 = *sold;
  const float fresh = fmaxf(__fdiv_rn(amax, 448.0f), 0x1p-126f);
  const bool grow = slot > 0 && !(__fdiv_rn(amax, s0) <= 448.0f);  // NaN (0/0) grows
  const float s = (slot == 0 || grow) ? fresh : s0;
  if (grow) {
    // requantise the page's earlier slots [0, slot) of every head
    if constexpr (IS_K) {
      // K: one 16-byte chunk (16 dims of one slot) per task
      const int chunks = p.num_kv_heads * (d / 16);
      for (int task = threadIdx.x; task < chunks * slot; task += kAppendThreads) {
        const int c = task / slot, t = task - c * slot;
        u32x4* q = (u32x4*)(page + ((int64_t)c * P + t) * 16);
        u32x4 w = *q;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          uint32_t out = 0;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float old = e4m3_to_f32((w[k] >> (8 * j)) & 0xFFu) * s0;
            out |= f32_to_e4m3(__fdiv_rn(old, s)) << (8 * j);
          }
          w[k] = out;
        }
        *q = w;
      }
    } else {
      // V: one byte per task (slot bytes of each (head, dim) row)
      for (int task = threadIdx.x; task < n * slot; task += kAppendThreads) {
        const int row = task / slot, t = task - row * slot;
        uint8_t* q = page + (int64_t)row * P + t;
        const float old = e4m3_to_f32(*q) * s0;
        *q = (uint8_t)f32_to_e4m3(__fdiv_rn(old, s));
      }
    }
  }
  // the token's codes
  if constexpr (IS_K) {
    for (int c = threadIdx.x; c < n / 16; c += kAppendThreads) {
      const int e = 16 * c, h = e / d, i = e - h * d;
      u32x4 w;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        uint32_t out = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j)
          out |= f32_to_e4m3(__fdiv_rn(bf16_bits_to_f32(x[e + 4 * k + j]), s)) << (8 * j);
        w[k] = out;
      }
      *(u32x4*)(page + k_offset<1>(d, P, h, slot, i)) = w;
    }
  } else {
    for (int e = threadIdx.x; e < n; e += kAppendThreads) {
      const int h = e / d, i = e - h * d;
      page[v_offset<1>(d, P, h, slot, i)] =
          (uint8_t)f32_to_e4m3(__fdiv_rn(bf16_bits_to_f32(x[e]), s));
    }
  }
  if (threadIdx.x == 0) *scale = s;
}

template <bool FP8>
__global__ __launch_bounds__(kAppendThreads) void append_kernel(AppendParams p) {
  __shared__ float sred[kAppendThreads / 64];
  __shared__ float sold[2];  // the K and the V page's scale before this token
  const int b = blockIdx.x;
  const int L = p.seq_lens[b];
  if (L <= 0) return;  // nothing to append
  const int t = L - 1, j = t / p.page_size, slot = t - j * p.page_size;
  bool ok = L <= p.stride * p.page_size;
  const int64_t page = ok ? (int64_t)p.block_table[(int64_t)b * p.stride + j] : -1;
  ok = ok && page >= 0 && page < p.num_pages;
  if (ok && p.page_owner && p.version_ids) ok = p.page_owner[page] == p.version_ids[b];
  if (!ok) {  // never write outside the pool or into another version's page
    if (threadIdx.x == 0 && p.dev_status) *p.dev_status = (int32_t)DORA_ERR_DEVICE_CHECK;
    return;
  }
  const int64_t n = (int64_t)p.num_kv_heads * p.head_dim;
  const int64_t pb = n * p.page_size * (FP8 ? 1 : 2);
  store_token<FP8, true>(p, p.k_new + b * n, p.k_pages + page * pb,
                         FP8 ? p.k_scales + page : nullptr, slot, sred, &sold[0]);
  store_token<FP8, false>(p, p.v_new + b * n, p.v_pages + page * pb,
                          FP8 ? p.v_scales + page : nullptr, slot, sred, &sold[1]);
}

hipError_t launch_append(const AppendParams& p, bool fp8, hipStream_t s) {
  if (p.num_seqs <= 0) return hipSuccess;
  if (p.dev_status) {
    const hipError_t e = launch_fill_i32(p.dev_status, (int32_t)DORA_OK, 1, s);
    if (e != hipSuccess) return e;
  }
  if (fp8)
    hipLaunchKernelGGL(append_kernel<true>, dim3(p.num_seqs), dim3(kAppendThreads), 0, s, p);
  else
    hipLaunchKernelGGL(append_kernel<false>, dim3(p.num_seqs), dim3(kAppendThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace dora
