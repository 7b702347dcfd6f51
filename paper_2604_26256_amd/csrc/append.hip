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
//   slot > 0, not fresh <= s0:       s = fresh, and every earlier code c of
//                                    the page (all heads) becomes
//                                    enc((dec(c) * s0) / s)
//   otherwise:                       s = s0
// (comparing the scales, a token with the page's own maximum does not grow it;
// an unset NaN scale does grow)
//   the token's codes are enc(x / s), and the page's scale becomes s.
// All steps round in fp32 (IEEE, one operation at a time); enc is the nearest
// OCP E4M3FN code, ties to even, saturating at +-448.
//
// The work is a few KiB per sequence, so the kernel is bound by latency: it
// keeps the chain of dependent memory round trips short (length, block-table
// entry, then the token and the page scales at once), holds the token in
// registers from load to store, and writes K in 8- or 16-byte pieces (V's
// layout puts a token's values P elements apart).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dora_internal.h"

namespace dora {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kAppendMaxThreads = 1024;

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

__device__ __forceinline__ float chunk_amax(uint4 c) {
  float m = 0.f;
  const uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    m = fmaxf(m, fabsf(bf16_bits_to_f32((uint16_t)(w[k] & 0xFFFFu))));
    m = fmaxf(m, fabsf(bf16_bits_to_f32((uint16_t)(w[k] >> 16))));
  }
  return m;
}

// 8 codes enc(x / s) of a chunk of 8 bf16 values, packed little-endian.
__device__ __forceinline__ uint2 chunk_encode(uint4 c, float s) {
  const uint32_t w[4] = {c.x, c.y, c.z, c.w};
  uint32_t out[2] = {0u, 0u};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t lo = f32_to_e4m3(__fdiv_rn(bf16_bits_to_f32((uint16_t)(w[k] & 0xFFFFu)), s));
    const uint32_t hi = f32_to_e4m3(__fdiv_rn(bf16_bits_to_f32((uint16_t)(w[k] >> 16)), s));
    out[k >> 1] |= (lo | (hi << 8)) << (16 * (k & 1));
  }
  return make_uint2(out[0], out[1]);
}

// Store chunk c (8 consecutive dims) of one token into slot `slot` of a page.
template <bool FP8, bool IS_K>
__device__ __forceinline__ void store_chunk(uint8_t* __restrict__ page, int d, int P, int slot,
                                            int e, uint4 x, float s) {
  const int h = e / d, i = e - h * d;
  if constexpr (!FP8) {
    if constexpr (IS_K) {
      *(uint4*)(page + k_offset<2>(d, P, h, slot, i)) = x;  // a whole 16-byte chunk
    } else {
      const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
      for (int k = 0; k < 8; ++k)
        *(uint16_t*)(page + v_offset<2>(d, P, h, slot, i + k)) =
            (uint16_t)(w[k >> 1] >> (16 * (k & 1)));
    }
  } else {
    const uint2 q = chunk_encode(x, s);
    if constexpr (IS_K) {
      *(uint2*)(page + k_offset<1>(d, P, h, slot, i)) = q;  // half a 16-byte chunk
    } else {
      const uint32_t w[2] = {q.x, q.y};
#pragma unroll
      for (int k = 0; k < 8; ++k)
        page[v_offset<1>(d, P, h, slot, i + k)] = (uint8_t)(w[k >> 2] >> (8 * (k & 3)));
    }
  }
}

// Requantise slots [0, slot) of every head of one fp8 page from scale s0 to s.
template <bool IS_K>
__device__ void requantise(uint8_t* __restrict__ page, int n, int P, int slot, float s0,
                           float s) {
  if constexpr (IS_K) {
    // K: one 16-byte chunk (16 dims of one slot) per task
    const int chunks = n / 16;
    for (int task = threadIdx.x; task < chunks * slot; task += blockDim.x) {
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
    // V: the first `slot` bytes of each (head, dim) row
    for (int task = threadIdx.x; task < n * slot; task += blockDim.x) {
      const int row = task / slot, t = task - row * slot;
      uint8_t* q = page + (int64_t)row * P + t;
      const float old = e4m3_to_f32(*q) * s0;
      *q = (uint8_t)f32_to_e4m3(__fdiv_rn(old, s));
    }
  }
}

// One workgroup per sequence, blockDim.x threads (a multiple of 64): thread i
// holds 8-value chunk i of the token's K and of its V in registers (chunks
// beyond blockDim.x, for very wide tokens, are read again when stored).  The
// dependent memory rounds are: length, block-table entry, then the chunks and
// the page scales together.
template <bool FP8>
__global__ __launch_bounds__(kAppendMaxThreads) void append_kernel(AppendParams p) {
  __shared__ float sred[2][kAppendMaxThreads / 64];
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
  const int d = p.head_dim, P = p.page_size;
  const int n = p.num_kv_heads * d, nchunks = n / 8;
  const int64_t pb = (int64_t)n * P * (FP8 ? 1 : 2);
  const uint16_t* kx = p.k_new + (int64_t)b * n;
  const uint16_t* vx = p.v_new + (int64_t)b * n;
  uint8_t* kpage = p.k_pages + page * pb;
  uint8_t* vpage = p.v_pages + page * pb;
  const int c0 = threadIdx.x;
  uint4 kc = make_uint4(0, 0, 0, 0), vc = make_uint4(0, 0, 0, 0);
  if (c0 < nchunks) {
    kc = *(const uint4*)(kx + 8 * c0);
    vc = *(const uint4*)(vx + 8 * c0);
  }
  float sk = 0.f, sv = 0.f;
  if constexpr (FP8) {
    // Thread 0 reads the page scales and publishes them in LDS before the
    // reduction's barrier; it alone stores the new ones, at the end.
    if (threadIdx.x == 0) {
      sold[0] = slot > 0 ? p.k_scales[page] : 0.f;
      sold[1] = slot > 0 ? p.v_scales[page] : 0.f;
    }
    float mk = chunk_amax(kc), mv = chunk_amax(vc);
    for (int c = c0 + blockDim.x; c < nchunks; c += blockDim.x) {
      mk = fmaxf(mk, chunk_amax(*(const uint4*)(kx + 8 * c)));
      mv = fmaxf(mv, chunk_amax(*(const uint4*)(vx + 8 * c)));
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      mk = fmaxf(mk, __shfl_xor(mk, off));
      mv = fmaxf(mv, __shfl_xor(mv, off));
    }
    const int waves = blockDim.x >> 6;
    if ((threadIdx.x & 63) == 0) {
      sred[0][threadIdx.x >> 6] = mk;
      sred[1][threadIdx.x >> 6] = mv;
    }
    __syncthreads();
    for (int i = 0; i < waves; ++i) {
      mk = fmaxf(mk, sred[0][i]);
      mv = fmaxf(mv, sred[1][i]);
    }
    const float k0 = sold[0], v0 = sold[1];
    const float kfresh = fmaxf(__fdiv_rn(mk, 448.0f), 0x1p-126f);
    const float vfresh = fmaxf(__fdiv_rn(mv, 448.0f), 0x1p-126f);
    const bool kgrow = slot > 0 && !(kfresh <= k0);  // an unset (NaN) scale grows
    const bool vgrow = slot > 0 && !(vfresh <= v0);
    sk = (slot == 0 || kgrow) ? kfresh : k0;
    sv = (slot == 0 || vgrow) ? vfresh : v0;
    if (kgrow) requantise<true>(kpage, n, P, slot, k0, sk);
    if (vgrow) requantise<false>(vpage, n, P, slot, v0, sv);
    if (threadIdx.x == 0) {
      p.k_scales[page] = sk;
      p.v_scales[page] = sv;
    }
  }
  if (c0 < nchunks) {
    store_chunk<FP8, true>(kpage, d, P, slot, 8 * c0, kc, sk);
    store_chunk<FP8, false>(vpage, d, P, slot, 8 * c0, vc, sv);
  }
  for (int c = c0 + blockDim.x; c < nchunks; c += blockDim.x) {
    store_chunk<FP8, true>(kpage, d, P, slot, 8 * c, *(const uint4*)(kx + 8 * c), sk);
    store_chunk<FP8, false>(vpage, d, P, slot, 8 * c, *(const uint4*)(vx + 8 * c), sv);
  }
}

int append_threads(int num_kv_heads, int head_dim) {
  const int chunks = num_kv_heads * head_dim / 8;
  int t = (chunks + 63) / 64 * 64;
  return t < 64 ? 64 : (t > kAppendMaxThreads ? kAppendMaxThreads : t);
}

hipError_t launch_append(const AppendParams& p, bool fp8, hipStream_t s) {
  if (p.num_seqs <= 0) return hipSuccess;
  if (p.dev_status) {
    const hipError_t e = launch_fill_i32(p.dev_status, (int32_t)DORA_OK, 1, s);
    if (e != hipSuccess) return e;
  }
  const dim3 block(append_threads(p.num_kv_heads, p.head_dim));
  if (fp8)
    hipLaunchKernelGGL(append_kernel<true>, dim3(p.num_seqs), block, 0, s, p);
  else
    hipLaunchKernelGGL(append_kernel<false>, dim3(p.num_seqs), block, 0, s, p);
  return hipGetLastError();
}

}  // namespace dora
