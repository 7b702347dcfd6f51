// Device building blocks of the decode-attention kernels, shared by the
// stream-K decode kernel and the group-prefix kernel: the register image of
// one (page, KV head) tile, its loads, the per-page MFMA + online-softmax
// step and the query operand.  Included by HIP sources only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace dora {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// decode
// ---------------------------------------------------------------------------

// Butterflies across the 16-lane rows of a wave (each lane with lane ^ 16, or
// with lane ^ 32) on gfx950's row-swap permutes, VALU operations instead of
// an LDS-routed shuffle.  A swap of a value with itself returns, in its two
// results, the lane's value and its partner's (in an order that depends on
// the row), so their max or sum is the butterfly's, bit for bit.
__device__ __forceinline__ float max_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Raw bytes of one page's K and V tiles for one KV head, as each lane loads them.
template <int D, int P, bool FP8>
struct PageRegs {
  static constexpr int NT = P / 16;                               // 16-token sub-tiles
  static constexpr int NK = FP8 ? NT * (D / 64) : NT * (D / 32);  // 16-byte K loads
  static constexpr int VB = (P == 16 ? 4 : 8) * (FP8 ? 1 : 2);    // bytes per V load
  u32x4 k[NK];
  typedef typename std::conditional<
      VB == 16, u32x4, typename std::conditional<VB == 8, u32x2, uint32_t>::type>::type vraw_t;
  vraw_t v[D / 16];
};

// Token slot (within the page) that MFMA row r of sub-tile t holds.  With 32-token
// pages the rows interleave so that the QK^T accumulator rows of lane row-group
// q are tokens 8q..8q+7, exactly the k-range that lane supplies to the PV MFMA.
template <int P>
__device__ __forceinline__ int tile_token(int t, int r) {
  return P == 16 ? r : 8 * (r >> 2) + 4 * t + (r & 3);
}

__device__ __forceinline__ bf16x8 fp8x8_to_bf16(uint32_t w0, uint32_t w1) {
  const bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, false);
  const bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, true);
  const bf16x2 c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w1, 1.0f, false);
  const bf16x2 d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w1, 1.0f, true);
  return bf16x8{a[0], a[1], b[0], b[1], c[0], c[1], d[0], d[1]};
}

__device__ __forceinline__ bf16x4 fp8x4_to_bf16(uint32_t w0) {
  const bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, false);
  const bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, true);
  return bf16x4{a[0], a[1], b[0], b[1]};
}

// K: lane reads token tile_token(t, col) of 16-byte chunk (4s + grp); the chunk
// and sub-tile strides are compile-time constants, so every K load is the
// lane's base offset plus an immediate.  V: 16 head-dim rows per load, rows
// 16 * P elements apart.  Every KV byte is read once per call, so the loads
// are non-temporal (no cache allocation for streaming data).
template <int D, int P, bool FP8>
__device__ __forceinline__ void load_page(PageRegs<D, P, FP8>& r, const uint8_t* kbase,
                                          const uint8_t* vbase, uint32_t koff, uint32_t voff) {
  typedef PageRegs<D, P, FP8> R;
  constexpr int per_t = R::NK / R::NT;
#pragma unroll
  for (int t = 0; t < R::NT; ++t)
#pragma unroll
    for (int s = 0; s < per_t; ++s)
      r.k[t * per_t + s] =
          __builtin_nontemporal_load((const u32x4*)(kbase + koff + (4 * s * P + 4 * t) * 16));
  constexpr int vrow = P * (FP8 ? 1 : 2) * 16;  // bytes between 16-row blocks of V
#pragma unroll
  for (int i = 0; i < D / 16; ++i)
    r.v[i] = __builtin_nontemporal_load((const typename R::vraw_t*)(vbase + voff + i * vrow));
}

// One page of one segment: scores S^T = K Q^T for the 16 query columns of the
// lane layout, online-softmax update in the log2 domain, then O^T += V^T P^T.
// NC column tiles of 16 share the page's operands (each K and V register
// feeds NC MFMAs); tile c has its own query operand, accumulator and running
// max / sum.  `r` holds the page as each lane loaded it (from HBM or LDS);
// nvalid tokens of the page count; ksc folds the softmax scale (and the fp8 K
// page scale), vsc the fp8 V page scale.
template <int D, int P, bool FP8, int NC>
__device__ __forceinline__ void consume_page_tiles(const PageRegs<D, P, FP8>& r, int nvalid,
                                                   float ksc, float vsc,
                                                   const bf16x8 (&qop)[NC][D / 32],
                                                   f32x4 (&acc)[NC][D / 16], float (&m_run)[NC],
                                                   float (&l_run)[NC]) {
  constexpr int NT = PageRegs<D, P, FP8>::NT;
  constexpr int KSTEPS = D / 32;
  constexpr int DBLK = D / 16;
  const int grp = (threadIdx.x & 63) >> 4;

  // scores S^T: lane holds tokens of its row group for head `col`
  f32x4 sc[NC][NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
#pragma unroll
    for (int c = 0; c < NC; ++c) sc[c][t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      bf16x8 a;
      if constexpr (FP8) {
        const u32x4& wd = r.k[t * (D / 64) + (ks >> 1)];
        a = (ks & 1) ? fp8x8_to_bf16(wd[2], wd[3]) : fp8x8_to_bf16(wd[0], wd[1]);
      } else {
        a = __builtin_bit_cast(bf16x8, r.k[t * KSTEPS + ks]);
      }
#pragma unroll
      for (int c = 0; c < NC; ++c)
        sc[c][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qop[c][ks], sc[c][t], 0, 0, 0);
    }
  }
  float alpha[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    float mx = -__builtin_inff();
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float x = sc[c][t][i] * ksc;
        const int tok = P == 16 ? 4 * grp + i : 8 * grp + 4 * t + i;
        if (nvalid < P && tok >= nvalid) x = -__builtin_inff();
        sc[c][t][i] = x;
        mx = fmaxf(mx, x);
      }
    mx = max_xor32(max_xor16(mx));
    const float m_new = fmaxf(m_run[c], mx);
    alpha[c] = __builtin_amdgcn_exp2f(m_run[c] - m_new);
    m_run[c] = m_new;
    float psum = 0.f;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = __builtin_amdgcn_exp2f(sc[c][t][i] - m_new);
        psum += e;
        sc[c][t][i] = e * vsc;
      }
    l_run[c] = l_run[c] * alpha[c] + psum;
    if (__ballot(alpha[c] != 1.f)) {
#pragma unroll
      for (int i = 0; i < DBLK; ++i) acc[c][i] *= alpha[c];
    }
  }
  // P^T operand, then O^T += V^T P^T per 16-row block of the head dim
  if constexpr (P == 16) {
    bf16x4 pb4[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c)
      pb4[c] = bf16x4{(__bf16)sc[c][0][0], (__bf16)sc[c][0][1], (__bf16)sc[c][0][2],
                      (__bf16)sc[c][0][3]};
#pragma unroll
    for (int i = 0; i < DBLK; ++i) {
      bf16x4 a;
      if constexpr (FP8)
        a = fp8x4_to_bf16(r.v[i]);
      else
        a = __builtin_bit_cast(bf16x4, r.v[i]);
      if (nvalid < P) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (4 * grp + e >= nvalid) a[e] = (__bf16)0.f;
      }
#pragma unroll
      for (int c = 0; c < NC; ++c)
        acc[c][i] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, pb4[c], acc[c][i], 0, 0, 0);
    }
  } else {
    bf16x8 pb8[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c)
      pb8[c] = bf16x8{(__bf16)sc[c][0][0], (__bf16)sc[c][0][1], (__bf16)sc[c][0][2],
                      (__bf16)sc[c][0][3], (__bf16)sc[c][1][0], (__bf16)sc[c][1][1],
                      (__bf16)sc[c][1][2], (__bf16)sc[c][1][3]};
#pragma unroll
    for (int i = 0; i < DBLK; ++i) {
      bf16x8 a;
      if constexpr (FP8)
        a = fp8x8_to_bf16(r.v[i][0], r.v[i][1]);
      else
        a = __builtin_bit_cast(bf16x8, r.v[i]);
      if (nvalid < P) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (8 * grp + e >= nvalid) a[e] = (__bf16)0.f;
      }
#pragma unroll
      for (int c = 0; c < NC; ++c)
        acc[c][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb8[c], acc[c][i], 0, 0, 0);
    }
  }
}

// The step for one column tile (the decode kernel's case).
template <int D, int P, bool FP8>
__device__ __forceinline__ void consume_page(const PageRegs<D, P, FP8>& r, int nvalid, float ksc,
                                             float vsc, const bf16x8 (&qop)[D / 32],
                                             f32x4 (&acc)[D / 16], float& m_run, float& l_run) {
  consume_page_tiles<D, P, FP8, 1>(r, nvalid, ksc, vsc,
                                   reinterpret_cast<const bf16x8(&)[1][D / 32]>(qop),
                                   reinterpret_cast<f32x4(&)[1][D / 16]>(acc),
                                   reinterpret_cast<float(&)[1]>(m_run),
                                   reinterpret_cast<float(&)[1]>(l_run));
}

// Query operand: lane supplies q[row][8 head-dim values] per k-step, in the
// head-dim order the K chunks are consumed in (zero when the column is unused).
template <int D, bool FP8>
__device__ __forceinline__ void load_q_operand(bf16x8 (&dst)[D / 32], const uint16_t* qrow,
                                               bool valid) {
  const int grp = (threadIdx.x & 63) >> 4;
#pragma unroll
  for (int s = 0; s < D / 32; ++s) {
    const int d0 = FP8 ? 64 * (s >> 1) + 16 * grp + 8 * (s & 1) : 32 * s + 8 * grp;
    dst[s] = valid ? *(const bf16x8*)(qrow + d0) : bf16x8{0, 0, 0, 0, 0, 0, 0, 0};
  }
}

}  // namespace dora
