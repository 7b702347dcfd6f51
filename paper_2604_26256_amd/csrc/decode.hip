// Split-KV decode attention over a paged, multi-version KV pool, for gfx950.
//
// The operation is scaled dot-product attention of one decode query per head
// over a sequence's cached tokens (the per-token decode step whose time enters
// the paper's step-time model, Sec. 2.2 Eq. (1); sequences of several policy
// versions share one pool, Sec. 3.2).  Decode is memory-bound (Sec. 1,
// Sec. 2.2), so the kernels are built around streaming every K/V byte once:
//
//   plan     one workgroup: pages per split C from the batch's total pages,
//            per-sequence split counts and partial-slot bases, and a work list
//            ordered longest-first (counting sort on split size).
//   split    one wavefront per (sequence, KV head, split).  The G query heads
//            of the KV head are packed into the 16 columns of MFMA tiles, so
//            each K/V byte is read once for the whole group:
//              S^T[16 tok x 16 head] = K[16 tok x d] * Q^T   (mfma 16x16x32 bf16)
//              O^T[16 d x 16 head]  += V^T[16 d x tok] * P^T  (mfma 16x16x{16,32} bf16)
//            The page layouts (K: 16-byte head-dim chunks, token-major inside a
//            chunk; V: tokens contiguous per head-dim index) make every lane's
//            global load land directly in its MFMA operand registers, so pages
//            stream HBM -> VGPRs with no LDS round trip; the next page is in
//            flight while the current one is consumed.  Online softmax in the
//            log2 domain; max and sum reductions across the four 16-lane rows
//            use cross-lane shuffles.  fp8 (OCP E4M3FN) pages are converted to
//            bf16 in registers (exact) and the per-page scales are folded into
//            the scores (K) and the probabilities (V).
//   combine  log-sum-exp merge of the partial results of split sequences.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dora_internal.h"

namespace dora {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// plan
// ---------------------------------------------------------------------------

__device__ __forceinline__ int pages_of(int L, int P, int stride) {
  if (L <= 0) return 0;
  int n = (L + P - 1) / P;
  return n < stride ? n : stride;  // a contract violation stays in bounds
}

// Inclusive block-wide prefix sum over kPlanThreads ints (Hillis-Steele).
__device__ int block_inclusive_scan(int v, int* sh) {
  const int t = threadIdx.x;
  sh[t] = v;
  __syncthreads();
  for (int off = 1; off < kPlanThreads; off <<= 1) {
    int add = t >= off ? sh[t - off] : 0;
    __syncthreads();
    sh[t] += add;
    __syncthreads();
  }
  int r = sh[t];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(PlanParams p) {
  __shared__ long long red[kPlanThreads / 64];
  __shared__ int scan[kPlanThreads];
  __shared__ int hist[kPlanBins];
  __shared__ int cursor[kPlanBins];
  __shared__ int s_chunk;
  __shared__ int s_tile;
  const int t = threadIdx.x;
  const int B = p.num_seqs, P = p.page_size;

  // 1. total pages of the batch
  long long local = 0;
  for (int b = t; b < B; b += kPlanThreads) local += pages_of(p.seq_lens[b], P, p.stride);
  for (int off = 32; off > 0; off >>= 1) local += __shfl_xor(local, off);
  if ((t & 63) == 0) red[t >> 6] = local;
  if (t < kPlanBins) hist[t] = 0;
  __syncthreads();
  if (t == 0) {
    long long total = 0;
    for (int w = 0; w < kPlanThreads / 64; ++w) total += red[w];
    long long c;
    if (p.force_pages > 0) {
      c = p.force_pages;
    } else {
      long long work = total * p.num_kv_heads;
      c = (work + p.target_units - 1) / p.target_units;
      if (c < p.min_pages) c = p.min_pages;
    }
    if (c > 0x3fffffff) c = 0x3fffffff;
    s_chunk = (int)c;
  }
  __syncthreads();
  const int C = s_chunk;

  // 2. splits per sequence, their partial-slot bases, and a size histogram
  int carry = 0;
  for (int base = 0; base < B; base += kPlanThreads) {
    const int b = base + t;
    int n = 0, ns = 0;
    if (b < B) {
      n = pages_of(p.seq_lens[b], P, p.stride);
      ns = n == 0 ? 1 : (n + C - 1) / C;
    }
    int incl = block_inclusive_scan(ns, scan);
    if (b < B) {
      p.seqinfo[b] = make_int2(carry + incl - ns, ns);
      int last = n - (ns - 1) * C;  // pages of the final split (0 for an empty sequence)
      if (ns > 1) atomicAdd(&hist[0], ns - 1);
      atomicAdd(&hist[(int)((long long)(C - last) * (kPlanBins - 1) / C)], 1);
    }
    if (t == kPlanThreads - 1) s_tile = incl;  // splits in this tile of sequences
    __syncthreads();
    carry += s_tile;
    __syncthreads();
  }
  // 3. bins in order of decreasing split size -> first work-list position
  if (t == 0) {
    int acc = 0;
    for (int i = 0; i < kPlanBins; ++i) {
      cursor[i] = acc;
      acc += hist[i];
    }
    p.hdr[0] = acc;
    p.hdr[1] = C;
  }
  __syncthreads();
  // 4. scatter the work items
  for (int b = t; b < B; b += kPlanThreads) {
    const int n = pages_of(p.seq_lens[b], P, p.stride);
    const int2 si = p.seqinfo[b];
    const int ns = si.y;
    if (ns > 1) {
      int pos = atomicAdd(&cursor[0], ns - 1);
      for (int s = 0; s < ns - 1; ++s)
        p.items[pos + s] = make_int4(b, s * C, (s + 1) * C, si.x + s);
    }
    const int last = n - (ns - 1) * C;
    int pos = atomicAdd(&cursor[(int)((long long)(C - last) * (kPlanBins - 1) / C)], 1);
    p.items[pos] = make_int4(b, (ns - 1) * C, n, ns > 1 ? si.x + ns - 1 : -1);
  }
}

// ---------------------------------------------------------------------------
// split decode
// ---------------------------------------------------------------------------

// Raw bytes of one page's K and V tiles for one KV head, as each lane loads them.
template <int D, int P, bool FP8>
struct PageRegs {
  static constexpr int NT = P / 16;                         // 16-token sub-tiles
  static constexpr int NK = FP8 ? NT * (D / 64) : NT * (D / 32);  // 16-byte K loads
  static constexpr int VB = (P == 16 ? 4 : 8) * (FP8 ? 1 : 2);   // bytes per V load
  u32x4 k[NK];
  typedef typename std::conditional<VB == 16, u32x4,
          typename std::conditional<VB == 8, u32x2, uint32_t>::type>::type vraw_t;
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
  bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, false);
  bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, true);
  bf16x2 c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w1, 1.0f, false);
  bf16x2 d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w1, 1.0f, true);
  return bf16x8{a[0], a[1], b[0], b[1], c[0], c[1], d[0], d[1]};
}

__device__ __forceinline__ bf16x4 fp8x4_to_bf16(uint32_t w0) {
  bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, false);
  bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w0, 1.0f, true);
  return bf16x4{a[0], a[1], b[0], b[1]};
}

template <int D, int P, bool FP8>
__device__ __forceinline__ void load_page(PageRegs<D, P, FP8>& r, const uint8_t* kbase,
                                          const uint8_t* vbase, const uint32_t* koff,
                                          uint32_t voff) {
  typedef PageRegs<D, P, FP8> R;
#pragma unroll
  for (int i = 0; i < R::NK; ++i) r.k[i] = *(const u32x4*)(kbase + koff[i]);
  constexpr int vrow = P * (FP8 ? 1 : 2) * 16;  // bytes between 16-row blocks of V
#pragma unroll
  for (int i = 0; i < D / 16; ++i)
    r.v[i] = *(const typename R::vraw_t*)(vbase + voff + i * vrow);
}

template <int D, int P, bool FP8>
__global__ __launch_bounds__(64) void split_decode_kernel(DecodeParams p) {
  typedef PageRegs<D, P, FP8> R;
  constexpr int NT = R::NT;
  constexpr int KSTEPS = D / 32;
  constexpr int DBLK = D / 16;
  constexpr int E = FP8 ? 1 : 2;
  constexpr int TILE_BYTES = P * D * E;  // one KV head of one page

  const int lane = threadIdx.x;
  const int col = lane & 15;  // MFMA row/column index of this lane
  const int grp = lane >> 4;  // 16-lane row group
  const int Hkv = p.num_kv_heads;
  const int u = blockIdx.x / Hkv;
  const int g = blockIdx.x - u * Hkv;
  if (u >= p.hdr[0]) return;
  const int4 it = p.items[u];
  const int b = it.x, j0 = it.y, j1 = it.z, slot = it.w;
  const int L = p.seq_lens[b];
  const int G = p.group;
  const int Hq = p.num_q_heads;

  f32x4 acc[DBLK];
#pragma unroll
  for (int i = 0; i < DBLK; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -__builtin_inff();
  float l_run = 0.f;

  if (j1 > j0) {
    // Query operand: lane supplies q[head col][8 head-dim values] per k-step.
    bf16x8 qop[KSTEPS];
    const uint16_t* qrow = p.q + ((int64_t)b * Hq + (int64_t)g * G + col) * D;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      const int dst = FP8 ? 64 * (s >> 1) + 16 * grp + 8 * (s & 1) : 32 * s + 8 * grp;
      if (col < G)
        qop[s] = *(const bf16x8*)(qrow + dst);
      else
        qop[s] = bf16x8{0, 0, 0, 0, 0, 0, 0, 0};
    }
    // Per-lane byte offsets inside a (page, KV head) tile.
    uint32_t koff[R::NK];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int tok = tile_token<P>(t, col);
      constexpr int per_t = R::NK / NT;
#pragma unroll
      for (int s = 0; s < per_t; ++s) koff[t * per_t + s] = ((4 * s + grp) * P + tok) * 16;
    }
    const uint32_t voff = (uint32_t)((col * P + (P == 16 ? 4 : 8) * grp) * E);

    const int32_t* bt = p.block_table + (int64_t)b * p.stride;
    const uint8_t* kpool = p.k_pages + (int64_t)g * TILE_BYTES;
    const uint8_t* vpool = p.v_pages + (int64_t)g * TILE_BYTES;
    const int64_t pb = p.page_bytes;

    // Page ids are fetched 64 at a time with one vector load and read with
    // readlane (wave-uniform), so no scalar-load latency sits in the loop.
    int bt_base = j0;
    int bt_vec = (j0 + lane < j1) ? bt[j0 + lane] : 0;
    int bt_next = (j0 + 64 + lane < j1) ? bt[j0 + 64 + lane] : 0;
    auto page_id = [&](int j) -> int {
      if (j - bt_base >= 64) {
        bt_base += 64;
        bt_vec = bt_next;
        bt_next = (bt_base + 64 + lane < j1) ? bt[bt_base + 64 + lane] : 0;
      }
      return __builtin_amdgcn_readlane(bt_vec, j - bt_base);
    };

    auto consume = [&](const R& r, int j, int pid) {
      // scores S^T: lane holds tokens of its row group for head `col`
      f32x4 sc[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
          bf16x8 a;
          if constexpr (FP8) {
            const u32x4& w = r.k[t * (D / 64) + (ks >> 1)];
            a = (ks & 1) ? fp8x8_to_bf16(w[2], w[3]) : fp8x8_to_bf16(w[0], w[1]);
          } else {
            a = __builtin_bit_cast(bf16x8, r.k[t * KSTEPS + ks]);
          }
          s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qop[ks], s, 0, 0, 0);
        }
        sc[t] = s;
      }
      float ksc = p.scale_log2;
      float vsc = 1.f;
      if constexpr (FP8) {
        ksc *= p.k_scales[pid];
        vsc = p.v_scales[pid];
      }
      const int nvalid = L - j * P;  // >= 1; < P only on a sequence's last page
      float mx = -__builtin_inff();
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float x = sc[t][i] * ksc;
          const int tok = P == 16 ? 4 * grp + i : 8 * grp + 4 * t + i;
          if (nvalid < P && tok >= nvalid) x = -__builtin_inff();
          sc[t][i] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      float psum = 0.f;
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float e = __builtin_amdgcn_exp2f(sc[t][i] - m_new);
          psum += e;
          sc[t][i] = e * vsc;
        }
      l_run = l_run * alpha + psum;
      if (__ballot(alpha != 1.f)) {
#pragma unroll
        for (int i = 0; i < DBLK; ++i) acc[i] *= alpha;
      }
      // P^T operand, then O^T += V^T P^T per 16-row block of the head dim
      if constexpr (P == 16) {
        bf16x4 pb4 = bf16x4{(__bf16)sc[0][0], (__bf16)sc[0][1], (__bf16)sc[0][2],
                            (__bf16)sc[0][3]};
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
          acc[i] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, pb4, acc[i], 0, 0, 0);
        }
      } else {
        bf16x8 pb8 = bf16x8{(__bf16)sc[0][0], (__bf16)sc[0][1], (__bf16)sc[0][2],
                            (__bf16)sc[0][3], (__bf16)sc[1][0], (__bf16)sc[1][1],
                            (__bf16)sc[1][2], (__bf16)sc[1][3]};
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
          acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb8, acc[i], 0, 0, 0);
        }
      }
    };

    // Two register buffers; the load of page j+1 is issued before page j is
    // consumed.  Past the end the last page is re-requested (a cache hit) so
    // that every iteration issues the same loads.
    R ra, rb;
    int pid_a = page_id(j0);
    load_page<D, P, FP8>(ra, kpool + (int64_t)pid_a * pb, vpool + (int64_t)pid_a * pb, koff,
                         voff);
    int j = j0;
    while (true) {
      const int pid_b = page_id(min(j + 1, j1 - 1));
      load_page<D, P, FP8>(rb, kpool + (int64_t)pid_b * pb, vpool + (int64_t)pid_b * pb, koff,
                           voff);
      consume(ra, j, pid_a);
      if (++j >= j1) break;
      pid_a = page_id(min(j + 1, j1 - 1));
      load_page<D, P, FP8>(ra, kpool + (int64_t)pid_a * pb, vpool + (int64_t)pid_a * pb, koff,
                           voff);
      consume(rb, j, pid_b);
      if (++j >= j1) break;
    }
  }

  // Sum of exponentials over the four row groups (same head, other tokens).
  float l_tot = l_run + __shfl_xor(l_run, 16);
  l_tot += __shfl_xor(l_tot, 32);
  if (col >= G) return;
  const int h = g * G + col;
  if (slot < 0) {
    const float inv = j1 > j0 ? 1.f / l_tot : 0.f;
    uint16_t* o = p.out + ((int64_t)b * Hq + h) * D + 4 * grp;
#pragma unroll
    for (int i = 0; i < DBLK; ++i) {
      bf16x4 v = bf16x4{(__bf16)(acc[i][0] * inv), (__bf16)(acc[i][1] * inv),
                        (__bf16)(acc[i][2] * inv), (__bf16)(acc[i][3] * inv)};
      *(bf16x4*)(o + 16 * i) = v;
    }
  } else {
    float* po = p.part_o + (((int64_t)slot * Hkv + g) * G + col) * D + 4 * grp;
#pragma unroll
    for (int i = 0; i < DBLK; ++i) *(f32x4*)(po + 16 * i) = acc[i];
    if (grp == 0) p.part_ml[((int64_t)slot * Hkv + g) * G + col] = make_float2(m_run, l_tot);
  }
}

// ---------------------------------------------------------------------------
// combine: out = sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void combine_kernel(CombineParams p) {
  const int Hkv = p.num_kv_heads;
  const int b = blockIdx.x / Hkv;
  const int g = blockIdx.x - b * Hkv;
  const int2 si = p.seqinfo[b];
  const int ns = si.y;
  if (ns <= 1) return;
  const int G = p.group, D = p.head_dim;
  const int64_t split_stride = (int64_t)Hkv * G;
  for (int e = threadIdx.x; e < G * D; e += blockDim.x) {
    const int n = e / D, d = e - n * D;
    const int64_t r0 = ((int64_t)si.x * Hkv + g) * G + n;
    float M = -__builtin_inff();
    for (int s = 0; s < ns; ++s) M = fmaxf(M, p.part_ml[r0 + s * split_stride].x);
    float den = 0.f, num = 0.f;
    for (int s = 0; s < ns; ++s) {
      const float2 ml = p.part_ml[r0 + s * split_stride];
      const float w = __builtin_amdgcn_exp2f(ml.x - M);
      den += w * ml.y;
      num += w * p.part_o[(r0 + s * split_stride) * D + d];
    }
    const __bf16 v = (__bf16)(num / den);
    p.out[((int64_t)b * p.num_q_heads + g * G + n) * D + d] = __builtin_bit_cast(uint16_t, v);
  }
}

// ---------------------------------------------------------------------------
// validate (DORA_FLAG_VALIDATE): page ids in range and owned by the version
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void validate_kernel(ValidateParams p) {
  const int b = blockIdx.x;
  const int L = p.seq_lens[b];
  if (L < 0 || (int64_t)L > (int64_t)p.stride * p.page_size) {
    if (threadIdx.x == 0) atomicOr(p.err, 1);
    return;
  }
  const int n = (L + p.page_size - 1) / p.page_size;
  const int32_t* bt = p.block_table + (int64_t)b * p.stride;
  for (int j = threadIdx.x; j < n; j += blockDim.x) {
    const int32_t pid = bt[j];
    if (pid < 0 || pid >= p.num_pages) {
      atomicOr(p.err, 2);
    } else if (p.page_owner && p.page_owner[pid] != p.version_ids[b]) {
      atomicOr(p.err, 4);
    }
  }
}

__global__ void fill_i32_kernel(int32_t* dst, int32_t value, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = value;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

hipError_t launch_plan(const PlanParams& p, hipStream_t s) {
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, s, p);
  return hipGetLastError();
}

template <int D, int P, bool FP8>
static hipError_t launch_split_t(const DecodeParams& p, int64_t grid, hipStream_t s) {
  hipLaunchKernelGGL((split_decode_kernel<D, P, FP8>), dim3((unsigned)grid), dim3(64), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_split_decode(const DecodeParams& p, int head_dim, int page_size, bool fp8,
                               int64_t grid, hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  if (head_dim == 128) {
    if (page_size == 16) return fp8 ? launch_split_t<128, 16, true>(p, grid, s)
                                    : launch_split_t<128, 16, false>(p, grid, s);
    return fp8 ? launch_split_t<128, 32, true>(p, grid, s)
               : launch_split_t<128, 32, false>(p, grid, s);
  }
  if (page_size == 16) return fp8 ? launch_split_t<64, 16, true>(p, grid, s)
                                  : launch_split_t<64, 16, false>(p, grid, s);
  return fp8 ? launch_split_t<64, 32, true>(p, grid, s)
             : launch_split_t<64, 32, false>(p, grid, s);
}

hipError_t launch_combine(const CombineParams& p, hipStream_t s) {
  const int64_t grid = (int64_t)p.num_seqs * p.num_kv_heads;
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(combine_kernel, dim3((unsigned)grid), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_validate(const ValidateParams& p, hipStream_t s) {
  if (p.num_seqs <= 0) return hipSuccess;
  hipLaunchKernelGGL(validate_kernel, dim3(p.num_seqs), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* dst, int32_t value, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_i32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, dst,
                     value, n);
  return hipGetLastError();
}

}  // namespace dora
