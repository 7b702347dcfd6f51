// Decode attention over a paged, multi-version KV pool, for gfx950.
//
// The operation is scaled dot-product attention of one decode query per head
// over a sequence's cached tokens (the per-token decode step whose time enters
// the paper's step-time model, Sec. 2.2 Eq. (1); sequences of several policy
// versions share one pool, Sec. 3.2).  Decode is memory-bound (Sec. 1,
// Sec. 2.2) and the batch is long-tailed (Sec. 2.2, "Workload skewness"), so
// the kernels stream every K/V byte exactly once and give every wavefront the
// same number of bytes whatever the length mix:
//
//   decode   stream-K over the flattened work list.  The work is the sequence
//            of (sequence b, KV head g, page j) "page-heads", ordered by b,
//            then g, then j; a segment is the run of pages of one (b, g).
//            Every wavefront first computes the page prefix of the batch
//            itself (no separate plan launch), then takes the contiguous range
//            [w*T/W, (w+1)*T/W) of the T page-heads.  A segment that lies
//            inside one range is finished in place; only the first and the
//            last segment of a range can be cut, so each wavefront writes at
//            most two partial results (unnormalised output, running max and
//            sum), to slots 2w and 2w+1.
//            Per page, the G query heads of the KV head are packed into the 16
//            columns of MFMA tiles, so each K/V byte is read once per group:
//              S^T[16 tok x 16 head] = K[16 tok x d] * Q^T   (mfma 16x16x32 bf16)
//              O^T[16 d x 16 head]  += V^T[16 d x tok] * P^T  (mfma 16x16x{16,32} bf16)
//            The page layouts (K: 16-byte head-dim chunks, token-major inside a
//            chunk; V: tokens contiguous per head-dim index) make every lane's
//            global load land directly in its MFMA operand registers: pages
//            stream HBM -> VGPRs with no LDS round trip, with the next pages in
//            flight while the current one is consumed.  Online softmax in the
//            log2 domain; max and sum reductions across the four 16-lane row
//            groups use cross-lane shuffles.  fp8 (OCP E4M3FN) pages are
//            converted to bf16 in registers (exact) and the per-page scales are
//            folded into the scores (K) and the probabilities (V).
//            Each wavefront records the one cut segment whose first piece it
//            holds (at most one: its last segment), and writes the zero output
//            of a share of the empty sequences.  When the batch has no more
//            segments than wavefronts the records are kept per segment
//            instead (every segment's record written every call).
//   combine  one workgroup per record: the log-sum-exp merge of the pieces
//            of a cut segment.  The grouped decode's variant has one
//            workgroup per segment and also folds every row with the
//            partials of its group's shared prefix.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "decode_core.h"
#include "dora_internal.h"

namespace dora {

// ---------------------------------------------------------------------------
// shared helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ int pages_of(int L, int P, int stride) {
  if (L <= 0) return 0;
  const int n = (L + P - 1) / P;
  return n < stride ? n : stride;  // a contract violation stays in bounds
}

__device__ __forceinline__ int wave_inclusive_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(v, off);
    if (lane >= off) v += y;
  }
  return v;
}

// A wave-uniform value, kept in a scalar register.
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Number of wavefronts that take part: at most the launched count, and few
// enough that every range holds at least min_range (>= 1) page-heads, so no
// range is empty (W <= T).
__device__ __forceinline__ int effective_waves(int T, int launched, int min_range) {
  const int want = (T + min_range - 1) / min_range;
  return want < launched ? (want > 0 ? want : 1) : launched;
}

// Equal split of T page-heads into W ranges: with q = T / W and rem = T % W,
// ranges 0 .. rem-1 hold q + 1 page-heads and the others q (q >= 1).
struct Split {
  int q, rem;
  __device__ int begin(int w) const { return w * q + (w < rem ? w : rem); }
  // the range that holds page-head x
  __device__ int range_of(int x) const {
    const int big = rem * (q + 1);
    return x < big ? x / (q + 1) : rem + (x - big) / q;
  }
};

// Page-head descriptor word: j (19 bits) | g << 19 (7 bits) | last << 26 |
// (tokens valid in the page - 1) << 27.
__device__ __forceinline__ int desc_j(uint32_t d) { return (int)(d & 0x7FFFFu); }
__device__ __forceinline__ int desc_g(uint32_t d) { return (int)((d >> 19) & 0x7Fu); }
__device__ __forceinline__ bool desc_last(uint32_t d) { return (d >> 26) & 1u; }
__device__ __forceinline__ int desc_nvalid(uint32_t d) { return (int)(d >> 27) + 1; }

// SUFFIX: the decode of the grouped path.  Each sequence starts after the
// pages its group shares (skip[(skip_seq0 + b) / skip_group] pages, which the
// group-prefix kernel covers), and the kernel writes normalised fp32 rows and
// their log-sum-exp (out32, lse) instead of bf16 rows.  A separate
// instantiation, so the plain kernel is unchanged.
template <int D, int P, bool FP8, int NBUF, bool SUFFIX>
__global__ __launch_bounds__(64, 2) void decode_kernel(DecodeParams p) {
  typedef PageRegs<D, P, FP8> R;
  constexpr int KSTEPS = D / 32;
  constexpr int DBLK = D / 16;
  constexpr int E = FP8 ? 1 : 2;
  constexpr int TILE_BYTES = P * D * E;  // one KV head of one page
  // Query operands.  bf16 pages: each page buffer carries the query operand
  // of its own (b, g), loaded with the page, so a page's first MFMA never
  // waits on a load issued after the next pages' (a query load under a
  // branch would be waited for together with everything issued before it).
  // fp8 pages: one operand per segment, the next segment's fetched with its
  // first page; the extra query loads of the per-page form cost the fp8
  // kernel more than its waits (measured: bf16 batches 0.5-1.2% faster with
  // per-page operands, the fp8 batch 2% slower).
  constexpr bool QSLOT = !FP8;
  extern __shared__ int sN[];            // page prefix over sequences, [B + 1]

  const int lane = threadIdx.x;
  const int col = lane & 15;  // MFMA row/column index of this lane
  const int grp = lane >> 4;  // 16-lane row group
  const int B = p.num_seqs, Hkv = p.num_kv_heads, G = p.group, Hq = p.num_q_heads;

  // 0. small block tables: the wavefronts of each XCD (workgroups go to the
  // XCDs round-robin) pull the whole table into their L2 while the lengths
  // load, so the first descriptor loads hit there.  Larger tables: one line.
  // (7B-class batch, 512 KiB table: kernel 0.5 us shorter, outputs bitwise
  // equal.)
  uint32_t bt_sink;
  {
    const int bt_lines = (int)(((int64_t)B * p.stride + 31) / 32);
    const int cover = (int)(gridDim.x >> 3) * 64;
    const int line = bt_lines <= cover ? (int)(blockIdx.x >> 3) * 64 + lane : 0;
    bt_sink = (uint32_t)p.block_table[(int64_t)(line < bt_lines ? line : bt_lines - 1) * 32];
  }

  // 1. page prefix N(b) = pages of the sequences before b, in LDS
  int carry = 0;
  for (int base = 0; base < B; base += 64 * 8) {
    int n[8], tsum = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      // lanes past the batch load the last length and drop it: no branch
      // around the load, so the eight loads issue back to back and are
      // waited for once (a load under a branch is waited for on its own)
      const int b = base + lane * 8 + k;
      const int bc = b < B ? b : B - 1;
      const int L = p.seq_lens[bc];
      int n_b = pages_of(L, P, p.stride);
      if constexpr (SUFFIX) n_b -= p.skip[(p.skip_seq0 + bc) / p.skip_group];
      n[k] = b < B ? n_b : 0;
      tsum += n[k];
    }
    const int incl = wave_inclusive_scan(tsum);
    int excl = carry + incl - tsum;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int b = base + lane * 8 + k;
      if (b < B) sN[b] = excl;
      excl += n[k];
    }
    carry += __shfl(incl, 63);
  }
  if (lane == 0) sN[B] = carry;
  __syncthreads();
  const int64_t w = blockIdx.x;
  // empty sequences: zero output, shared out over the launched wavefronts
  for (int b = (int)w; b < B; b += gridDim.x) {
    if (sN[b + 1] != sN[b]) continue;
    if constexpr (SUFFIX) {  // fp32 outputs: zero, and an empty softmax (lse -inf)
      float* o = p.out32 + (int64_t)b * Hq * D;
      for (int e = lane; e < Hq * D; e += 64) o[e] = 0.f;
      for (int e = lane; e < Hq; e += 64) p.lse[(int64_t)b * Hq + e] = -__builtin_inff();
      for (int e = lane; e < Hkv; e += 64) p.cuts[(int64_t)b * Hkv + e] = make_int4(-1, 0, 0, 0);
      continue;
    }
    uint32_t* o = (uint32_t*)(p.out + (int64_t)b * Hq * D);
    for (int e = lane; e < Hq * D / 2; e += 64) o[e] = 0u;
    if (p.seg_records)
      for (int e = lane; e < Hkv; e += 64) p.cuts[(int64_t)b * Hkv + e] = make_int4(-1, 0, 0, 0);
  }

  // 2. this wavefront's range of page-heads
  const int T = uni(Hkv * carry);  // fits in 32 bits: the host bounds batch x stride x Hkv
  const int W = uni(effective_waves(T, (int)gridDim.x, p.min_range));
  if (T == 0 || w >= W) {
    if (lane == 0 && !p.seg_records) p.cuts[w] = make_int4(-1, 0, 0, 0);
    return;
  }
  Split split;
  split.q = uni(T / W);
  split.rem = T - split.q * W;
  const int x0 = split.begin((int)w), x1 = split.begin((int)w + 1);

  // Descriptors of 64 consecutive page-heads, one per lane: sequence, page id,
  // packed (j, g, last, valid tokens).
  auto describe = [&](int cbase, int& db, int& dpid, uint32_t& dinfo) {
    const int x = cbase + lane;
    db = 0;
    dpid = 0;
    dinfo = 0;
    if (x < x1) {
      int lo = 0, hi = B;  // largest b with Hkv * N(b) <= x
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (Hkv * sN[mid] <= x) lo = mid; else hi = mid;
      }
      const int nb = sN[lo + 1] - sN[lo];
      const int r = x - Hkv * sN[lo];
      const int g = r / nb;
      const int j = r - g * nb;
      const int jt = SUFFIX ? j + p.skip[(p.skip_seq0 + lo) / p.skip_group] : j;  // table index
      int nv = p.seq_lens[lo] - jt * P;
      nv = nv > P ? P : nv;
      db = lo;
      dpid = p.block_table[(int64_t)lo * p.stride + jt];
      dinfo = (uint32_t)j | ((uint32_t)g << 19) | ((uint32_t)(j == nb - 1) << 26) |
              ((uint32_t)(nv - 1) << 27);
    }
  };

  // Per-lane byte offsets inside a (page, KV head) tile (sub-tile 0, k-step 0).
  const uint32_t koff = (uint32_t)((grp * P + tile_token<P>(0, col)) * 16);
  const uint32_t voff = (uint32_t)((col * P + (P == 16 ? 4 : 8) * grp) * E);
  const int64_t pb = p.page_bytes;

  // running state of the current segment
  f32x4 acc[DBLK];
  bf16x8 qop[QSLOT ? 1 : KSTEPS];
  float m_run = -__builtin_inff(), l_run = 0.f;
  int seg_b = 0, seg_g = 0;
  bool seg_whole = false, seg_here = false, first_seg = true;
  int4 cut = make_int4(-1, 0, 0, 0);  // the cut segment whose first piece is here

  // Query operand of (b, g): lane supplies q[head col][8 head-dim values] per
  // k-step, in the head-dim order the K chunks are consumed in.
  auto load_q = [&](bf16x8(&dst)[KSTEPS], int b, int g) {
    load_q_operand<D, FP8>(dst, p.q + ((int64_t)b * Hq + (int64_t)g * G + col) * D, col < G);
  };
  // fp8: the query of the next segment is fetched together with that
  // segment's first page (q_next, tagged with the page-head where the
  // segment starts).
  bf16x8 q_next[QSLOT ? 1 : KSTEPS];
  int q_next_at = -1;

  auto start_segment = [&](int b, int g, bool whole, int x) {
    seg_b = b;
    seg_g = g;
    seg_whole = whole;
    seg_here = whole;  // the segment's first page is in this range
    m_run = -__builtin_inff();
    l_run = 0.f;
#pragma unroll
    for (int i = 0; i < DBLK; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (!QSLOT) {
      if (x == x0) return;  // the range's first query was loaded up front
      if (q_next_at == x) {
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) qop[s] = q_next[s];
      } else {
        load_q(qop, b, g);  // a second segment start inside the prefetch window
      }
    }
  };

  auto finish_segment = [&]() {
    // Sum of exponentials over the four row groups (same head, other tokens).
    const float l_tot = sum_xor32(sum_xor16(l_run));
    if (col < G) {
      if (seg_whole) {
        const float inv = 1.f / l_tot;
        const int64_t row = (int64_t)seg_b * Hq + seg_g * G + col;
        if constexpr (SUFFIX) {  // normalised fp32 output and its base-2 log-sum-exp
#pragma unroll
          for (int i = 0; i < DBLK; ++i)
            *(f32x4*)(p.out32 + row * D + 4 * grp + 16 * i) = acc[i] * inv;
          if (grp == 0) p.lse[row] = m_run + __builtin_amdgcn_logf(l_tot);
        } else {
          uint16_t* o = p.out + row * D + 4 * grp;
#pragma unroll
          for (int i = 0; i < DBLK; ++i)
            *(bf16x4*)(o + 16 * i) =
                bf16x4{(__bf16)(acc[i][0] * inv), (__bf16)(acc[i][1] * inv),
                       (__bf16)(acc[i][2] * inv), (__bf16)(acc[i][3] * inv)};
        }
      } else {
        const int64_t slot = 2 * w + (first_seg ? 0 : 1);
        float* po = p.part_o + (slot * G + col) * D + 4 * grp;
#pragma unroll
        for (int i = 0; i < DBLK; ++i) *(f32x4*)(po + 16 * i) = acc[i];
        if (grp == 0) p.part_ml[slot * G + col] = make_float2(m_run, l_tot);
      }
    }
    if (!seg_whole && seg_here) {
      // pieces of this segment: ranges w .. the range of its last page-head
      const int nb = sN[seg_b + 1] - sN[seg_b];
      const int s0 = Hkv * sN[seg_b] + seg_g * nb;
      const int np = split.range_of(s0 + nb - 1) - (int)w + 1;
      cut = make_int4(seg_b, seg_g, np, first_seg ? 0 : 1);
    }
    if (p.seg_records && lane == 0 && (seg_whole || seg_here))  // the segment's record
      p.cuts[(int64_t)seg_b * Hkv + seg_g] =
          seg_whole ? make_int4(-1, 0, 0, 0) : make_int4((int)w, cut.z, cut.w, 0);
    first_seg = false;
  };

  auto consume = [&](const R& r, const bf16x8(&qo)[KSTEPS], int nvalid, float ksc, float vsc) {
    consume_page<D, P, FP8>(r, nvalid, ksc, vsc, qo, acc, m_run, l_run);
  };

  // 3. stream the range.  Descriptors come in chunks of 64 (current and next);
  // NBUF page buffers rotate so that NBUF-1 pages are in flight while one is
  // consumed; every iteration issues the same loads.
  int cb_b, cb_pid, nb_b, nb_pid;
  uint32_t cb_info, nb_info;
  describe(x0, cb_b, cb_pid, cb_info);
  describe(x0 + 64, nb_b, nb_pid, nb_info);
  int chunk = x0;  // first page-head of the current descriptor chunk
  asm volatile("" ::"v"(bt_sink));  // keeps the table prefetch

  R buf[NBUF];
  bf16x8 qb[QSLOT ? NBUF : 1][KSTEPS];  // bf16: each page's query operand
  int s_b[NBUF];
  uint32_t s_info[NBUF];
  float s_ks[NBUF], s_vs[NBUF];

  auto prefetch = [&](int r, int x) {
    // Past the end of the range the loads still issue (uniform load count per
    // iteration) but every lane reads the same address of the last tile, so
    // each load is a single cache-line request.
    const bool past = x >= x1;
    if (past) x = x1 - 1;
    if (x - chunk >= 64) {
      chunk += 64;
      cb_b = nb_b;
      cb_pid = nb_pid;
      cb_info = nb_info;
      describe(chunk + 64, nb_b, nb_pid, nb_info);
    }
    const int i = x - chunk;
    const int b = __builtin_amdgcn_readlane(cb_b, i);
    const int pid = __builtin_amdgcn_readlane(cb_pid, i);
    const uint32_t info = (uint32_t)__builtin_amdgcn_readlane((int)cb_info, i);
    s_b[r] = b;
    s_info[r] = info;
    if constexpr (QSLOT) {
      load_q(qb[r], b, desc_g(info));
    } else if (desc_j(info) == 0 && x > x0 && x > q_next_at) {
      load_q(q_next, b, desc_g(info));
      q_next_at = x;
    }
    const int64_t tile = (int64_t)pid * pb + (int64_t)desc_g(info) * TILE_BYTES;
    if constexpr (FP8) {
      s_ks[r] = p.k_scales[pid] * p.scale_log2;
      s_vs[r] = p.v_scales[pid];
    } else {
      s_ks[r] = p.scale_log2;
      s_vs[r] = 1.f;
    }
    load_page<D, P, FP8>(buf[r], p.k_pages + tile, p.v_pages + tile, past ? 0u : koff,
                         past ? 0u : voff);
  };

  if constexpr (!QSLOT)
    load_q(qop, __builtin_amdgcn_readlane(cb_b, 0),
           desc_g((uint32_t)__builtin_amdgcn_readlane((int)cb_info, 0)));
#pragma unroll
  for (int k = 0; k < NBUF - 1; ++k) prefetch(k, x0 + k);
  int x = x0;
  while (true) {
#pragma unroll
    for (int r = 0; r < NBUF; ++r) {
      prefetch((r + NBUF - 1) % NBUF, x + NBUF - 1);
      const uint32_t info = s_info[r];
      const int j = desc_j(info);
      if (x == x0 || j == 0) start_segment(s_b[r], desc_g(info), j == 0, x);
      if constexpr (QSLOT)
        consume(buf[r], qb[r], desc_nvalid(info), s_ks[r], s_vs[r]);
      else
        consume(buf[r], qop, desc_nvalid(info), s_ks[r], s_vs[r]);
      if (desc_last(info) || x == x1 - 1) {
        seg_whole = seg_whole && desc_last(info);
        finish_segment();
      }
      if (++x >= x1) goto done;
    }
  }
done:
  if (lane == 0 && !p.seg_records) p.cuts[w] = cut;
}

// ---------------------------------------------------------------------------
// combine
// ---------------------------------------------------------------------------

constexpr int kCombineThreads = 1024;
constexpr int kCombineBatch = 4;  // pieces whose loads a thread issues together

// Online log-sum-exp merge of one piece (max in log2 units, sum, unnormalised
// weighted values) into a running (M, S, acc).
__device__ __forceinline__ void merge_piece(float2 ml, f32x4 o, float& M, float& S, f32x4& acc) {
  if (ml.x > M) {
    const float sc = __builtin_amdgcn_exp2f(M - ml.x);
    acc = acc * sc + o;
    S = S * sc + ml.y;
    M = ml.x;
  } else if (ml.x > -__builtin_inff()) {
    const float w = __builtin_amdgcn_exp2f(ml.x - M);
    acc += w * o;
    S += w * ml.y;
  }
}

// Grouped decode: thread group sg of `groups` folds chunks c = sg, sg +
// groups, ... of the prefix partials of (member, head n) of segment (b, g)
// into its running (M, S, acc); Sk is the group's shared page count.
__device__ __forceinline__ void fold_prefix_chunks(const CombineParams& p, int b, int g, int n,
                                                   int d4, int Sk, int sg, int groups, float& M,
                                                   float& S, f32x4& acc) {
  const int G = p.group, D = p.head_dim, Mg = p.group_size, MG = Mg * G;
  const int64_t bb = (int64_t)p.seq0 + b;  // index in the whole batch
  const int k = (int)(bb / Mg), m = (int)(bb - (int64_t)k * Mg);
  const int64_t item0 = ((int64_t)k * p.num_kv_heads + g) * p.cmax;
  const int chunk = prefix_chunk_of(Sk, p.pre_kh);
  const int chunks = (Sk + chunk - 1) / chunk;
  for (int c0 = sg; c0 < chunks; c0 += groups * kCombineBatch) {
    float2 ml[kCombineBatch];
    f32x4 o[kCombineBatch];
#pragma unroll
    for (int i = 0; i < kCombineBatch; ++i) {  // all loads of the batch first
      const int c = c0 + i * groups;
      ml[i] = make_float2(-__builtin_inff(), 0.f);
      o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (c < chunks) {
        const int64_t slot = (item0 + c) * MG + m * G + n;
        ml[i] = p.pre_ml[slot];
        o[i] = *(const f32x4*)(p.pre_o + slot * D + 4 * d4);
      }
    }
#pragma unroll
    for (int i = 0; i < kCombineBatch; ++i) merge_piece(ml[i], o[i], M, S, acc);
  }
}

// One workgroup per cut record: per decode wavefront w, or per segment when
// the records are kept per segment (batches with no more segments than
// wavefronts, so the launch is smaller).  A cut segment's np pieces sit in
// the slots of wavefronts wa .. wa+np-1, wa the wavefront holding its first
// piece: wa's in 2wa + first_off, every later one's in 2w'.  Threads are
// (head, 4 head-dim values) tasks x piece groups; each folds its pieces into
// a running (max, normaliser, weighted sum) with one pass of loads, and the
// groups are merged in LDS.
template <int THREADS>
__global__ __launch_bounds__(THREADS) void combine_kernel(CombineParams p) {
  __shared__ float sM[THREADS], sS[THREADS];
  __shared__ f32x4 sAcc[THREADS];
  const int4 cut = p.cuts[blockIdx.x];
  if (cut.x < 0) return;
  int64_t wa = blockIdx.x;
  int b = cut.x, g = cut.y, np = cut.z, first_off = cut.w;
  if (p.seg_records) {  // workgroup per segment (b, g); the record names its first wavefront
    const int Hkv = p.num_q_heads / p.group;
    wa = cut.x;
    np = cut.y;
    first_off = cut.z;
    b = (int)blockIdx.x / Hkv;
    g = (int)blockIdx.x - b * Hkv;
  }
  const int t = threadIdx.x;
  const int G = p.group, D = p.head_dim;
  const int tasks = G * (D / 4);
  const int tasks_r = (tasks + 63) & ~63;
  const int groups = THREADS / tasks_r;  // >= 1 since tasks <= 512
  const int task = t % tasks_r, sg = t / tasks_r;
  const bool active = task < tasks && sg < groups;
  const int n = active ? task / (D / 4) : 0, d4 = active ? task - n * (D / 4) : 0;
  float M = -__builtin_inff(), S = 0.f;
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  if (active) {
    for (int k0 = sg; k0 < np; k0 += groups * kCombineBatch) {
      float2 ml[kCombineBatch];
      f32x4 o[kCombineBatch];
#pragma unroll
      for (int i = 0; i < kCombineBatch; ++i) {  // all loads of the batch first
        const int k = k0 + i * groups;
        ml[i] = make_float2(-__builtin_inff(), 0.f);
        o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (k < np) {
          const int64_t row = (2 * (wa + k) + (k == 0 ? first_off : 0)) * G + n;
          ml[i] = p.part_ml[row];
          o[i] = *(const f32x4*)(p.part_o + row * D + 4 * d4);
        }
      }
#pragma unroll
      for (int i = 0; i < kCombineBatch; ++i) {
        if (ml[i].x > M) {
          const float sc = __builtin_amdgcn_exp2f(M - ml[i].x);
          acc = acc * sc + o[i];
          S = S * sc + ml[i].y;
          M = ml[i].x;
        } else if (ml[i].x > -__builtin_inff()) {
          const float wgt = __builtin_amdgcn_exp2f(ml[i].x - M);
          acc += wgt * o[i];
          S += wgt * ml[i].y;
        }
      }
    }
  }
  sM[t] = M;
  sS[t] = S;
  sAcc[t] = acc;
  __syncthreads();
  if (sg == 0 && task < tasks) {
    float Mx = M;
    for (int k = 1; k < groups; ++k) Mx = fmaxf(Mx, sM[k * tasks_r + task]);
    f32x4 num = f32x4{0.f, 0.f, 0.f, 0.f};
    float den = 0.f;
    for (int k = 0; k < groups; ++k) {
      const int i = k * tasks_r + task;
      if (sM[i] == -__builtin_inff()) continue;  // a group with no pieces
      const float sc = __builtin_amdgcn_exp2f(sM[i] - Mx);
      num += sc * sAcc[i];
      den += sc * sS[i];
    }
    const float inv = 1.f / den;
    const int64_t row = (int64_t)b * p.num_q_heads + g * G + n;
    uint16_t* o = p.out + row * D + 4 * d4;
    *(bf16x4*)o = bf16x4{(__bf16)(num[0] * inv), (__bf16)(num[1] * inv),
                         (__bf16)(num[2] * inv), (__bf16)(num[3] * inv)};
  }
}

// The combine of the grouped decode's suffix: one workgroup per segment (b, g)
// of the launch, with the segment's cut record.  A cut segment's pieces are
// merged as in combine_kernel; a segment the decode finished whole (or an
// empty one) starts from its normalised rows in out32 with weight 2^lse
// (loaded with the record, and dropped if the segment was cut).  Either way
// the chunk partials of the group's shared prefix are folded in as further
// pieces before the bf16 store.
__global__ __launch_bounds__(kCombineThreads) void combine_grouped_kernel(CombineParams p) {
  __shared__ float sM[kCombineThreads], sS[kCombineThreads];
  __shared__ f32x4 sAcc[kCombineThreads];
  const int t = threadIdx.x;
  const int G = p.group, D = p.head_dim;
  const int tasks = G * (D / 4);
  const int tasks_r = (tasks + 63) & ~63;
  const int groups = kCombineThreads / tasks_r;  // >= 2 since tasks <= 512
  const int task = t % tasks_r, sg = t / tasks_r;
  const bool active = task < tasks && sg < groups;
  const int n = active ? task / (D / 4) : 0, d4 = active ? task - n * (D / 4) : 0;
  const int b = (int)blockIdx.x / p.num_kv_heads, g = (int)blockIdx.x - b * p.num_kv_heads;
  const int64_t row = (int64_t)b * p.num_q_heads + g * G + n;
  const int4 cut = p.cuts[blockIdx.x];
  const int Sk = p.group_shared[(p.seq0 + b) / p.group_size];
  float M = -__builtin_inff(), S = 0.f;
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  if (active) {
    float lse = -__builtin_inff();
    f32x4 o32 = f32x4{0.f, 0.f, 0.f, 0.f};
    if (sg == 0) {
      lse = p.lse[row];
      o32 = *(const f32x4*)(p.out32 + row * D + 4 * d4);
    }
    if (cut.x >= 0) {  // uniform: a cut segment's pieces
      const int64_t wa = cut.x;
      const int np = cut.y, first_off = cut.z;
      for (int k0 = sg; k0 < np; k0 += groups * kCombineBatch) {
        float2 ml[kCombineBatch];
        f32x4 o[kCombineBatch];
#pragma unroll
        for (int i = 0; i < kCombineBatch; ++i) {  // all loads of the batch first
          const int k = k0 + i * groups;
          ml[i] = make_float2(-__builtin_inff(), 0.f);
          o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
          if (k < np) {
            const int64_t r = (2 * (wa + k) + (k == 0 ? first_off : 0)) * G + n;
            ml[i] = p.part_ml[r];
            o[i] = *(const f32x4*)(p.part_o + r * D + 4 * d4);
          }
        }
#pragma unroll
        for (int i = 0; i < kCombineBatch; ++i) merge_piece(ml[i], o[i], M, S, acc);
      }
    } else if (sg == 0) {  // finished whole by the decode
      M = lse;
      S = lse > -__builtin_inff() ? 1.f : 0.f;
      acc = o32;
    }
    fold_prefix_chunks(p, b, g, n, d4, Sk, sg, groups, M, S, acc);
  }
  sM[t] = M;
  sS[t] = S;
  sAcc[t] = acc;
  __syncthreads();
  if (sg == 0 && task < tasks) {
    float Mx = M;
    for (int k = 1; k < groups; ++k) Mx = fmaxf(Mx, sM[k * tasks_r + task]);
    f32x4 num = f32x4{0.f, 0.f, 0.f, 0.f};
    float den = 0.f;
    for (int k = 0; k < groups; ++k) {
      const int i = k * tasks_r + task;
      if (sM[i] == -__builtin_inff()) continue;  // a group with no pieces
      const float sc = __builtin_amdgcn_exp2f(sM[i] - Mx);
      num += sc * sAcc[i];
      den += sc * sS[i];
    }
    const float inv = den > 0.f ? 1.f / den : 0.f;  // an empty row with no prefix is zero
    *(bf16x4*)(p.out + row * D + 4 * d4) =
        bf16x4{(__bf16)(num[0] * inv), (__bf16)(num[1] * inv), (__bf16)(num[2] * inv),
               (__bf16)(num[3] * inv)};
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

// Register buffers per wave (NBUF - 1 pages in flight).  32-token pages of
// head dim 128 keep one page in flight: for bf16 the register budget of two
// waves per SIMD allows no more; for fp8 one page was 0.2-0.3% faster per
// step than two (MoE batch, two boxes) with 190 instead of 224 registers.
// The other geometries keep two.
template <int D, int P, bool FP8>
constexpr int page_buffers() {
  return (P == 32 && D == 128) ? 2 : 3;
}

template <int D, int P, bool FP8>
static const void* decode_fn(bool out32) {
  constexpr int NBUF = page_buffers<D, P, FP8>();
  return out32 ? (const void*)&decode_kernel<D, P, FP8, NBUF, true>
               : (const void*)&decode_kernel<D, P, FP8, NBUF, false>;
}

static const void* decode_symbol(int head_dim, int page_size, bool fp8, bool out32) {
  if (head_dim == 128) {
    if (page_size == 16)
      return fp8 ? decode_fn<128, 16, true>(out32) : decode_fn<128, 16, false>(out32);
    return fp8 ? decode_fn<128, 32, true>(out32) : decode_fn<128, 32, false>(out32);
  }
  if (page_size == 16) return fp8 ? decode_fn<64, 16, true>(out32) : decode_fn<64, 16, false>(out32);
  return fp8 ? decode_fn<64, 32, true>(out32) : decode_fn<64, 32, false>(out32);
}

size_t decode_lds_bytes(int num_seqs) { return (size_t)(num_seqs + 1) * sizeof(int); }

hipError_t decode_waves_per_cu(int head_dim, int page_size, bool fp8, int num_seqs, int* out) {
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(
      out, decode_symbol(head_dim, page_size, fp8, false), 64, decode_lds_bytes(num_seqs));
}

hipError_t launch_decode(const DecodeParams& p, int head_dim, int page_size, bool fp8,
                         int64_t waves, hipStream_t s) {
  if (waves <= 0) return hipSuccess;
  DecodeParams arg = p;
  void* args[] = {(void*)&arg};
  return hipLaunchKernel(decode_symbol(head_dim, page_size, fp8, p.out32 != nullptr),
                         dim3((unsigned)waves),
                         dim3(64), args, decode_lds_bytes(p.num_seqs), s);
}

// Records per segment (a segment's pieces can be many): 1,024 threads.
// Records per wavefront (batches with more segments than wavefronts, whose
// cut segments mostly have two pieces): 512 threads, one piece group fewer
// to wait for (multi-version batch: combine 8.8 -> 6.2 us; the per-segment
// case is slower with 512, 6.8 -> 7.4 us on the 7B-class batch).
hipError_t launch_combine(const CombineParams& p, int64_t waves, hipStream_t s) {
  if (waves <= 0) return hipSuccess;
  if (p.seg_records)
    hipLaunchKernelGGL(combine_kernel<kCombineThreads>, dim3((unsigned)waves),
                       dim3(kCombineThreads), 0, s, p);
  else
    hipLaunchKernelGGL(combine_kernel<512>, dim3((unsigned)waves), dim3(512), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_combine_grouped(const CombineParams& p, int64_t grid, hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(combine_grouped_kernel, dim3((unsigned)grid), dim3(kCombineThreads), 0, s,
                     p);
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
