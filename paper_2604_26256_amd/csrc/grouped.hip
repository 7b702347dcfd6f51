// Decode attention for batches of response groups that share a prompt (the
// GRPO groups of the paper's rollouts: several responses sampled per prompt,
// App. B).  Within a group the members' block tables start with the same page
// ids for the prompt's full pages.  Those shared pages are read from HBM once
// per group instead of once per member.  Everything is planned on the device
// from the block tables, so a call makes no host round trip:
//
//   prefix   one workgroup per (group, KV head, chunk of the group's shared
//            pages).  It finds the group's shared prefix S (leading page ids
//            equal in every member's row, full pages of every member), then
//            its waves stage the pages' K and V tiles in LDS (double-buffered,
//            one barrier per step); each computing wave applies them to a tile
//            of 16 of the group's (member, query head) columns with the decode
//            kernel's MFMA/online-softmax step, and writes an unnormalised
//            partial (o, running max, sum) per column.
//   suffix   the decode kernel over each member's pages past S, writing fp32
//            rows and their log-sum-exp for the segments it finishes whole;
//            its combine merges the cut ones and folds every row with the
//            chunk partials of its group's prefix into the bf16 output.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "decode_core.h"
#include "dora_internal.h"

namespace dora {

constexpr int kPrefixThreads = 64 * kPrefixMaxWaves;
constexpr int kStageSets = 2;  // steps in flight per workgroup (register staging)
constexpr int NCW = 1;         // column tiles per computing wave (2 measured no faster)

// Shared prefix of group k (all threads of the workgroup get it): the number
// of leading pages that every member holds in full (floor(len / P), at most
// the table's width) and whose page id equals the leader's; a group of one
// shares nothing.  Returns early, with a value <= `enough`, once every
// member's full pages number at most `enough`.
//   The loads of the common case (at most kDetectBatch members) issue at
// once, so that the detection costs one round trip: each thread reads the
// members' lengths itself (the same few lines for all threads: the cap needs
// no barrier and no atomics), then the entries j = threadIdx.x of every
// member's row (entries past a member's pages are read and ignored: the rows
// are stride wide).  The lengths go first, so a workgroup whose chunk lies
// past the cap leaves as soon as they arrive.  More members, and prefixes
// longer than the workgroup, are compared in further passes.
constexpr int kDetectBatch = 16;
template <int P>
__device__ int shared_prefix(const GroupedParams& p, int k, int enough) {
  __shared__ int s_min;
  const int M = p.group_size, stride = p.stride;
  const int64_t b0 = (int64_t)k * M;
  if (M == 1) return 0;
  const int32_t* __restrict__ bt = p.block_table + b0 * stride;
  const int j = (int)threadIdx.x < stride ? (int)threadIdx.x : stride - 1;
  int L[kDetectBatch];
  int32_t e[kDetectBatch];
#pragma unroll
  for (int i = 0; i < kDetectBatch; ++i) L[i] = p.seq_lens[b0 + (i < M ? i : M - 1)];
  const int32_t lead = bt[j];
#pragma unroll
  for (int i = 0; i < kDetectBatch; ++i) e[i] = bt[(int64_t)(i < M ? i : M - 1) * stride + j];
  int cap = stride;
#pragma unroll
  for (int i = 0; i < kDetectBatch; ++i) cap = min(cap, L[i] > 0 ? L[i] / P : 0);
  for (int m = kDetectBatch; m < M; ++m) {
    const int Lm = p.seq_lens[b0 + m];
    cap = min(cap, Lm > 0 ? Lm / P : 0);
  }
  if (cap <= enough) return cap;  // uniform: every thread read the same lengths
  bool diff = false;
#pragma unroll
  for (int i = 0; i < kDetectBatch; ++i) diff |= e[i] != lead;
  for (int m = kDetectBatch; m < M; ++m) diff |= bt[(int64_t)m * stride + j] != lead;
  if (threadIdx.x == 0) s_min = cap;
  __syncthreads();
  int first = diff && (int)threadIdx.x < cap ? (int)threadIdx.x : cap;  // smallest mismatch
  for (int jj = threadIdx.x + blockDim.x; jj < cap; jj += blockDim.x) {
    const int32_t ld = bt[jj];
    bool d = false;
    for (int m = 1; m < M; ++m) d |= bt[(int64_t)m * stride + jj] != ld;
    if (d && jj < first) first = jj;
  }
  if (first < cap) atomicMin(&s_min, first);
  __syncthreads();
  return s_min;
}

// The split of a group's shared pages into work items: prefix_chunk_of.
__device__ __forceinline__ int prefix_chunk(int S, const GroupedParams& p) {
  return prefix_chunk_of(S, (int64_t)(p.num_seqs / p.group_size) * p.num_kv_heads);
}

// One step consumes PAIR consecutive pages as one virtual page of VP = PAIR * P
// tokens (bf16 16-token pages go in pairs: half the softmax reductions and
// barriers; fp8 pages keep their own scales, one page per step).  LDS holds a
// step in the layout of a VP-token page, so the decode's lane operands apply:
// K [d/8][VP][8] and V [d][VP] for bf16.
template <int D, int P, bool FP8>
__global__ __launch_bounds__(kPrefixThreads) void prefix_kernel(GroupedParams p) {
  constexpr int PAIR = (!FP8 && P == 16) ? 2 : 1;
  constexpr int VP = PAIR * P;
  typedef PageRegs<D, VP, FP8> R;
  typedef typename R::vraw_t vraw_t;
  constexpr int E = FP8 ? 1 : 2;
  constexpr int TILE = P * D * E;  // bytes of one (page, KV head) K tile; V's is the same
  constexpr int PIECES = 2 * PAIR * TILE / 16;  // 16-byte pieces per step
  constexpr int PER = (PIECES + kPrefixThreads - 1) / kPrefixThreads;
  constexpr int per_t = R::NK / R::NT;
  // V rows in LDS are padded by 16 bytes where the lanes' row-strided reads
  // would otherwise meet in the same banks.
  constexpr int VROW = VP * E >= 32 ? VP * E + 16 : VP * E;
  constexpr int vrow = 16 * VROW;                 // bytes between 16-row blocks of V
  constexpr int KBYTES = PAIR * TILE;             // K part of a step in LDS
  __shared__ __align__(16) uint8_t lds[2][KBYTES + D * VROW];
  __shared__ int s_pid[kPrefixMaxChunk];
  __shared__ float s_ksc[FP8 ? kPrefixMaxChunk : 1], s_vsc[FP8 ? kPrefixMaxChunk : 1];

  // chunk-major order: the blocks that have work (low chunk indices) come
  // first and are dispatched first
  const int KH = p.num_seqs / p.group_size * p.num_kv_heads;
  const int c = blockIdx.x / KH, kg = blockIdx.x - c * KH;
  const int k = kg / p.num_kv_heads, g = kg - k * p.num_kv_heads;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, grp = lane >> 4;
  const int G = p.group, MG = p.group_size * G;
  // A computing wave takes NCW tiles of 16 (member, query head) columns (each
  // K and V operand read from LDS then feeds NCW MFMAs).  Waves past the
  // columns only stage.
  const bool computes = wave * 16 * NCW < MG;
  bf16x8 qop[NCW][D / 32];  // issued first: it does not depend on the prefix
#pragma unroll
  for (int t = 0; t < NCW; ++t) {
    const int cg = (wave * NCW + t) * 16 + col;  // column among (member, head) pairs
    const int m = cg < MG ? cg / G : 0, h = cg < MG ? cg - m * G : 0;
    const int64_t b = (int64_t)k * p.group_size + m;
    load_q_operand<D, FP8>(qop[t], p.q + (b * p.num_q_heads + (int64_t)g * G + h) * D, cg < MG);
  }

  // The group's shared prefix; the first workgroup of each group publishes it
  // for the suffix decode and its combine.  A chunk that starts past every
  // member's full pages has no work whatever the prefix is.
  const int S = shared_prefix<P>(p, k, c * kPrefixMinChunk);
  if (c == 0 && g == 0 && threadIdx.x == 0) {
    p.group_shared[k] = S;
    if (p.shared_out) p.shared_out[k] = S;
  }
  const int chunk = prefix_chunk(S, p);
  const int j0 = c * chunk;
  if (j0 >= S) return;  // uniform: this chunk is past the group's prefix
  const int j1 = j0 + chunk < S ? j0 + chunk : S;
  // The item's page ids (and fp8 scales) go to LDS first: a page load that
  // waited on a block-table load would wait on every load issued before it.
  f32x4 acc[NCW][D / 16];
  float m_run[NCW], l_run[NCW];
#pragma unroll
  for (int t = 0; t < NCW; ++t) {
#pragma unroll
    for (int i = 0; i < D / 16; ++i) acc[t][i] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_run[t] = -__builtin_inff();
    l_run[t] = 0.f;
  }

  const int32_t* bt = p.block_table + (int64_t)k * p.group_size * p.stride;  // the leader's row
  for (int t = threadIdx.x; t < j1 - j0; t += kPrefixThreads) {
    const int pid = bt[j0 + t];
    s_pid[t] = pid;
    if constexpr (FP8) {
      s_ksc[t] = p.scale_log2 * p.k_scales[pid];
      s_vsc[t] = p.v_scales[pid];
    }
  }
  __syncthreads();
  const uint32_t koff = (uint32_t)((grp * VP + tile_token<VP>(0, col)) * 16);
  const uint32_t voff = (uint32_t)(col * VROW + (VP == 16 ? 4 : 8) * grp * E);

  // Piece o of a step: page h = o / (2 TILE / 16) of the step, then its K tile
  // and V tile in 16-byte pieces.  lds_of maps it into the VP-token layout.
  auto lds_of = [&](int o) -> int {
    const int hh = o / (2 * TILE / 16), w = o - hh * (2 * TILE / 16);
    if (w < TILE / 16) {  // K piece (dx, token) -> (dx, hh * P + token)
      const int dx = w / P, t = w - dx * P;
      return (dx * VP + hh * P + t) * 16;
    }
    constexpr int RP = P * E / 16 > 0 ? P * E / 16 : 1;  // 16-byte pieces per V row of a page
    const int v = w - TILE / 16;  // V piece (row, r) -> row of the step, after page hh
    const int row = v / RP;
    return KBYTES + row * VROW + hh * P * E + (v - row * RP) * 16;
  };
  // Loads are never skipped, so the compiler's in-order wait counts stay exact
  // (a load under a branch makes it wait for everything): a step past the end
  // re-reads the last step, a missing second page re-reads the last page, and
  // pieces past the step (fp8 16-token pages) re-read an earlier piece.  None
  // of these duplicates reach a score: LDS only takes the real pieces, and the
  // tokens of a missing page are masked.
  u32x4 st[kStageSets][PER];
  const int n_steps = (j1 - j0 + PAIR - 1) / PAIR;
  auto fetch = [&](u32x4(&dst)[PER], int step) {
    step = step < n_steps ? step : n_steps - 1;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int o = (threadIdx.x + i * kPrefixThreads) % PIECES;
      const int hh = o / (2 * TILE / 16), w = (o - hh * (2 * TILE / 16)) * 16;
      int j = j0 + step * PAIR + hh;
      j = j < j1 ? j : j1 - 1;
      const int64_t pid = s_pid[j - j0];
      const uint8_t* src = (w < TILE ? p.k_pages + w : p.v_pages + (w - TILE)) +
                           pid * p.page_bytes + (int64_t)g * TILE;
      dst[i] = *(const u32x4*)src;
    }
  };
  auto put = [&](const u32x4(&src)[PER], int buf, int step) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int o = threadIdx.x + i * kPrefixThreads;
      const int j = j0 + step * PAIR + o / (2 * TILE / 16);
      if (o < PIECES && j < j1) *(u32x4*)&lds[buf][lds_of(o)] = src[i];
    }
  };

#pragma unroll
  for (int r = 0; r < kStageSets; ++r) fetch(st[r], r);
  put(st[0], 0, 0);
  __syncthreads();
  for (int base = 0; base < n_steps; base += kStageSets) {
#pragma unroll
    for (int r = 0; r < kStageSets; ++r) {
      const int u = base + r;  // step u sits in LDS buffer u & 1; its register set r is free
      fetch(st[r], u + kStageSets);
      if (u < n_steps) {
        if (computes) {
          const int buf = u & 1;
          R pr;
#pragma unroll
          for (int t = 0; t < R::NT; ++t)
#pragma unroll
            for (int s = 0; s < per_t; ++s)
              pr.k[t * per_t + s] = *(const u32x4*)&lds[buf][koff + (4 * s * VP + 4 * t) * 16];
#pragma unroll
          for (int i = 0; i < D / 16; ++i)
            pr.v[i] = *(const vraw_t*)&lds[buf][KBYTES + voff + i * vrow];
          const int jj = j0 + u * PAIR;
          float ksc = p.scale_log2, vsc = 1.f;
          if constexpr (FP8) {
            ksc = s_ksc[jj - j0];
            vsc = s_vsc[jj - j0];
          }
          const int nvalid = (j1 - jj < PAIR ? j1 - jj : PAIR) * P;  // shared pages are full
          consume_page_tiles<D, VP, FP8, NCW>(pr, nvalid, ksc, vsc, qop, acc, m_run, l_run);
        }
        if (u + 1 < n_steps) put(st[(r + 1) % kStageSets], (u + 1) & 1, u + 1);
        __syncthreads();
      }
    }
  }

#pragma unroll
  for (int t = 0; t < NCW; ++t) {
    const float l_tot = sum_xor32(sum_xor16(l_run[t]));
    const int cg = (wave * NCW + t) * 16 + col;
    if (cg < MG) {
      const int64_t slot = ((int64_t)kg * p.cmax + c) * MG + cg;
      float* po = p.part_o + slot * D + 4 * grp;
#pragma unroll
      for (int i = 0; i < D / 16; ++i) *(f32x4*)(po + 16 * i) = acc[t][i];
      if (grp == 0) p.part_ml[slot] = make_float2(m_run[t], l_tot);
    }
  }
}

template <int D, int P, bool FP8>
static const void* prefix_fn() {
  return (const void*)&prefix_kernel<D, P, FP8>;
}

hipError_t launch_grouped_prefix(const GroupedParams& p, int grid, bool fp8, hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  const void* fn;
  if (p.head_dim == 128)
    fn = p.page_size == 16 ? (fp8 ? prefix_fn<128, 16, true>() : prefix_fn<128, 16, false>())
                           : (fp8 ? prefix_fn<128, 32, true>() : prefix_fn<128, 32, false>());
  else
    fn = p.page_size == 16 ? (fp8 ? prefix_fn<64, 16, true>() : prefix_fn<64, 16, false>())
                           : (fp8 ? prefix_fn<64, 32, true>() : prefix_fn<64, 32, false>());
  GroupedParams arg = p;
  void* args[] = {(void*)&arg};
  return hipLaunchKernel(fn, dim3((unsigned)grid), dim3(kPrefixThreads), args, 0, s);
}

}  // namespace dora
