// C-ABI front end: argument validation (before any launch, no side effects),
// workspace layout, and the launch sequence of each entry point.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "dora_internal.h"

using namespace dora;

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool geometry_supported(const dora_decode_desc& d) {
  if (d.head_dim != 64 && d.head_dim != 128) return false;
  if (d.page_size != 16 && d.page_size != 32) return false;
  if (d.kv_dtype != DORA_KV_BF16 && d.kv_dtype != DORA_KV_FP8_E4M3) return false;
  const int G = d.num_q_heads / d.num_kv_heads;
  // the decode kernel's page-head descriptor holds g in 7 bits and j in 19, and
  // its page prefix and page-head indices are 32-bit
  const int64_t seqs = d.num_seqs < kMaxSeqsPerLaunch ? d.num_seqs : kMaxSeqsPerLaunch;
  return G >= 1 && G <= 16 && d.num_kv_heads <= 127 && d.block_table_stride < (1 << 19) &&
         seqs * d.block_table_stride * d.num_kv_heads < ((int64_t)1 << 31);
}

// Host-checkable validity of a descriptor (pointers are checked separately).
dora_status check_desc(const dora_decode_desc* d) {
  if (!d) return DORA_ERR_INVALID_ARG;
  if (d->num_seqs < 0 || d->num_kv_heads < 1 || d->num_q_heads < 1 ||
      d->num_q_heads % d->num_kv_heads != 0 || d->block_table_stride < 1 ||
      d->num_pages < 1 || d->head_dim < 1 || d->page_size < 1 || !(d->sm_scale >= 0.f) ||
      d->num_waves < 0 || d->min_range_pages < 0 || (d->flags & ~DORA_FLAG_VALIDATE) != 0)
    return DORA_ERR_INVALID_ARG;
  if (!geometry_supported(*d)) return DORA_ERR_UNSUPPORTED;
  return DORA_OK;
}

int min_range_of(const dora_decode_desc& d) {
  return d.min_range_pages > 0 ? d.min_range_pages : kMinRangePages;
}

}  // namespace

namespace dora {

// Decode wavefronts per launch.  bf16 pages take at most kBf16WavesPerCu per
// CU, one per SIMD: past that the kernel is bound by HBM, and each extra
// wavefront only adds cuts, partials and combine work (4 per CU against 5:
// 1.2-1.8% faster per step on every bf16 batch; 4.5 per CU, which leaves
// some SIMDs two wavefronts and others one, is slower than both).  fp8 pages
// take at most kFp8WavesPerCu: their per-page conversion work needs the
// occupancy (4 per CU: 20% slower), and 7 per CU is 0.7% faster per step than
// every resident slot (8).  Never more than the batch can use: at most
// B * Hkv * stride page-heads, min_range each.
int64_t decode_waves(const dora_decode_desc& d) {
  if (d.num_waves > 0) return d.num_waves;
  int dev = 0, cus = 0, per_cu = 0;
  const bool fp8 = d.kv_dtype == DORA_KV_FP8_E4M3;
  const int seqs = d.num_seqs < kMaxSeqsPerLaunch ? d.num_seqs : kMaxSeqsPerLaunch;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      decode_waves_per_cu(d.head_dim, d.page_size, fp8, seqs, &per_cu) != hipSuccess ||
      cus <= 0 || per_cu <= 0) {
    (void)hipGetLastError();  // no device here: size for a 256-CU part at 8 waves per CU
    cus = 256;
    per_cu = 8;
  }
  const int cap = fp8 ? kFp8WavesPerCu : kBf16WavesPerCu;
  if (per_cu > cap) per_cu = cap;
  const int64_t slots = (int64_t)cus * per_cu;
  const int64_t most = (int64_t)seqs * d.num_kv_heads * d.block_table_stride;
  const int64_t need = (most + min_range_of(d) - 1) / min_range_of(d);
  return need < slots ? (need > 0 ? need : 1) : slots;
}

bool ws_layout(const dora_decode_desc& d, int64_t waves, WsLayout* out) {
  const int64_t G = d.num_q_heads / d.num_kv_heads;
  WsLayout w;
  w.waves = waves;
  size_t off = kWsHeaderBytes;
  w.cuts_off = off;
  off = align_up(off + (size_t)waves * 16);
  w.part_o_off = off;
  off = align_up(off + (size_t)(2 * waves) * G * d.head_dim * 4);
  w.part_ml_off = off;
  off = align_up(off + (size_t)(2 * waves) * G * 8);
  w.total = off;
  *out = w;
  return true;
}

}  // namespace dora

extern "C" {

const char* dora_status_string(int status) {
  switch (status) {
    case DORA_OK: return "ok";
    case DORA_ERR_INVALID_ARG: return "invalid argument";
    case DORA_ERR_UNSUPPORTED: return "unsupported geometry or dtype";
    case DORA_ERR_WORKSPACE_TOO_SMALL: return "workspace or buffer too small";
    case DORA_ERR_VERSION_MISMATCH: return "policy version mismatch";
    case DORA_ERR_POOL_EXHAUSTED: return "page pool exhausted";
    case DORA_ERR_DEVICE_CHECK: return "device data check failed";
    case DORA_ERR_HIP: return "HIP runtime error";
    case DORA_ERR_NOT_FOUND: return "sequence not found";
  }
  return "unknown status";
}

size_t dora_decode_workspace_bytes(const dora_decode_desc* desc) {
  if (check_desc(desc) != DORA_OK) return 0;
  WsLayout w;
  if (!ws_layout(*desc, decode_waves(*desc), &w)) return 0;
  return w.total;
}

int64_t dora_decode_num_waves(const dora_decode_desc* desc) {
  if (check_desc(desc) != DORA_OK) return 0;
  return decode_waves(*desc);
}

}  // extern "C"

namespace dora {

// DORA_FLAG_VALIDATE: range- and ownership-check every page id the call will
// read, synchronously (err: one device int32 of scratch).
dora_status validate_tables(const dora_decode_desc& d, const int32_t* block_table,
                            const int32_t* seq_lens, const int32_t* version_ids, int32_t* err,
                            hipStream_t s) {
  if (launch_fill_i32(err, 0, 1, s) != hipSuccess) return DORA_ERR_HIP;
  ValidateParams vp{block_table, seq_lens, version_ids, d.page_owner, d.num_seqs,
                    d.page_size, d.block_table_stride, d.num_pages, err};
  if (launch_validate(vp, s) != hipSuccess) return DORA_ERR_HIP;
  int32_t host_err = 0;
  if (hipMemcpyAsync(&host_err, err, 4, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return DORA_ERR_HIP;
  return host_err ? DORA_ERR_DEVICE_CHECK : DORA_OK;
}

// Grouped decode: where each piece lives in the workspace (the decode
// workspace first).  The shared prefixes are found on the device, so the
// prefix launch and its partials are sized for the most chunks any group can
// have: with chunk = clamp(ceil(S * K * Hkv / T), kPrefixMinChunk,
// kPrefixMaxChunk), T = kPrefixTargetItems, and S <= stride, a (group, KV
// head) has at most min(ceil(stride / kPrefixMinChunk),
// max(ceil(T / (K * Hkv)), ceil(stride / kPrefixMaxChunk))) chunks.
struct GroupedLayout {
  WsLayout dec;
  size_t gshared_off, part_o_off, part_ml_off, out32_off, lse_off, seg_rec_off, total;
  int64_t cmax, items;
};

bool grouped_layout(const dora_decode_desc& d, int32_t group_size, GroupedLayout* L) {
  const int64_t G = d.num_q_heads / d.num_kv_heads;
  const int64_t n_groups = d.num_seqs / group_size;
  const int64_t MG = group_size * G;
  const int64_t kh = n_groups * d.num_kv_heads;
  auto cdiv = [](int64_t a, int64_t b) { return (a + b - 1) / b; };
  const int64_t lo = cdiv(d.block_table_stride, kPrefixMinChunk);
  int64_t hi = kh > 0 ? cdiv(kPrefixTargetItems, kh) : 1;
  const int64_t big = cdiv(d.block_table_stride, kPrefixMaxChunk);
  hi = hi > big ? hi : big;
  L->cmax = lo < hi ? lo : hi;
  L->items = kh * L->cmax;
  if (L->items > INT32_MAX / 2) return false;
  if (!ws_layout(d, decode_waves(d), &L->dec)) return false;
  size_t off = L->dec.total;
  L->gshared_off = off;
  off = align_up(off + (size_t)n_groups * 4);
  L->part_o_off = off;
  off = align_up(off + (size_t)L->items * MG * d.head_dim * 4);
  L->part_ml_off = off;
  off = align_up(off + (size_t)L->items * MG * 8);
  L->out32_off = off;
  off = align_up(off + (size_t)d.num_seqs * d.num_q_heads * d.head_dim * 4);
  L->lse_off = off;
  off = align_up(off + (size_t)d.num_seqs * d.num_q_heads * 4);
  L->seg_rec_off = off;  // one launch's segment records: reused by every launch
  const int64_t seqs = d.num_seqs < kMaxSeqsPerLaunch ? d.num_seqs : kMaxSeqsPerLaunch;
  off = align_up(off + (size_t)seqs * d.num_kv_heads * 16);
  L->total = off;
  return true;
}

// Host-checkable validity of the group arguments.
dora_status check_groups(const dora_decode_desc& d, int32_t group_size) {
  if (group_size < 1 || d.num_seqs % group_size != 0) return DORA_ERR_INVALID_ARG;
  if ((int64_t)group_size * (d.num_q_heads / d.num_kv_heads) > 16 * kPrefixMaxWaves)
    return DORA_ERR_UNSUPPORTED;
  return DORA_OK;
}

// The decode launches of one call on validated arguments: per 8192 sequences,
// the decode kernel and the combine kernel.  Outputs go to `out` (bf16), or,
// when out32 is set (the grouped path's suffix), to out32 (fp32, normalised)
// and lse (base-2 log-sum-exp), each sequence b starting at page
// skip[b / skip_group].
dora_status enqueue_decode(const dora_decode_desc& d, const void* q, const void* k_pages,
                           const void* v_pages, const int32_t* block_table,
                           const int32_t* seq_lens, uint16_t* out, const GroupedSuffix* gs,
                           uint8_t* ws, const WsLayout& w, hipStream_t s, hipEvent_t* ev) {
  const GroupedParams* gp = gs ? gs->gp : nullptr;
  const bool fp8 = d.kv_dtype == DORA_KV_FP8_E4M3;
  const int G = d.num_q_heads / d.num_kv_heads;
  const int e = fp8 ? 1 : 2;
  const float scale = d.sm_scale > 0.f ? d.sm_scale : 1.0f / sqrtf((float)d.head_dim);
  const int64_t qrow = (int64_t)d.num_q_heads * d.head_dim;  // elements per sequence
  if (ev && hipEventRecord(ev[0], s) != hipSuccess) return DORA_ERR_HIP;
  for (int c0 = 0; c0 < d.num_seqs; c0 += kMaxSeqsPerLaunch) {
    const int nb = d.num_seqs - c0 < kMaxSeqsPerLaunch ? d.num_seqs - c0 : kMaxSeqsPerLaunch;
    DecodeParams dp;
    dp.q = (const uint16_t*)q + c0 * qrow;
    dp.k_pages = (const uint8_t*)k_pages;
    dp.v_pages = (const uint8_t*)v_pages;
    dp.k_scales = d.k_scales;
    dp.v_scales = d.v_scales;
    dp.block_table = block_table + (int64_t)c0 * d.block_table_stride;
    dp.seq_lens = seq_lens + c0;
    dp.out = gp ? nullptr : out + c0 * qrow;
    dp.out32 = gp ? gp->out32 + c0 * qrow : nullptr;
    dp.lse = gp ? gp->lse + (int64_t)c0 * d.num_q_heads : nullptr;
    dp.skip = gp ? gp->group_shared : nullptr;
    dp.skip_seq0 = c0;
    dp.skip_group = gp ? gp->group_size : 1;
    // Cut records per segment where that is the smaller combine launch (the
    // grouped combine always works per segment); per wavefront otherwise.
    const int64_t segs = (int64_t)nb * d.num_kv_heads;
    dp.seg_records = (gp || segs <= w.waves) ? 1 : 0;
    dp.cuts = gs ? gs->seg_rec : (int4*)(ws + w.cuts_off);
    dp.part_o = (float*)(ws + w.part_o_off);
    dp.part_ml = (float2*)(ws + w.part_ml_off);
    dp.num_seqs = nb;
    dp.num_q_heads = d.num_q_heads;
    dp.num_kv_heads = d.num_kv_heads;
    dp.group = G;
    dp.stride = d.block_table_stride;
    dp.min_range = min_range_of(d);
    dp.page_bytes = (int64_t)d.num_kv_heads * d.page_size * d.head_dim * e;
    dp.scale_log2 = scale * 1.4426950408889634f;
    if (launch_decode(dp, d.head_dim, d.page_size, fp8, w.waves, s) != hipSuccess)
      return DORA_ERR_HIP;
    if (ev && c0 == 0 && hipEventRecord(ev[1], s) != hipSuccess) return DORA_ERR_HIP;
    CombineParams cp{};
    cp.cuts = dp.cuts;
    cp.seg_records = dp.seg_records;
    cp.part_o = dp.part_o;
    cp.part_ml = dp.part_ml;
    cp.num_q_heads = d.num_q_heads;
    cp.group = G;
    cp.head_dim = d.head_dim;
    if (!gp) {
      cp.out = dp.out;
      if (launch_combine(cp, dp.seg_records ? segs : w.waves, s) != hipSuccess)
        return DORA_ERR_HIP;
    } else {
      cp.out = gp->out + c0 * qrow;
      cp.out32 = dp.out32;
      cp.lse = dp.lse;
      cp.group_shared = gp->group_shared;
      cp.pre_o = gp->part_o;
      cp.pre_ml = gp->part_ml;
      cp.num_seqs = nb;
      cp.seq0 = c0;
      cp.num_kv_heads = d.num_kv_heads;
      cp.group_size = gp->group_size;
      cp.cmax = gp->cmax;
      cp.pre_kh = (int64_t)(d.num_seqs / gp->group_size) * d.num_kv_heads;
      if (launch_combine_grouped(cp, segs, s) != hipSuccess)
        return DORA_ERR_HIP;
    }
  }
  if (ev && hipEventRecord(ev[2], s) != hipSuccess) return DORA_ERR_HIP;
  return DORA_OK;
}

// dora_decode_attn with optional timing events (ev: NULL or three events).
dora_status decode_attn(const dora_decode_desc* desc, const void* q, const void* k_pages,
                        const void* v_pages, const int32_t* block_table, const int32_t* seq_lens,
                        const int32_t* version_ids, void* out, void* workspace,
                        size_t workspace_bytes, hipStream_t s, hipEvent_t* ev) {
  dora_status st = check_desc(desc);
  if (st != DORA_OK) return st;
  const dora_decode_desc& d = *desc;
  if (d.num_seqs == 0) return DORA_OK;
  const bool fp8 = d.kv_dtype == DORA_KV_FP8_E4M3;
  const bool validate = (d.flags & DORA_FLAG_VALIDATE) != 0;
  if (!q || !k_pages || !v_pages || !block_table || !seq_lens || !out || !workspace)
    return DORA_ERR_INVALID_ARG;
  if (fp8 && (!d.k_scales || !d.v_scales)) return DORA_ERR_INVALID_ARG;
  if (validate && (!version_ids && d.page_owner)) return DORA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k_pages) || !aligned16(v_pages) || !aligned16(out) ||
      !aligned16(workspace))
    return DORA_ERR_INVALID_ARG;
  WsLayout w;
  ws_layout(d, decode_waves(d), &w);
  if (workspace_bytes < w.total) return DORA_ERR_WORKSPACE_TOO_SMALL;

  uint8_t* ws = (uint8_t*)workspace;
  if (validate) {
    st = validate_tables(d, block_table, seq_lens, version_ids, (int32_t*)ws, s);
    if (st != DORA_OK) return st;
  }

  return enqueue_decode(d, q, k_pages, v_pages, block_table, seq_lens, (uint16_t*)out, nullptr,
                        ws, w, s, ev);
}

}  // namespace dora

extern "C" {

dora_status dora_decode_attn(const dora_decode_desc* desc, const void* q, const void* k_pages,
                             const void* v_pages, const int32_t* block_table,
                             const int32_t* seq_lens, const int32_t* version_ids, void* out,
                             void* workspace, size_t workspace_bytes, dora_stream_t stream) {
  return decode_attn(desc, q, k_pages, v_pages, block_table, seq_lens, version_ids, out,
                     workspace, workspace_bytes, (hipStream_t)stream, nullptr);
}

size_t dora_decode_grouped_workspace_bytes(const dora_decode_desc* desc, int32_t group_size) {
  if (check_desc(desc) != DORA_OK || check_groups(*desc, group_size) != DORA_OK) return 0;
  GroupedLayout L;
  if (!grouped_layout(*desc, group_size, &L)) return 0;
  return L.total;
}

dora_status dora_decode_attn_grouped(const dora_decode_desc* desc, const void* q,
                                     const void* k_pages, const void* v_pages,
                                     const int32_t* block_table, const int32_t* seq_lens,
                                     const int32_t* version_ids, void* out, int32_t group_size,
                                     int32_t* shared_pages_out, void* workspace,
                                     size_t workspace_bytes, dora_stream_t stream) {
  dora_status st = check_desc(desc);
  if (st != DORA_OK) return st;
  const dora_decode_desc& d = *desc;
  st = check_groups(d, group_size);
  if (st != DORA_OK) return st;
  if (d.num_seqs == 0) return DORA_OK;
  const bool fp8 = d.kv_dtype == DORA_KV_FP8_E4M3;
  if (!q || !k_pages || !v_pages || !block_table || !seq_lens || !out || !workspace)
    return DORA_ERR_INVALID_ARG;
  if (fp8 && (!d.k_scales || !d.v_scales)) return DORA_ERR_INVALID_ARG;
  if ((d.flags & DORA_FLAG_VALIDATE) && !version_ids && d.page_owner)
    return DORA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k_pages) || !aligned16(v_pages) || !aligned16(out) ||
      !aligned16(workspace))
    return DORA_ERR_INVALID_ARG;
  GroupedLayout L;
  if (!grouped_layout(d, group_size, &L)) return DORA_ERR_INVALID_ARG;
  if (workspace_bytes < L.total) return DORA_ERR_WORKSPACE_TOO_SMALL;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)workspace;
  if (d.flags & DORA_FLAG_VALIDATE) {
    st = validate_tables(d, block_table, seq_lens, version_ids, (int32_t*)ws, s);
    if (st != DORA_OK) return st;
  }

  const int e = fp8 ? 1 : 2;
  const float scale = d.sm_scale > 0.f ? d.sm_scale : 1.0f / sqrtf((float)d.head_dim);
  GroupedParams gp;
  gp.q = (const uint16_t*)q;
  gp.k_pages = (const uint8_t*)k_pages;
  gp.v_pages = (const uint8_t*)v_pages;
  gp.k_scales = d.k_scales;
  gp.v_scales = d.v_scales;
  gp.block_table = block_table;
  gp.seq_lens = seq_lens;
  gp.group_shared = (int32_t*)(ws + L.gshared_off);
  gp.shared_out = shared_pages_out;
  gp.part_o = (float*)(ws + L.part_o_off);
  gp.part_ml = (float2*)(ws + L.part_ml_off);
  gp.out32 = (float*)(ws + L.out32_off);
  gp.lse = (float*)(ws + L.lse_off);
  gp.out = (uint16_t*)out;
  gp.num_seqs = d.num_seqs;
  gp.num_q_heads = d.num_q_heads;
  gp.num_kv_heads = d.num_kv_heads;
  gp.group = d.num_q_heads / d.num_kv_heads;
  gp.stride = d.block_table_stride;
  gp.group_size = group_size;
  gp.page_size = d.page_size;
  gp.head_dim = d.head_dim;
  gp.cmax = (int32_t)L.cmax;
  gp.page_bytes = (int64_t)d.num_kv_heads * d.page_size * d.head_dim * e;
  gp.scale_log2 = scale * 1.4426950408889634f;
  if (launch_grouped_prefix(gp, (int)L.items, fp8, s) != hipSuccess) return DORA_ERR_HIP;
  const GroupedSuffix gs{&gp, (int4*)(ws + L.seg_rec_off)};
  return enqueue_decode(d, q, k_pages, v_pages, block_table, seq_lens, nullptr, &gs, ws, L.dec, s,
                        nullptr);
}

dora_status dora_kv_append(const dora_decode_desc* desc, const void* k_new, const void* v_new,
                           const int32_t* block_table, const int32_t* seq_lens,
                           const int32_t* version_ids, void* k_pages, void* v_pages,
                           float* k_scales, float* v_scales, int32_t* dev_status,
                           dora_stream_t stream) {
  dora_status st = check_desc(desc);
  if (st != DORA_OK) return st;
  const dora_decode_desc& d = *desc;
  if (d.num_seqs == 0) return DORA_OK;
  const bool fp8 = d.kv_dtype == DORA_KV_FP8_E4M3;
  const bool validate = (d.flags & DORA_FLAG_VALIDATE) != 0;
  if (!k_new || !v_new || !block_table || !seq_lens || !k_pages || !v_pages)
    return DORA_ERR_INVALID_ARG;
  if (fp8 && (!k_scales || !v_scales)) return DORA_ERR_INVALID_ARG;
  if (validate && d.page_owner && !version_ids) return DORA_ERR_INVALID_ARG;
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_pages) || !aligned16(v_pages))
    return DORA_ERR_INVALID_ARG;
  AppendParams p;
  p.k_new = (const uint16_t*)k_new;
  p.v_new = (const uint16_t*)v_new;
  p.block_table = block_table;
  p.seq_lens = seq_lens;
  p.version_ids = validate ? version_ids : nullptr;
  p.page_owner = validate ? d.page_owner : nullptr;
  p.k_pages = (uint8_t*)k_pages;
  p.v_pages = (uint8_t*)v_pages;
  p.k_scales = fp8 ? k_scales : nullptr;
  p.v_scales = fp8 ? v_scales : nullptr;
  p.dev_status = dev_status;
  p.num_seqs = d.num_seqs;
  p.num_kv_heads = d.num_kv_heads;
  p.head_dim = d.head_dim;
  p.page_size = d.page_size;
  p.stride = d.block_table_stride;
  p.num_pages = d.num_pages;
  return launch_append(p, fp8, (hipStream_t)stream) == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}

// ---------------------------------------------------------------------------
// pack / unpack
// ---------------------------------------------------------------------------

static dora_status check_pack_desc(const dora_pack_desc* d) {
  if (!d) return DORA_ERR_INVALID_ARG;
  if (d->num_kv_heads < 1 || d->page_size < 1 || d->head_dim < 1 || d->num_pages < 1)
    return DORA_ERR_INVALID_ARG;
  if (d->kv_dtype != DORA_KV_BF16 && d->kv_dtype != DORA_KV_FP8_E4M3)
    return DORA_ERR_UNSUPPORTED;
  const int e = d->kv_dtype == DORA_KV_BF16 ? 2 : 1;
  if (((int64_t)d->num_kv_heads * d->page_size * d->head_dim * e) % 16 != 0)
    return DORA_ERR_UNSUPPORTED;
  return DORA_OK;
}

size_t dora_kv_packed_bytes(const dora_pack_desc* desc, int64_t n_pages) {
  if (check_pack_desc(desc) != DORA_OK || n_pages < 0) return 0;
  const int e = desc->kv_dtype == DORA_KV_BF16 ? 2 : 1;
  const int64_t pb = (int64_t)desc->num_kv_heads * desc->page_size * desc->head_dim * e;
  size_t total = 256 + (size_t)(2 * n_pages * pb);
  if (desc->kv_dtype == DORA_KV_FP8_E4M3) total += (size_t)(2 * n_pages * 4);
  return total;
}

dora_status dora_kv_page_pack(const dora_pack_desc* desc, const void* k_pages,
                              const void* v_pages, const float* k_scales,
                              const float* v_scales, const int32_t* src_pages, int64_t n_pages,
                              void* packed, size_t packed_bytes, dora_stream_t stream) {
  dora_status st = check_pack_desc(desc);
  if (st != DORA_OK) return st;
  if (n_pages < 0 || !packed) return DORA_ERR_INVALID_ARG;
  if (n_pages > 0 && (!k_pages || !v_pages || !src_pages)) return DORA_ERR_INVALID_ARG;
  const bool fp8 = desc->kv_dtype == DORA_KV_FP8_E4M3;
  if (fp8 && n_pages > 0 && (!k_scales || !v_scales)) return DORA_ERR_INVALID_ARG;
  if (!aligned16(packed) || (n_pages > 0 && (!aligned16(k_pages) || !aligned16(v_pages))))
    return DORA_ERR_INVALID_ARG;
  if (packed_bytes < dora_kv_packed_bytes(desc, n_pages)) return DORA_ERR_WORKSPACE_TOO_SMALL;
  PackParams p;
  memset(&p, 0, sizeof p);
  p.k_pages = (const uint8_t*)k_pages;
  p.v_pages = (const uint8_t*)v_pages;
  p.k_scales = k_scales;
  p.v_scales = v_scales;
  p.pages = src_pages;
  p.n_pages = n_pages;
  p.num_pages = desc->num_pages;
  p.page_bytes = (int64_t)desc->num_kv_heads * desc->page_size * desc->head_dim * (fp8 ? 1 : 2);
  p.packed = (uint8_t*)packed;
  p.has_scales = fp8 ? 1 : 0;
  make_pack_header(*desc, n_pages, &p.hdr);
  return launch_pack(p, (hipStream_t)stream) == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}

dora_status dora_kv_page_unpack(const dora_pack_desc* desc, int32_t src_version,
                                const void* packed, size_t packed_bytes,
                                const int32_t* dst_pages, int64_t n_pages, void* k_pages,
                                void* v_pages, float* k_scales, float* v_scales,
                                int32_t* dev_status, dora_stream_t stream) {
  dora_status st = check_pack_desc(desc);
  if (st != DORA_OK) return st;
  if (src_version != desc->policy_version) return DORA_ERR_VERSION_MISMATCH;
  if (n_pages < 0 || !packed) return DORA_ERR_INVALID_ARG;
  if (n_pages > 0 && (!k_pages || !v_pages || !dst_pages)) return DORA_ERR_INVALID_ARG;
  const bool fp8 = desc->kv_dtype == DORA_KV_FP8_E4M3;
  if (fp8 && n_pages > 0 && (!k_scales || !v_scales)) return DORA_ERR_INVALID_ARG;
  if (!aligned16(packed) || (n_pages > 0 && (!aligned16(k_pages) || !aligned16(v_pages))))
    return DORA_ERR_INVALID_ARG;
  if (packed_bytes < dora_kv_packed_bytes(desc, n_pages)) return DORA_ERR_WORKSPACE_TOO_SMALL;
  PackParams p;
  memset(&p, 0, sizeof p);
  p.pages = dst_pages;
  p.n_pages = n_pages;
  p.num_pages = desc->num_pages;
  p.page_bytes = (int64_t)desc->num_kv_heads * desc->page_size * desc->head_dim * (fp8 ? 1 : 2);
  p.packed_in = (const uint8_t*)packed;
  p.k_out = (uint8_t*)k_pages;
  p.v_out = (uint8_t*)v_pages;
  p.ks_out = k_scales;
  p.vs_out = v_scales;
  p.dev_status = dev_status;
  p.has_scales = fp8 ? 1 : 0;
  make_pack_header(*desc, n_pages, &p.hdr);
  return launch_unpack(p, (hipStream_t)stream) == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}

}  // extern "C"
