// Internal declarations shared by the C-ABI front end and the HIP kernels of
// the decode-attention library.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "dora.h"

namespace dora {

// Decode wavefronts per compute unit, at most, for bf16 and for fp8 pages (and
// never more than the resident slots).  One equal range per wavefront.
constexpr int kBf16WavesPerCu = 4;
constexpr int kFp8WavesPerCu = 7;
// Smallest range (page-heads) a wavefront gets by default: a range must carry
// enough bytes to amortise the wavefront's start-up (page prefix, first loads).
constexpr int kMinRangePages = 8;
// Largest batch one decode launch takes: its page prefix ((B + 1) ints) lives
// in each wavefront's LDS.  Larger batches are cut into launches of this size.
constexpr int kMaxSeqsPerLaunch = 8192;
// Bytes reserved at the start of the workspace for flags.
constexpr size_t kWsHeaderBytes = 256;

// Workspace carve-up for one geometry (offsets in bytes from the base).
struct WsLayout {
  int64_t waves;       // decode wavefronts launched (2 partial slots each)
  size_t cuts_off;     // int4 [waves] cut segment owned by each wavefront
  size_t part_o_off;   // float [2 * waves][G][D] unnormalised partial outputs
  size_t part_ml_off;  // float2 [2 * waves][G] {running max (log2 units), sum}
  size_t total;
};

// Decode wavefronts to launch for this descriptor on the current device
// (desc->num_waves if set).  Falls back to a 256-CU, 8-wave estimate when no
// device can be queried.
int64_t decode_waves(const dora_decode_desc& d);
bool ws_layout(const dora_decode_desc& d, int64_t waves, WsLayout* out);

struct DecodeParams {
  const uint16_t* q;
  const uint8_t* k_pages;
  const uint8_t* v_pages;
  const float* k_scales;
  const float* v_scales;
  const int32_t* block_table;
  const int32_t* seq_lens;
  uint16_t* out;
  float* out32;        // grouped suffix: normalised fp32 rows [B][Hq][d] of the segments
  float* lse;          // finished whole (not `out`), their base-2 log-sum-exp [B][Hq],
  const int32_t* skip; // and sequence b starts at page skip[(skip_seq0 + b) / skip_group]
  int32_t skip_seq0, skip_group;
  int4* cuts;          // cut records, per wavefront or per segment (seg_records)
  float* part_o;
  float2* part_ml;
  int32_t num_seqs, num_q_heads, num_kv_heads, group, stride;
  int32_t min_range;   // smallest range in page-heads
  int64_t page_bytes;  // bytes of one K (or V) page, all KV heads
  float scale_log2;    // softmax scale times log2(e)
  // 0: cuts[w] = {b, g, pieces, first-slot offset} of the cut segment whose
  // first piece wavefront w holds, or b = -1.  1: cuts[b * Hkv + g] = {w,
  // pieces, first-slot offset, 0} for a cut segment, w = -1 for a segment
  // finished whole or empty (every segment's record is written every call).
  int32_t seg_records;
};

struct CombineParams {
  const int4* cuts;             // as DecodeParams::cuts, with seg_records
  const float* part_o;
  const float2* part_ml;
  uint16_t* out;                // bf16 rows of this launch's sequences
  int32_t num_q_heads, group, head_dim;
  int32_t seg_records;
  // Grouped decode only (records per segment): every row of this launch's
  // sequences is folded with its group's prefix partials before the bf16
  // store.  Rows the decode finished whole come from out32 / lse; cut ones
  // from the pieces.
  const float* out32;
  const float* lse;
  const int32_t* group_shared;  // per group: shared full pages
  const float* pre_o;           // prefix partials, as GroupedParams::part_o
  const float2* pre_ml;
  int32_t num_seqs, seq0, num_kv_heads, group_size, cmax;
  int64_t pre_kh;               // groups x KV heads of the whole batch
};

// Grouped decode (groups of sequences sharing a prompt's pages).
constexpr int kPrefixMaxWaves = 8;      // (member, head) columns per group <= 128
constexpr int kPrefixMinChunk = 16;     // shared pages per prefix work item, at least ...
constexpr int kPrefixMaxChunk = 512;    // ... and at most
constexpr int kPrefixTargetItems = 512; // prefix work items aimed at (2 per CU)

// Pages per prefix work item of a group sharing S pages, with kh (group, KV
// head) pairs in the batch: about kPrefixTargetItems items over all pairs,
// clamped to [kPrefixMinChunk, kPrefixMaxChunk].  Item (k, g, c) covers pages
// [c * chunk, min((c + 1) * chunk, S)); its partials sit at item index
// (k * Hkv + g) * cmax + c.  The prefix kernel and the folding combine both
// derive the split from here.
__host__ __device__ inline int prefix_chunk_of(int S, int64_t kh) {
  const int64_t want = ((int64_t)S * kh + kPrefixTargetItems - 1) / kPrefixTargetItems;
  return want < kPrefixMinChunk ? kPrefixMinChunk
                                : (want > kPrefixMaxChunk ? kPrefixMaxChunk : (int)want);
}

struct GroupedParams {
  const uint16_t* q;
  const uint8_t* k_pages;
  const uint8_t* v_pages;
  const float* k_scales;
  const float* v_scales;
  const int32_t* block_table;
  const int32_t* seq_lens;
  int32_t* group_shared;      // per group: shared full pages (prefix kernel)
  int32_t* shared_out;        // optional caller copy of group_shared
  float* part_o;              // [items][columns][d] unnormalised prefix partials
  float2* part_ml;            // [items][columns] {max (log2 units), sum}
  float* out32;               // suffix rows [B][Hq][d] (normalised) ...
  float* lse;                 // ... and their base-2 log-sum-exp [B][Hq]
  uint16_t* out;
  int32_t num_seqs, num_q_heads, num_kv_heads, group, stride, group_size, page_size, head_dim;
  int32_t cmax;               // prefix items per (group, KV head), at most
  int64_t page_bytes;
  float scale_log2;
};

hipError_t launch_grouped_prefix(const GroupedParams& p, int grid, bool fp8, hipStream_t s);
// The suffix decode of the grouped path: out32 / lse hold rows the decode
// finishes whole, seg_rec every segment's cut record; the combine then
// writes every row to gp.out folded with the prefix partials.
struct GroupedSuffix {
  const GroupedParams* gp;
  int4* seg_rec;  // [min(B, kMaxSeqsPerLaunch)][Hkv], reused per launch
};
dora_status enqueue_decode(const dora_decode_desc& d, const void* q, const void* k_pages,
                           const void* v_pages, const int32_t* block_table,
                           const int32_t* seq_lens, uint16_t* out, const GroupedSuffix* gs,
                           uint8_t* ws, const WsLayout& w, hipStream_t s, hipEvent_t* ev);
// dora_decode_attn, with three timing events recorded on `s` when ev is set:
// before the first decode kernel, after it, and after the last combine kernel.
dora_status decode_attn(const dora_decode_desc* desc, const void* q, const void* k_pages,
                        const void* v_pages, const int32_t* block_table, const int32_t* seq_lens,
                        const int32_t* version_ids, void* out, void* workspace,
                        size_t workspace_bytes, hipStream_t s, hipEvent_t* ev);

struct ValidateParams {
  const int32_t* block_table;
  const int32_t* seq_lens;
  const int32_t* version_ids;
  const int16_t* page_owner;
  int32_t num_seqs, page_size, stride;
  int64_t num_pages;
  int32_t* err;
};

size_t decode_lds_bytes(int num_seqs);
hipError_t decode_waves_per_cu(int head_dim, int page_size, bool fp8, int num_seqs, int* out);
hipError_t launch_decode(const DecodeParams& p, int head_dim, int page_size, bool fp8,
                         int64_t waves, hipStream_t s);
hipError_t launch_combine(const CombineParams& p, int64_t waves, hipStream_t s);
hipError_t launch_combine_grouped(const CombineParams& p, int64_t grid, hipStream_t s);
hipError_t launch_validate(const ValidateParams& p, hipStream_t s);

struct AppendParams {
  const uint16_t* k_new;       // bf16 [B][Hkv][d]
  const uint16_t* v_new;
  const int32_t* block_table;
  const int32_t* seq_lens;
  const int32_t* version_ids;  // ownership check when page_owner is set
  const int16_t* page_owner;
  uint8_t* k_pages;
  uint8_t* v_pages;
  float* k_scales;             // fp8 only
  float* v_scales;
  int32_t* dev_status;         // may be null
  int32_t num_seqs, num_kv_heads, head_dim, page_size, stride;
  int64_t num_pages;
};

hipError_t launch_append(const AppendParams& p, bool fp8, hipStream_t s);
hipError_t launch_fill_i32(int32_t* dst, int32_t value, int64_t n, hipStream_t s);

// 256-byte pack header, written by the pack kernel and checked by unpack.
struct PackHeader {
  uint32_t words[64];
};
void make_pack_header(const dora_pack_desc& d, int64_t n_pages, PackHeader* h);

struct PackParams {
  const uint8_t* k_pages;
  const uint8_t* v_pages;
  const float* k_scales;
  const float* v_scales;
  const int32_t* pages;   // source (pack) or destination (unpack) page ids
  int64_t n_pages, num_pages, page_bytes;
  uint8_t* packed;        // pack: destination buffer
  const uint8_t* packed_in;  // unpack: source buffer
  uint8_t* k_out;         // unpack destinations
  uint8_t* v_out;
  float* ks_out;
  float* vs_out;
  int32_t* dev_status;
  int32_t has_scales;
  PackHeader hdr;
};

hipError_t launch_pack(const PackParams& p, hipStream_t s);
hipError_t launch_unpack(const PackParams& p, hipStream_t s);

}  // namespace dora
