// Internal declarations shared by the C-ABI front end and the HIP kernels of
// the decode-attention library.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "dora.h"

namespace dora {

// Default target number of (sequence, KV head, split) work units per call: 16
// units per compute unit of a 256-CU device, enough for the grid's tail to be
// a small fraction of the call even when one sequence holds most of the pages.
constexpr int kDefaultTargetUnits = 4096;
// Smallest split (pages) chosen automatically: a split must carry enough bytes
// to amortise its start-up latency and its partial-result write.
constexpr int kMinSplitPages = 4;
// Threads of the single-workgroup plan kernel.
constexpr int kPlanThreads = 1024;
// Size-ordering bins of the plan kernel (longest work units dispatched first).
constexpr int kPlanBins = 256;
// Bytes reserved at the start of the workspace for plan counters / flags.
constexpr size_t kWsHeaderBytes = 256;

// Workspace carve-up for one geometry (offsets in bytes from the base).
struct WsLayout {
  int64_t max_items;   // upper bound on (sequence, split) items
  size_t seqinfo_off;  // int2 [B]      {first partial slot, number of splits}
  size_t items_off;    // int4 [max_items] {b, first page, end page, slot or -1}
  size_t part_o_off;   // float [max_items][Hkv][G][D] unnormalised partial outputs
  size_t part_ml_off;  // float2 [max_items][Hkv][G] {running max (log2 units), sum}
  size_t total;
};

bool ws_layout(const dora_decode_desc& d, WsLayout* out);

struct PlanParams {
  const int32_t* seq_lens;
  int32_t num_seqs, page_size, num_kv_heads, stride;
  int32_t target_units, min_pages, force_pages;
  int32_t* hdr;        // hdr[0] = number of items, hdr[1] = pages per split
  int2* seqinfo;
  int4* items;
};

struct DecodeParams {
  const uint16_t* q;
  const uint8_t* k_pages;
  const uint8_t* v_pages;
  const float* k_scales;
  const float* v_scales;
  const int32_t* block_table;
  const int32_t* seq_lens;
  uint16_t* out;
  const int32_t* hdr;
  const int4* items;
  float* part_o;
  float2* part_ml;
  int32_t num_q_heads, num_kv_heads, group, stride;
  int64_t page_bytes;  // bytes of one K (or V) page, all KV heads
  float scale_log2;    // softmax scale times log2(e)
};

struct CombineParams {
  const int2* seqinfo;
  const float* part_o;
  const float2* part_ml;
  uint16_t* out;
  int32_t num_seqs, num_q_heads, num_kv_heads, group, head_dim;
};

struct ValidateParams {
  const int32_t* block_table;
  const int32_t* seq_lens;
  const int32_t* version_ids;
  const int16_t* page_owner;
  int32_t num_seqs, page_size, stride;
  int64_t num_pages;
  int32_t* err;
};

hipError_t launch_plan(const PlanParams& p, hipStream_t s);
hipError_t launch_split_decode(const DecodeParams& p, int head_dim, int page_size, bool fp8,
                               int64_t grid, hipStream_t s);
hipError_t launch_combine(const CombineParams& p, hipStream_t s);
hipError_t launch_validate(const ValidateParams& p, hipStream_t s);
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
