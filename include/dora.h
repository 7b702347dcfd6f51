/*
 * dora.h — C ABI of the MI355X (gfx950) decode-attention hot path of DORA's
 * rollout stage ("DORA: A Scalable Asynchronous Reinforcement Learning System
 * for Language Model Training", arXiv 2604.26256).
 *
 * What the paper fixes and this library implements:
 *   - Rollout decode is memory-bound and dominates the RL step (Sec. 1;
 *     Sec. 2.2, Eq. (1) and the TPOT term tau in it).  Each decode step attends
 *     every active sequence's cached keys and values; response lengths are
 *     heavily long-tailed (Sec. 2.2, "Workload skewness").
 *   - Sequences of several policy versions coexist in one rollout instance;
 *     every request carries the version tag it was dispatched under (Sec. 3.2,
 *     "Multi-version policy management").  Here: one shared page pool, one
 *     block-table row per sequence, and version_ids[b] per sequence.
 *   - KV states of a trajectory are identical on every instance that hosts its
 *     version, so migration moves the KV pages instead of re-running prefill
 *     (Sec. 3.4, "KV-Cache Reuse", two-phase state transfer).  Here: the page
 *     gather/scatter dora_kv_page_pack / dora_kv_page_unpack, bit-exact.
 *
 * Conventions shared by every entry point:
 *   - Every pointer named "device" is a HIP device pointer owned by the caller.
 *     The library never allocates, frees or retains device memory.
 *   - Every device-side entry point enqueues work on `stream` and returns
 *     without synchronising (graph-capturable), except where a flag says so.
 *   - All host-checkable errors (null pointers, unsupported shapes, a too-small
 *     workspace or packed buffer, version mismatch) are reported BEFORE any
 *     launch and leave every buffer untouched.  Nothing throws or aborts across
 *     this ABI.  Device-data errors (a page id outside the pool, a page not
 *     owned by the sequence's version, seq_lens[b] > block_table_stride *
 *     page_size) are undefined behaviour unless DORA_FLAG_VALIDATE is set.
 *   - No global mutable state, with one exception: the fixed per-GPU
 *     workspace of dora_decode_attn_noalloc (calls of that entry point that
 *     overlap on one GPU race on it).  Pool objects are single-threaded.
 *
 * Data layouts (row-major, innermost index last; e = 2 bytes for bf16, 1 for
 * fp8; X = 16 / e, i.e. one 16-byte chunk of the head dimension):
 *   q, out       [num_seqs][num_q_heads][head_dim]                       bf16
 *   k_pages      [num_pages][num_kv_heads][head_dim / X][page_size][X]   bf16 | fp8
 *                (each token's key is cut into 16-byte chunks; chunk c of all
 *                 page_size tokens is stored contiguously)
 *   v_pages      [num_pages][num_kv_heads][head_dim][page_size]          bf16 | fp8
 *                (values stored transposed: the page_size tokens of one
 *                 head-dim index are contiguous)
 *   k_scales, v_scales  [num_pages] fp32 (fp8 only): stored value times the
 *                page's scale is the key/value (one scale per page, shared by
 *                all heads and tokens of that page)
 *   block_table  [num_seqs][block_table_stride] int32 page ids, logical order
 *   seq_lens     [num_seqs] int32, tokens to attend (>= 0)
 *   version_ids  [num_seqs] int32 policy version of each sequence
 * fp8 is OCP E4M3FN (bias 7, max 448, S.1111.111 = NaN, no infinity).
 * GQA mapping: query head h reads KV head h / (num_q_heads / num_kv_heads).
 * Slots of the last page beyond seq_lens[b] are never used in the arithmetic
 * (they may hold any bytes, NaN included).
 *
 * The operation (dora_decode_attn), for every sequence b and query head h,
 * with G = num_q_heads / num_kv_heads, g = h / G, L = seq_lens[b]:
 *   K_t, V_t = key/value of token t < L, read from page block_table[b][t / P]
 *              at slot t % P, KV head g (times the page scale for fp8)
 *   s_t      = sm_scale * <q[b][h], K_t>
 *   out[b][h] = sum_t exp(s_t - max s) V_t / sum_t exp(s_t - max s)
 *   L = 0 gives out[b][h] = 0.
 */
#ifndef DORA_H
#define DORA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Opaque stream handle: a hipStream_t (NULL = the legacy default stream). */
typedef void* dora_stream_t;

typedef enum {
  DORA_OK = 0,
  DORA_ERR_INVALID_ARG = 1,          /* null pointer, bad count or bad geometry */
  DORA_ERR_UNSUPPORTED = 2,          /* head_dim / page_size / group size / dtype not built */
  DORA_ERR_WORKSPACE_TOO_SMALL = 3,  /* workspace or packed buffer smaller than required */
  DORA_ERR_VERSION_MISMATCH = 4,     /* pages of one policy version sent to another */
  DORA_ERR_POOL_EXHAUSTED = 5,       /* pool has too few free pages (state unchanged) */
  DORA_ERR_DEVICE_CHECK = 6,         /* DORA_FLAG_VALIDATE found bad device data */
  DORA_ERR_HIP = 7,                  /* a HIP runtime call failed */
  DORA_ERR_NOT_FOUND = 8             /* unknown sequence id in a pool call */
} dora_status;

typedef enum {
  DORA_KV_BF16 = 0,
  DORA_KV_FP8_E4M3 = 1
} dora_kv_dtype;

/* Flags for dora_decode_desc.flags. */
#define DORA_FLAG_VALIDATE    0x1u  /* range- and ownership-check every page id read;
                                       synchronises the stream and returns
                                       DORA_ERR_DEVICE_CHECK on bad device data */

/* Geometry and options of one decode-attention call.  Supported builds:
 * head_dim in {64, 128}; page_size in {16, 32}; group size num_q_heads /
 * num_kv_heads in [1, 16]; kv_dtype bf16 or fp8 e4m3. */
typedef struct {
  int32_t num_seqs;            /* B >= 0 */
  int32_t num_q_heads;         /* Hq, multiple of num_kv_heads */
  int32_t num_kv_heads;        /* Hkv >= 1 */
  int32_t head_dim;            /* d */
  int32_t page_size;           /* P tokens per page */
  int32_t block_table_stride;  /* int32 entries per block-table row (>= 1) */
  int64_t num_pages;           /* pool capacity in pages (for VALIDATE range checks) */
  int32_t kv_dtype;            /* dora_kv_dtype */
  float   sm_scale;            /* softmax scale; 0 means 1/sqrt(head_dim) */
  const float* k_scales;       /* device [num_pages] fp32, fp8 only (else NULL) */
  const float* v_scales;       /* device [num_pages] fp32, fp8 only (else NULL) */
  const int16_t* page_owner;   /* device [num_pages] owning version, or NULL; read
                                  only under DORA_FLAG_VALIDATE */
  uint32_t flags;              /* DORA_FLAG_* */
  int32_t num_waves;           /* decode wavefronts to launch; 0 = library
                                  default: per compute unit of the current
                                  device at most 4 for bf16 pages and 7 for
                                  fp8 pages, within the resident wavefront
                                  slots; never more than the batch can use
                                  (B x Hkv x stride page-heads over the minimum
                                  range) */
  int32_t min_range_pages;     /* smallest work range per wavefront, in
                                  (page, KV head) units; 0 = library default */
} dora_decode_desc;

/* Human-readable name of a status code (static storage); "unknown status" for
 * a value that is no dora_status.  The code is passed as an int, so any value
 * is a valid argument. */
const char* dora_status_string(int status);

/* Bytes of device workspace dora_decode_attn needs for this geometry on the
 * current device (valid for every seq_lens the call may see).  Returns 0 for an
 * invalid or unsupported descriptor.  The workspace holds a 256-byte flag
 * header, one cut record per decode wavefront (or per (sequence, KV head)
 * segment, when there are no more segments than wavefronts) and two partial
 * results per wavefront (unnormalised output, running max and sum in fp32);
 * the batch's page prefix is built in each wavefront's LDS. */
size_t dora_decode_workspace_bytes(const dora_decode_desc* desc);

/* Decode wavefronts dora_decode_attn launches per launch for this descriptor on
 * the current device: desc->num_waves when it is set, else the library default
 * described at dora_decode_desc.num_waves.  Wavefront w takes page-heads
 * [w*T/W', (w+1)*T/W') of the launch's T (sequence, KV head, page) work items
 * in (sequence, head, page) order, where W' = min(W, ceil(T / m)), m being
 * desc->min_range_pages or 8 when that is 0, and the first T mod W' ranges hold
 * one extra item; so a caller can tell which (sequence, KV head) segments a
 * call cuts across wavefronts.  Each launch covers at most 8192 sequences.
 * Returns 0 for an invalid or unsupported descriptor. */
int64_t dora_decode_num_waves(const dora_decode_desc* desc);

/* Decode-step attention over the paged, multi-version KV pool (the operation
 * defined at the top of this file; the step the paper times as tau per output
 * token, Sec. 2.2 Eq. (1); version tags per Sec. 3.2).
 *   q            device bf16 [B][Hq][d]
 *   k_pages      device, layout above
 *   v_pages      device, layout above
 *   block_table  device int32 [B][block_table_stride]
 *   seq_lens     device int32 [B]
 *   version_ids  device int32 [B]; does not enter the arithmetic.  Under
 *                DORA_FLAG_VALIDATE every page b reads must satisfy
 *                page_owner[page] == version_ids[b].  May be NULL without it.
 *   out          device bf16 [B][Hq][d], written for every (b, h)
 *   workspace    device, >= dora_decode_workspace_bytes(desc) bytes, 16-byte
 *                aligned; contents on entry are ignored
 * Launches the decode kernel and a log-sum-exp combine kernel on `stream` (per
 * 8192 sequences).  Every decode wavefront takes an equal share of the batch's
 * (page, KV head) work, whatever the length mix.  Results do not depend on the
 * number of wavefronts beyond fp32 rounding, and repeated calls on the same
 * inputs and device are bitwise identical. */
dora_status dora_decode_attn(const dora_decode_desc* desc,
                             const void* q, const void* k_pages, const void* v_pages,
                             const int32_t* block_table, const int32_t* seq_lens,
                             const int32_t* version_ids, void* out,
                             void* workspace, size_t workspace_bytes,
                             dora_stream_t stream);

/* Size of the fixed device array dora_decode_attn_noalloc uses as its
 * workspace, one per GPU. */
#define DORA_NOALLOC_WORKSPACE_BYTES ((size_t)48 << 20)

/* dora_decode_attn for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * Same arguments, results and errors as dora_decode_attn, without the
 * workspace: the call uses a fixed array of DORA_NOALLOC_WORKSPACE_BYTES in
 * device memory that the library holds on each GPU it runs on, from load until
 * the process ends.  It allocates and frees nothing; its first call on a device
 * looks the array's address up.
 *   DORA_ERR_WORKSPACE_TOO_SMALL  dora_decode_workspace_bytes(desc) exceeds the
 *                                 array (e.g. a large desc->num_waves)
 *   DORA_ERR_INVALID_ARG          DORA_FLAG_VALIDATE set (it synchronises and
 *                                 copies to the host); plus dora_decode_attn's
 * Every call on one GPU uses that GPU's array, and the array keeps the last
 * call's contents (the decode ignores them): calls that overlap on one GPU (on
 * different streams or from different threads) race, and the caller must
 * order them. */
dora_status dora_decode_attn_noalloc(const dora_decode_desc* desc,
                                     const void* q, const void* k_pages, const void* v_pages,
                                     const int32_t* block_table, const int32_t* seq_lens,
                                     const int32_t* version_ids, void* out,
                                     dora_stream_t stream);

/* Decode attention for a batch made of response groups that share a prompt
 * (the responses sampled per prompt for GRPO-style advantages, App. B).  The
 * result equals dora_decode_attn's on the same arguments (up to fp32 rounding);
 * what changes is that each group's shared prompt pages are read from HBM once
 * instead of once per member.
 *   group_size    M >= 1; sequences [k*M, (k+1)*M) form group k; num_seqs must
 *                 be a multiple of M; M * (num_q_heads / num_kv_heads) <= 128
 *                 (else DORA_ERR_UNSUPPORTED)
 *   shared_pages_out  device int32 [num_seqs / M] or NULL: receives each
 *                 group's shared prefix S_k (below)
 *   other arguments as for dora_decode_attn; the workspace must hold
 *   dora_decode_grouped_workspace_bytes(desc, group_size) bytes.
 * Sharing is read off the block tables on the device: S_k is the number of
 * leading pages that every member of group k holds in full (j < seq_len /
 * page_size) under the same page id as the group's first member; a group of
 * one shares nothing.  Any batch is valid input (S_k = 0 where nothing is
 * shared).  Steps, all enqueued on `stream`, no host round trip: a prefix
 * kernel (per group, KV head and chunk of shared pages: finds S_k, stages the
 * pages in LDS once and applies them to every member's query heads); the
 * ordinary decode over each member's remaining pages; its combine, which
 * merges cut segments and folds every row with its group's prefix into out. */
size_t dora_decode_grouped_workspace_bytes(const dora_decode_desc* desc, int32_t group_size);
dora_status dora_decode_attn_grouped(const dora_decode_desc* desc, const void* q,
                                     const void* k_pages, const void* v_pages,
                                     const int32_t* block_table, const int32_t* seq_lens,
                                     const int32_t* version_ids, void* out, int32_t group_size,
                                     int32_t* shared_pages_out, void* workspace,
                                     size_t workspace_bytes, dora_stream_t stream);

/* Store every sequence's current-token K and V into its page slot: the write
 * that precedes each decode step (the per-token step of Sec. 2.2; seq_lens
 * counts that token, so dora_decode_attn with the same seq_lens then attends
 * over it).  Token t = seq_lens[b] - 1 of sequence b goes to page
 * block_table[b][t / P], token slot t % P; seq_lens[b] = 0 appends nothing.
 *   desc         the decode descriptor (num_seqs, num_kv_heads, head_dim,
 *                page_size, block_table_stride, num_pages, kv_dtype; flags may
 *                hold DORA_FLAG_VALIDATE; num_q_heads must be valid for it)
 *   k_new, v_new device bf16 [B][Hkv][d], 16-byte aligned
 *   block_table, seq_lens, version_ids  as for dora_decode_attn
 *   k_pages, v_pages  device, the layouts above, written in place
 *   k_scales, v_scales  device fp32 [num_pages], fp8 only (else ignored),
 *                updated in place
 *   dev_status   device int32 or NULL: receives DORA_OK, or
 *                DORA_ERR_DEVICE_CHECK if some sequence was skipped because its
 *                page id is out of range, its length exceeds its block-table
 *                row, or (under DORA_FLAG_VALIDATE with desc->page_owner) its
 *                page belongs to another version.  Skipped sequences write
 *                nothing; no write ever leaves the pool.
 * bf16 pages take the values as given.  fp8 pages: the paper fixes no
 * quantisation policy; this library keeps one fp32 scale per page for K and one
 * for V, grow-only, computed in fp32 with IEEE rounding:
 *   amax = max |x| over the token's Hkv x d values
 *   fresh = max(amax / 448, 2^-126)   (a normal fp32 number)
 *   slot 0:                           s = fresh
 *   slot > 0, not fresh <= s0:        s = fresh, and every earlier code c of
 *                                     the page (all heads) becomes
 *                                     enc((dec(c) * s0) / s)
 *   otherwise:                        s = s0       (s0: the page's scale)
 *   codes of the token: enc(x / s); the page's scale becomes s.
 * enc is the nearest OCP E4M3FN code, ties to even, saturating at +-448.
 * The pages of one call must belong to distinct sequences (a page is never
 * appended to by two sequences at once).  Enqueued on `stream`; one launch
 * (two with dev_status). */
dora_status dora_kv_append(const dora_decode_desc* desc, const void* k_new, const void* v_new,
                           const int32_t* block_table, const int32_t* seq_lens,
                           const int32_t* version_ids, void* k_pages, void* v_pages,
                           float* k_scales, float* v_scales, int32_t* dev_status,
                           dora_stream_t stream);

/* ---------------------------------------------------------------------------
 * KV page pack / unpack: the device half of the paper's two-phase state
 * transfer for same-version migration (Sec. 3.4: request metadata travels by
 * RPC, the KV data by collectives; KV states are equal on every instance of
 * the version, so no re-prefill).
 *
 * Packed buffer format (all integers little-endian):
 *   bytes [0, 256)   header:
 *       0  char[8]  magic "DORAKV01"
 *       8  int32    format (= 1)
 *      12  int32    policy_version
 *      16  int32    kv_dtype
 *      20  int32    page_size
 *      24  int32    num_kv_heads
 *      28  int32    head_dim
 *      32  int64    n_pages
 *      40  int64    page_bytes   (= num_kv_heads * page_size * head_dim * e)
 *      48  int32    n_seqs       (caller's count of sequences in the list)
 *      52  int32    reserved (0); bytes 56..255 are 0
 *   then n_pages K pages (page_bytes each) in list order,
 *   then n_pages V pages in list order,
 *   then, for fp8 only, n_pages fp32 k scales and n_pages fp32 v scales.
 * Pages are copied whole, tail slots included; the copy is bit-exact.
 * ------------------------------------------------------------------------- */

typedef struct {
  int32_t kv_dtype;        /* dora_kv_dtype */
  int32_t page_size;
  int32_t num_kv_heads;
  int32_t head_dim;
  int64_t num_pages;       /* capacity of the pool the page ids index */
  int32_t policy_version;  /* version tag of the pages (pack: source, unpack: destination) */
  int32_t n_seqs;          /* recorded in the header by pack; informational */
} dora_pack_desc;

/* Size in bytes of a packed buffer holding n_pages pages (0 if invalid). */
size_t dora_kv_packed_bytes(const dora_pack_desc* desc, int64_t n_pages);

/* Gather pages src_pages[0..n_pages) (device int32, logical order) of a pool
 * into `packed` (>= dora_kv_packed_bytes bytes, 16-byte aligned) and write the
 * header.  k_scales/v_scales: device [num_pages], fp8 only.
 * `packed` may be device memory, or pinned host memory from hipHostMalloc
 * (mapped: the kernel writes it over the host link).  The latter is the
 * offload half of the paper's hierarchical memory management (Sec. 3.4: KV
 * caches moved to host memory under VRAM pressure and restored for deferred
 * generation); no device staging buffer is needed. */
dora_status dora_kv_page_pack(const dora_pack_desc* desc,
                              const void* k_pages, const void* v_pages,
                              const float* k_scales, const float* v_scales,
                              const int32_t* src_pages, int64_t n_pages,
                              void* packed, size_t packed_bytes,
                              dora_stream_t stream);

/* Scatter a packed buffer into pages dst_pages[0..n_pages) (device int32) of
 * the destination pool described by `desc`.  src_version is the version tag the
 * request metadata carries; it must equal desc->policy_version, else
 * DORA_ERR_VERSION_MISMATCH before any launch (KV states are only equivalent
 * within one policy version).  On the device the header is checked against
 * desc and n_pages; on any mismatch nothing is written to the pool and, if
 * dev_status (device int32, may be NULL) is given, it receives a non-zero
 * dora_status code; it receives DORA_OK otherwise.  `packed` may be device
 * memory or pinned host memory from hipHostMalloc (restore from host: the
 * kernel reads it over the host link). */
dora_status dora_kv_page_unpack(const dora_pack_desc* desc, int32_t src_version,
                                const void* packed, size_t packed_bytes,
                                const int32_t* dst_pages, int64_t n_pages,
                                void* k_pages, void* v_pages,
                                float* k_scales, float* v_scales,
                                int32_t* dev_status, dora_stream_t stream);

/* ---------------------------------------------------------------------------
 * Orchestrator planners (host, integer arithmetic; Sec. 3.3).  Versions are
 * indexed oldest first; the last index is the latest version.
 * ------------------------------------------------------------------------- */

/* Resource partitioning plan: DP groups per version in proportion to its
 * workload (active plus pending requests).  A version with work keeps at least
 * one group; the other groups go by the largest-remainder method on the
 * quotas (n_groups - busy versions) * workload / total, equal remainders to the
 * newer version; with no work, every group goes to the latest version.
 *   workload    host int64 [n_versions], >= 0
 *   groups_out  host int32 [n_versions], sums to n_groups
 * DORA_ERR_INVALID_ARG for null pointers, negative workload, n_groups < 1, or
 * more versions with work than groups. */
dora_status dora_plan_partition(const int64_t* workload, int32_t n_versions, int32_t n_groups,
                                int32_t* groups_out);

/* Staleness-aware data supplementation: prompts to inject per version.  The
 * latest version gets min(latest_quota, its idle slots), latest_quota being
 * what its rollout batch still needs; every legacy version gets exactly its
 * residual idle slots (groups * slots_per_group - active, at least 0).
 *   groups, active  host int32 [n_versions], >= 0
 *   inject_out      host int32 [n_versions] */
dora_status dora_plan_supplement(const int32_t* groups, const int32_t* active,
                                 int32_t n_versions, int32_t slots_per_group,
                                 int64_t latest_quota, int32_t* inject_out);

/* ---------------------------------------------------------------------------
 * Host page pool: page allocator plus per-version sequence tables for one
 * shared pool (Sec. 3.2: every request carries its version tag; Sec. 3.3: the
 * orchestrator reads per-version KV-cache utilisation; Sec. 3.4: migration
 * only between instances of the same version, locality first).  Metadata only:
 * the pool never touches device memory.  Not thread-safe.
 * ------------------------------------------------------------------------- */

typedef struct dora_pool dora_pool;

/* num_pages >= 1, page_size >= 1, num_versions >= 1.  seed != 0 shuffles the
 * free list with a seeded generator so that pages are scattered in the pool;
 * seed == 0 hands pages out in increasing order. */
dora_status dora_pool_create(int64_t num_pages, int32_t page_size,
                             int32_t num_versions, uint64_t seed, dora_pool** out);
void        dora_pool_destroy(dora_pool* pool);

/* Register a sequence of `version` holding num_tokens tokens and allocate its
 * ceil(num_tokens / page_size) pages.  DORA_ERR_POOL_EXHAUSTED leaves the pool
 * unchanged. */
dora_status dora_pool_add_seq(dora_pool* pool, int32_t version, int32_t num_tokens,
                              int64_t* seq_id_out);
/* Grow a sequence to new_num_tokens (>= current), allocating pages as needed. */
dora_status dora_pool_extend_seq(dora_pool* pool, int64_t seq_id, int32_t new_num_tokens);
/* Release a sequence and all of its pages. */
dora_status dora_pool_free_seq(dora_pool* pool, int64_t seq_id);
/* Tokens, version and page count of a sequence (any out pointer may be NULL). */
dora_status dora_pool_seq_info(const dora_pool* pool, int64_t seq_id, int32_t* num_tokens,
                               int32_t* version, int32_t* num_pages);
/* Copy a sequence's page ids in logical order into pages_out[cap]. */
dora_status dora_pool_seq_pages(const dora_pool* pool, int64_t seq_id,
                                int32_t* pages_out, int32_t cap, int32_t* n_out);
/* Fill host arrays for a decode batch: table_out[n][stride] (unused entries
 * set to 0), lens_out[n], versions_out[n].  INVALID_ARG if a sequence needs
 * more than `stride` pages. */
dora_status dora_pool_block_table(const dora_pool* pool, const int64_t* seq_ids, int32_t n,
                                  int32_t stride, int32_t* table_out, int32_t* lens_out,
                                  int32_t* versions_out);
/* owner_out[num_pages]: owning version of each page, -1 if free. */
dora_status dora_pool_page_owner(const dora_pool* pool, int16_t* owner_out);
/* Pages held by `version` (version = -1: all versions) and pages free. */
dora_status dora_pool_stats(const dora_pool* pool, int32_t version, int64_t* pages_used,
                            int64_t* pages_free);
/* Migrate a sequence from `src` to `dst` (same-version instances): allocates
 * pages in dst for dst_version and registers the sequence there; writes the
 * source page list and the destination page list (logical order, n_out
 * entries each) for pack/unpack, and the new id.  dst_version must equal the
 * sequence's version (DORA_ERR_VERSION_MISMATCH otherwise).  If src == dst the
 * sequence stays where it is (locality: no pages move, n_out = 0 and
 * dst_seq_id = seq_id).  The source sequence is kept until the caller frees it
 * after the copy. */
dora_status dora_pool_migrate_seq(dora_pool* src, int64_t seq_id, dora_pool* dst,
                                  int32_t dst_version, int64_t* dst_seq_id,
                                  int32_t* src_pages, int32_t* dst_pages, int32_t cap,
                                  int32_t* n_out);

#ifdef __cplusplus
}
#endif

#endif /* DORA_H */
