/* A C client of the library on the GPU: raw hipMalloc'd buffers and the HIP
 * runtime's C API, no torch.  Built as a small shared library whose one entry
 * point the GPU test calls in its own process.  It builds a small ragged bf16
 * batch in the header's page layouts (pages scattered over the pool, tail
 * slots of last pages NaN), runs dora_decode_attn, first under
 * DORA_FLAG_VALIDATE and then plain, and compares every output with the fp64
 * oracle (liboracle: test infrastructure) within 2e-2, empty sequences
 * exactly zero.  Then it packs the pages of two sequences, unpacks them into
 * other page ids of a second, zeroed pool, and compares those pages with the
 * source pages byte for byte (and the pages it must not touch with zero).
 * Prints "ok" and returns 0 when every check passes, else prints the failed
 * check and returns 1.
 *
 * dora_c_gpu_step_loop drives a few rollout steps of an fp8 batch the way a C
 * serving loop would: the host pool places the sequences of two versions,
 * each step grows every sequence by one token (dora_pool_extend_seq), rebuilds
 * the block tables and page owners from the pool, appends the new token's K
 * and V under DORA_FLAG_VALIDATE (pools and page scales compared byte for byte
 * with the oracle's append on host copies) and decodes (oracle, 5e-2; the
 * no-allocation entry point bitwise equal to the plain one).  Then it migrates
 * one sequence to a second pool (same version; another version is refused,
 * a same-pool move is a no-op) with pack and unpack, compares the moved pages
 * and scales with the source, and checks that the moved sequence decodes
 * bitwise as it did in the first pool. */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "dora.h"

/* The oracle's entry point (oracle/dora_oracle.c). */
int oracle_decode(int B, int Hq, int Hkv, int d, int P, int64_t num_pages, int stride,
                  int kv_dtype, double scale, const uint16_t* q, const void* k_pages,
                  const void* v_pages, const float* k_scales, const float* v_scales,
                  const int32_t* block_table, const int32_t* seq_lens,
                  const int32_t* version_ids, const int16_t* page_owner, double* out,
                  int nthreads);
int oracle_kv_append(int B, int Hkv, int d, int P, int64_t num_pages, int stride, int kv_dtype,
                     const int32_t* block_table, const int32_t* seq_lens,
                     const uint16_t* k_new, const uint16_t* v_new, uint8_t* k_pages,
                     uint8_t* v_pages, float* k_scales, float* v_scales);
uint8_t oracle_f32_to_e4m3(float x);

#define CHECK(c)                                      \
  do {                                                \
    if (!(c)) {                                       \
      printf("failed: %s (line %d)\n", #c, __LINE__); \
      fflush(stdout);                                 \
      return 1;                                       \
    }                                                 \
  } while (0)
#define HIP(c) CHECK((c) == hipSuccess)

enum { B = 6, HQ = 14, HKV = 2, D = 128, P = 16, NPAGES = 512, STRIDE = 160, X = 8 };
static const int32_t kLens[B] = {0, 1, 17, 300, 1000, 2049};

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) { /* xorshift64* (Vigna) */
  rng_state ^= rng_state >> 12;
  rng_state ^= rng_state << 25;
  rng_state ^= rng_state >> 27;
  return (uint32_t)((rng_state * 0x2545F4914F6CDD1Dull) >> 32);
}
/* roughly N(0, 1): sum of four uniforms, centred and scaled */
static float next_normal(void) {
  float s = 0.f;
  for (int i = 0; i < 4; ++i) s += (float)next_u32() / 4294967296.0f;
  return (s - 2.0f) * 1.7320508f;
}
static uint16_t to_bf16(float f) { /* round to nearest even */
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
static double bf16_to_double(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

int dora_c_gpu_client(void) {
  const size_t page_elems = (size_t)HKV * P * D; /* per pool page, K or V */
  const size_t pool_elems = (size_t)NPAGES * page_elems;
  uint16_t* k = malloc(pool_elems * 2);
  uint16_t* v = malloc(pool_elems * 2);
  uint16_t* q = malloc((size_t)B * HQ * D * 2);
  uint16_t* out = malloc((size_t)B * HQ * D * 2);
  double* ref = malloc((size_t)B * HQ * D * sizeof(double));
  int32_t* table = calloc((size_t)B * STRIDE, 4);
  int32_t perm[NPAGES], versions[B];
  CHECK(k && v && q && out && ref && table);

  /* pool contents, query, and a scattered page placement */
  for (size_t i = 0; i < pool_elems; ++i) k[i] = to_bf16(next_normal());
  for (size_t i = 0; i < pool_elems; ++i) v[i] = to_bf16(next_normal());
  for (int i = 0; i < B * HQ * D; ++i) q[i] = to_bf16(next_normal());
  for (int i = 0; i < NPAGES; ++i) perm[i] = i;
  for (int i = NPAGES - 1; i > 0; --i) {
    const int j = (int)(next_u32() % (uint32_t)(i + 1));
    const int t = perm[i];
    perm[i] = perm[j];
    perm[j] = t;
  }
  int used = 0;
  for (int b = 0; b < B; ++b) {
    versions[b] = 0;
    const int n = (kLens[b] + P - 1) / P;
    CHECK(n <= STRIDE && used + n <= NPAGES);
    for (int j = 0; j < n; ++j) table[b * STRIDE + j] = perm[used++];
    /* slots past the length in the last page: NaN, never to be read */
    for (int t = kLens[b]; n > 0 && t < n * P; ++t) {
      const size_t page = (size_t)table[b * STRIDE + n - 1];
      for (int g = 0; g < HKV; ++g)
        for (int i = 0; i < D; ++i) {
          /* K [page][g][i / X][slot][i % X], V [page][g][i][slot] */
          k[page * page_elems + ((size_t)g * (D / X) + i / X) * P * X + (t % P) * X + i % X] = 0x7FC0;
          v[page * page_elems + ((size_t)g * D + i) * P + t % P] = 0x7FC0;
        }
    }
  }
  CHECK(oracle_decode(B, HQ, HKV, D, P, NPAGES, STRIDE, DORA_KV_BF16, 0.0, q, k, v, NULL, NULL,
                      table, kLens, versions, NULL, ref, 0) == 0);

  int ndev = 0;
  HIP(hipGetDeviceCount(&ndev));
  CHECK(ndev > 0);
  HIP(hipSetDevice(0));
  void *dk, *dv, *dq, *dout, *dws;
  int32_t *dtable, *dlens, *dvers;
  HIP(hipMalloc(&dk, pool_elems * 2));
  HIP(hipMalloc(&dv, pool_elems * 2));
  HIP(hipMalloc(&dq, (size_t)B * HQ * D * 2));
  HIP(hipMalloc(&dout, (size_t)B * HQ * D * 2));
  HIP(hipMalloc((void**)&dtable, (size_t)B * STRIDE * 4));
  HIP(hipMalloc((void**)&dlens, B * 4));
  HIP(hipMalloc((void**)&dvers, B * 4));
  HIP(hipMemcpy(dk, k, pool_elems * 2, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dv, v, pool_elems * 2, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dq, q, (size_t)B * HQ * D * 2, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dtable, table, (size_t)B * STRIDE * 4, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dlens, kLens, B * 4, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dvers, versions, B * 4, hipMemcpyHostToDevice));
  HIP(hipMemset(dout, 0xFF, (size_t)B * HQ * D * 2));

  dora_decode_desc desc;
  memset(&desc, 0, sizeof desc);
  desc.num_seqs = B;
  desc.num_q_heads = HQ;
  desc.num_kv_heads = HKV;
  desc.head_dim = D;
  desc.page_size = P;
  desc.block_table_stride = STRIDE;
  desc.num_pages = NPAGES;
  desc.kv_dtype = DORA_KV_BF16;
  const size_t ws_bytes = dora_decode_workspace_bytes(&desc);
  CHECK(ws_bytes > 0);
  HIP(hipMalloc(&dws, ws_bytes));

  desc.flags = DORA_FLAG_VALIDATE;
  CHECK(dora_decode_attn(&desc, dq, dk, dv, dtable, dlens, dvers, dout, dws, ws_bytes, NULL) ==
        DORA_OK);
  desc.flags = 0;
  HIP(hipMemset(dout, 0xFF, (size_t)B * HQ * D * 2));
  CHECK(dora_decode_attn(&desc, dq, dk, dv, dtable, dlens, dvers, dout, dws, ws_bytes, NULL) ==
        DORA_OK);
  HIP(hipDeviceSynchronize());
  HIP(hipMemcpy(out, dout, (size_t)B * HQ * D * 2, hipMemcpyDeviceToHost));
  double err = 0.0;
  for (int i = 0; i < B * HQ * D; ++i) {
    const double o = bf16_to_double(out[i]);
    CHECK(isfinite(o));
    const double e = fabs(o - ref[i]);
    err = e > err ? e : err;
  }
  for (int i = 0; i < HQ * D; ++i) CHECK(out[i] == 0); /* sequence 0 is empty */
  printf("decode max-abs error vs oracle %.3e\n", err);
  CHECK(err <= 2e-2);

  /* pack sequences 4 and 5, unpack into a second pool at other page ids */
  const int n4 = (kLens[4] + P - 1) / P, n5 = (kLens[5] + P - 1) / P, n = n4 + n5;
  int32_t* src = malloc((size_t)n * 4);
  int32_t* dst = malloc((size_t)n * 4);
  CHECK(src && dst);
  for (int j = 0; j < n4; ++j) src[j] = table[4 * STRIDE + j];
  for (int j = 0; j < n5; ++j) src[n4 + j] = table[5 * STRIDE + j];
  for (int j = 0; j < n; ++j) dst[j] = perm[NPAGES - 1 - j]; /* distinct ids */
  dora_pack_desc pd;
  memset(&pd, 0, sizeof pd);
  pd.kv_dtype = DORA_KV_BF16;
  pd.page_size = P;
  pd.num_kv_heads = HKV;
  pd.head_dim = D;
  pd.num_pages = NPAGES;
  pd.policy_version = 0;
  pd.n_seqs = 2;
  const size_t packed_bytes = dora_kv_packed_bytes(&pd, n);
  CHECK(packed_bytes > 0);
  void *dpacked, *dk2, *dv2;
  int32_t *dsrc, *ddst, *dstatus;
  HIP(hipMalloc(&dpacked, packed_bytes));
  HIP(hipMalloc(&dk2, pool_elems * 2));
  HIP(hipMalloc(&dv2, pool_elems * 2));
  HIP(hipMalloc((void**)&dsrc, (size_t)n * 4));
  HIP(hipMalloc((void**)&ddst, (size_t)n * 4));
  HIP(hipMalloc((void**)&dstatus, 4));
  HIP(hipMemset(dk2, 0, pool_elems * 2));
  HIP(hipMemset(dv2, 0, pool_elems * 2));
  HIP(hipMemset(dstatus, 0xFF, 4));
  HIP(hipMemcpy(dsrc, src, (size_t)n * 4, hipMemcpyHostToDevice));
  HIP(hipMemcpy(ddst, dst, (size_t)n * 4, hipMemcpyHostToDevice));
  CHECK(dora_kv_page_pack(&pd, dk, dv, NULL, NULL, dsrc, n, dpacked, packed_bytes, NULL) ==
        DORA_OK);
  CHECK(dora_kv_page_unpack(&pd, 0, dpacked, packed_bytes, ddst, n, dk2, dv2, NULL, NULL, dstatus,
                            NULL) == DORA_OK);
  CHECK(dora_kv_page_unpack(&pd, 1, dpacked, packed_bytes, ddst, n, dk2, dv2, NULL, NULL, dstatus,
                            NULL) == DORA_ERR_VERSION_MISMATCH);
  HIP(hipDeviceSynchronize());
  int32_t status = -1;
  HIP(hipMemcpy(&status, dstatus, 4, hipMemcpyDeviceToHost));
  CHECK(status == DORA_OK);
  uint16_t* k2 = malloc(pool_elems * 2);
  uint16_t* v2 = malloc(pool_elems * 2);
  char* written = calloc(NPAGES, 1);
  CHECK(k2 && v2 && written);
  HIP(hipMemcpy(k2, dk2, pool_elems * 2, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(v2, dv2, pool_elems * 2, hipMemcpyDeviceToHost));
  for (int j = 0; j < n; ++j) {
    written[dst[j]] = 1;
    CHECK(memcmp(k2 + (size_t)dst[j] * page_elems, k + (size_t)src[j] * page_elems,
                 page_elems * 2) == 0);
    CHECK(memcmp(v2 + (size_t)dst[j] * page_elems, v + (size_t)src[j] * page_elems,
                 page_elems * 2) == 0);
  }
  for (int p = 0; p < NPAGES; ++p) {
    if (written[p]) continue;
    for (size_t i = 0; i < page_elems; ++i) {
      CHECK(k2[(size_t)p * page_elems + i] == 0);
      CHECK(v2[(size_t)p * page_elems + i] == 0);
    }
  }
  printf("pack/unpack of %d pages bit-exact\n", n);

  HIP(hipFree(dk));
  HIP(hipFree(dv));
  HIP(hipFree(dq));
  HIP(hipFree(dout));
  HIP(hipFree(dws));
  HIP(hipFree(dtable));
  HIP(hipFree(dlens));
  HIP(hipFree(dvers));
  HIP(hipFree(dpacked));
  HIP(hipFree(dk2));
  HIP(hipFree(dv2));
  HIP(hipFree(dsrc));
  HIP(hipFree(ddst));
  HIP(hipFree(dstatus));
  free(k);
  free(v);
  free(q);
  free(out);
  free(ref);
  free(table);
  free(src);
  free(dst);
  free(k2);
  free(v2);
  free(written);
  printf("ok\n");
  fflush(stdout);
  return 0;
}

/* ------------------------------------------------------------------------- */

enum { SB = 5, SHQ = 16, SHKV = 2, SD = 128, SP = 32, SNPAGES = 1024, SSTRIDE = 64, STEPS = 3 };
static const int32_t kStepLens[SB] = {31, 32, 33, 700, 1500};
static const int32_t kStepVers[SB] = {0, 1, 0, 1, 0};
static const float kStepGain[STEPS] = {1.0f, 2.5f, 0.5f}; /* step 2 grows page scales */

static int32_t* dev_i32(const int32_t* h, size_t n) {
  void* d = NULL;
  if (hipMalloc(&d, n * 4) != hipSuccess) return NULL;
  if (hipMemcpy(d, h, n * 4, hipMemcpyHostToDevice) != hipSuccess) return NULL;
  return (int32_t*)d;
}

int dora_c_gpu_step_loop(void) {
  const size_t page_bytes = (size_t)SHKV * SP * SD; /* fp8: one byte per element */
  const size_t pool_bytes = (size_t)SNPAGES * page_bytes;
  const size_t qn = (size_t)SB * SHQ * SD, tn = (size_t)SB * SHKV * SD;
  uint8_t* k = malloc(pool_bytes);
  uint8_t* v = malloc(pool_bytes);
  uint8_t* kc = malloc(pool_bytes);
  uint8_t* vc = malloc(pool_bytes);
  float* ks = malloc(SNPAGES * 4);
  float* vs = malloc(SNPAGES * 4);
  float* ksc = malloc(SNPAGES * 4);
  float* vsc = malloc(SNPAGES * 4);
  uint16_t* q = malloc(qn * 2);
  uint16_t* out = malloc(qn * 2);
  uint16_t* out_na = malloc(qn * 2);
  uint16_t* knew = malloc(tn * 2);
  uint16_t* vnew = malloc(tn * 2);
  double* ref = malloc(qn * sizeof(double));
  int32_t* table = malloc((size_t)SB * SSTRIDE * 4);
  int16_t* owner = malloc(SNPAGES * 2);
  int32_t lens[SB], vers[SB];
  CHECK(k && v && kc && vc && ks && vs && ksc && vsc && q && out && out_na && knew && vnew &&
        ref && table && owner);

  /* pool contents: N(0, 1) values quantised with per-page scales */
  for (int p = 0; p < SNPAGES; ++p) {
    ks[p] = (4.0f / 448.0f) * (0.5f + (float)next_u32() / 4294967296.0f);
    vs[p] = (4.0f / 448.0f) * (0.5f + (float)next_u32() / 4294967296.0f);
    for (size_t i = 0; i < page_bytes; ++i) {
      k[(size_t)p * page_bytes + i] = oracle_f32_to_e4m3(next_normal() / ks[p]);
      v[(size_t)p * page_bytes + i] = oracle_f32_to_e4m3(next_normal() / vs[p]);
    }
  }
  for (size_t i = 0; i < qn; ++i) q[i] = to_bf16(next_normal());

  dora_pool *pa = NULL, *pb = NULL;
  CHECK(dora_pool_create(SNPAGES, SP, 2, 0x5EEDull, &pa) == DORA_OK);
  CHECK(dora_pool_create(SNPAGES, SP, 2, 0xB0B0ull, &pb) == DORA_OK);
  int64_t ids[SB];
  for (int b = 0; b < SB; ++b)
    CHECK(dora_pool_add_seq(pa, kStepVers[b], kStepLens[b], &ids[b]) == DORA_OK);

  HIP(hipSetDevice(0));
  void *dk, *dv, *dq, *dout, *dknew, *dvnew, *dws;
  float *dks, *dvs;
  int32_t *dtable, *dlens, *dvers, *dstatus;
  int16_t* downer;
  HIP(hipMalloc(&dk, pool_bytes));
  HIP(hipMalloc(&dv, pool_bytes));
  HIP(hipMalloc((void**)&dks, SNPAGES * 4));
  HIP(hipMalloc((void**)&dvs, SNPAGES * 4));
  HIP(hipMalloc(&dq, qn * 2));
  HIP(hipMalloc(&dout, qn * 2));
  HIP(hipMalloc(&dknew, tn * 2));
  HIP(hipMalloc(&dvnew, tn * 2));
  HIP(hipMalloc((void**)&dtable, (size_t)SB * SSTRIDE * 4));
  HIP(hipMalloc((void**)&dlens, SB * 4));
  HIP(hipMalloc((void**)&dvers, SB * 4));
  HIP(hipMalloc((void**)&downer, SNPAGES * 2));
  HIP(hipMalloc((void**)&dstatus, 4));
  HIP(hipMemcpy(dk, k, pool_bytes, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dv, v, pool_bytes, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dks, ks, SNPAGES * 4, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dvs, vs, SNPAGES * 4, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dq, q, qn * 2, hipMemcpyHostToDevice));

  dora_decode_desc desc;
  memset(&desc, 0, sizeof desc);
  desc.num_seqs = SB;
  desc.num_q_heads = SHQ;
  desc.num_kv_heads = SHKV;
  desc.head_dim = SD;
  desc.page_size = SP;
  desc.block_table_stride = SSTRIDE;
  desc.num_pages = SNPAGES;
  desc.kv_dtype = DORA_KV_FP8_E4M3;
  desc.k_scales = dks;
  desc.v_scales = dvs;
  desc.page_owner = downer;
  const size_t ws_bytes = dora_decode_workspace_bytes(&desc);
  CHECK(ws_bytes > 0);
  HIP(hipMalloc(&dws, ws_bytes));

  for (int step = 0; step < STEPS; ++step) {
    for (int b = 0; b < SB; ++b) {
      int32_t L = -1;
      CHECK(dora_pool_seq_info(pa, ids[b], &L, NULL, NULL) == DORA_OK);
      CHECK(dora_pool_extend_seq(pa, ids[b], L + 1) == DORA_OK);
    }
    CHECK(dora_pool_block_table(pa, ids, SB, SSTRIDE, table, lens, vers) == DORA_OK);
    CHECK(dora_pool_page_owner(pa, owner) == DORA_OK);
    for (int b = 0; b < SB; ++b) CHECK(lens[b] == kStepLens[b] + step + 1 && vers[b] == kStepVers[b]);
    for (size_t i = 0; i < tn; ++i) knew[i] = to_bf16(kStepGain[step] * next_normal());
    for (size_t i = 0; i < tn; ++i) vnew[i] = to_bf16(kStepGain[step] * next_normal());
    HIP(hipMemcpy(dtable, table, (size_t)SB * SSTRIDE * 4, hipMemcpyHostToDevice));
    HIP(hipMemcpy(dlens, lens, SB * 4, hipMemcpyHostToDevice));
    HIP(hipMemcpy(dvers, vers, SB * 4, hipMemcpyHostToDevice));
    HIP(hipMemcpy(downer, owner, SNPAGES * 2, hipMemcpyHostToDevice));
    HIP(hipMemcpy(dknew, knew, tn * 2, hipMemcpyHostToDevice));
    HIP(hipMemcpy(dvnew, vnew, tn * 2, hipMemcpyHostToDevice));
    HIP(hipMemset(dstatus, 0xFF, 4));

    /* append: device against the oracle on the host copies, whole pools */
    desc.flags = DORA_FLAG_VALIDATE;
    CHECK(dora_kv_append(&desc, dknew, dvnew, dtable, dlens, dvers, dk, dv, dks, dvs, dstatus,
                         NULL) == DORA_OK);
    CHECK(oracle_kv_append(SB, SHKV, SD, SP, SNPAGES, SSTRIDE, DORA_KV_FP8_E4M3, table, lens,
                           knew, vnew, k, v, ks, vs) == 0);
    HIP(hipDeviceSynchronize());
    int32_t status = -1;
    HIP(hipMemcpy(&status, dstatus, 4, hipMemcpyDeviceToHost));
    CHECK(status == DORA_OK);
    HIP(hipMemcpy(kc, dk, pool_bytes, hipMemcpyDeviceToHost));
    HIP(hipMemcpy(vc, dv, pool_bytes, hipMemcpyDeviceToHost));
    HIP(hipMemcpy(ksc, dks, SNPAGES * 4, hipMemcpyDeviceToHost));
    HIP(hipMemcpy(vsc, dvs, SNPAGES * 4, hipMemcpyDeviceToHost));
    CHECK(memcmp(kc, k, pool_bytes) == 0 && memcmp(vc, v, pool_bytes) == 0);
    CHECK(memcmp(ksc, ks, SNPAGES * 4) == 0 && memcmp(vsc, vs, SNPAGES * 4) == 0);

    /* decode (ownership checked), then the no-allocation entry point */
    HIP(hipMemset(dout, 0xFF, qn * 2));
    CHECK(dora_decode_attn(&desc, dq, dk, dv, dtable, dlens, dvers, dout, dws, ws_bytes, NULL) ==
          DORA_OK);
    CHECK(oracle_decode(SB, SHQ, SHKV, SD, SP, SNPAGES, SSTRIDE, DORA_KV_FP8_E4M3, 0.0, q, k, v,
                        ks, vs, table, lens, vers, owner, ref, 0) == 0);
    HIP(hipDeviceSynchronize());
    HIP(hipMemcpy(out, dout, qn * 2, hipMemcpyDeviceToHost));
    double err = 0.0;
    for (size_t i = 0; i < qn; ++i) {
      const double o = bf16_to_double(out[i]);
      CHECK(isfinite(o));
      const double e = fabs(o - ref[i]);
      err = e > err ? e : err;
    }
    printf("step %d: append bit-exact, decode max-abs error vs oracle %.3e\n", step, err);
    CHECK(err <= 5e-2);
    desc.flags = 0;
    HIP(hipMemset(dout, 0xFF, qn * 2));
    CHECK(dora_decode_attn_noalloc(&desc, dq, dk, dv, dtable, dlens, dvers, dout, NULL) ==
          DORA_OK);
    HIP(hipDeviceSynchronize());
    HIP(hipMemcpy(out_na, dout, qn * 2, hipMemcpyDeviceToHost));
    CHECK(memcmp(out_na, out, qn * 2) == 0);
  }

  /* migrate sequence 4 (version 0) to the second pool */
  int32_t src_pages[SSTRIDE], dst_pages[SSTRIDE], n = -1, n_here = -1;
  int64_t moved = -1, here = -1;
  CHECK(dora_pool_migrate_seq(pa, ids[4], pb, 1, &moved, src_pages, dst_pages, SSTRIDE, &n) ==
        DORA_ERR_VERSION_MISMATCH);
  CHECK(dora_pool_migrate_seq(pa, ids[2], pa, 0, &here, src_pages, dst_pages, SSTRIDE,
                              &n_here) == DORA_OK);
  CHECK(n_here == 0 && here == ids[2]);
  CHECK(dora_pool_migrate_seq(pa, ids[4], pb, 0, &moved, src_pages, dst_pages, SSTRIDE, &n) ==
        DORA_OK);
  CHECK(n == (lens[4] + SP - 1) / SP);
  dora_pack_desc pd;
  memset(&pd, 0, sizeof pd);
  pd.kv_dtype = DORA_KV_FP8_E4M3;
  pd.page_size = SP;
  pd.num_kv_heads = SHKV;
  pd.head_dim = SD;
  pd.num_pages = SNPAGES;
  pd.policy_version = 0;
  pd.n_seqs = 1;
  const size_t packed_bytes = dora_kv_packed_bytes(&pd, n);
  CHECK(packed_bytes > 0);
  void *dpacked, *dk2, *dv2;
  float *dks2, *dvs2;
  HIP(hipMalloc(&dpacked, packed_bytes));
  HIP(hipMalloc(&dk2, pool_bytes));
  HIP(hipMalloc(&dv2, pool_bytes));
  HIP(hipMalloc((void**)&dks2, SNPAGES * 4));
  HIP(hipMalloc((void**)&dvs2, SNPAGES * 4));
  HIP(hipMemset(dk2, 0, pool_bytes));
  HIP(hipMemset(dv2, 0, pool_bytes));
  HIP(hipMemset(dks2, 0, SNPAGES * 4));
  HIP(hipMemset(dvs2, 0, SNPAGES * 4));
  HIP(hipMemset(dstatus, 0xFF, 4));
  int32_t* dsrc = dev_i32(src_pages, (size_t)n);
  int32_t* ddst = dev_i32(dst_pages, (size_t)n);
  CHECK(dsrc && ddst);
  CHECK(dora_kv_page_pack(&pd, dk, dv, dks, dvs, dsrc, n, dpacked, packed_bytes, NULL) ==
        DORA_OK);
  CHECK(dora_kv_page_unpack(&pd, 0, dpacked, packed_bytes, ddst, n, dk2, dv2, dks2, dvs2,
                            dstatus, NULL) == DORA_OK);
  HIP(hipDeviceSynchronize());
  int32_t status = -1;
  HIP(hipMemcpy(&status, dstatus, 4, hipMemcpyDeviceToHost));
  CHECK(status == DORA_OK);
  HIP(hipMemcpy(kc, dk2, pool_bytes, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(vc, dv2, pool_bytes, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(ksc, dks2, SNPAGES * 4, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(vsc, dvs2, SNPAGES * 4, hipMemcpyDeviceToHost));
  for (int j = 0; j < n; ++j) {
    const size_t s = (size_t)src_pages[j], d = (size_t)dst_pages[j];
    CHECK(memcmp(kc + d * page_bytes, k + s * page_bytes, page_bytes) == 0);
    CHECK(memcmp(vc + d * page_bytes, v + s * page_bytes, page_bytes) == 0);
    CHECK(memcmp(&ksc[d], &ks[s], 4) == 0 && memcmp(&vsc[d], &vs[s], 4) == 0);
  }
  printf("migrated %d pages bit-exact\n", n);

  /* the moved sequence decodes bitwise as before, on either pool */
  int32_t row_a[SSTRIDE], row_b[SSTRIDE], len_a, len_b, ver_a, ver_b;
  CHECK(dora_pool_block_table(pa, &ids[4], 1, SSTRIDE, row_a, &len_a, &ver_a) == DORA_OK);
  CHECK(dora_pool_block_table(pb, &moved, 1, SSTRIDE, row_b, &len_b, &ver_b) == DORA_OK);
  CHECK(len_a == len_b && ver_a == 0 && ver_b == 0);
  int16_t* owner_b = malloc(SNPAGES * 2);
  CHECK(owner_b && dora_pool_page_owner(pb, owner_b) == DORA_OK);
  int32_t* drow_a = dev_i32(row_a, SSTRIDE);
  int32_t* drow_b = dev_i32(row_b, SSTRIDE);
  int32_t* dlen1 = dev_i32(&len_a, 1);
  int32_t* dver1 = dev_i32(&ver_a, 1);
  CHECK(drow_a && drow_b && dlen1 && dver1);
  int16_t* downer_b;
  HIP(hipMalloc((void**)&downer_b, SNPAGES * 2));
  HIP(hipMemcpy(downer_b, owner_b, SNPAGES * 2, hipMemcpyHostToDevice));
  uint16_t one_a[SHQ * SD], one_b[SHQ * SD];
  const void* dq4 = (const uint16_t*)dq + (size_t)4 * SHQ * SD;
  dora_decode_desc d1 = desc;
  d1.num_seqs = 1;
  d1.flags = DORA_FLAG_VALIDATE;
  CHECK(dora_decode_attn(&d1, dq4, dk, dv, drow_a, dlen1, dver1, dout, dws, ws_bytes, NULL) ==
        DORA_OK);
  HIP(hipMemcpy(one_a, dout, sizeof one_a, hipMemcpyDeviceToHost));
  d1.k_scales = dks2;
  d1.v_scales = dvs2;
  d1.page_owner = downer_b;
  HIP(hipMemset(dout, 0xFF, sizeof one_b));
  CHECK(dora_decode_attn(&d1, dq4, dk2, dv2, drow_b, dlen1, dver1, dout, dws, ws_bytes, NULL) ==
        DORA_OK);
  HIP(hipMemcpy(one_b, dout, sizeof one_b, hipMemcpyDeviceToHost));
  CHECK(memcmp(one_a, one_b, sizeof one_a) == 0);
  int64_t used_before = -1, used_after = -1;
  CHECK(dora_pool_stats(pa, -1, &used_before, NULL) == DORA_OK);
  CHECK(dora_pool_free_seq(pa, ids[4]) == DORA_OK);
  CHECK(dora_pool_stats(pa, -1, &used_after, NULL) == DORA_OK);
  CHECK(used_before - used_after == n);
  printf("moved sequence decodes bitwise equal on both pools\n");

  void* dev_bufs[] = {dk, dv, dks, dvs, dq, dout, dknew, dvnew, dtable, dlens, dvers, downer,
                      dstatus, dws, dpacked, dk2, dv2, dks2, dvs2, dsrc, ddst, drow_a, drow_b,
                      dlen1, dver1, downer_b};
  for (size_t i = 0; i < sizeof dev_bufs / sizeof dev_bufs[0]; ++i) HIP(hipFree(dev_bufs[i]));
  dora_pool_destroy(pa);
  dora_pool_destroy(pb);
  void* host_bufs[] = {k, v, kc, vc, ks, vs, ksc, vsc, q, out, out_na, knew, vnew, ref, table,
                       owner, owner_b};
  for (size_t i = 0; i < sizeof host_bufs / sizeof host_bufs[0]; ++i) free(host_bufs[i]);
  printf("ok\n");
  fflush(stdout);
  return 0;
}
