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
 * check and returns 1. */
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
