/* A C99 client of the library's C ABI: compiled with a C compiler against the
 * public headers and linked with libdora.so, it drives the host-side entry
 * points (status strings, descriptor checks and sizing, the page pool and the
 * planners) with no GPU.  Prints "ok" and exits 0 when every check passes,
 * else prints the failed check and exits 1. */
#include <stdio.h>
#include <string.h>

#include "dora.h"
#include "dora_measure.h"

#define CHECK(c)                                      \
  do {                                                \
    if (!(c)) {                                       \
      printf("failed: %s (line %d)\n", #c, __LINE__); \
      return 1;                                       \
    }                                                 \
  } while (0)

int main(void) {
  dora_decode_desc d;
  dora_pool* pool = NULL;
  int64_t a = -1, b = -1, used = -1, free_pages = -1;
  int32_t table[2 * 4], lens[2], vers[2];
  int64_t ids[2];
  int64_t workload[3] = {5, 0, 3};
  int32_t groups[3];

  CHECK(strcmp(dora_status_string(DORA_OK), "ok") == 0);
  CHECK(strcmp(dora_status_string(12345), "unknown status") == 0);

  memset(&d, 0, sizeof d);
  d.num_seqs = 3;
  d.num_q_heads = 28;
  d.num_kv_heads = 4;
  d.head_dim = 128;
  d.page_size = 16;
  d.num_pages = 1024;
  d.block_table_stride = 64;
  d.kv_dtype = DORA_KV_BF16;
  CHECK(dora_decode_workspace_bytes(&d) > 0);
  CHECK(dora_decode_num_waves(&d) >= 1);
  d.head_dim = 96; /* not built */
  CHECK(dora_decode_workspace_bytes(&d) == 0);
  CHECK(dora_decode_attn(&d, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0, NULL) !=
        DORA_OK);

  CHECK(dora_pool_create(16, 16, 2, 7, &pool) == DORA_OK && pool != NULL);
  CHECK(dora_pool_add_seq(pool, 0, 40, &a) == DORA_OK); /* 3 pages */
  CHECK(dora_pool_add_seq(pool, 1, 16, &b) == DORA_OK); /* 1 page */
  CHECK(dora_pool_stats(pool, -1, &used, &free_pages) == DORA_OK);
  CHECK(used == 4 && free_pages == 12);
  ids[0] = a;
  ids[1] = b;
  CHECK(dora_pool_block_table(pool, ids, 2, 4, table, lens, vers) == DORA_OK);
  CHECK(lens[0] == 40 && lens[1] == 16 && vers[0] == 0 && vers[1] == 1);
  CHECK(table[3] == 0 && table[5] == 0); /* unused entries are 0 */
  CHECK(dora_pool_add_seq(pool, 0, 16 * 13, &a) == DORA_ERR_POOL_EXHAUSTED);
  CHECK(dora_pool_free_seq(pool, b) == DORA_OK);
  CHECK(dora_pool_stats(pool, 1, &used, &free_pages) == DORA_OK && used == 0);
  dora_pool_destroy(pool);

  /* two busy versions keep a group each; the rest goes by workload */
  CHECK(dora_plan_partition(workload, 3, 8, groups) == DORA_OK);
  CHECK(groups[0] == 5 && groups[1] == 0 && groups[2] == 3);
  printf("ok\n");
  return 0;
}
