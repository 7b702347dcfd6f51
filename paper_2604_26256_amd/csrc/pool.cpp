// Host page pool: page allocator, page -> owning-version map and per-sequence
// page lists for one KV pool shared by several policy versions (Sec. 3.2:
// every request carries its version tag; Sec. 3.3: per-version KV-cache
// utilisation drives re-balancing; Sec. 3.4: same-version migration with
// locality first).  Metadata only; device memory is the caller's.
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <unordered_map>
#include <vector>

#include "dora.h"

struct dora_pool {
  int64_t num_pages = 0;
  int32_t page_size = 0;
  int32_t num_versions = 0;
  std::vector<int32_t> free_list;  // stack; back() is handed out next
  std::vector<int16_t> owner;      // -1 = free
  std::vector<int64_t> used_by_version;
  struct Seq {
    int32_t version;
    int32_t num_tokens;
    std::vector<int32_t> pages;
  };
  std::unordered_map<int64_t, Seq> seqs;
  int64_t next_id = 1;
};

namespace {

// splitmix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
// generators", OOPSLA 2014): the free-list shuffle's generator.
uint64_t splitmix64(uint64_t& x) {
  uint64_t z = (x += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

int64_t pages_for(const dora_pool* p, int64_t tokens) {
  return (tokens + p->page_size - 1) / p->page_size;
}

// Take n pages for `version`; all or nothing.
bool take_pages(dora_pool* p, int32_t version, int64_t n, std::vector<int32_t>* dst) {
  if (n > (int64_t)p->free_list.size()) return false;
  for (int64_t i = 0; i < n; ++i) {
    int32_t pg = p->free_list.back();
    p->free_list.pop_back();
    p->owner[pg] = (int16_t)version;
    dst->push_back(pg);
  }
  p->used_by_version[version] += n;
  return true;
}

}  // namespace

extern "C" {

dora_status dora_pool_create(int64_t num_pages, int32_t page_size, int32_t num_versions,
                             uint64_t seed, dora_pool** out) {
  if (!out || num_pages < 1 || num_pages > INT32_MAX || page_size < 1 || num_versions < 1 ||
      num_versions > INT16_MAX)
    return DORA_ERR_INVALID_ARG;
  dora_pool* p = new (std::nothrow) dora_pool;
  if (!p) return DORA_ERR_POOL_EXHAUSTED;
  p->num_pages = num_pages;
  p->page_size = page_size;
  p->num_versions = num_versions;
  p->owner.assign((size_t)num_pages, (int16_t)-1);
  p->used_by_version.assign((size_t)num_versions, 0);
  p->free_list.resize((size_t)num_pages);
  // back() is handed out first: store in decreasing order so that an unshuffled
  // pool gives pages 0, 1, 2, ...
  for (int64_t i = 0; i < num_pages; ++i) p->free_list[(size_t)i] = (int32_t)(num_pages - 1 - i);
  if (seed != 0) {  // Fisher-Yates
    uint64_t st = seed;
    for (int64_t i = num_pages - 1; i > 0; --i) {
      int64_t j = (int64_t)(splitmix64(st) % (uint64_t)(i + 1));
      std::swap(p->free_list[(size_t)i], p->free_list[(size_t)j]);
    }
  }
  *out = p;
  return DORA_OK;
}

void dora_pool_destroy(dora_pool* pool) { delete pool; }

dora_status dora_pool_add_seq(dora_pool* pool, int32_t version, int32_t num_tokens,
                              int64_t* seq_id_out) {
  if (!pool || !seq_id_out || num_tokens < 0 || version < 0 || version >= pool->num_versions)
    return DORA_ERR_INVALID_ARG;
  dora_pool::Seq s;
  s.version = version;
  s.num_tokens = num_tokens;
  if (!take_pages(pool, version, pages_for(pool, num_tokens), &s.pages))
    return DORA_ERR_POOL_EXHAUSTED;
  const int64_t id = pool->next_id++;
  pool->seqs.emplace(id, std::move(s));
  *seq_id_out = id;
  return DORA_OK;
}

dora_status dora_pool_extend_seq(dora_pool* pool, int64_t seq_id, int32_t new_num_tokens) {
  if (!pool) return DORA_ERR_INVALID_ARG;
  auto it = pool->seqs.find(seq_id);
  if (it == pool->seqs.end()) return DORA_ERR_NOT_FOUND;
  dora_pool::Seq& s = it->second;
  if (new_num_tokens < s.num_tokens) return DORA_ERR_INVALID_ARG;
  const int64_t need = pages_for(pool, new_num_tokens) - (int64_t)s.pages.size();
  if (need > 0 && !take_pages(pool, s.version, need, &s.pages)) return DORA_ERR_POOL_EXHAUSTED;
  s.num_tokens = new_num_tokens;
  return DORA_OK;
}

dora_status dora_pool_free_seq(dora_pool* pool, int64_t seq_id) {
  if (!pool) return DORA_ERR_INVALID_ARG;
  auto it = pool->seqs.find(seq_id);
  if (it == pool->seqs.end()) return DORA_ERR_NOT_FOUND;
  dora_pool::Seq& s = it->second;
  // Return pages so that the most recently freed page is reused first.
  for (auto r = s.pages.rbegin(); r != s.pages.rend(); ++r) {
    pool->owner[*r] = -1;
    pool->free_list.push_back(*r);
  }
  pool->used_by_version[s.version] -= (int64_t)s.pages.size();
  pool->seqs.erase(it);
  return DORA_OK;
}

dora_status dora_pool_seq_info(const dora_pool* pool, int64_t seq_id, int32_t* num_tokens,
                               int32_t* version, int32_t* num_pages) {
  if (!pool) return DORA_ERR_INVALID_ARG;
  auto it = pool->seqs.find(seq_id);
  if (it == pool->seqs.end()) return DORA_ERR_NOT_FOUND;
  if (num_tokens) *num_tokens = it->second.num_tokens;
  if (version) *version = it->second.version;
  if (num_pages) *num_pages = (int32_t)it->second.pages.size();
  return DORA_OK;
}

dora_status dora_pool_seq_pages(const dora_pool* pool, int64_t seq_id, int32_t* pages_out,
                                int32_t cap, int32_t* n_out) {
  if (!pool || !n_out || cap < 0 || (cap > 0 && !pages_out)) return DORA_ERR_INVALID_ARG;
  auto it = pool->seqs.find(seq_id);
  if (it == pool->seqs.end()) return DORA_ERR_NOT_FOUND;
  const auto& pg = it->second.pages;
  if ((int64_t)pg.size() > cap) return DORA_ERR_WORKSPACE_TOO_SMALL;
  std::copy(pg.begin(), pg.end(), pages_out);
  *n_out = (int32_t)pg.size();
  return DORA_OK;
}

dora_status dora_pool_block_table(const dora_pool* pool, const int64_t* seq_ids, int32_t n,
                                  int32_t stride, int32_t* table_out, int32_t* lens_out,
                                  int32_t* versions_out) {
  if (!pool || n < 0 || stride < 1 || (n > 0 && (!seq_ids || !table_out || !lens_out)))
    return DORA_ERR_INVALID_ARG;
  for (int32_t i = 0; i < n; ++i) {  // check everything before writing anything
    auto it = pool->seqs.find(seq_ids[i]);
    if (it == pool->seqs.end()) return DORA_ERR_NOT_FOUND;
    if ((int64_t)it->second.pages.size() > stride) return DORA_ERR_INVALID_ARG;
  }
  for (int32_t i = 0; i < n; ++i) {
    const auto& s = pool->seqs.find(seq_ids[i])->second;
    int32_t* row = table_out + (int64_t)i * stride;
    std::fill(row, row + stride, 0);
    std::copy(s.pages.begin(), s.pages.end(), row);
    lens_out[i] = s.num_tokens;
    if (versions_out) versions_out[i] = s.version;
  }
  return DORA_OK;
}

dora_status dora_pool_page_owner(const dora_pool* pool, int16_t* owner_out) {
  if (!pool || !owner_out) return DORA_ERR_INVALID_ARG;
  memcpy(owner_out, pool->owner.data(), pool->owner.size() * sizeof(int16_t));
  return DORA_OK;
}

dora_status dora_pool_stats(const dora_pool* pool, int32_t version, int64_t* pages_used,
                            int64_t* pages_free) {
  if (!pool || version < -1 || version >= pool->num_versions) return DORA_ERR_INVALID_ARG;
  if (pages_used) {
    if (version < 0)
      *pages_used = pool->num_pages - (int64_t)pool->free_list.size();
    else
      *pages_used = pool->used_by_version[version];
  }
  if (pages_free) *pages_free = (int64_t)pool->free_list.size();
  return DORA_OK;
}

dora_status dora_pool_migrate_seq(dora_pool* src, int64_t seq_id, dora_pool* dst,
                                  int32_t dst_version, int64_t* dst_seq_id, int32_t* src_pages,
                                  int32_t* dst_pages, int32_t cap, int32_t* n_out) {
  if (!src || !dst || !dst_seq_id || !n_out || cap < 0) return DORA_ERR_INVALID_ARG;
  auto it = src->seqs.find(seq_id);
  if (it == src->seqs.end()) return DORA_ERR_NOT_FOUND;
  const dora_pool::Seq& s = it->second;
  if (dst_version != s.version) return DORA_ERR_VERSION_MISMATCH;
  if (dst_version < 0 || dst_version >= dst->num_versions) return DORA_ERR_INVALID_ARG;
  if (src == dst) {  // locality: the request stays on its instance, nothing moves
    *dst_seq_id = seq_id;
    *n_out = 0;
    return DORA_OK;
  }
  if (dst->page_size != src->page_size) return DORA_ERR_INVALID_ARG;
  const int64_t n = (int64_t)s.pages.size();
  if (n > cap || (n > 0 && (!src_pages || !dst_pages))) return DORA_ERR_WORKSPACE_TOO_SMALL;
  dora_pool::Seq t;
  t.version = s.version;
  t.num_tokens = s.num_tokens;
  if (!take_pages(dst, dst_version, n, &t.pages)) return DORA_ERR_POOL_EXHAUSTED;
  std::copy(s.pages.begin(), s.pages.end(), src_pages);
  std::copy(t.pages.begin(), t.pages.end(), dst_pages);
  const int64_t id = dst->next_id++;
  dst->seqs.emplace(id, std::move(t));
  *dst_seq_id = id;
  *n_out = (int32_t)n;
  return DORA_OK;
}

}  // extern "C"
