// Host-side page allocator of a paged KV pool: per-session (per-tag) page
// lists over one shared set of pages (Algorithm 1's per-tag isolated KV state,
// with the session's cache created, grown each step, cut back to the accepted
// prefix and released).  Host memory only; the pages themselves are device
// buffers the caller owns.
#include <stdint.h>

#include <new>
#include <unordered_map>
#include <vector>

#include "sdverify.h"

struct sd_kv_pool {
  int32_t num_pages;
  int32_t page_size;
  std::vector<int32_t> free_list;  // back() is handed out next
  std::unordered_map<int32_t, std::vector<int32_t>> tags;
};

namespace {

bool pow2_page(int32_t p) { return p >= 64 && p <= 4096 && (p & (p - 1)) == 0; }

int64_t pages_for(const sd_kv_pool* pool, int32_t length) {
  return (static_cast<int64_t>(length) + pool->page_size - 1) / pool->page_size;
}

}  // namespace

extern "C" {

sd_kv_pool_t* sd_kv_pool_create(int32_t num_pages, int32_t page_size) {
  if (num_pages < 1 || !pow2_page(page_size)) return nullptr;
  sd_kv_pool* pool = new (std::nothrow) sd_kv_pool;
  if (pool == nullptr) return nullptr;
  pool->num_pages = num_pages;
  pool->page_size = page_size;
  pool->free_list.reserve(num_pages);
  for (int32_t i = num_pages - 1; i >= 0; --i) pool->free_list.push_back(i);
  return pool;
}

void sd_kv_pool_destroy(sd_kv_pool_t* pool) { delete pool; }

int sd_kv_pool_reserve(sd_kv_pool_t* pool, int32_t tag, int32_t length) {
  if (pool == nullptr || tag < 0 || length < 0) return SD_ERR_INVALID_ARGUMENT;
  std::vector<int32_t>& pages = pool->tags[tag];
  const int64_t need = pages_for(pool, length) - static_cast<int64_t>(pages.size());
  if (need <= 0) return SD_OK;
  if (need > static_cast<int64_t>(pool->free_list.size())) {
    if (pages.empty()) pool->tags.erase(tag);
    return SD_ERR_CAPACITY;
  }
  for (int64_t i = 0; i < need; ++i) {
    pages.push_back(pool->free_list.back());
    pool->free_list.pop_back();
  }
  return SD_OK;
}

int sd_kv_pool_truncate(sd_kv_pool_t* pool, int32_t tag, int32_t length) {
  if (pool == nullptr || tag < 0 || length < 0) return SD_ERR_INVALID_ARGUMENT;
  auto it = pool->tags.find(tag);
  if (it == pool->tags.end()) return SD_OK;
  std::vector<int32_t>& pages = it->second;
  const int64_t keep = pages_for(pool, length);
  while (static_cast<int64_t>(pages.size()) > keep) {
    pool->free_list.push_back(pages.back());
    pages.pop_back();
  }
  return SD_OK;
}

int sd_kv_pool_release(sd_kv_pool_t* pool, int32_t tag) {
  if (pool == nullptr || tag < 0) return SD_ERR_INVALID_ARGUMENT;
  auto it = pool->tags.find(tag);
  if (it == pool->tags.end()) return SD_OK;
  for (auto p = it->second.rbegin(); p != it->second.rend(); ++p) pool->free_list.push_back(*p);
  pool->tags.erase(it);
  return SD_OK;
}

int32_t sd_kv_pool_free_pages(const sd_kv_pool_t* pool) {
  return pool == nullptr ? 0 : static_cast<int32_t>(pool->free_list.size());
}

int32_t sd_kv_pool_tag_pages(const sd_kv_pool_t* pool, int32_t tag) {
  if (pool == nullptr) return 0;
  auto it = pool->tags.find(tag);
  return it == pool->tags.end() ? 0 : static_cast<int32_t>(it->second.size());
}

int sd_kv_pool_block_table(const sd_kv_pool_t* pool, const int32_t* tags, int32_t n, int32_t max_pages,
                           int32_t* table) {
  if (pool == nullptr || n < 0 || max_pages < 1 || (n > 0 && (tags == nullptr || table == nullptr)))
    return SD_ERR_INVALID_ARGUMENT;
  for (int32_t i = 0; i < n; ++i) {
    if (tags[i] < 0) return SD_ERR_INVALID_ARGUMENT;
    if (sd_kv_pool_tag_pages(pool, tags[i]) > max_pages) return SD_ERR_INVALID_ARGUMENT;
  }
  for (int32_t i = 0; i < n; ++i) {
    int32_t* row = table + static_cast<int64_t>(i) * max_pages;
    auto it = pool->tags.find(tags[i]);
    int32_t j = 0;
    if (it != pool->tags.end())
      for (int32_t p : it->second) row[j++] = p;
    for (; j < max_pages; ++j) row[j] = -1;
  }
  return SD_OK;
}

}  // extern "C"
