// Host-side page allocator for the paged KV cache.
//
// The cache of every running trajectory lives in fixed-size pages drawn from
// a pool of bounded size (the KV-cache budget the paper's snapshot tracks,
// Sec. 5.2): a sequence takes one more page each time its length crosses a
// multiple of 16 tokens and returns all of them when it leaves. The free list
// is a stack, so the page released last is the first handed out again (its
// tiles are the most likely to still sit in a cache); a new pool hands pages
// out in increasing id order. Every call checks all of its arguments before
// it changes anything.
#include <cstdint>
#include <new>
#include <vector>

#include "sf_internal.h"

struct sf_page_pool {
  int32_t num_pages;
  std::vector<int32_t> stack;   // free pages; the top is the back
  std::vector<uint8_t> in_use;  // per page
  std::vector<uint8_t> mark;    // scratch for duplicate checks, all zero between calls
};

namespace {

// True if pages[0..n) are distinct, in range and each has in_use == want.
bool check_pages(sf_page_pool* p, const int32_t* pages, int32_t n, uint8_t want) {
  bool ok = true;
  int32_t i = 0;
  for (; i < n; ++i) {
    const int32_t pg = pages[i];
    if (pg < 0 || pg >= p->num_pages || p->in_use[size_t(pg)] != want || p->mark[size_t(pg)]) {
      ok = false;
      break;
    }
    p->mark[size_t(pg)] = 1;
  }
  for (int32_t j = 0; j < i; ++j) p->mark[size_t(pages[j])] = 0;
  return ok;
}

}  // namespace

extern "C" sf_status sf_page_pool_create(int32_t num_pages, sf_page_pool** pool) {
  if (!pool || num_pages < 0) return SF_ERR_INVALID_ARG;
  *pool = nullptr;
  sf_page_pool* p = new (std::nothrow) sf_page_pool;
  if (!p) return SF_ERR_CAPACITY;
  try {
    p->num_pages = num_pages;
    p->stack.resize(size_t(num_pages));
    for (int32_t i = 0; i < num_pages; ++i) p->stack[size_t(i)] = num_pages - 1 - i;
    p->in_use.assign(size_t(num_pages), 0);
    p->mark.assign(size_t(num_pages), 0);
  } catch (...) {
    delete p;
    return SF_ERR_CAPACITY;
  }
  *pool = p;
  return SF_OK;
}

extern "C" void sf_page_pool_destroy(sf_page_pool* pool) { delete pool; }

extern "C" int32_t sf_page_pool_available(const sf_page_pool* pool) {
  return pool ? int32_t(pool->stack.size()) : -1;
}

extern "C" sf_status sf_page_pool_claim(sf_page_pool* pool, const int32_t* pages, int32_t n) {
  if (!pool || n < 0 || (n > 0 && !pages)) return SF_ERR_INVALID_ARG;
  if (!check_pages(pool, pages, n, 0)) return SF_ERR_INVALID_ARG;
  for (int32_t i = 0; i < n; ++i) pool->in_use[size_t(pages[i])] = 1;
  size_t w = 0;  // keep the order of the pages still free
  for (size_t r = 0; r < pool->stack.size(); ++r)
    if (!pool->in_use[size_t(pool->stack[r])]) pool->stack[w++] = pool->stack[r];
  pool->stack.resize(w);
  return SF_OK;
}

extern "C" sf_status sf_page_pool_alloc(sf_page_pool* pool, int32_t n, int32_t* pages) {
  if (!pool || n < 0 || (n > 0 && !pages)) return SF_ERR_INVALID_ARG;
  if (size_t(n) > pool->stack.size()) return SF_ERR_CAPACITY;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t pg = pool->stack.back();
    pool->stack.pop_back();
    pool->in_use[size_t(pg)] = 1;
    pages[i] = pg;
  }
  return SF_OK;
}

extern "C" sf_status sf_page_pool_release(sf_page_pool* pool, const int32_t* pages, int32_t n) {
  if (!pool || n < 0 || (n > 0 && !pages)) return SF_ERR_INVALID_ARG;
  if (!check_pages(pool, pages, n, 1)) return SF_ERR_INVALID_ARG;
  for (int32_t i = 0; i < n; ++i) {
    pool->in_use[size_t(pages[i])] = 0;
    pool->stack.push_back(pages[i]);
  }
  return SF_OK;
}

using sf::kPage;

extern "C" sf_status sf_page_table_step(sf_page_pool* pool, int32_t* block_table, int32_t stride,
                                        int32_t num_seqs, const int32_t* prev_lens, const int32_t* lens,
                                        int32_t appending, int32_t* new_pages) {
  if (!pool || !block_table || stride < 1 || num_seqs < 0) return SF_ERR_INVALID_ARG;
  if (num_seqs > 0 && (!prev_lens || !lens || !new_pages)) return SF_ERR_INVALID_ARG;
  const int64_t max_len = int64_t(stride) * kPage;
  thread_local std::vector<int32_t> gone;
  gone.clear();
  int64_t opens = 0;
  for (int32_t s = 0; s < num_seqs; ++s) {
    const int32_t prev = prev_lens[s], len = lens[s];
    if (prev < 0 || len < 0 || prev > max_len || len > max_len) return SF_ERR_INVALID_ARG;
    if (prev > 0 && len == 0) {
      const int32_t* row = block_table + int64_t(s) * stride;
      for (int32_t j = 0; j < (prev + kPage - 1) / kPage; ++j) gone.push_back(row[j]);
    }
    if (appending && len > 0 && (len - 1) % kPage == 0) ++opens;
  }
  if (!check_pages(pool, gone.data(), int32_t(gone.size()), 1)) return SF_ERR_INVALID_ARG;
  if (opens > int64_t(pool->stack.size() + gone.size())) return SF_ERR_CAPACITY;
  for (int32_t pg : gone) {
    pool->in_use[size_t(pg)] = 0;
    pool->stack.push_back(pg);
  }
  for (int32_t s = 0; s < num_seqs; ++s) {
    const int32_t len = lens[s];
    int32_t page = -1;
    if (appending && len > 0 && (len - 1) % kPage == 0) {
      page = pool->stack.back();
      pool->stack.pop_back();
      pool->in_use[size_t(page)] = 1;
      block_table[int64_t(s) * stride + (len - 1) / kPage] = page;
    }
    new_pages[s] = page;
  }
  return SF_OK;
}

extern "C" sf_status sf_check_block_table(const sf_attn_desc* desc, const int32_t* block_table_host,
                                          const int32_t* seq_lens_host, int32_t* bad_seq) {
  if (bad_seq) *bad_seq = -1;
  if (sf::validate_desc(desc) != SF_OK) return SF_ERR_INVALID_ARG;
  if (desc->num_seqs > 0 && (!block_table_host || !seq_lens_host)) return SF_ERR_INVALID_ARG;
  for (int32_t s = 0; s < desc->num_seqs; ++s) {
    const int64_t len = seq_lens_host[s];
    if (len <= 0) continue;
    const int64_t pages = (len + sf::kPage - 1) / sf::kPage;
    bool ok = pages <= desc->block_table_stride;
    const int32_t* row = block_table_host + int64_t(s) * desc->block_table_stride;
    for (int64_t j = 0; ok && j < pages; ++j) ok = row[j] >= 0 && row[j] < desc->num_pages;
    if (!ok) {
      if (bad_seq) *bad_seq = s;
      return SF_ERR_INVALID_ARG;
    }
  }
  return SF_OK;
}
