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
