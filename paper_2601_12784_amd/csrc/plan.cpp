// Host-side length-aware split-K planner (pure integer work, no device calls).
//
// Rollout batches mix a few very long trajectories with many short ones
// (Sec. 2.3 of the paper); the paper balances that skew across rollout
// instances by routing and migration (Sec. 5.2). Inside one GPU the same job
// falls to this planner: it cuts every (sequence, KV head) range of pages into
// balanced page-aligned chunks no longer than a target derived from the
// batch's total KV pages and the number of compute units, so that long
// sequences are read by many workgroups at once. The exact rule is stated in
// sf_decode_attn.h next to sf_decode_attn_plan.
#include <algorithm>
#include <cstring>
#include <vector>

#include "sf_internal.h"

namespace sf {

uint64_t align256(uint64_t x) { return (x + 255u) & ~uint64_t(255u); }

sf_status validate_desc(const sf_attn_desc* d) {
  if (!d) return SF_ERR_INVALID_ARG;
  if (d->num_seqs < 0 || d->num_q_heads < 1 || d->num_kv_heads < 1) return SF_ERR_INVALID_ARG;
  if (d->num_q_heads % d->num_kv_heads != 0) return SF_ERR_INVALID_ARG;
  if (d->block_table_stride < 1 || d->num_pages < 0) return SF_ERR_INVALID_ARG;
  if (!(d->softmax_scale == d->softmax_scale) ||
      d->softmax_scale > 3.0e38f || d->softmax_scale < -3.0e38f) return SF_ERR_INVALID_ARG;
  if (d->head_dim != 64 && d->head_dim != 128) return SF_ERR_UNSUPPORTED;
  if (d->page_size != kPage) return SF_ERR_UNSUPPORTED;
  if (d->num_q_heads / d->num_kv_heads > kMaxGroup) return SF_ERR_UNSUPPORTED;
  return SF_OK;
}

uint64_t desc_key(const sf_attn_desc* d) {
  // FNV-1a over the shape fields a plan depends on.
  const int32_t f[8] = {0x5f440001, d->num_seqs, d->num_q_heads, d->num_kv_heads,
                        d->head_dim, d->page_size, d->block_table_stride, d->num_pages};
  uint64_t h = 1469598103934665603ull;
  const unsigned char* p = reinterpret_cast<const unsigned char*>(f);
  for (size_t i = 0; i < sizeof f; ++i) {
    h ^= p[i];
    h *= 1099511628211ull;
  }
  return h;
}

Workspace carve_workspace(void* base, int32_t slots, int32_t g, int32_t d) {
  Workspace w;
  char* b = static_cast<char*>(base);
  w.part_o = reinterpret_cast<float*>(b);
  w.part_lse = reinterpret_cast<float*>(b + align256(uint64_t(slots) * g * d * 4));
  return w;
}

}  // namespace sf

using namespace sf;

extern "C" sf_status sf_decode_attn_plan(const sf_attn_desc* desc, const int32_t* seq_lens_host,
                                         const sf_plan_opts* opts, int32_t* work_host,
                                         uint64_t work_capacity_bytes, sf_plan_info* info) {
  sf_status st = validate_desc(desc);
  if (st != SF_OK) return st;
  if (!info || (desc->num_seqs > 0 && !seq_lens_host)) return SF_ERR_INVALID_ARG;

  const int32_t B = desc->num_seqs;
  const int32_t hkv = desc->num_kv_heads;
  int32_t num_cus = kDefaultNumCus, forced = 0, upc = kDefaultUnitsPerCu;
  int32_t mn = kDefaultMinChunk, mx = kDefaultMaxChunk;
  if (opts) {
    if (opts->num_cus < 0 || opts->chunk_pages < 0 || opts->units_per_cu < 0 ||
        opts->min_chunk_pages < 0 || opts->max_chunk_pages < 0) return SF_ERR_INVALID_ARG;
    if (opts->num_cus) num_cus = opts->num_cus;
    forced = opts->chunk_pages;
    if (opts->units_per_cu) upc = opts->units_per_cu;
    if (opts->min_chunk_pages) mn = opts->min_chunk_pages;
    if (opts->max_chunk_pages) mx = opts->max_chunk_pages;
  }
  if (mn > mx) return SF_ERR_INVALID_ARG;

  int64_t total = 0, max_pages = 0;
  for (int32_t s = 0; s < B; ++s) {
    const int32_t L = seq_lens_host[s];
    if (L < 0 || (L > 0 && desc->num_pages == 0)) return SF_ERR_INVALID_ARG;
    const int64_t npg = (int64_t(L) + kPage - 1) / kPage;
    if (npg > desc->block_table_stride) return SF_ERR_INVALID_ARG;
    total += npg * hkv;
    max_pages = std::max(max_pages, npg);
  }
  int64_t chunk;
  if (forced > 0) {
    chunk = forced;
  } else {
    const int64_t units = int64_t(upc) * num_cus;
    chunk = (total + units - 1) / units;
    chunk = std::min<int64_t>(std::max<int64_t>(chunk, mn), mx);
  }
  auto pages_of = [&](int32_t s) { return (int64_t(seq_lens_host[s]) + kPage - 1) / kPage; };
  auto chunks_of = [&](int64_t npg) { return npg ? (npg + chunk - 1) / chunk : int64_t(1); };

  // Sizes first: items, combine rows, partial slots.
  int64_t n_work = 0, n_comb = 0, n_part = 0;
  for (int32_t s = 0; s < B; ++s) {
    const int64_t n = chunks_of(pages_of(s));
    n_work += n * hkv;
    if (n > 1) {
      n_comb += hkv;
      n_part += n * hkv;
    }
  }
  if (n_work + n_comb > INT32_MAX / kItemInts || n_part > INT32_MAX) return SF_ERR_INVALID_ARG;
  const int32_t g = desc->num_q_heads / hkv;
  info->num_work = int32_t(n_work);
  info->num_combine = int32_t(n_comb);
  info->num_partials = int32_t(n_part);
  info->chunk_pages = int32_t(std::min<int64_t>(chunk, INT32_MAX));
  info->work_bytes = uint64_t(n_work + n_comb) * kItemInts * 4;
  info->workspace_bytes =
      n_part ? align256(uint64_t(n_part) * g * desc->head_dim * 4) + align256(uint64_t(n_part) * g * 4) : 0;
  info->desc_key = desc_key(desc);
  if (!work_host) return SF_OK;
  if (work_capacity_bytes < info->work_bytes) return SF_ERR_CAPACITY;

  // Items are generated in (s, kvh, c) order and placed by a stable counting
  // sort on page count, largest first. Chunk c of a pair spans
  // floor((c+1)*npg/n) - floor(c*npg/n) <= chunk pages.
  const int64_t max_size = std::min<int64_t>(chunk, max_pages);
  // Scratch reused across calls on this thread; raw pointers keep the loops
  // free of per-access thread-local lookups.
  thread_local std::vector<int64_t> pos_buf;
  thread_local std::vector<int32_t> bounds_buf;
  pos_buf.assign(size_t(max_size) + 2, 0);
  int64_t* pos = pos_buf.data();
  // Chunk sizes of a pair are q = floor(npg/n) or q + 1; the bounds
  // floor(c*npg/n) follow by stepping a remainder (one division per sequence).
  int32_t* bounds = nullptr;
  auto fill_bounds = [&](int64_t npg, int64_t n) {
    if (bounds_buf.size() < size_t(n) + 1) bounds_buf.resize(size_t(n) + 1);
    bounds = bounds_buf.data();
    const int64_t q = npg / n, r = npg % n;
    int64_t e = 0, rem = 0;
    bounds[0] = 0;
    for (int64_t c = 1; c <= n; ++c) {
      e += q;
      rem += r;
      if (rem >= n) {
        rem -= n;
        ++e;
      }
      bounds[c] = int32_t(e);
    }
  };
  for (int32_t s = 0; s < B; ++s) {
    const int64_t npg = pages_of(s);
    const int64_t n = chunks_of(npg);
    if (n == 1) {
      pos[npg] += hkv;
      continue;
    }
    const int64_t q = npg / n, r = npg % n;  // r chunks of q + 1 pages, n - r of q
    pos[q + 1] += r * hkv;
    pos[q] += (n - r) * hkv;
  }
  int64_t start = 0;  // descending sizes: the largest size starts at row 0
  for (int64_t sz = max_size; sz >= 0; --sz) {
    const int64_t cnt = pos[sz];
    pos[sz] = start;
    start += cnt;
  }
  int32_t* comb = work_host + n_work * kItemInts;
  int32_t slot = 0, comb_idx = 0;
  for (int32_t s = 0; s < B; ++s) {
    const int64_t npg = pages_of(s);
    const int64_t n = chunks_of(npg);
    const int32_t L = seq_lens_host[s];
    fill_bounds(npg, n);
    for (int32_t kvh = 0; kvh < hkv; ++kvh) {
      for (int64_t c = 0; c < n; ++c) {
        const int32_t b = bounds[c];
        const int32_t e = bounds[c + 1];
        int32_t* row = work_host + pos[e - b]++ * kItemInts;
        row[0] = s;
        row[1] = kvh;
        row[2] = b;
        row[3] = e;
        row[4] = L;
        row[5] = n > 1 ? slot + int32_t(c) : -1;
        row[6] = n > 1 ? comb_idx : -1;
        row[7] = int32_t(n);
      }
      if (n > 1) {
        const int32_t c8[kItemInts] = {s, kvh, slot, int32_t(n), 0, 0, 0, 0};
        std::memcpy(comb, c8, sizeof c8);
        comb += kItemInts;
        slot += int32_t(n);
        ++comb_idx;
      }
    }
  }
  return SF_OK;
}
