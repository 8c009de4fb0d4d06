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
  const int32_t f[7] = {0x5f440001, d->num_seqs, d->num_q_heads, d->num_kv_heads,
                        d->head_dim, d->page_size, d->block_table_stride};
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

  std::vector<int64_t> pages(B);
  int64_t total = 0;
  for (int32_t s = 0; s < B; ++s) {
    const int32_t L = seq_lens_host[s];
    if (L < 0) return SF_ERR_INVALID_ARG;
    pages[s] = (int64_t(L) + kPage - 1) / kPage;
    if (pages[s] > desc->block_table_stride) return SF_ERR_INVALID_ARG;
    total += pages[s] * hkv;
  }
  int64_t chunk;
  if (forced > 0) {
    chunk = forced;
  } else {
    const int64_t units = int64_t(upc) * num_cus;
    chunk = (total + units - 1) / units;
    chunk = std::min<int64_t>(std::max<int64_t>(chunk, mn), mx);
  }

  // Sizes first: items, combine rows, partial slots.
  int64_t n_work = 0, n_comb = 0, n_part = 0;
  for (int32_t s = 0; s < B; ++s) {
    const int64_t n = pages[s] ? (pages[s] + chunk - 1) / chunk : 1;
    n_work += n * hkv;
    if (n > 1) {
      n_comb += hkv;
      n_part += n * hkv;
    }
  }
  if (n_work > INT32_MAX / kItemInts || n_part > INT32_MAX) return SF_ERR_INVALID_ARG;
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

  // Rows in (s, kvh, c) order, then a stable sort by page count (descending)
  // keeps that order among equal sizes.
  struct Row {
    int32_t size;
    int32_t f[kItemInts];
  };
  std::vector<Row> rows;
  rows.reserve(size_t(n_work));
  int32_t* comb = work_host + n_work * kItemInts;
  int32_t slot = 0;
  for (int32_t s = 0; s < B; ++s) {
    const int64_t npg = pages[s];
    const int32_t L = seq_lens_host[s];
    for (int32_t kvh = 0; kvh < hkv; ++kvh) {
      if (npg == 0) {
        rows.push_back(Row{0, {s, kvh, 0, 0, L, -1, 0, 1}});
        continue;
      }
      const int64_t n = (npg + chunk - 1) / chunk;
      for (int64_t c = 0; c < n; ++c) {
        const int32_t b = int32_t(c * npg / n);
        const int32_t e = int32_t((c + 1) * npg / n);
        rows.push_back(Row{e - b, {s, kvh, b, e, L, n > 1 ? slot + int32_t(c) : -1, int32_t(c), int32_t(n)}});
      }
      if (n > 1) {
        const int32_t c8[kItemInts] = {s, kvh, slot, int32_t(n), 0, 0, 0, 0};
        std::memcpy(comb, c8, sizeof c8);
        comb += kItemInts;
        slot += int32_t(n);
      }
    }
  }
  std::stable_sort(rows.begin(), rows.end(), [](const Row& a, const Row& b) { return a.size > b.size; });
  for (size_t i = 0; i < rows.size(); ++i) std::memcpy(work_host + i * kItemInts, rows[i].f, sizeof rows[i].f);
  return SF_OK;
}
