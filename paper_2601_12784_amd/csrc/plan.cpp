// Host-side length-aware split-K planner (pure integer work, no device calls).
//
// Rollout batches mix a few very long trajectories with many short ones
// (Sec. 2.3 of the paper); the paper balances that skew across rollout
// instances by routing and migration (Sec. 5.3). Inside one GPU the same job
// falls to this planner: it lays every (sequence, KV head) page range end to
// end and gives each resident attention wave (a worker) an equal slice of the
// pages, cut at pair boundaries into segments. Long sequences are then read
// by many waves at once and every wave finishes at about the same time,
// whatever the skew. The exact rule is stated in sf_decode_attn.h next to
// sf_decode_attn_plan.
#include <algorithm>
#include <cfloat>
#include <cmath>
#include <cstring>
#include <vector>

#include "sf_internal.h"

static_assert(sizeof(sf_attn_desc) == 32, "sf_attn_desc layout is part of the ABI");
static_assert(sizeof(sf_plan_opts) == 20, "sf_plan_opts layout is part of the ABI");
static_assert(sizeof(sf_plan_info) == 48, "sf_plan_info layout is part of the ABI");
static_assert(sizeof(sf_cost_model) == 48 && sizeof(sf_instance_state) == 24 && sizeof(sf_trajectory) == 16,
              "cost-model structs are part of the ABI");

namespace sf {

uint64_t align256(uint64_t x) { return (x + 255u) & ~uint64_t(255u); }

sf_status validate_desc(const sf_attn_desc* d) {
  if (!d) return SF_ERR_INVALID_ARG;
  if (d->num_seqs < 0 || d->num_q_heads < 1 || d->num_kv_heads < 1) return SF_ERR_INVALID_ARG;
  if (d->num_q_heads % d->num_kv_heads != 0) return SF_ERR_INVALID_ARG;
  if (d->block_table_stride < 1 || d->num_pages < 0) return SF_ERR_INVALID_ARG;
  // The kernels scale scores by |softmax_scale| * log2(e) in float, which must
  // be finite (false for NaN as well).
  if (!(std::fabs(double(d->softmax_scale)) * 1.4426950408889634074 <= double(FLT_MAX))) return SF_ERR_INVALID_ARG;
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
  int32_t num_cus = kDefaultNumCus, forced = 0, wpc = kDefaultWorkersPerCu, mn = kDefaultMinChunk;
  int32_t skew = 0;
  if (opts) {
    if (opts->num_cus < 0 || opts->chunk_pages < 0 || opts->workers_per_cu < 0 ||
        opts->min_chunk_pages < 0 || opts->xcd_parity_skew < -kMaxParitySkew ||
        opts->xcd_parity_skew > kMaxParitySkew)
      return SF_ERR_INVALID_ARG;
    if (opts->num_cus) num_cus = opts->num_cus;
    forced = opts->chunk_pages;
    if (opts->workers_per_cu) wpc = opts->workers_per_cu;
    if (opts->min_chunk_pages) mn = opts->min_chunk_pages;
    skew = opts->xcd_parity_skew;
  }

  // Pages per sequence (every KV head of a sequence has the same count).
  thread_local std::vector<int32_t> spg_buf;
  spg_buf.resize(size_t(B));
  int32_t* spg = spg_buf.data();
  int64_t total = 0;
  for (int32_t s = 0; s < B; ++s) {
    const int32_t L = seq_lens_host[s];
    if (L < 0 || (L > 0 && desc->num_pages == 0)) return SF_ERR_INVALID_ARG;
    const int64_t npg = (int64_t(L) + kPage - 1) / kPage;
    if (npg > desc->block_table_stride) return SF_ERR_INVALID_ARG;
    spg[s] = int32_t(npg);
    total += npg * hkv;
  }
  if (total > (int64_t(1) << 40)) return SF_ERR_INVALID_ARG;
  const int64_t num_pairs = int64_t(B) * hkv;
  int64_t workers;
  if (num_pairs == 0) {
    workers = 0;
  } else if (total == 0) {
    workers = 1;  // only empty pairs: one worker writes their zero rows
  } else if (forced > 0) {
    workers = (total + forced - 1) / forced;
  } else {
    workers = std::min<int64_t>(int64_t(wpc) * num_cus, (total + mn - 1) / mn);
  }
  if (workers > INT32_MAX / 2) return SF_ERR_INVALID_ARG;

  // The attention launch runs workers G b .. G b + G - 1 as workgroup b
  // (one wave each), and workgroup b runs on XCD b mod 8. G is the largest
  // of 8, 4, 2 that packs the workers into whole rounds of one workgroup per
  // CU (W a multiple of G num_cus), else 1: a partial round would leave some
  // CUs with one group more than others.
  int32_t group = 1;
  for (const int32_t g : {8, 4, 2})
    if (workers >= g * int64_t(num_cus) && workers % (g * int64_t(num_cus)) == 0) {
      group = g;
      break;
    }

  // Worker range starts lo(w) = floor(T C(w) / C(W)) with the cumulative
  // weight C(v) = 1000 v + p D(v), D(v) = v mod G if floor(v / G) is even,
  // else G - v mod G: a worker of an even group weighs 1000 + p, of an odd
  // group 1000 - p (|p| <= 250; p = 0 for a forced slice size). Walked
  // forward without divisions: T C(v) grows by T (1000 + p) or T (1000 - p),
  // each positive and below 2^51, and quotient and remainder advance by
  // those over C(W) > 0.
  if (forced > 0) skew = 0;
  struct Cuts {
    int64_t q = 0, r = 0, den = 1, idx = 0, g = 1;
    int64_t dq[2] = {0, 0}, dr[2] = {0, 0};   // [group parity of v]: step from C(v) to C(v + 1)
    void init(int64_t t, int64_t w, int64_t p, int64_t grp) {
      q = r = idx = 0;
      g = grp;
      const int64_t rem = w % g;
      den = w > 0 ? 1000 * w + p * (((w / g) & 1) ? g - rem : rem) : 1;
      for (int k = 0; k < 2; ++k) {
        const int64_t inc = t * (k == 0 ? 1000 + p : 1000 - p);
        dq[k] = inc / den;
        dr[k] = inc % den;
      }
    }
    void next() {
      const int k = int((idx / g) & 1);
      q += dq[k];
      r += dr[k];
      if (r >= den) {
        r -= den;
        ++q;
      }
      ++idx;
    }
  };

  // Pass 1: segments per pair. Worker ranges are cut at pair boundaries; a
  // pair spanning k worker boundaries has k + 1 segments. Pairs are walked in
  // order (s-major, kvh-minor) with a worker cursor that only moves forward.
  // Returns the number of cut pairs.
  auto segments = [&](int64_t p_skew, int32_t* nseg) -> int64_t {
    Cuts next_lo;           // lo(cur + 1)
    next_lo.init(total, workers, p_skew, group);
    next_lo.next();
    int64_t cur = 0;        // worker whose range holds `start`
    int64_t start = 0;      // global page where the current pair starts
    int64_t p = 0, cut = 0;
    for (int32_t s = 0; s < B; ++s) {
      const int64_t npg = spg[s];
      for (int32_t h = 0; h < hkv; ++h, ++p) {
        if (npg == 0) {
          nseg[p] = 1;
          continue;
        }
        while (cur + 1 < workers && next_lo.q <= start) {
          ++cur;
          next_lo.next();
        }
        // boundaries lo(w) inside (start, start + npg) each add a segment
        int32_t k = 1;
        while (cur + 1 < workers && next_lo.q < start + npg) {
          ++cur;
          next_lo.next();
          ++k;
        }
        nseg[p] = k;
        cut += k > 1;
        start += npg;
      }
    }
    return cut;
  };
  if (skew != 0 && workers > 1) {
    // Slices near one page: a skew that would leave a worker without a page
    // falls back to equal slices (which give every worker at least one, since
    // W <= T), so every worker has a segment.
    Cuts c;
    c.init(total, workers, skew, group);
    int64_t prev = 0;
    for (int64_t w = 0; w < workers; ++w) {
      c.next();
      if (c.q == prev) {
        skew = 0;
        break;
      }
      prev = c.q;
    }
  }
  thread_local std::vector<int32_t> nseg_buf, nseg_alt;
  nseg_buf.resize(size_t(num_pairs));
  int32_t* nseg = nseg_buf.data();
  if (skew != 0 && workers > 1) {
    // The skew moves every boundary off the equal cuts; where those fall on
    // pair boundaries (equal lengths, page-aligned) it would cut pairs the
    // equal slices leave whole. Keep it unless it cuts more than W / 8 pairs
    // more than they do.
    nseg_alt.resize(size_t(num_pairs));
    const int64_t cut_skew = segments(skew, nseg);
    const int64_t cut_equal = segments(0, nseg_alt.data());
    if (cut_skew - cut_equal > workers / 8) {
      skew = 0;
      nseg_buf.swap(nseg_alt);
      nseg = nseg_buf.data();
    }
  } else {
    segments(skew, nseg);
  }
  int64_t n_work = 0, n_comb = 0, n_part = 0;
  for (int64_t p = 0; p < num_pairs; ++p) {
    n_work += nseg[p];
    if (nseg[p] > 1) {
      ++n_comb;
      n_part += nseg[p];
    }
  }
  const int64_t table_rows = workers;   // one row per worker
  if (table_rows + n_work + n_comb > INT32_MAX / kItemInts || n_part > INT32_MAX) return SF_ERR_INVALID_ARG;
  const int32_t g = desc->num_q_heads / hkv;
  info->num_workers = int32_t(workers);
  info->num_work = int32_t(n_work);
  info->num_combine = int32_t(n_comb);
  info->num_partials = int32_t(n_part);
  {
    // the widest slice (an even group's worker's when the slices are skewed)
    Cuts c;
    c.init(total, workers, skew, group);
    int64_t prev = 0, widest = 0;
    for (int64_t w = 0; w < workers; ++w) {
      c.next();
      widest = std::max(widest, c.q - prev);
      prev = c.q;
    }
    info->chunk_pages = int32_t(widest);
  }
  info->workers_per_group = group;
  info->work_bytes = uint64_t(table_rows + n_work + n_comb) * kItemInts * 4;
  info->workspace_bytes =
      n_part ? align256(uint64_t(n_part) * g * desc->head_dim * 4) + align256(uint64_t(n_part) * g * 4) : 0;
  info->desc_key = desc_key(desc);
  if (!work_host) return SF_OK;
  if (work_capacity_bytes < info->work_bytes) return SF_ERR_CAPACITY;

  // Pass 2: partial slots and combine rows (pairs with several segments, in pair order).
  int32_t* table = work_host;
  int32_t* items = work_host + table_rows * kItemInts;
  int32_t* comb = items + n_work * kItemInts;
  std::memset(table, 0, size_t(table_rows) * kItemInts * 4);
  thread_local std::vector<int32_t> base_buf, cidx_buf;
  base_buf.assign(size_t(num_pairs), -1);
  cidx_buf.assign(size_t(num_pairs), -1);
  {
    int32_t slot = 0, ci = 0;
    int64_t p = 0;
    for (int32_t s = 0; s < B; ++s) {
      for (int32_t h = 0; h < hkv; ++h, ++p) {
        if (nseg[p] <= 1) continue;
        base_buf[size_t(p)] = slot;
        cidx_buf[size_t(p)] = ci;
        const int32_t c8[kItemInts] = {s, h, slot, nseg[p], seq_lens_host[s], 0, 0, 0};
        std::memcpy(comb + int64_t(ci) * kItemInts, c8, sizeof c8);
        slot += nseg[p];
        ++ci;
      }
    }
  }
  const int32_t* base = base_buf.data();
  const int32_t* cidx = cidx_buf.data();

  // Pass 3: items, worker by worker; a worker's segments in pair order, then
  // the empty pairs e with e mod workers == w.
  thread_local std::vector<int64_t> empty_buf;
  empty_buf.clear();
  int64_t n_empty = 0;
  for (int32_t s = 0; s < B; ++s) n_empty += spg[s] == 0 ? hkv : 0;
  empty_buf.reserve(size_t(n_empty));
  for (int32_t s = 0; s < B; ++s)
    if (spg[s] == 0)
      for (int32_t h = 0; h < hkv; ++h) empty_buf.push_back(int64_t(s) * hkv + h);
  // Cursor over the non-empty pairs: pair p = (ps, ph).
  int64_t p = 0;
  int32_t ps = 0, ph = 0;
  auto skip_empty = [&]() {
    while (ps < B && spg[ps] == 0) {
      ++ps;
      p = int64_t(ps) * hkv;
      ph = 0;
    }
  };
  auto advance = [&]() {
    ++p;
    if (++ph == hkv) {
      ph = 0;
      ++ps;
    }
    skip_empty();
  };
  skip_empty();
  int64_t row = 0, pstart = 0;
  int32_t seg_c = 0;  // segment index within the current pair
  Cuts lo_w, hi_w;
  lo_w.init(total, workers, skew, group);
  hi_w.init(total, workers, skew, group);
  hi_w.next();
  for (int64_t w = 0; w < workers; ++w, lo_w.next(), hi_w.next()) {
    const int64_t lo = lo_w.q, hi = hi_w.q;
    const int64_t first = row;
    int64_t cnt = 0;
    while (ps < B && pstart < hi) {
      const int64_t npg = spg[ps];
      const int64_t b = std::max(lo, pstart) - pstart, e = std::min(hi, pstart + npg) - pstart;
      int32_t* r = items + row * kItemInts;
      r[0] = ps;
      r[1] = ph;
      r[2] = int32_t(b);
      r[3] = int32_t(e);
      r[4] = seq_lens_host[ps];
      r[5] = nseg[p] > 1 ? base[p] + seg_c : -1;
      r[6] = cidx[p];
      r[7] = nseg[p];
      ++row;
      ++cnt;
      if (pstart + npg <= hi) {  // pair finished inside this worker
        pstart += npg;
        seg_c = 0;
        advance();
      } else {
        ++seg_c;
        break;
      }
    }
    for (size_t e = size_t(w); e < empty_buf.size(); e += size_t(workers)) {
      const int64_t q = empty_buf[e];
      int32_t* r = items + row * kItemInts;
      const int32_t r8[kItemInts] = {int32_t(q / hkv), int32_t(q % hkv), 0, 0, 0, -1, -1, 1};
      std::memcpy(r, r8, sizeof r8);
      ++row;
      ++cnt;
    }
    // the worker's row: first item, item count, the first item's fields
    int32_t* t = table + w * kItemInts;
    t[0] = int32_t(first);
    t[1] = int32_t(cnt);
    if (cnt > 0) std::memcpy(t + 2, items + first * kItemInts, 6 * sizeof(int32_t));
  }
  return row == n_work ? SF_OK : SF_ERR_INVALID_ARG;
}
