// Extend (re-prefill) attention: host planner and entry point.
//
// A re-prefill recomputes a resumed trajectory's KV cache (Sec. 2.3, partial
// rollout and migration). Its cost per new token grows with the token's
// position, so a sequence's new tokens are cut into blocks of
// floor(384 / g) tokens, one work item per (sequence, KV head, block), and
// the items are launched longest first: the GPU starts the longest key walks
// early and fills the tail with the short ones. The rule is stated in
// sf_decode_attn.h next to sf_extend_attn_plan.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "sf_internal.h"

static_assert(sizeof(sf_extend_info) == 32, "sf_extend_info layout is part of the ABI");

using namespace sf;

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

struct Item {
  int32_t seq, kvh, t0, nt, prefix, qrow0, steps;
};

}  // namespace

extern "C" sf_status sf_extend_attn_plan(const sf_attn_desc* desc, const int32_t* seq_lens_host,
                                         const int32_t* q_lens_host, int32_t* work_host,
                                         uint64_t work_capacity_bytes, sf_extend_info* info) {
  sf_status st = validate_desc(desc);
  if (st != SF_OK) return st;
  if (!info || (desc->num_seqs > 0 && (!seq_lens_host || !q_lens_host))) return SF_ERR_INVALID_ARG;
  const int32_t g = desc->num_q_heads / desc->num_kv_heads;
  const int32_t per_item = kExtendRows / g;
  int64_t rows = 0;
  for (int32_t s = 0; s < desc->num_seqs; ++s) {
    const int32_t L = seq_lens_host[s], e = q_lens_host[s];
    if (e < 0 || L < e || int64_t(L) > int64_t(kPage) * desc->block_table_stride) return SF_ERR_INVALID_ARG;
    if (L > 0 && desc->num_pages == 0) return SF_ERR_INVALID_ARG;
    rows += e;
  }
  if (rows > INT32_MAX / (int64_t(desc->num_q_heads) * desc->head_dim)) return SF_ERR_INVALID_ARG;

  std::vector<Item> items;
  int32_t qrow0 = 0;
  for (int32_t s = 0; s < desc->num_seqs; ++s) {
    const int32_t L = seq_lens_host[s], e = q_lens_host[s];
    for (int32_t kvh = 0; kvh < desc->num_kv_heads; ++kvh)
      for (int32_t t0 = 0; t0 < e; t0 += per_item) {
        const int32_t nt = std::min(per_item, e - t0);
        const int32_t prefix = L - e;
        items.push_back({s, kvh, t0, nt, prefix, qrow0, (prefix + t0 + nt + 2 * kPage - 1) / (2 * kPage)});
      }
    qrow0 += e;
  }
  // Longest key walk first; ties keep (sequence, KV head, block) order.
  std::stable_sort(items.begin(), items.end(), [](const Item& x, const Item& y) { return x.steps > y.steps; });

  info->num_items = int32_t(items.size());
  info->tokens_per_item = per_item;
  info->num_q_rows = int32_t(rows);
  info->reserved = 0;
  info->work_bytes = uint64_t(items.size()) * kItemInts * 4;
  info->desc_key = desc_key(desc);
  if (!work_host) return SF_OK;
  if (work_capacity_bytes < info->work_bytes) return SF_ERR_CAPACITY;
  for (size_t i = 0; i < items.size(); ++i) {
    const Item& it = items[i];
    int32_t* r = work_host + i * kItemInts;
    r[0] = it.seq;
    r[1] = it.kvh;
    r[2] = it.t0;
    r[3] = it.nt;
    r[4] = it.prefix;
    r[5] = it.qrow0;
    r[6] = it.steps;
    r[7] = 0;
  }
  return SF_OK;
}

extern "C" sf_status sf_extend_attn(const sf_attn_desc* desc, const sf_extend_info* info,
                                    const int32_t* work_host, int32_t* work_dev, const void* q,
                                    const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                                    const int32_t* block_table, float* out, float* lse, void* stream) {
  sf_status st = validate_desc(desc);
  if (st != SF_OK) return st;
  if (!info) return SF_ERR_INVALID_ARG;
  if (info->desc_key != desc_key(desc)) return SF_ERR_PLAN_MISMATCH;
  if (info->num_items < 0 || info->num_q_rows < 0 || info->reserved != 0 ||
      info->work_bytes != uint64_t(info->num_items) * kItemInts * 4 ||
      info->tokens_per_item != kExtendRows / (desc->num_q_heads / desc->num_kv_heads))
    return SF_ERR_PLAN_MISMATCH;
  if (info->num_items == 0) return SF_OK;
  if ((k_new == nullptr) != (v_new == nullptr)) return SF_ERR_INVALID_ARG;
  if (!work_dev || !q || !k_pool || !v_pool || !block_table || !out) return SF_ERR_INVALID_ARG;
  if (!aligned16(work_dev) || !aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(out) ||
      !aligned4(block_table) || (lse && !aligned4(lse)) || (k_new && (!aligned16(k_new) || !aligned16(v_new))))
    return SF_ERR_INVALID_ARG;

  hipStream_t s = static_cast<hipStream_t>(stream);
  if (work_host) {
    hipError_t e = hipMemcpyAsync(work_dev, work_host, info->work_bytes, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return SF_ERR_HIP;
  }
  ExtendArgs a;
  a.items = work_dev;
  a.num_items = info->num_items;
  a.q = static_cast<const uint16_t*>(q);
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.block_table = block_table;
  a.out = out;
  a.lse = lse;
  a.num_q_heads = desc->num_q_heads;
  a.num_kv_heads = desc->num_kv_heads;
  a.group = desc->num_q_heads / desc->num_kv_heads;
  a.head_dim = desc->head_dim;
  a.bt_stride = desc->block_table_stride;
  // Negating bf16 queries is exact, so a negative scale becomes a positive one.
  a.scale_log2 = float(std::fabs(double(desc->softmax_scale)) * 1.4426950408889634074);
  a.q_sign = desc->softmax_scale < 0.f ? 0x80008000u : 0u;
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.k_dst = static_cast<uint16_t*>(k_pool);
  a.v_dst = static_cast<uint16_t*>(v_pool);
  return launch_extend(a, s) == hipSuccess ? SF_OK : SF_ERR_HIP;
}
