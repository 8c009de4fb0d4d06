// C entry points: argument checks on the host, then stream-ordered launches.
// Nothing here allocates device memory or keeps state between calls.
#include <cmath>
#include <cstdint>

#include "sf_internal.h"

using namespace sf;

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

sf_status check_plan(const sf_attn_desc* d, const sf_plan_info* info) {
  if (!info) return SF_ERR_INVALID_ARG;
  if (info->desc_key != desc_key(d)) return SF_ERR_PLAN_MISMATCH;
  if (info->num_workers < 0 || info->num_work < 0 || info->num_combine < 0 || info->num_partials < 0)
    return SF_ERR_INVALID_ARG;
  const int32_t grp = info->workers_per_group;
  if ((grp != 1 && grp != 2 && grp != 4 && grp != 8) ||
      info->work_bytes != uint64_t(table_rows(info->num_workers) + info->num_work +
                                                          info->num_combine) * kItemInts * 4)
    return SF_ERR_PLAN_MISMATCH;
  return SF_OK;
}

sf_status from_hip(hipError_t e) { return e == hipSuccess ? SF_OK : SF_ERR_HIP; }

}  // namespace

namespace {

struct AppendArgs {
  const void* q;
  const void* k_new;
  const void* v_new;
  const int32_t* new_pages;
  const int32_t* single_rows;   // optional (see decode_attn_append_rows)
  int32_t num_single;
};

// Merge rows of a plan; with `app`, also the newest-token stores. rows: the
// combine rows' device copy (NULL: read them from the work list).
CombineArgs combine_args(const sf_attn_desc* desc, const sf_plan_info* info, const int32_t* work_dev,
                         void* workspace, float* out, float* lse, const AppendArgs* app, void* k_pool,
                         void* v_pool, int32_t* block_table, const int32_t* rows = nullptr) {
  const int32_t g = desc->num_q_heads / desc->num_kv_heads;
  Workspace ws = carve_workspace(workspace, info->num_partials, g, desc->head_dim);
  CombineArgs a = {};
  a.items = rows ? rows : work_dev + (table_rows(info->num_workers) + info->num_work) * kItemInts;
  a.num_items = info->num_combine;
  a.part_o = info->num_partials ? ws.part_o : nullptr;
  a.part_lse = info->num_partials ? ws.part_lse : nullptr;
  a.out = out;
  a.lse = lse;
  a.num_q_heads = desc->num_q_heads;
  a.group = g;
  a.head_dim = desc->head_dim;
  if (app) {
    a.work_items = work_dev + table_rows(info->num_workers) * kItemInts;
    a.num_work = info->num_work;
    a.q = static_cast<const uint16_t*>(app->q);
    a.scale_log2 = float(double(desc->softmax_scale) * 1.4426950408889634074);
    a.k_new = static_cast<const uint16_t*>(app->k_new);
    a.v_new = static_cast<const uint16_t*>(app->v_new);
    a.new_pages = app->new_pages;
    a.block_table = block_table;
    a.bt_dst = block_table;
    a.k_dst = static_cast<uint16_t*>(k_pool);
    a.v_dst = static_cast<uint16_t*>(v_pool);
    a.num_kv_heads = desc->num_kv_heads;
    a.bt_stride = desc->block_table_stride;
    a.single_rows = app->single_rows;
    a.num_single = app->num_single;
  }
  return a;
}

}  // namespace

// Every host-side check of a decode step's arguments except the workspace.
sf_status sf::check_step_args(const sf_attn_desc* desc, const sf_plan_info* info, const int32_t* work_dev,
                              const void* q, const void* k_pool, const void* v_pool, const int32_t* block_table,
                              const float* out, const float* lse, const void* k_new, const void* v_new,
                              const int32_t* new_pages, const float* k_scale, const float* v_scale) {
  sf_status st = validate_desc(desc);
  if (st != SF_OK) return st;
  if ((st = check_plan(desc, info)) != SF_OK) return st;
  if (info->num_workers == 0) return SF_OK;
  if (!work_dev || !q || !block_table || !out) return SF_ERR_INVALID_ARG;
  // An empty pool (num_pages == 0) only backs plans whose sequences are all empty.
  if (desc->num_pages > 0 && (!k_pool || !v_pool)) return SF_ERR_INVALID_ARG;
  if (!aligned16(work_dev) || !aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool) ||
      !aligned16(out) || !aligned4(block_table) || (lse && !aligned4(lse)))
    return SF_ERR_INVALID_ARG;
  if ((k_scale == nullptr) != (v_scale == nullptr)) return SF_ERR_INVALID_ARG;
  if (k_scale && desc->num_pages > 0 && (!aligned4(k_scale) || !aligned4(v_scale))) return SF_ERR_INVALID_ARG;
  if ((k_new || v_new) && (!k_new || !v_new || !aligned16(k_new) || !aligned16(v_new) ||
                           (new_pages && !aligned4(new_pages)) || !lse))
    return SF_ERR_INVALID_ARG;
  return SF_OK;
}

namespace {

// Shared by sf_decode_attn and sf_decode_attn_append: checks, optional
// work-list upload, the attention launch; when appending, also the merge
// launch that stores the newest tokens.
sf_status attend(const sf_attn_desc* desc, const sf_plan_info* info, const int32_t* work_host,
                 int32_t* work_dev, const void* q, const void* k_pool, const void* v_pool,
                 const int32_t* block_table, float* out, float* lse, void* workspace,
                 uint64_t workspace_bytes, void* stream, const AppendArgs* app,
                 const float* k_scale = nullptr, const float* v_scale = nullptr, const RowCopy* copy = nullptr,
                 void* attn_start = nullptr, void* attn_end = nullptr) {
  sf_status st = check_step_args(desc, info, work_dev, q, k_pool, v_pool, block_table, out, lse,
                                 app ? app->k_new : nullptr, app ? app->v_new : nullptr,
                                 app ? app->new_pages : nullptr, k_scale, v_scale);
  if (st != SF_OK) return st;
  if (info->num_workers == 0) return SF_OK;
  // An appending step must name both new-token arrays.
  if (app && (!app->k_new || !app->v_new)) return SF_ERR_INVALID_ARG;
  if (workspace_bytes < info->workspace_bytes) return SF_ERR_CAPACITY;
  if (info->workspace_bytes && (!workspace || !aligned16(workspace))) return SF_ERR_INVALID_ARG;

  hipStream_t s = static_cast<hipStream_t>(stream);
  if (work_host) {
    hipError_t e = hipMemcpyAsync(work_dev, work_host, info->work_bytes, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return SF_ERR_HIP;
  }
  const int32_t g = desc->num_q_heads / desc->num_kv_heads;
  Workspace ws = carve_workspace(workspace, info->num_partials, g, desc->head_dim);
  AttnArgs a;
  a.worker_table = work_dev;
  a.items = work_dev + table_rows(info->num_workers) * kItemInts;
  a.num_workers = info->num_workers;
  a.workers_per_group = info->workers_per_group;
  a.q = static_cast<const uint16_t*>(q);
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.block_table = block_table;
  a.out = out;
  a.lse = lse;
  a.part_o = info->num_partials ? ws.part_o : nullptr;
  a.part_lse = info->num_partials ? ws.part_lse : nullptr;
  a.num_q_heads = desc->num_q_heads;
  a.num_kv_heads = desc->num_kv_heads;
  a.group = g;
  a.head_dim = desc->head_dim;
  a.bt_stride = desc->block_table_stride;
  a.scale_log2 = float(double(desc->softmax_scale) * 1.4426950408889634074);
  a.k_new = app ? static_cast<const uint16_t*>(app->k_new) : nullptr;
  a.v_new = app ? static_cast<const uint16_t*>(app->v_new) : nullptr;
  a.new_pages = app ? app->new_pages : nullptr;
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  const bool copying = copy && copy->ints > 0 && copy->ints <= int64_t(64) * info->num_workers;
  a.copy_src = copying ? copy->src : nullptr;
  a.copy_dst = copying ? copy->dst : nullptr;
  a.copy_ints = copying ? copy->ints : 0;
  if ((st = from_hip(launch_attention(a, s, static_cast<hipEvent_t>(attn_start),
                                      static_cast<hipEvent_t>(attn_end)))) != SF_OK || !app)
    return st;
  AppendArgs app_rows = *app;
  if (copying && app->single_rows && copy->single_off >= 0) app_rows.single_rows = copy->dst + copy->single_off;
  if (copying && app->new_pages && copy->pages_off >= 0) app_rows.new_pages = copy->dst + copy->pages_off;
  const CombineArgs m = combine_args(desc, info, work_dev, workspace, out, lse, &app_rows,
                                     const_cast<void*>(k_pool), const_cast<void*>(v_pool),
                                     const_cast<int32_t*>(block_table), copying ? copy->dst : nullptr);
  return from_hip(launch_combine(m, s));
}

}  // namespace

sf_status sf::decode_attn_append_rows(const sf_attn_desc* desc, const sf_plan_info* info, int32_t* work_dev,
                                      const void* q, const void* k_new, const void* v_new,
                                      const int32_t* new_pages, const int32_t* single_rows, int32_t num_single,
                                      void* k_pool, void* v_pool, int32_t* block_table, float* out, float* lse,
                                      void* workspace, uint64_t workspace_bytes, void* stream,
                                      const RowCopy* copy, void* attn_start, void* attn_end) {
  if (num_single < 0 || (info && num_single > info->num_work) || (num_single > 0 && !single_rows) ||
      (single_rows && !aligned16(single_rows)))
    return SF_ERR_INVALID_ARG;
  const AppendArgs app = {q, k_new, v_new, new_pages, single_rows, num_single};
  return attend(desc, info, nullptr, work_dev, q, k_pool, v_pool, block_table, out, lse, workspace,
                workspace_bytes, stream, &app, nullptr, nullptr, copy, attn_start, attn_end);
}

sf_status sf::decode_attn_rows(const sf_attn_desc* desc, const sf_plan_info* info, int32_t* work_dev, const void* q,
                               const void* k_pool, const void* v_pool, const float* k_scale, const float* v_scale,
                               const int32_t* block_table, float* out, float* lse, void* workspace,
                               uint64_t workspace_bytes, void* stream, const RowCopy* copy, void* attn_start,
                               void* attn_end) {
  sf_status st = attend(desc, info, nullptr, work_dev, q, k_pool, v_pool, block_table, out, lse, workspace,
                        workspace_bytes, stream, nullptr, k_scale, v_scale, copy, attn_start, attn_end);
  if (st != SF_OK) return st;
  if (info->num_workers == 0 || info->num_combine == 0) return st;
  const bool copying = copy && copy->ints > 0 && copy->ints <= int64_t(64) * info->num_workers;
  const CombineArgs a = combine_args(desc, info, work_dev, workspace, out, lse, nullptr, nullptr, nullptr, nullptr,
                                     copying ? copy->dst : nullptr);
  return from_hip(launch_combine(a, static_cast<hipStream_t>(stream)));
}

sf_status sf::decode_attn_and_combine(const sf_attn_desc* desc, const sf_plan_info* info, const int32_t* work_dev,
                                     const void* q, const void* k_pool, const void* v_pool,
                                     const int32_t* block_table, float* out, float* lse, void* workspace,
                                     uint64_t workspace_bytes, void* stream) {
  int32_t* wd = const_cast<int32_t*>(work_dev);   // read only: no work_host, so nothing is copied into it
  sf_status st = attend(desc, info, nullptr, wd, q, k_pool, v_pool, block_table, out, lse, workspace,
                        workspace_bytes, stream, nullptr);
  if (st != SF_OK || info->num_workers == 0 || info->num_combine == 0) return st;
  const CombineArgs a = combine_args(desc, info, wd, workspace, out, lse, nullptr, nullptr, nullptr, nullptr);
  return from_hip(launch_combine(a, static_cast<hipStream_t>(stream)));
}

extern "C" sf_status sf_decode_attn(const sf_attn_desc* desc, const sf_plan_info* info,
                                    const int32_t* work_host, int32_t* work_dev, const void* q,
                                    const void* k_pool, const void* v_pool,
                                    const int32_t* block_table, float* out, float* lse,
                                    void* workspace, uint64_t workspace_bytes, void* stream) {
  return attend(desc, info, work_host, work_dev, q, k_pool, v_pool, block_table, out, lse, workspace,
                workspace_bytes, stream, nullptr);
}

extern "C" sf_status sf_decode_attn_append(const sf_attn_desc* desc, const sf_plan_info* info,
                                           const int32_t* work_host, int32_t* work_dev, const void* q,
                                           const void* k_new, const void* v_new, const int32_t* new_pages,
                                           void* k_pool, void* v_pool, int32_t* block_table, float* out,
                                           float* lse, void* workspace, uint64_t workspace_bytes,
                                           void* stream) {
  const AppendArgs app = {q, k_new, v_new, new_pages, nullptr, 0};
  return attend(desc, info, work_host, work_dev, q, k_pool, v_pool, block_table, out, lse, workspace,
                workspace_bytes, stream, &app);
}

extern "C" sf_status sf_decode_attn_fp8(const sf_attn_desc* desc, const sf_plan_info* info,
                                        const int32_t* work_host, int32_t* work_dev, const void* q,
                                        const void* k_pool8, const void* v_pool8, const float* k_scale,
                                        const float* v_scale, const int32_t* block_table, float* out,
                                        float* lse, void* workspace, uint64_t workspace_bytes, void* stream) {
  if (desc && desc->num_pages > 0 && (!k_scale || !v_scale)) return SF_ERR_INVALID_ARG;
  // With no pages there is nothing to scale; any non-NULL pointer marks the fp8 path.
  static const float kNoScale = 1.f;
  return attend(desc, info, work_host, work_dev, q, k_pool8, v_pool8, block_table, out, lse, workspace,
                workspace_bytes, stream, nullptr, k_scale ? k_scale : &kNoScale, v_scale ? v_scale : &kNoScale);
}

extern "C" sf_status sf_kv_quantize_fp8(const sf_attn_desc* desc, const void* k_pool, const void* v_pool,
                                        const int32_t* pages, const int32_t* valid_slots, int32_t num_pages,
                                        void* k_pool8, void* v_pool8, float* k_scale, float* v_scale,
                                        void* stream) {
  sf_status st = validate_desc(desc);
  if (st != SF_OK) return st;
  if (num_pages < 0) return SF_ERR_INVALID_ARG;
  if (num_pages == 0) return SF_OK;
  if (desc->num_pages == 0 || !k_pool || !v_pool || !pages || !valid_slots || !k_pool8 || !v_pool8 || !k_scale ||
      !v_scale)
    return SF_ERR_INVALID_ARG;
  if (!aligned16(k_pool) || !aligned16(v_pool) || !aligned16(k_pool8) || !aligned16(v_pool8) || !aligned4(pages) ||
      !aligned4(valid_slots) || !aligned4(k_scale) || !aligned4(v_scale))
    return SF_ERR_INVALID_ARG;
  QuantArgs a;
  a.k_src = static_cast<const uint16_t*>(k_pool);
  a.v_src = static_cast<const uint16_t*>(v_pool);
  a.pages = pages;
  a.valid = valid_slots;
  a.num_pages = num_pages;
  a.k_dst = static_cast<uint8_t*>(k_pool8);
  a.v_dst = static_cast<uint8_t*>(v_pool8);
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.num_kv_heads = desc->num_kv_heads;
  a.head_dim = desc->head_dim;
  return from_hip(launch_quantize_fp8(a, static_cast<hipStream_t>(stream)));
}

extern "C" sf_status sf_decode_attn_combine(const sf_attn_desc* desc, const sf_plan_info* info,
                                            const int32_t* work_dev, const void* workspace,
                                            uint64_t workspace_bytes, float* out, float* lse,
                                            void* stream) {
  sf_status st = validate_desc(desc);
  if (st != SF_OK) return st;
  if ((st = check_plan(desc, info)) != SF_OK) return st;
  if (info->num_combine == 0) return SF_OK;
  if (!work_dev || !workspace || !out) return SF_ERR_INVALID_ARG;
  if (!aligned16(work_dev) || !aligned16(workspace) || !aligned16(out) || (lse && !aligned4(lse)))
    return SF_ERR_INVALID_ARG;
  if (workspace_bytes < info->workspace_bytes) return SF_ERR_CAPACITY;
  const CombineArgs a = combine_args(desc, info, work_dev, const_cast<void*>(workspace), out, lse, nullptr,
                                     nullptr, nullptr, nullptr);
  return from_hip(launch_combine(a, static_cast<hipStream_t>(stream)));
}

extern "C" sf_status sf_debug_gather_kv(const sf_attn_desc* desc, const void* k_pool,
                                        const void* v_pool, const int32_t* block_table,
                                        int32_t seq, int32_t kv_head, int32_t len, void* k_dense,
                                        void* v_dense, void* stream) {
  sf_status st = validate_desc(desc);
  if (st != SF_OK) return st;
  if (seq < 0 || seq >= desc->num_seqs || kv_head < 0 || kv_head >= desc->num_kv_heads || len < 0)
    return SF_ERR_INVALID_ARG;
  if ((int64_t(len) + kPage - 1) / kPage > desc->block_table_stride) return SF_ERR_INVALID_ARG;
  if (len == 0) return SF_OK;
  if (!k_pool || !v_pool || !block_table || !k_dense || !v_dense) return SF_ERR_INVALID_ARG;
  if (!aligned16(k_pool) || !aligned16(v_pool) || !aligned4(block_table) || !aligned16(k_dense) ||
      !aligned16(v_dense))
    return SF_ERR_INVALID_ARG;
  GatherArgs a;
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.block_table = block_table;
  a.k_dense = static_cast<uint16_t*>(k_dense);
  a.v_dense = static_cast<uint16_t*>(v_dense);
  a.seq = seq;
  a.kv_head = kv_head;
  a.len = len;
  a.num_kv_heads = desc->num_kv_heads;
  a.head_dim = desc->head_dim;
  a.bt_stride = desc->block_table_stride;
  return from_hip(launch_gather(a, static_cast<hipStream_t>(stream)));
}

extern "C" sf_status sf_debug_stream_read(const void* buf, uint64_t bytes, void* sink, int32_t blocks,
                                          void* stream, void* start_event, void* stop_event) {
  if (bytes == 0) return SF_OK;
  if (!buf || !sink || !aligned16(buf) || !aligned16(sink) || bytes % 16 != 0 || blocks < 1 || blocks > 65536)
    return SF_ERR_INVALID_ARG;
  return from_hip(launch_stream_read(buf, bytes, sink, blocks, static_cast<hipStream_t>(stream),
                                     static_cast<hipEvent_t>(start_event), static_cast<hipEvent_t>(stop_event)));
}

extern "C" const char* sf_status_string(sf_status s) {
  switch (s) {
    case SF_OK: return "ok";
    case SF_ERR_INVALID_ARG: return "invalid argument";
    case SF_ERR_UNSUPPORTED: return "unsupported shape (head_dim must be 64 or 128, page_size 16, Hq/Hkv <= 16)";
    case SF_ERR_CAPACITY: return "buffer, workspace or page pool too small";
    case SF_ERR_PLAN_MISMATCH: return "plan was built for a different descriptor";
    case SF_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

extern "C" int32_t sf_version(void) { return (1 << 16) | 0; }
