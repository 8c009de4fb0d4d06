// Internal declarations shared by the host-side API, the planner and the
// kernel launchers of the decode-attention library.
#pragma once

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "sf_decode_attn.h"

namespace sf {

constexpr int kPage = 16;       // tokens per KV page
constexpr int kItemInts = 8;    // int32 fields per work-list row
constexpr int kMaxGroup = 16;   // query heads per KV head handled by one MFMA column block

// Defaults of the length-aware chunk rule (see sf_decode_attn_plan).
constexpr int kDefaultNumCus = 256;
constexpr int kDefaultWorkersPerCu = 4;  // attention waves per CU (one per SIMD)
constexpr int kDefaultMinChunk = 8;      // pages: fewer workers rather than thinner slices
// Largest per-mille shift of page share between even- and odd-indexed
// workers (sf_plan_opts.xcd_parity_skew; none by default).
constexpr int kMaxParitySkew = 250;

sf_status validate_desc(const sf_attn_desc* d);
inline int64_t table_rows(int64_t workers) { return workers; }   // worker-table rows of a plan
uint64_t desc_key(const sf_attn_desc* d);
uint64_t align256(uint64_t x);

// Partial-result workspace: o [slots][g][D] fp32, then lse [slots][g] fp32 (log2 units).
struct Workspace {
  float* part_o;
  float* part_lse;
};
Workspace carve_workspace(void* base, int32_t slots, int32_t g, int32_t d);

struct AttnArgs {
  const int32_t* worker_table;  // (first item, item count) per worker
  const int32_t* items;         // segment rows
  int32_t num_workers;
  int32_t workers_per_group;    // waves per workgroup (1, 4 or 8; the plan's choice)
  const uint16_t* q;
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* block_table;
  float* out;
  float* lse;
  float* part_o;
  float* part_lse;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;
  int32_t head_dim;
  int32_t bt_stride;
  float scale_log2;   // softmax_scale * log2(e)
  // Appending step (sf_decode_attn_append only; k_new is NULL otherwise):
  // the newest tokens, read straight into registers.
  const uint16_t* k_new;      // [B][Hkv][D] newest token's keys
  const uint16_t* v_new;      // [B][Hkv][D] and values
  const int32_t* new_pages;   // [B] page newly given to that token, -1 = none; may be NULL
  // fp8 cache (sf_decode_attn_fp8 only; NULL otherwise): k_pool / v_pool then
  // hold E4M3 codes, and these the per-(page, KV head) scales.
  const float* k_scale;
  const float* v_scale;
  // Optional side job: copy_ints ints from copy_src (the merge rows in
  // pinned host memory) to copy_dst (device), 64 per worker, so that the
  // launch after this one reads its rows from device memory. NULL dst: none.
  const int32_t* copy_src;
  int32_t* copy_dst;
  int32_t copy_ints;
};

// The row copy an attention launch makes for the merge launch after it:
// the plan's combine rows, then (appending) the single-segment rows at int
// single_off and new_pages at int pages_off of dst (-1: not in the copy).
struct RowCopy {
  const int32_t* src;   // device-accessible (mapped pinned host memory)
  int32_t* dst;         // device memory
  int32_t ints;         // at most 64 per worker
  int32_t single_off;
  int32_t pages_off;
};

struct CombineArgs {
  const int32_t* items;       // merge rows
  int32_t num_items;
  const float* part_o;
  const float* part_lse;
  float* out;
  float* lse;
  int32_t num_q_heads;
  int32_t group;
  int32_t head_dim;
  // Appending step (k_new NULL otherwise): the newest tokens join the
  // softmax and go to the pool.
  const int32_t* work_items;  // segment rows
  int32_t num_work;
  const uint16_t* q;
  float scale_log2;
  const uint16_t* k_new;
  const uint16_t* v_new;
  const int32_t* new_pages;
  const int32_t* block_table;
  int32_t* bt_dst;            // the block table, writable
  uint16_t* k_dst;            // the pools, writable
  uint16_t* v_dst;
  int32_t num_kv_heads;
  int32_t bt_stride;
  // Optional: copies of just the segment rows of pairs with one segment and
  // len > 0 (the rows the merge launch acts on); NULL: walk all work_items.
  const int32_t* single_rows;
  int32_t num_single;
};

struct QuantArgs {
  const uint16_t* k_src;      // bf16 pools
  const uint16_t* v_src;
  const int32_t* pages;       // [num_pages] pages to quantize
  const int32_t* valid;       // [num_pages] valid slots of each (1 .. 16)
  int32_t num_pages;
  uint8_t* k_dst;             // fp8 pools
  uint8_t* v_dst;
  float* k_scale;             // [pool pages][Hkv]
  float* v_scale;
  int32_t num_kv_heads;
  int32_t head_dim;
};

struct GatherArgs {
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* block_table;
  uint16_t* k_dense;
  uint16_t* v_dense;
  int32_t seq;
  int32_t kv_head;
  int32_t len;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t bt_stride;
};

// Extend (re-prefill) attention and the store of the new tokens.
struct ExtendArgs {
  const int32_t* items;       // rows: seq, kv_head, t0, nt, prefix, q_row0, key steps, 0
  int32_t num_items;
  const uint16_t* q;          // [T][Hq][D]
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* block_table;
  float* out;                 // [T][Hq][D]
  float* lse;                 // [T][Hq] or NULL
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;
  int32_t head_dim;
  int32_t bt_stride;
  float scale_log2;           // |softmax_scale| * log2(e)
  uint32_t q_sign;            // 0x80008000 for a negative scale: query bf16 sign flips
  // Store launch first when k_new is not NULL.
  const uint16_t* k_new;      // [T][Hkv][D]
  const uint16_t* v_new;
  uint16_t* k_dst;            // the pools, writable
  uint16_t* v_dst;
};

// Rows (tokens x query heads of a group) of one extend work item.
constexpr int kExtendRows = 384;

// start / stop (hipEvent_t, may be NULL) take the kernel's own start and end
// times: the launch records them from its dispatch (hipExtLaunchKernel), so
// their difference is the kernel's duration without queue time.
hipError_t launch_attention(const AttnArgs& a, hipStream_t stream, hipEvent_t start = nullptr,
                            hipEvent_t stop = nullptr);

// sf_decode_attn_append with the merge launch restricted to single_rows
// (num_single copies, in work-item format, of the rows of pairs that have one
// segment and len > 0; device-accessible). The native runner's path. With
// `copy`, the attention launch copies the merge rows to copy->dst (the plan's
// combine rows, then the single rows) and the merge launch reads them there.
sf_status decode_attn_append_rows(const sf_attn_desc* desc, const sf_plan_info* info, int32_t* work_dev,
                                  const void* q, const void* k_new, const void* v_new, const int32_t* new_pages,
                                  const int32_t* single_rows, int32_t num_single, void* k_pool, void* v_pool,
                                  int32_t* block_table, float* out, float* lse, void* workspace,
                                  uint64_t workspace_bytes, void* stream, const RowCopy* copy,
                                  void* attn_start = nullptr, void* attn_end = nullptr);

// sf_decode_attn (k_scale NULL) or sf_decode_attn_fp8, then the combine of
// split pairs, on a device-resident or mapped work list; with `copy`, the
// attention launch copies the plan's combine rows to copy->dst and the
// combine launch reads them there. The native runner's other path.
// attn_start / attn_end (hipEvent_t, may be NULL) take the attention
// kernel's own start and end times (launch_attention).
sf_status decode_attn_rows(const sf_attn_desc* desc, const sf_plan_info* info, int32_t* work_dev, const void* q,
                           const void* k_pool, const void* v_pool, const float* k_scale, const float* v_scale,
                           const int32_t* block_table, float* out, float* lse, void* workspace,
                           uint64_t workspace_bytes, void* stream, const RowCopy* copy, void* attn_start,
                           void* attn_end);
hipError_t launch_extend(const ExtendArgs& a, hipStream_t stream);

// Every host-side check of a decode step's arguments except the workspace
// (k_new / v_new / new_pages: an appending step; k_scale / v_scale: fp8).
sf_status check_step_args(const sf_attn_desc* desc, const sf_plan_info* info, const int32_t* work_dev,
                          const void* q, const void* k_pool, const void* v_pool, const int32_t* block_table,
                          const float* out, const float* lse, const void* k_new, const void* v_new,
                          const int32_t* new_pages, const float* k_scale, const float* v_scale);

// sf_decode_attn (work list already on the device) then
// sf_decode_attn_combine, both on `workspace`; the body of
// sf_decode_attn_scratch.
sf_status decode_attn_and_combine(const sf_attn_desc* desc, const sf_plan_info* info, const int32_t* work_dev,
                                  const void* q, const void* k_pool, const void* v_pool, const int32_t* block_table,
                                  float* out, float* lse, void* workspace, uint64_t workspace_bytes, void* stream);
hipError_t launch_combine(const CombineArgs& a, hipStream_t stream);
hipError_t launch_gather(const GatherArgs& a, hipStream_t stream);
// Streaming-read probe: reads bytes (a multiple of 16) of buf once; sink: 16 B.
// start / stop: as for launch_attention.
hipError_t launch_stream_read(const void* buf, uint64_t bytes, void* sink, int blocks, hipStream_t stream,
                              hipEvent_t start = nullptr, hipEvent_t stop = nullptr);
hipError_t launch_quantize_fp8(const QuantArgs& a, hipStream_t stream);

}  // namespace sf
