/*
 * sf_decode_attn.h -- C ABI of the gfx950 (MI355X) paged decode-attention library.
 *
 * The operation. In the paper's rollout phase every running trajectory emits
 * one token per batched decode step, and the step's attention reads each
 * trajectory's whole KV cache, so its latency grows linearly with the cached
 * bytes (App. B.1, attention-latency term of the per-step cost model; the
 * decode share of rollout time is in Table "time_breakdown"). For a batch of
 * B sequences, sequence s holding L_s cached tokens (the current token
 * included), query head h and g = Hq / Hkv query heads per KV head:
 *
 *   kvh      = h / g                                   (contiguous GQA groups)
 *   z_t      = softmax_scale * sum_d q[s,h,d] * K_s[t,d]     t = 0 .. L_s-1
 *   out[s,h] = sum_t exp(z_t) V_s[t] / sum_t exp(z_t)
 *   lse[s,h] = ln sum_t exp(z_t)                        (natural log)
 *
 * K_s[t] / V_s[t] are found through the block table: physical page
 * block_table[s][t / 16], slot t % 16. L_s = 0 yields out = 0, lse = -inf.
 * Trajectory lengths in a rollout batch are heavily skewed (Sec. 2.3); the
 * library splits long (sequence, KV head) ranges into page-aligned chunks
 * (split-K) and merges the chunk results with a log-sum-exp combine, so one
 * GPU's compute units stay busy while stragglers are read.
 *
 * Memory layouts (row-major, every device pointer 16-byte aligned):
 *   q            bf16  [B][Hq][D]
 *   k_pool       bf16  [num_pages][Hkv][16][D]   a page tile is token-major
 *   v_pool       bf16  [num_pages][Hkv][D][16]   a page tile is dim-major
 *   block_table  int32 [B][block_table_stride]   entries 0 .. ceil(L_s/16)-1 are read
 *   out          fp32  [B][Hq][D]
 *   lse          fp32  [B][Hq]                   optional (NULL = not written)
 * A (page, KV head) tile is 16*D*2 bytes (4 KiB at D = 128) and contiguous.
 * Supported: D in {64, 128}, page_size 16, 1 <= g <= 16. The pools may be NULL
 * only when num_pages == 0, and then every sequence length must be 0.
 *
 * Ownership and ordering. The caller allocates every buffer; the library
 * allocates nothing, keeps no state between calls and is reentrant. Device
 * work is enqueued on the caller's HIP stream (void* = hipStream_t, NULL =
 * the default stream) and is asynchronous. A host work list handed to
 * sf_decode_attn must stay unmodified until the stream has passed the call.
 *
 * Errors. Every entry point returns an sf_status. Arguments visible on the
 * host are checked before anything is enqueued; on an error nothing is
 * launched. Block-table entries and pool contents live on the device and are
 * trusted: page ids must be in [0, num_pages).
 */
#ifndef SF_DECODE_ATTN_H
#define SF_DECODE_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sf_status {
  SF_OK = 0,
  SF_ERR_INVALID_ARG = 1,   /* null/misaligned pointer, bad shape or length */
  SF_ERR_UNSUPPORTED = 2,   /* valid but not built: D, page size or g out of range */
  SF_ERR_CAPACITY = 3,      /* work-list buffer or workspace smaller than the plan needs */
  SF_ERR_PLAN_MISMATCH = 4, /* plan was built for a different descriptor */
  SF_ERR_HIP = 5            /* the HIP runtime reported an error */
} sf_status;

/* Shape of one decode step. */
typedef struct sf_attn_desc {
  int32_t num_seqs;            /* B >= 0 */
  int32_t num_q_heads;         /* Hq >= 1 */
  int32_t num_kv_heads;        /* Hkv >= 1, Hq % Hkv == 0 */
  int32_t head_dim;            /* D: 64 or 128 */
  int32_t page_size;           /* tokens per page: 16 */
  int32_t block_table_stride;  /* int32 entries per block-table row, >= max_s ceil(L_s/16) */
  int32_t num_pages;           /* pages in each pool (0: all lengths must be 0) */
  float softmax_scale;         /* multiplies q.k; must be finite */
} sf_attn_desc;

/* Planner knobs; a zero field takes its default. */
typedef struct sf_plan_opts {
  int32_t num_cus;          /* compute units of the target GPU (default 256) */
  int32_t chunk_pages;      /* > 0 forces this chunk size (pages) */
  int32_t units_per_cu;     /* default 8 */
  int32_t min_chunk_pages;  /* default 16 */
  int32_t max_chunk_pages;  /* default 4096 */
} sf_plan_opts;

/* Filled by the planner; passed back unchanged to the other calls. */
typedef struct sf_plan_info {
  int32_t num_work;          /* attention work items */
  int32_t num_combine;       /* (seq, KV head) pairs cut into more than one chunk */
  int32_t num_partials;      /* partial-result slots = sum of their chunk counts */
  int32_t chunk_pages;       /* chunk size the plan used */
  uint64_t work_bytes;       /* bytes of the work list: (num_work + num_combine) * 32 */
  uint64_t workspace_bytes;  /* device scratch sf_decode_attn needs (0 if no partials) */
  uint64_t desc_key;         /* fingerprint of the descriptor's shape and pool-size fields */
} sf_plan_info;

/*
 * Builds the work list on the host (no device calls).
 *
 * Rule (the length-aware split-K partition; the paper balances skewed
 * trajectory lengths across rollout instances, Sec. 5.2, and this balances
 * them across the compute units of one GPU):
 *   pages_s = ceil(L_s / 16);  T = sum_s pages_s * Hkv
 *   C   = opts.chunk_pages if > 0, else
 *         clamp(ceil(T / (units_per_cu * num_cus)), min_chunk_pages, max_chunk_pages)
 *   n_s = ceil(pages_s / C); chunk c of (s, kvh) covers pages
 *         [floor(c * pages_s / n_s), floor((c + 1) * pages_s / n_s))
 *   A sequence with L_s = 0 gets one item per KV head with an empty range.
 *   Items are ordered by page count, largest first, ties by (s, kvh, c).
 *   Pairs with n_s > 1 get consecutive partial slots in (s, kvh) order
 *   (chunk c -> slot_base + c) and one combine item each, in (s, kvh) order.
 * Work list, int32 rows of 8: attention items, then combine items:
 *   attention: seq, kv_head, page_begin, page_end, seq_len,
 *              slot (-1 = write out directly), combine index (-1 if n_s = 1), n_s
 *   combine:   seq, kv_head, slot_base, n_s, 0, 0, 0, 0
 *
 * seq_lens_host: B lengths on the host. opts may be NULL (all defaults).
 * work_host: host buffer of work_capacity_bytes; NULL only reports the sizes
 * in *info. Returns SF_ERR_CAPACITY (with *info filled) if it is too small.
 */
sf_status sf_decode_attn_plan(const sf_attn_desc* desc, const int32_t* seq_lens_host,
                              const sf_plan_opts* opts, int32_t* work_host,
                              uint64_t work_capacity_bytes, sf_plan_info* info);

/*
 * Enqueues the attention pass for one decode step.
 *
 * If work_host is not NULL its info->work_bytes are first copied to work_dev
 * on the stream (work_host should be pinned memory for an asynchronous copy);
 * if it is NULL, work_dev must already hold this plan. Items whose sequence
 * fits in one chunk write out (and lse) directly; the others write partial
 * results into workspace, which sf_decode_attn_combine then merges. Calls
 * that share a work_dev or workspace must not overlap on the device.
 * workspace: device buffer of workspace_bytes >= info->workspace_bytes
 * (may be NULL when that is 0). q, k_pool, v_pool, block_table, out: device
 * pointers in the layouts above. lse: device pointer or NULL.
 */
sf_status sf_decode_attn(const sf_attn_desc* desc, const sf_plan_info* info,
                         const int32_t* work_host, int32_t* work_dev,
                         const void* q, const void* k_pool, const void* v_pool,
                         const int32_t* block_table, float* out, float* lse,
                         void* workspace, uint64_t workspace_bytes, void* stream);

/*
 * Enqueues the log-sum-exp merge of split sequences (after sf_decode_attn on
 * the same stream, same plan, same workspace):
 *   M = max_c lse_c;  out = sum_c e^(lse_c - M) o_c / sum_c e^(lse_c - M);
 *   lse = M + ln sum_c e^(lse_c - M)
 * merging chunks in chunk order. A no-op when info->num_combine == 0.
 */
sf_status sf_decode_attn_combine(const sf_attn_desc* desc, const sf_plan_info* info,
                                 const int32_t* work_dev, const void* workspace,
                                 uint64_t workspace_bytes, float* out, float* lse, void* stream);

/*
 * Test support: copies the cached keys and values of tokens 0 .. len-1 of
 * (seq, kv_head) through the same address translation the attention kernel
 * uses, into device buffers k_dense and v_dense, bf16 [len][D] token-major.
 */
sf_status sf_debug_gather_kv(const sf_attn_desc* desc, const void* k_pool, const void* v_pool,
                             const int32_t* block_table, int32_t seq, int32_t kv_head,
                             int32_t len, void* k_dense, void* v_dense, void* stream);

/* Static description of a status code. */
const char* sf_status_string(sf_status status);

/* Library version, (major << 16) | minor. */
int32_t sf_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SF_DECODE_ATTN_H */
