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
 *   k_pool       bf16  [num_pages][Hkv][D/8][16][8]  key of slot t, dim d at [..][d/8][t][d%8]
 *   v_pool       bf16  [num_pages][Hkv][D][16]       value of slot t, dim d at [..][d][t]
 *   block_table  int32 [B][block_table_stride]       entries 0 .. ceil(L_s/16)-1 are read
 *   out          fp32  [B][Hq][D]
 *   lse          fp32  [B][Hq]                       optional (NULL = not written)
 * A (page, KV head) tile is 16*D*2 bytes (4 KiB at D = 128) and contiguous in
 * both pools. Inside a K tile each group of 8 dims holds the 16 tokens' 8-dim
 * pieces back to back; a V tile is dim-major. (Both are what the gfx950
 * matrix-core operands of one page read as contiguous runs.)
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
  SF_ERR_CAPACITY = 3,      /* work-list buffer or workspace smaller than the plan needs, or too few free pages */
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
  float softmax_scale;         /* multiplies q.k; |scale| * log2(e) must be a finite float
                                  (|scale| <= 2.35e38) */
} sf_attn_desc;

/* Planner knobs; a zero field takes its default. */
typedef struct sf_plan_opts {
  int32_t num_cus;          /* compute units of the target GPU (default 256) */
  int32_t chunk_pages;      /* > 0 forces the pages per worker: workers = ceil(T / chunk_pages) */
  int32_t workers_per_cu;   /* default 4: attention waves per CU (one per SIMD) */
  int32_t min_chunk_pages;  /* default 8: fewer workers rather than slices thinner than this */
  int32_t xcd_parity_skew;  /* p in the slice rule below, per mille, -250 .. 250: default 0
                               (equal slices); ignored when chunk_pages > 0 */
} sf_plan_opts;

/* Filled by the planner; passed back unchanged to the other calls. */
typedef struct sf_plan_info {
  int32_t num_workers;       /* attention waves to launch (one per worker) */
  int32_t num_work;          /* segments (work items) */
  int32_t num_combine;       /* (seq, KV head) pairs cut into more than one segment */
  int32_t num_partials;      /* partial-result slots = sum of their segment counts */
  int32_t chunk_pages;       /* the most pages any worker owns (0 if T = 0) */
  int32_t workers_per_group; /* G: waves per attention workgroup, 1, 2, 4 or 8 (rule below) */
  uint64_t work_bytes;       /* bytes of the work list:
                                (num_workers + num_work + num_combine) * 32 */
  uint64_t workspace_bytes;  /* device scratch sf_decode_attn needs (0 if no partials) */
  uint64_t desc_key;         /* fingerprint of the descriptor's shape and pool-size fields */
} sf_plan_info;

/*
 * Builds the work list on the host (no device calls).
 *
 * Rule (the length-aware partition; the paper balances skewed trajectory
 * lengths across rollout instances, Sec. 5.3, and this balances them across
 * the compute units of one GPU). The pairs p = (s, kvh), in order s-major,
 * kvh-minor, have pages_p = ceil(L_s / 16); laid end to end they form
 * T = sum_p pages_p global pages. With
 *   W = ceil(T / chunk_pages)                                   if chunk_pages > 0
 *   W = min(workers_per_cu * num_cus, ceil(T / min_chunk_pages)) otherwise
 * (W = 1 if T = 0 but B * Hkv > 0), and G the largest of 8, 4, 2 for which
 * W is a positive multiple of G num_cus (else G = 1), worker w owns the global pages
 * [floor(T C(w) / C(W)), floor(T C(w + 1) / C(W))) with C(v) = 1000 v +
 * p D(v), D(v) = v mod G if floor(v / G) is even, else G - v mod G: every
 * worker reads its share of the pages however skewed the lengths are, 1000 + p
 * per mille of the mean if floor(w / G) is even, 1000 - p if it is odd
 * (p = opts->xcd_parity_skew, default 0: equal slices, within one page; p is
 * also 0 when chunk_pages is forced, when the skewed slices would leave a
 * worker without a page (slices near one page; the equal ones give each
 * worker at least one, so every worker has a segment), and when they would
 * cut more than floor(W / 8) more pairs than the equal ones: equal lengths can
 * put every equal boundary on a pair boundary). The attention launch runs workers
 * G b .. G b + G - 1 as workgroup b, and workgroup b runs on XCD b mod 8: a
 * GPU whose odd (p > 0) or even (p < 0) XCDs are slower on the same work can
 * give them less. How much slower, and which, differs from one MI355X to the
 * next. A worker's range is
 * cut at pair boundaries into segments, each a work item on one pair; a pair
 * crossing k worker boundaries has n_p = k + 1 segments. Empty pairs
 * (L_s = 0) get one item each, handed to worker e mod W for the e-th empty
 * pair, after that worker's segments; their rows are written as zeros.
 * Pairs with n_p > 1 get consecutive partial slots in pair order (segment c,
 * counted in page order, -> slot_base + c) and one combine item each.
 *
 * Work list, int32 rows of 8:
 *   W rows of worker table, row w: first item, item count (the worker's
 *     items are consecutive), then ints 0 .. 5 of its first item's row
 *     (all zero for a worker without items)
 *   num_work item rows, worker by worker:
 *     seq, kv_head, page_begin, page_end (pages of the pair), seq_len,
 *     slot (-1 = write out directly), combine index (-1 if n_p = 1), n_p
 *   num_combine rows: seq, kv_head, slot_base, n_p, seq_len, 0, 0, 0
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
 * if it is NULL, work_dev must already hold this plan. One wave runs per
 * worker and walks its segments in order. A pair with a single segment
 * writes out (and lse) directly; segments of cut pairs write partial results
 * into workspace, which sf_decode_attn_combine then merges. Calls that share
 * a work_dev or workspace must not overlap on the device.
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
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the decode
 * step of sf_decode_attn followed by sf_decode_attn_combine, with the split-K
 * partial results in a device array the library owns (SF_SCRATCH_BYTES per
 * device, set up on the first call on that device and held until the
 * process ends) instead of a caller workspace. The plan must come from
 * sf_decode_attn_plan for desc and already sit in device memory at work_dev
 * (the call copies nothing to it); the other arguments are as for
 * sf_decode_attn and sf_decode_attn_combine. The call allocates nothing
 * (no hipMalloc, no hipFree). The stream's device must be the current device.
 * Every call on one device shares that device's array: calls that overlap
 * on one device (other streams, other threads) race and give wrong results.
 * Nothing in the array needs to start at zero: the attention launch writes
 * every partial result the combine launch reads.
 * Errors as sf_decode_attn; SF_ERR_CAPACITY if info->workspace_bytes exceeds
 * SF_SCRATCH_BYTES (plan with fewer workers, e.g. the default options).
 */
#define SF_SCRATCH_BYTES (32ull << 20)
sf_status sf_decode_attn_scratch(const sf_attn_desc* desc, const sf_plan_info* info, const int32_t* work_dev,
                                 const void* q, const void* k_pool, const void* v_pool,
                                 const int32_t* block_table, float* out, float* lse, void* stream);

/*
 * Append, then attend: the decode step of a growing cache. Each step of a
 * batched decode produces one new token per running trajectory (App. B.1),
 * whose key and value join the trajectory's cache before its query attends.
 *
 * Same as sf_decode_attn over the plan's lengths L_s, where for every
 * sequence with L_s >= 1 the newest token (index t = L_s - 1) is not yet in
 * the pool: its key and value are k_new[s][kvh][:] and v_new[s][kvh][:]
 * (bf16 [B][Hkv][D], device). The call also stores them into the pool, at
 * slot t % 16 of page P = new_pages[s] if new_pages is not NULL and
 * new_pages[s] >= 0 (P is then also written to block_table[s][t / 16]),
 * else of page P = block_table[s][t / 16].
 * new_pages: device int32 [B] or NULL; the caller allocates the pages (see
 * sf_page_pool_* and sf_page_table_step) and passes -1 where the token lands
 * in a page the sequence already holds. Sequences with L_s = 0 store nothing.
 * Two launches on the stream: the attention pass over the L_s - 1 cached
 * tokens, then a merge pass that adds the newest token as one more softmax
 * term, merges split sequences and stores the tokens. The call thus also
 * does sf_decode_attn_combine's work: do not call that for this step. lse is
 * required (not NULL): the merge reads it back. The pools and the block
 * table are written, so they must not be read by other work on the device
 * until the call's stream has passed it. Errors as sf_decode_attn, plus
 * SF_ERR_INVALID_ARG for NULL or misaligned (16 bytes) k_new / v_new or a
 * NULL lse.
 */
sf_status sf_decode_attn_append(const sf_attn_desc* desc, const sf_plan_info* info,
                                const int32_t* work_host, int32_t* work_dev, const void* q,
                                const void* k_new, const void* v_new, const int32_t* new_pages,
                                void* k_pool, void* v_pool, int32_t* block_table, float* out,
                                float* lse, void* workspace, uint64_t workspace_bytes, void* stream);

/*
 * Native per-step runner. A rollout instance runs one batched decode step
 * after another (App. B.1), so host work between steps is on the critical
 * path once the kernels are short. sf_runner_step does, in one call: plan
 * (sf_decode_attn_plan with the runner's options) into a pinned, device-
 * mapped host buffer, then on the caller's stream the attention (plain,
 * appending or fp8) and the merge of split sequences, whose kernels read that
 * work list in place (no separate upload). The runner owns a ring of 32 such
 * buffers, the split-K workspace and a few events, one recorded after every
 * 16th step: a buffer is rewritten only after the step that read it has
 * ended, so the host plans ahead while the kernels of earlier steps run. One runner serves one device (the current one at
 * creation) and one caller stream at a time; steps on different streams, or
 * calls that overlap, are not supported.
 */
typedef struct sf_runner sf_runner;

typedef struct sf_runner_extras {
  const void* k_new;             /* appending step (sf_decode_attn_append's arguments) */
  const void* v_new;
  const int32_t* new_pages_host; /* host int32 [num_seqs], copied next to the work list */
  const float* k_scale;          /* fp8 cache (sf_decode_attn_fp8's scales); not with k_new */
  const float* v_scale;
  void* attn_start;              /* optional hipEvent_t: takes the attention kernel's own start time */
  void* attn_end;                /* optional hipEvent_t: takes its end time (before the merge) */
} sf_runner_extras;

/* *runner = a runner for the shape's head counts, head_dim and page size
 * (the per-step fields of shape are ignored); opts may be NULL (defaults).
 * Allocates host and device resources; free with sf_runner_destroy. */
sf_status sf_runner_create(const sf_attn_desc* shape, const sf_plan_opts* opts, sf_runner** runner);
/* Waits for the runner's work to finish, then frees everything it owns. */
void sf_runner_destroy(sf_runner* runner);
/* Sizes the runner's buffers ahead of its steps: the split-K workspace to at
 * least workspace_bytes, and every ring buffer to hold a work list of
 * work_bytes plus an appending step's extras for up to max_num_seqs
 * sequences; workspace_bytes and work_bytes as sf_decode_attn_plan reports
 * them (work_host NULL) for the largest batch the caller will step, with the
 * runner's options. Growing the workspace synchronizes `stream` first (the
 * old one may still be in use); a ring buffer grows after the step that last
 * read it has ended. A step whose plan needs more than the runner holds grows
 * it the same way inside sf_runner_step: a stall in that step, which a
 * reserve beforehand avoids. SF_ERR_INVALID_ARG for a NULL runner or a
 * negative max_num_seqs, SF_ERR_HIP if an allocation fails. */
sf_status sf_runner_reserve(sf_runner* runner, uint64_t workspace_bytes, uint64_t work_bytes,
                            int32_t max_num_seqs, void* stream);
/* One decode step: desc (its head counts, head_dim and page size as at
 * creation), seq_lens_host (host int32 [num_seqs]) and the device tensors as
 * for sf_decode_attn; extras may be NULL. *info (may be NULL) receives the
 * step's plan. lse is required for an appending step. An fp8 step whose
 * runner options leave workers_per_cu at 0 plans 8 workers per CU (two waves
 * per SIMD: its blocks move half the bytes). */
sf_status sf_runner_step(sf_runner* runner, const sf_attn_desc* desc, const int32_t* seq_lens_host,
                         const void* q, const void* k_pool, const void* v_pool, const int32_t* block_table,
                         float* out, float* lse, const sf_runner_extras* extras, void* stream,
                         sf_plan_info* info);

/*
 * fp8 KV cache. The paper lists KV-cache quantization among the
 * optimizations its design is compatible with (Sec. 7); this variant halves
 * the bytes a decode step reads. Keys and values are OCP FP8 E4M3 codes
 * (sign, 4 exponent bits with bias 7, 3 mantissa bits; 0x7F / 0xFF are NaN,
 * the largest finite magnitude is 448), one byte per element: k_pool8 and
 * v_pool8 are [num_pages][Hkv][16*D] bytes, and inside a tile the byte of
 * slot t, dim d sits at
 *   K: ((d/64 * 4 + (d%32)/8) * 16 + t) * 16 + (d/32 % 2) * 8 + d%8
 *   V: ((d/64 * 4 + t/4) * 16 + d%16) * 16 + (d/16 % 4) * 4 + t%4
 * (the gfx950 matrix-core operands of one lane are then 16-byte pieces and
 * each wave load a contiguous 1 KiB). Each (page, KV head) tile has one fp32 scale for
 * K and one for V: k_scale, v_scale [num_pages][Hkv]. The cached key of slot
 * t, dim d is value(code) * k_scale[page][kvh] (values likewise), and the
 * attention is the decode step's over those values.
 *
 * sf_decode_attn_fp8: as sf_decode_attn (same plan, work list and workspace;
 * follow it with sf_decode_attn_combine for split sequences) over an fp8
 * cache. SF_ERR_INVALID_ARG also for NULL scales when num_pages > 0.
 */
sf_status sf_decode_attn_fp8(const sf_attn_desc* desc, const sf_plan_info* info, const int32_t* work_host,
                             int32_t* work_dev, const void* q, const void* k_pool8, const void* v_pool8,
                             const float* k_scale, const float* v_scale, const int32_t* block_table,
                             float* out, float* lse, void* workspace, uint64_t workspace_bytes, void* stream);

/*
 * Quantizes pages of a bf16 cache (bf16 layouts) into an fp8 one (fp8 layouts above).
 * For each listed page p = pages[i] (device int32 [num_pages]) with
 * n = valid_slots[i] valid slots (device int32, 1 .. 16), and every KV head,
 * separately for the K tile and the V tile of the slots 0 .. n-1:
 *   amax = max |x|;  scale = amax / 448;  inv = 448 / amax   (fp32, correctly
 *   rounded; scale = inv = 1 for an all-zero tile)
 *   code = E4M3 round-to-nearest-even of the fp32 product x * inv
 * Slots n .. 15 get code 0. Writes k_pool8, v_pool8, k_scale[p][*] and
 * v_scale[p][*]; other pages are untouched. One launch on the stream. The
 * valid slots must hold finite values.
 */
sf_status sf_kv_quantize_fp8(const sf_attn_desc* desc, const void* k_pool, const void* v_pool,
                             const int32_t* pages, const int32_t* valid_slots, int32_t num_pages,
                             void* k_pool8, void* v_pool8, float* k_scale, float* v_scale, void* stream);

/*
 * Extend (re-prefill) attention. A trajectory interrupted for a model update
 * or migrated to another instance has its KV cache recomputed before its
 * generation resumes (partial rollout and migration, Sec. 2.3; prefill and
 * re-prefill are the second largest share of rollout time, Table
 * "time_breakdown"). Such a pass appends E_s = q_lens[s] new tokens to
 * sequence s, which then holds L_s = seq_lens[s] tokens in the pool: a prefix
 * of P_s = L_s - E_s tokens cached before (0 for a full re-prefill) and the
 * new tokens at positions P_s .. L_s - 1. New token j of sequence s has query
 * row r = cu_s + j, cu_s = E_0 + ... + E_{s-1}, and attends causally:
 *
 *   z_t      = softmax_scale * sum_d q[r,h,d] * K_s[t,d]     t = 0 .. P_s + j
 *   out[r,h] = sum_t exp(z_t) V_s[t] / sum_t exp(z_t)
 *   lse[r,h] = ln sum_t exp(z_t)
 *
 * Layouts: q bf16 [T][Hq][D], out fp32 [T][Hq][D], lse fp32 [T][Hq] (optional),
 * T = sum_s E_s; k_new and v_new bf16 [T][Hkv][D] (the new tokens' keys and
 * values, optional); pools and block table as for a decode step. Block-table
 * entries 0 .. ceil(L_s / 16) - 1 of every sequence with E_s > 0 are read.
 */
typedef struct sf_extend_info {
  int32_t num_items;        /* work items (one 768-thread block each, up to 384 rows) */
  int32_t tokens_per_item;  /* new tokens per item: floor(384 / g) */
  int32_t num_q_rows;       /* T */
  int32_t reserved;         /* 0 */
  uint64_t work_bytes;      /* num_items * 32 */
  uint64_t desc_key;        /* fingerprint of the descriptor */
} sf_extend_info;

/*
 * Builds the extend work list on the host (no device calls).
 *
 * Rule: each sequence's new tokens are cut into blocks of n = floor(384 / g)
 * (the last block shorter), and each (sequence, KV head, block) is one item,
 * whose rows are the block's tokens times the group's g query heads. An item
 * whose block starts at new token t0 with nt tokens reads the keys
 * [0, P_s + t0 + nt), i.e. steps = ceil((P_s + t0 + nt) / 32) blocks of 32
 * keys. Items are ordered by steps, largest first; equal steps keep the
 * order (sequence, KV head, t0) ascending.
 * Work list, int32 rows of 8: seq, kv_head, t0, nt, P_s, cu_s, steps, 0.
 * Lengths must satisfy 0 <= E_s <= L_s <= 16 * block_table_stride.
 * work_host NULL only reports the sizes in *info; SF_ERR_CAPACITY if
 * work_capacity_bytes < info->work_bytes.
 */
sf_status sf_extend_attn_plan(const sf_attn_desc* desc, const int32_t* seq_lens_host,
                              const int32_t* q_lens_host, int32_t* work_host,
                              uint64_t work_capacity_bytes, sf_extend_info* info);

/*
 * Enqueues extend attention on the stream. If work_host is not NULL its
 * info->work_bytes are first copied to work_dev (as for sf_decode_attn). If
 * k_new and v_new are not NULL, a first launch stores every new token's keys
 * and values into the pool, at slot p % 16 of page block_table[s][p / 16]
 * for position p = P_s + j, before the attention reads them; the pools are
 * then written, and the block table must already hold every page the new
 * tokens land in. With both NULL the pool must already hold them. One
 * launch of the attention kernel follows (one 512-thread block per item).
 * Numerics: scores from bf16 q and K with fp32 accumulation; the softmax
 * weights and the values enter the P.V product as fp16, with fp32
 * accumulation. Every bf16 V element of magnitude in [2^-17, 65280] is exact
 * in fp16 and smaller ones round by at most 2^-25; a V element of magnitude
 * 65536 or more at a position a row attends to makes that row's out
 * non-finite. Within that range out and lse meet
 * |err| <= 2e-3 + 1e-2 |exact| (the decode step's bound).
 * Errors as sf_decode_attn; SF_ERR_INVALID_ARG also if only one of k_new and
 * v_new is given, or either is not 16-byte aligned.
 */
sf_status sf_extend_attn(const sf_attn_desc* desc, const sf_extend_info* info, const int32_t* work_host,
                         int32_t* work_dev, const void* q, const void* k_new, const void* v_new,
                         void* k_pool, void* v_pool, const int32_t* block_table, float* out,
                         float* lse, void* stream);

/*
 * Host page allocator for the KV pool. A trajectory's cache grows by one
 * 16-token page at a time and is released when it leaves, within a pool of
 * fixed size (the KV-cache budget of Sec. 5.2). Pages are ids 0 .. N-1 of
 * the pool's first dimension. The free list is last in, first out: a new
 * pool hands out pages in increasing id order, and a released page is handed
 * out again before any page released earlier. Host memory only, no device
 * calls; calls on one pool must not overlap. Every call checks all of its
 * arguments before it changes anything.
 */
typedef struct sf_page_pool sf_page_pool;

/* *pool = a pool of num_pages >= 0 free pages; free with sf_page_pool_destroy. */
sf_status sf_page_pool_create(int32_t num_pages, sf_page_pool** pool);
void sf_page_pool_destroy(sf_page_pool* pool);
/* Free pages, or -1 for a NULL pool. */
int32_t sf_page_pool_available(const sf_page_pool* pool);
/* Marks the n given free pages as in use (e.g. a prompt's pages), keeping the
 * order of the rest. SF_ERR_INVALID_ARG if one is out of range, repeated or
 * already in use. */
sf_status sf_page_pool_claim(sf_page_pool* pool, const int32_t* pages, int32_t n);
/* Takes n pages into pages[0..n) (host), in hand-out order; SF_ERR_CAPACITY
 * if fewer than n are free. */
sf_status sf_page_pool_alloc(sf_page_pool* pool, int32_t n, int32_t* pages);
/* Returns n pages in use, in the given order (the last one is handed out
 * next). SF_ERR_INVALID_ARG if one is out of range, repeated or not in use. */
sf_status sf_page_pool_release(sf_page_pool* pool, const int32_t* pages, int32_t n);

/*
 * Host bookkeeping of one decode step over a growing cache, on a host copy of
 * the block table (int32 [num_seqs][stride]). Moving from lengths prev_lens
 * to lens (host int32 [num_seqs]; 0 for a sequence that is not running):
 *   1. every sequence with prev_lens > 0 and lens == 0 returns its
 *      ceil(prev_lens / 16) pages to the pool (ascending sequence order, each
 *      in block-table order);
 *   2. if appending != 0, every sequence whose newest token (index lens - 1)
 *      opens a page, i.e. lens > 0 and (lens - 1) % 16 == 0, takes one page,
 *      in ascending sequence order, recorded in the block table;
 *   3. new_pages[s] = that page, or -1: the array sf_decode_attn_append takes.
 * Appending steps expect lens = prev_lens + 1 for every running sequence.
 * All or nothing: SF_ERR_INVALID_ARG for a length outside [0, 16 * stride]
 * or a page to return that is not in use, SF_ERR_CAPACITY if the pool cannot
 * supply the pages; nothing changes then.
 */
sf_status sf_page_table_step(sf_page_pool* pool, int32_t* block_table, int32_t stride,
                             int32_t num_seqs, const int32_t* prev_lens, const int32_t* lens,
                             int32_t appending, int32_t* new_pages);

/*
 * Host check of a block table before it is used on the device: the kernels
 * read block-table entries without checking them (a bad page id is an
 * out-of-bounds device read), so a caller holding a host copy can check it
 * first. For every sequence s with seq_lens_host[s] = L > 0 (L <= 0 for a
 * sequence that reads nothing), the entries block_table_host[s][0 ..
 * ceil(L / 16) - 1] must lie in [0, desc->num_pages) and ceil(L / 16) must
 * not exceed desc->block_table_stride. Host memory only, no device calls.
 * Returns SF_OK, or SF_ERR_INVALID_ARG with *bad_seq (may be NULL) = the
 * first sequence that breaks the rule (-1 for a bad descriptor or a NULL
 * array).
 */
sf_status sf_check_block_table(const sf_attn_desc* desc, const int32_t* block_table_host,
                               const int32_t* seq_lens_host, int32_t* bad_seq);

/*
 * Throughput cost model and trajectory routing (host only, no device calls).
 *
 * The paper's coordinator charges a rollout instance's decode step as
 * attention linear in its KV-cache size, plus a matrix-multiplication term
 * that is memory bound for few running trajectories and compute bound for
 * many, plus a constant, and takes throughput as running trajectories over
 * that latency (App. B.1, final throughput equation):
 *   T_i = n / (k1 * kv + max(k2, k3 * n) + k4),  n = num_running (T_i = 0 if n = 0)
 * Routing a trajectory of length l to instance i (Sec. 5.3, marginal gain):
 *   it runs there iff kv + k5 * l <= kv_budget and num_waiting == 0 (then
 *   kv += k5 * l, n += 1), else it waits (num_waiting += 1);
 *   gain = T_i(after) - T_i(before);  ideal gain = 1 / (k1 * k5 * l + max(k2, k3) + k4).
 * kv_cache, kv_budget and k5 * l share one unit (bytes or tokens); k1 is
 * seconds per that unit, k2 and k4 seconds, k3 seconds per trajectory.
 */
typedef struct sf_cost_model {
  double k1, k2, k3, k4;     /* >= 0 */
  double k5;                 /* KV footprint per token, >= 0 */
  double kv_budget;          /* M */
} sf_cost_model;

typedef struct sf_instance_state {  /* one instance of a snapshot */
  int32_t version;           /* model version the instance runs */
  int32_t num_running;       /* |run_trajs| */
  int32_t num_waiting;       /* |wait_trajs| */
  int32_t reserved;          /* 0 */
  double kv_cache;           /* KV-cache size */
} sf_instance_state;

typedef struct sf_trajectory {
  int32_t version;           /* version it was generated with; < 0: initial (none yet) */
  int32_t reserved;          /* 0 */
  double length;             /* tokens, >= 0 */
} sf_trajectory;

/* T_i of one instance; NaN for an invalid model or state. */
double sf_cost_throughput(const sf_cost_model* model, const sf_instance_state* state);
/* Marginal gain of routing a trajectory of this length to the instance; NaN if invalid. */
double sf_cost_marginal_gain(const sf_cost_model* model, const sf_instance_state* state, double length);
/* Gain of routing it to an idle instance; NaN if invalid. */
double sf_cost_ideal_gain(const sf_cost_model* model, double length);

/*
 * Routing strategy (Sec. 5.3; App. D, check-routable and routing algorithms).
 * Trajectories form queues by version, oldest first, initial ones last,
 * arrival order inside a queue. For the head of the current queue:
 *   candidates = instances it may run on: initial trajectories on instances
 *   with version >= min_initial_version (the staleness manager's admission,
 *   given as this bound), others on instances with version >= its version;
 *   no candidate: stop. Candidates are grouped by increasing version; in the
 *   first group whose largest gain (first maximum in instance order) is
 *   >= mu * ideal gain, the trajectory goes to that instance, whose state is
 *   updated as above, and the walk goes on; if no group qualifies: stop.
 * inst (host, in/out): the snapshot, updated with every routed trajectory.
 * target[j] (host, out): instance of trajectory j, or -1 if it stays.
 * *num_routed: trajectories routed. SF_ERR_INVALID_ARG for a bad model (any
 * coefficient negative or not finite), mu not finite, negative counts or
 * lengths, or a NULL pointer where data is expected.
 */
sf_status sf_route(const sf_cost_model* model, double mu, int32_t min_initial_version,
                   sf_instance_state* inst, int32_t num_inst, const sf_trajectory* trajs,
                   int32_t num_trajs, int32_t* target, int32_t* num_routed);

/*
 * Test support: copies the cached keys and values of tokens 0 .. len-1 of
 * (seq, kv_head) through the same address translation the attention kernel
 * uses, into device buffers k_dense and v_dense, bf16 [len][D] token-major.
 */
sf_status sf_debug_gather_kv(const sf_attn_desc* desc, const void* k_pool, const void* v_pool,
                             const int32_t* block_table, int32_t seq, int32_t kv_head,
                             int32_t len, void* k_dense, void* v_dense, void* stream);

/* Measurement support: reads `bytes` of device memory at `buf` once, the way
 * a plain streaming kernel does (`blocks` workgroups of 512 threads, each
 * streaming its own contiguous range; every 16-byte piece loaded once,
 * nontemporal, eight in flight per lane), so that its
 * duration gives the bandwidth an HBM-bound kernel can reach in practice.
 * buf and sink (16 bytes of device memory, written at most once with a
 * meaningless value) must be 16-byte aligned; bytes a multiple of 16;
 * 1 <= blocks <= 65536. bytes == 0 launches nothing. Asynchronous on stream.
 * start_event / stop_event (hipEvent_t, may be NULL) take the kernel's own
 * start and end times, as sf_runner_extras.attn_start / attn_end do.
 * Errors: SF_ERR_INVALID_ARG for the cases above, SF_ERR_HIP on a launch error. */
sf_status sf_debug_stream_read(const void* buf, uint64_t bytes, void* sink, int32_t blocks, void* stream,
                               void* start_event, void* stop_event);

/* Static description of a status code. */
const char* sf_status_string(sf_status status);

/* Library version, (major << 16) | minor. */
int32_t sf_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SF_DECODE_ATTN_H */
