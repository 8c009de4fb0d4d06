// Native per-step runner: plan -> attention (-> merge) in one call.
//
// A rollout instance runs one batched decode step after another (App. B.1:
// each step generates one token per running trajectory), so the host work
// between two steps is on the critical path once the kernels are short:
// small batches, late steps of a long-tail batch, an fp8 cache. This object
// keeps that work native. It owns a ring of pinned host buffers that the
// planner writes into and the kernels read in place (mapped host memory,
// zero-copy), the split-K workspace, and a few events:
//   - a slot is rewritten only after the step that read it has ended;
//   - nothing else orders the steps, so the host plans step i + 1 while the
//     kernels of step i run.
// An event recorded on the stream after every step delayed the next step's
// first launch by ~4.4 us (the marker's own dispatch; 2 % of a long-tail
// step), so one event marks a run of kMarkEvery steps on one stream instead;
// the ring holds kRing > kMarkEvery slots, so the run that holds a slot's
// last step is always marked before the slot comes round again.
// A separate upload (a copy stream, a device work list and a cross-stream
// wait) cost more per step than the kernels' in-place reads of the list, and
// how much more depended on whether the two streams shared a hardware queue.
#include <hip/hip_runtime.h>

#include <cstring>
#include <new>

#include "sf_internal.h"

static_assert(sizeof(sf_runner_extras) == 56, "sf_runner_extras layout is part of the ABI");

namespace {

constexpr int kRing = 32;
constexpr int kMarkEvery = 16;
constexpr int kMarks = 4;
constexpr int kFp8WorkersPerCu = 8;
static_assert(kMarkEvery < kRing, "a slot's last step must be marked before the slot comes round again");

struct Pinned {
  int32_t* ptr = nullptr;          // host address (the planner writes here)
  const int32_t* dev = nullptr;    // the same memory as the kernels address it
  uint64_t bytes = 0;
  uint64_t last_step = 0;          // the step that last read it
  bool used = false;
};

// An event recorded on one stream after steps [begin, end), all on that stream.
struct Mark {
  hipEvent_t ev = nullptr;
  uint64_t begin = 0, end = 0;
  bool valid = false;
};

}  // namespace

struct sf_runner {
  sf_attn_desc shape;      // heads, head_dim, page size (per-step fields are overwritten)
  sf_plan_opts opts;
  int device = 0;
  Pinned ring[kRing];
  Mark marks[kMarks];
  uint64_t num_marks = 0;  // marks recorded so far (the next one reuses marks[num_marks % kMarks])
  uint64_t unmarked = 0;   // steps [unmarked, steps) have no mark yet
  hipStream_t last_stream = nullptr;
  void* workspace = nullptr;
  uint64_t workspace_bytes = 0;
  uint64_t steps = 0;
  sf_plan_info last;
};

namespace {

// Records a mark after the unmarked steps, on the stream they ran on. The
// mark it reuses is waited for first, so a recycled event never stands for
// steps of another run.
sf_status mark_steps(sf_runner* r) {
  if (r->unmarked == r->steps) return SF_OK;
  Mark& m = r->marks[r->num_marks % kMarks];
  if (m.valid && hipEventSynchronize(m.ev) != hipSuccess) return SF_ERR_HIP;
  m.valid = false;
  if (hipEventRecord(m.ev, r->last_stream) != hipSuccess) return SF_ERR_HIP;
  m.begin = r->unmarked;
  m.end = r->steps;
  m.valid = true;
  r->unmarked = r->steps;
  ++r->num_marks;
  return SF_OK;
}

// Returns once step u (< steps) has ended on the GPU.
sf_status wait_step(sf_runner* r, uint64_t u) {
  if (u >= r->unmarked) {
    sf_status st = mark_steps(r);
    if (st != SF_OK) return st;
  }
  for (auto& m : r->marks)
    if (m.valid && m.begin <= u && u < m.end) return hipEventSynchronize(m.ev) == hipSuccess ? SF_OK : SF_ERR_HIP;
  return SF_OK;  // its mark was waited for and reused: the step has ended
}

// Returns once every step so far has ended.
sf_status wait_all(sf_runner* r) {
  sf_status st = mark_steps(r);
  for (auto& m : r->marks)
    if (m.valid && hipEventSynchronize(m.ev) != hipSuccess) st = SF_ERR_HIP;
  return st;
}

// Called only when no step in flight reads the slot (its last step has ended).
sf_status grow_pinned(Pinned& p, uint64_t bytes) {
  if (p.bytes >= bytes) return SF_OK;
  if (p.ptr && hipHostFree(p.ptr) != hipSuccess) return SF_ERR_HIP;
  p.ptr = nullptr;
  p.dev = nullptr;
  p.bytes = 0;
  const uint64_t want = bytes + bytes / 4 + 4096;
  if (hipHostMalloc(reinterpret_cast<void**>(&p.ptr), want, hipHostMallocDefault) != hipSuccess) return SF_ERR_HIP;
  void* dev = nullptr;
  if (hipHostGetDevicePointer(&dev, p.ptr, 0) != hipSuccess) {
    (void)hipHostFree(p.ptr);
    p.ptr = nullptr;
    return SF_ERR_HIP;
  }
  p.dev = static_cast<const int32_t*>(dev);
  p.bytes = want;
  return SF_OK;
}

// The workspace grows only when nothing in flight can still use it: growing
// waits for the runner's steps and the stream (sf_runner_reserve does it
// ahead of the steps).
sf_status grow_device(sf_runner* r, void** ptr, uint64_t* have, uint64_t bytes, hipStream_t main) {
  if (*have >= bytes) return SF_OK;
  sf_status st = wait_all(r);
  if (st != SF_OK) return st;
  if (hipStreamSynchronize(main) != hipSuccess) return SF_ERR_HIP;
  if (*ptr && hipFree(*ptr) != hipSuccess) return SF_ERR_HIP;
  *ptr = nullptr;
  *have = 0;
  const uint64_t want = bytes + bytes / 4 + 4096;
  if (hipMalloc(ptr, want) != hipSuccess) return SF_ERR_HIP;
  *have = want;
  return SF_OK;
}

}  // namespace

extern "C" sf_status sf_runner_create(const sf_attn_desc* shape, const sf_plan_opts* opts, sf_runner** out) {
  if (!out) return SF_ERR_INVALID_ARG;
  *out = nullptr;
  if (!shape) return SF_ERR_INVALID_ARG;
  sf_attn_desc probe = *shape;
  probe.num_seqs = 0;
  probe.block_table_stride = probe.block_table_stride > 0 ? probe.block_table_stride : 1;
  probe.num_pages = probe.num_pages >= 0 ? probe.num_pages : 0;
  sf_status st = sf::validate_desc(&probe);
  if (st != SF_OK) return st;
  if (opts && (opts->xcd_parity_skew < -sf::kMaxParitySkew || opts->xcd_parity_skew > sf::kMaxParitySkew))
    return SF_ERR_INVALID_ARG;
  sf_runner* r = new (std::nothrow) sf_runner();
  if (!r) return SF_ERR_HIP;
  r->shape = probe;
  if (opts) r->opts = *opts;
  else std::memset(&r->opts, 0, sizeof r->opts);
  if (hipGetDevice(&r->device) != hipSuccess) {
    delete r;
    return SF_ERR_HIP;
  }
  // The events only order the host's reuse of a slot after the GPU's reads
  // of it; they publish no GPU writes, so they skip the system-scope fence.
  for (auto& m : r->marks)
    if (hipEventCreateWithFlags(&m.ev, hipEventDisableTiming | hipEventDisableSystemFence) != hipSuccess)
      st = SF_ERR_HIP;
  if (st != SF_OK) {
    sf_runner_destroy(r);
    return st;
  }
  *out = r;
  return SF_OK;
}

// Teardown cannot report errors: every call is made, whatever the others return.
extern "C" void sf_runner_destroy(sf_runner* r) {
  if (!r) return;
  // Steps not yet marked ran on the caller's stream, which may be gone by
  // now: nothing is recorded on it here, the device is waited for instead.
  if (r->unmarked < r->steps) (void)hipDeviceSynchronize();
  for (auto& m : r->marks) {
    if (m.ev && m.valid) (void)hipEventSynchronize(m.ev);
    if (m.ev) (void)hipEventDestroy(m.ev);
  }
  for (auto& p : r->ring)
    if (p.ptr) (void)hipHostFree(p.ptr);
  if (r->workspace) {
    (void)hipDeviceSynchronize();
    (void)hipFree(r->workspace);
  }
  delete r;
}

extern "C" sf_status sf_runner_step(sf_runner* r, const sf_attn_desc* desc, const int32_t* seq_lens_host,
                                    const void* q, const void* k_pool, const void* v_pool,
                                    const int32_t* block_table, float* out, float* lse,
                                    const sf_runner_extras* extras, void* stream, sf_plan_info* info_out) {
  if (!r || !desc || (desc->num_seqs > 0 && !seq_lens_host)) return SF_ERR_INVALID_ARG;
  if (desc->num_q_heads != r->shape.num_q_heads || desc->num_kv_heads != r->shape.num_kv_heads ||
      desc->head_dim != r->shape.head_dim || desc->page_size != r->shape.page_size)
    return SF_ERR_INVALID_ARG;
  const bool append = extras && extras->k_new;
  const bool fp8 = extras && extras->k_scale;
  if (extras && (append && fp8)) return SF_ERR_INVALID_ARG;
  if (append && !lse) return SF_ERR_INVALID_ARG;
  hipStream_t main = static_cast<hipStream_t>(stream);

  // 1. plan into the next ring slot (after the step that last read it has
  //    ended); grow it and plan again only if the plan does not fit
  Pinned& pin = r->ring[r->steps % kRing];
  sf_status st = pin.used ? wait_step(r, pin.last_step) : SF_OK;
  if (st != SF_OK) return st;
  pin.used = false;
  // A mark stands for steps of one stream: a new stream closes the run.
  if (r->unmarked < r->steps && main != r->last_stream && (st = mark_steps(r)) != SF_OK) return st;
  // Appending: after the work list, copies of the rows the merge launch acts
  // on (pairs with one segment and len > 0, at most one per item), then
  // new_pages. The work list ends with the combine rows, so the merge
  // launch's rows are one contiguous range, which the attention launch
  // copies to device memory (RowCopy).
  const uint64_t pages_bytes = append ? (uint64_t(desc->num_seqs) * 4 + 31) / 32 * 32 : 0;
  // An fp8 block moves half the bytes of a bf16 one: unless the caller chose,
  // fp8 steps plan two waves per SIMD (measured: kernel 129 us instead of 136
  // on the long-tail batch; bf16 is slower at 8).
  sf_plan_opts opts = r->opts;
  if (fp8 && opts.workers_per_cu == 0) opts.workers_per_cu = kFp8WorkersPerCu;
  sf_plan_info info;
  st = sf_decode_attn_plan(desc, seq_lens_host, &opts, pin.ptr, pin.bytes, &info);
  auto need = [&]() { return info.work_bytes + (append ? uint64_t(info.num_work) * 32 + pages_bytes : 0); };
  if (st == SF_ERR_CAPACITY || (st == SF_OK && pin.bytes < need())) {
    if ((st = grow_pinned(pin, need())) != SF_OK) return st;
    st = sf_decode_attn_plan(desc, seq_lens_host, &opts, pin.ptr, pin.bytes, &info);
  }
  if (st != SF_OK) return st;
  int32_t num_single = 0;
  uint64_t pages_off = info.work_bytes;
  if (append && desc->num_seqs > 0) {
    if (!extras->new_pages_host) return SF_ERR_INVALID_ARG;
    char* base = reinterpret_cast<char*>(pin.ptr);
    const int32_t* items = pin.ptr + sf::table_rows(info.num_workers) * sf::kItemInts;
    int32_t* singles = reinterpret_cast<int32_t*>(base + info.work_bytes);
    for (int32_t i = 0; i < info.num_work; ++i) {
      const int32_t* row = items + int64_t(i) * sf::kItemInts;
      if (row[7] == 1 && row[4] > 0)
        std::memcpy(singles + int64_t(num_single++) * sf::kItemInts, row, sf::kItemInts * 4);
    }
    pages_off = info.work_bytes + uint64_t(num_single) * 32;
    std::memcpy(base + pages_off, extras->new_pages_host, uint64_t(desc->num_seqs) * 4);
  }
  if (info_out) *info_out = info;
  r->last = info;
  if (info.num_workers == 0) return SF_OK;

  // 2. workspace (grown only while idle): the partial results, then the
  //    device copy of what the merge launch reads from the ring: the combine
  //    rows and, appending, the single rows and new_pages (contiguous there)
  const uint64_t rows_off = sf::align256(info.workspace_bytes);
  const int64_t rows_ints = (int64_t(info.num_combine) + (append ? num_single : 0)) * sf::kItemInts;
  const int64_t copy_ints = rows_ints + (append && desc->num_seqs > 0 ? int64_t(pages_bytes / 4) : 0);
  if ((st = grow_device(r, &r->workspace, &r->workspace_bytes, rows_off + uint64_t(copy_ints) * 4, main)) != SF_OK)
    return st;
  int32_t* work = const_cast<int32_t*>(pin.dev);
  const sf::RowCopy copy = {work + (sf::table_rows(info.num_workers) + info.num_work) * sf::kItemInts,
                            reinterpret_cast<int32_t*>(static_cast<char*>(r->workspace) + rows_off),
                            int32_t(copy_ints), append ? int32_t(info.num_combine) * sf::kItemInts : -1,
                            append && desc->num_seqs > 0 ? int32_t(rows_ints) : -1};
  const sf::RowCopy* cp = copy_ints > 0 ? &copy : nullptr;

  // 3. kernels on the caller's stream (the caller's events, if any, take the
  //    attention kernel's own start and end times)
  void* ev0 = extras ? extras->attn_start : nullptr;
  void* ev1 = extras ? extras->attn_end : nullptr;
  // From here on a launch may have been enqueued that reads the slot, so the
  // step counts (and is marked in its turn) whatever the launches return.
  if (append) {
    const char* wbase = reinterpret_cast<const char*>(work);
    st = sf::decode_attn_append_rows(desc, &info, work, q, extras->k_new, extras->v_new,
                                     reinterpret_cast<const int32_t*>(wbase + pages_off),
                                     reinterpret_cast<const int32_t*>(wbase + info.work_bytes), num_single,
                                     const_cast<void*>(k_pool), const_cast<void*>(v_pool),
                                     const_cast<int32_t*>(block_table), out, lse, r->workspace,
                                     r->workspace_bytes, stream, cp, ev0, ev1);
  } else {
    st = sf::decode_attn_rows(desc, &info, work, q, k_pool, v_pool, fp8 ? extras->k_scale : nullptr,
                              fp8 ? extras->v_scale : nullptr, block_table, out, lse, r->workspace,
                              r->workspace_bytes, stream, cp, ev0, ev1);
  }
  pin.used = true;
  pin.last_step = r->steps;
  r->last_stream = main;
  ++r->steps;
  if (r->steps - r->unmarked >= kMarkEvery && mark_steps(r) != SF_OK) {
    // Without the mark nothing orders a later rewrite of these slots after
    // the steps' reads: wait for the stream instead.
    (void)hipStreamSynchronize(main);
    for (auto& p : r->ring) p.used = false;
    r->unmarked = r->steps;
    if (st == SF_OK) st = SF_ERR_HIP;
  }
  return st;
}

extern "C" sf_status sf_runner_reserve(sf_runner* r, uint64_t workspace_bytes, uint64_t work_bytes,
                                       int32_t max_num_seqs, void* stream) {
  if (!r || max_num_seqs < 0) return SF_ERR_INVALID_ARG;
  hipStream_t main = static_cast<hipStream_t>(stream);
  // partials, then the device copy of the merge rows (at most the work
  // list's size) and new_pages
  sf_status st = grow_device(r, &r->workspace, &r->workspace_bytes,
                             sf::align256(workspace_bytes) + work_bytes + (uint64_t(max_num_seqs) * 4 + 31) / 32 * 32,
                             main);
  if (st != SF_OK) return st;
  // An appending step also keeps its new-page array (padded to 32 bytes) and
  // copies of at most one 32-byte row per row of the work list in the slot.
  const uint64_t pages = (uint64_t(max_num_seqs) * 4 + 31) / 32 * 32;
  const uint64_t slot = work_bytes + pages + work_bytes;
  for (auto& p : r->ring) {
    if (p.bytes >= slot) continue;
    if (p.used && (st = wait_step(r, p.last_step)) != SF_OK) return st;
    p.used = false;
    if ((st = grow_pinned(p, slot)) != SF_OK) return st;
  }
  return SF_OK;
}
