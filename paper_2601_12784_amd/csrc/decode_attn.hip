// gfx950 kernels of the paged decode-attention library.
//
// One decode step lets each running trajectory's new query attend over its
// whole cached K/V (App. B.1 of the paper, attention-latency term); the step is
// bound by reading that cache from HBM. A work item is one page-aligned
// segment of one (sequence, KV head) pair; one wave64 runs per worker, walks
// its segments in order and each segment two pages (32 tokens) at a time:
//
//   S^T[16 tok][16 heads] = K_page Q^T per page, (D/32) v_mfma_f32_16x16x32_bf16 each
//   online softmax in base 2 (wave64 max across the four 16-lane groups)
//   O^T[D][16 heads]     += V_blk^T P^T    (D/16) x 2 MFMAs, P split bf16 hi + lo
//
// The GQA group's g <= 16 query heads fill the 16 MFMA columns (zero padded),
// so K and V bytes are read exactly once per KV head. The page-tile layouts
// make every MFMA A operand a plain global load straight into registers (no
// LDS staging): a K tile stores, for each group of 8 dims, the 16 tokens'
// 8-dim pieces back to back, so the QK operand of one page (row = token slot,
// k-group = dim group) is one contiguous 1 KiB load per MFMA; a V tile is
// dim-major, so the PV operand (row = dim, k = tokens) is two 8-byte loads,
// 4 tokens from each page of the block. Each lane's eight scores are tokens
// 4*grp .. 4*grp+3 of both pages, exactly the eight P^T values its PV operand
// needs (the contraction order inside an MFMA is free as long as both
// operands agree).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sf_internal.h"

namespace sf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kLog2e = 1.44269504088896340736f;

// ---------------------------------------------------------------------------
// Block-table address translation, shared by the attention and gather kernels.
// Logical token t of sequence s lives in physical page bt[s][t / 16], slot t % 16.
// ---------------------------------------------------------------------------
__device__ __forceinline__ size_t tile_offset(int32_t page, int32_t num_kv_heads, int32_t kv_head,
                                              int32_t d) {
  return (size_t(page) * num_kv_heads + kv_head) * size_t(kPage * d);
}
// K tile: D/8 groups of 8 dims; inside a group the 16 slots' 8-dim pieces are
// consecutive (16 bytes each). V tile: dim-major, 16 slots per dim.
__device__ __forceinline__ int k_elem(int slot, int dim, int d) {
  (void)d;
  return ((dim >> 3) * kPage + slot) * 8 + (dim & 7);
}
__device__ __forceinline__ int v_elem(int slot, int dim) { return dim * kPage + slot; }

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// The work list and the block table are never written while a kernel runs.
// Reading them through the constant address space lets the compiler use
// scalar loads, whose completion is counted apart from the K/V vector loads
// (a vector load of a page id would make the wave wait for every K/V load
// issued before it).
typedef __attribute__((address_space(4))) const int32_t* const_i32_ptr;
__device__ __forceinline__ const_i32_ptr as_constant(const int32_t* p) {
  return (const_i32_ptr)(p);
}

__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ uint32_t bf16_bits(float x) {
  return uint32_t(__builtin_bit_cast(uint16_t, static_cast<__bf16>(x)));
}
__device__ __forceinline__ float bf16_value(uint32_t bits) {
  return __builtin_bit_cast(float, bits << 16);
}

// ---------------------------------------------------------------------------
// attention over one chunk per wave
// ---------------------------------------------------------------------------
// K and V are streamed once and never reused, so they are read with
// nontemporal loads. Each two-page block is fetched in two halves: the next
// block's K is issued before this block's scores are formed and its V before
// this block's P.V product, so 16 loads (16 KiB) stay in flight behind every
// wait while only three half-blocks occupy registers.
__device__ __forceinline__ u32x4 stream16(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

template <int D>
struct Shape {
  static constexpr int KB = D / 32;  // QK MFMA steps over the head dimension
  static constexpr int JB = D / 16;  // PV output blocks of 16 dims
};

template <int D>
struct KHalf {
  u32x4 k[2][Shape<D>::KB];
};

template <int D>
struct VHalf {
  u32x4 v[Shape<D>::JB];
};

template <int D>
struct ChunkCtx {
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const_i32_ptr bt;   // this sequence's block-table row
  int num_kv_heads;
  int kvh;
  int pe;             // end of this segment (pages)
  int k_off;          // element offset of this lane's K piece inside a tile
  int v_off;          // element offset of this lane's V^T piece inside a tile
  int empty_idx;      // appending: logical page that holds only the newest token (-1: none)
};

// Physical pages of the two-page block at logical page pg (a single page if
// pg + 1 == pe; the missing page then aliases the first and is masked later).
struct PagePair {
  int p0, p1;
};
// When appending, the newest token's page may be new in this very step and
// not yet in the block table. This pass leaves that token out, so a page
// that holds only it (the token opened the page) has no slot to read: it is
// replaced by a page already in the table (the one before it, or pool page 0
// for a one-token sequence), whose loads the block's token count masks.
template <int D, bool kAppend>
__device__ __forceinline__ int page_of(const ChunkCtx<D>& c, int pg) {
  if constexpr (kAppend) {
    if (pg == c.empty_idx) return pg > 0 ? c.bt[pg - 1] : 0;
  }
  return c.bt[pg];
}
template <int D, bool kAppend>
__device__ __forceinline__ PagePair block_pages(const ChunkCtx<D>& c, int pg) {
  PagePair pp;
  pp.p0 = page_of<D, kAppend>(c, pg);
  pp.p1 = pp.p0;
  if (pg + 1 < c.pe) pp.p1 = page_of<D, kAppend>(c, pg + 1);
  return pp;
}

// K operand of page h for MFMA step kb: row = token slot col, k-group = dims
// 32*kb + 8*grp .. +8; the wave reads one contiguous 1 KiB per step.
template <int D>
__device__ __forceinline__ void load_k(const ChunkCtx<D>& c, PagePair pp, KHalf<D>& b) {
  const uint16_t* k0 = c.k_pool + tile_offset(pp.p0, c.num_kv_heads, c.kvh, D) + c.k_off;
  const uint16_t* k1 = c.k_pool + tile_offset(pp.p1, c.num_kv_heads, c.kvh, D) + c.k_off;
#pragma unroll
  for (int kb = 0; kb < Shape<D>::KB; ++kb) {
    b.k[0][kb] = stream16(k0 + k_elem(0, 32 * kb, D));
    b.k[1][kb] = stream16(k1 + k_elem(0, 32 * kb, D));
  }
}

// V^T operand for dims 16*jb + col: tokens 4*grp .. +3 of each page (8 bytes
// each); the wave reads 512 contiguous bytes per page and step.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u32x2 stream8(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
}
template <int D>
__device__ __forceinline__ void load_v(const ChunkCtx<D>& c, PagePair pp, VHalf<D>& b) {
  const uint16_t* v0 = c.v_pool + tile_offset(pp.p0, c.num_kv_heads, c.kvh, D) + c.v_off;
  const uint16_t* v1 = c.v_pool + tile_offset(pp.p1, c.num_kv_heads, c.kvh, D) + c.v_off;
#pragma unroll
  for (int jb = 0; jb < Shape<D>::JB; ++jb) {
    const u32x2 x = stream8(v0 + v_elem(0, 16 * jb));
    const u32x2 y = stream8(v1 + v_elem(0, 16 * jb));
    b.v[jb] = u32x4{x[0], x[1], y[0], y[1]};
  }
}

// Block token (counted from the block's first token) of a lane's item e:
// items 0..3 are slots 4*grp + e of the first page, 4..7 of the second.
__device__ __forceinline__ int item_token(int grp, int e) { return (e < 4 ? 0 : kPage - 4) + 4 * grp + e; }

template <int D>
struct SoftmaxState {
  f32x4 o[Shape<D>::JB];  // O^T block jb: O[head col][16*jb + 4*grp + i]
  float m;                // running max of this lane's head, log2 units
  float lsum;             // this lane's share of sum_t 2^(z_t - m)
};

// Weights of one block as the P^T operand (bf16 hi + lo parts, about 16 bits
// of each weight) and the factor that rescales earlier accumulations.
struct BlockWeights {
  u32x4 phi, plo;
  float alpha;
};

// Scores and online-softmax update for one block.
// nvalid = tokens of the block (from its first token) inside the sequence.
// kMayBeEmpty: the block may hold no valid token (then nothing changes);
// without it every block holds at least one, as in a plain decode step.
// Per-page factors of a block for an fp8 cache: the score scale of each page
// (softmax scale * log2(e) * the page's K scale) and each page's V scale.
struct PageScales {
  float c0, c1, v0, v1;
};

template <int D, bool kMayBeEmpty = false, bool kScaled = false>
__device__ __forceinline__ BlockWeights score_block(const KHalf<D>& b, const u32x4* qf, int nvalid, int grp,
                                                    float scale_log2, SoftmaxState<D>& st,
                                                    PageScales scl = PageScales{0.f, 0.f, 0.f, 0.f}) {
  f32x4 s0 = {0.f, 0.f, 0.f, 0.f};
  f32x4 s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < Shape<D>::KB; ++kb) {
    s0 = mfma_bf16(b.k[0][kb], qf[kb], s0);
    s1 = mfma_bf16(b.k[1][kb], qf[kb], s1);
  }
  // This lane now holds head `col`: s0[e] = slot 4*grp + e of the first page,
  // s1[e] = the same slot of the second page.
  float sc[8];
  const float c0 = kScaled ? scl.c0 : scale_log2;
  const float c1 = kScaled ? scl.c1 : scale_log2;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    sc[e] = (item_token(grp, e) < nvalid) ? s0[e] * c0 : -__builtin_inff();
    sc[4 + e] = (item_token(grp, 4 + e) < nvalid) ? s1[e] * c1 : -__builtin_inff();
  }
  float mx = fmaxf(fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3])),
                   fmaxf(fmaxf(sc[4], sc[5]), fmaxf(sc[6], sc[7])));
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float mnew = fmaxf(st.m, mx);
  // With no token seen yet mnew is -inf: subtract 0 instead, so that
  // 2^(-inf - 0) = 0 rather than 2^(-inf + inf).
  const float mref = (kMayBeEmpty && mnew == -__builtin_inff()) ? 0.f : mnew;
  BlockWeights w;
  w.alpha = fast_exp2(st.m - mref);
  st.m = mnew;
  float ps = 0.f;
  uint32_t hi[4], lo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float p0 = fast_exp2(sc[2 * i] - mref);
    float p1 = fast_exp2(sc[2 * i + 1] - mref);
    ps += p0 + p1;
    if constexpr (kScaled) {
      // The P.V operand carries the page's V scale (the weight sum does not).
      const float vs = i < 2 ? scl.v0 : scl.v1;
      p0 *= vs;
      p1 *= vs;
    }
    const uint32_t h0 = bf16_bits(p0), h1 = bf16_bits(p1);
    const uint32_t l0 = bf16_bits(p0 - bf16_value(h0)), l1 = bf16_bits(p1 - bf16_value(h1));
    hi[i] = h0 | (h1 << 16);
    lo[i] = l0 | (l1 << 16);
  }
  st.lsum = st.lsum * w.alpha + ps;
  w.phi = u32x4{hi[0], hi[1], hi[2], hi[3]};
  w.plo = u32x4{lo[0], lo[1], lo[2], lo[3]};
  return w;
}

// P.V accumulation for one block.
template <int D>
__device__ __forceinline__ void accumulate_block(VHalf<D>& b, const BlockWeights& w, int nvalid, int grp,
                                                 SoftmaxState<D>& st) {
  if (nvalid < 2 * kPage) {
    // Slots past the sequence end may hold anything (even NaN): zero them,
    // since a zero weight times NaN would still be NaN.
    u32x4 mask;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      mask[i] = (item_token(grp, 2 * i) < nvalid ? 0x0000FFFFu : 0u) |
                (item_token(grp, 2 * i + 1) < nvalid ? 0xFFFF0000u : 0u);
#pragma unroll
    for (int jb = 0; jb < Shape<D>::JB; ++jb) b.v[jb] &= mask;
  }
#pragma unroll
  for (int jb = 0; jb < Shape<D>::JB; ++jb) {
    st.o[jb] *= w.alpha;
    st.o[jb] = mfma_bf16(b.v[jb], w.phi, st.o[jb]);
    st.o[jb] = mfma_bf16(b.v[jb], w.plo, st.o[jb]);
  }
}

// Stores the newest token of (seq, kvh) into its page slot: lane l < D/8
// writes key dims 8l .. 8l+7 (one 16-byte piece of the K tile), and every
// lane writes the value dims l, l + 64 (two bytes each, 32 bytes apart).
// Nontemporal stores: these scattered small writes, if left as ordinary
// dirty cache lines, slow the next attention pass by several percent.
template <int D>
__device__ __forceinline__ void store_token(uint16_t* k_dst, uint16_t* v_dst, const uint16_t* k_new,
                                            const uint16_t* v_new, int num_kv_heads, int seq, int kvh,
                                            int page, int slot, int lane) {
  const size_t row = (size_t(seq) * num_kv_heads + kvh) * D;
  const size_t tile = tile_offset(page, num_kv_heads, kvh, D);
  if (lane < D / 8)
    __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(k_new + row + 8 * lane),
                                reinterpret_cast<u32x4*>(k_dst + tile + k_elem(slot, 8 * lane, D)));
#pragma unroll
  for (int dim = lane; dim < D; dim += 64)
    __builtin_nontemporal_store(v_new[row + dim], v_dst + tile + v_elem(slot, dim));
}

// The fields of a segment row that the attention pass uses.
// Lane of the calling thread in its wave (a workgroup may hold several waves,
// one worker each).
__device__ __forceinline__ int lane_id() { return int(threadIdx.x) & 63; }

struct Segment {
  int seq, kvh, pb, pe, len, slot;
};

// A worker's segment rows. The worker's table row holds its first item's
// index, its item count and its first segment's fields, so one scalar load
// starts the worker: its first segment's loads go out right after it. The
// other rows come kRowsPerLoad at a time, one vector load each (lane l holds
// int l of the rows), requested behind the loads of the segment before them:
// vector memory completes in issue order, so the work list, read in place
// from pinned host memory, never holds up a K/V block requested before it.
constexpr int kRowsPerLoad = 64 / kItemInts;

__device__ __forceinline__ Segment segment_at(int v, int i) {
  Segment sg;
  sg.seq = __builtin_amdgcn_readlane(v, i * kItemInts + 0);
  sg.kvh = __builtin_amdgcn_readlane(v, i * kItemInts + 1);
  sg.pb = __builtin_amdgcn_readlane(v, i * kItemInts + 2);
  sg.pe = __builtin_amdgcn_readlane(v, i * kItemInts + 3);
  sg.len = __builtin_amdgcn_readlane(v, i * kItemInts + 4);
  sg.slot = __builtin_amdgcn_readlane(v, i * kItemInts + 5);
  return sg;
}

struct WorkerRows {
  int worker;     // this wave's worker: workgroup * waves per workgroup + wave
  int first;      // index of the worker's first item
  int count;      // its items
  Segment head;   // item 0, from the table row
  int v;          // rows of items 1 + kRowsPerLoad * group .. (lane l: int l)
  int group;      // the group v holds, -1 for none
  int copy_val;   // the launch's side job (AttnArgs::copy_*): this lane's int
};

// The side job: this worker's 64 ints of the merge rows, requested once its
// first segment's first loads are out (like the work-list rows) and stored
// after its last result.
__device__ __forceinline__ bool copies_rows(const AttnArgs& a, const WorkerRows& w) {
  return a.copy_dst != nullptr && w.worker * 64 + lane_id() < a.copy_ints;
}

__device__ __forceinline__ void row_copy_load(const AttnArgs& a, WorkerRows& w) {
  if (copies_rows(a, w)) w.copy_val = a.copy_src[w.worker * 64 + lane_id()];
}

__device__ __forceinline__ void row_copy_store(const AttnArgs& a, const WorkerRows& w) {
  if (copies_rows(a, w)) a.copy_dst[w.worker * 64 + lane_id()] = w.copy_val;
}

// The table rows of a workgroup's kWG workers are consecutive: with kWG > 1
// the first wave reads all of them in one vector load (one request of up to
// 256 bytes over PCIe instead of one per worker: at eight workers per CU the
// per-worker reads queued for several microseconds) and shares them through
// LDS. Returns false for a wave past the last worker (the last workgroup may
// be partial); it must then leave without touching anything else.
template <int kWG>
__device__ __forceinline__ bool worker_rows(const AttnArgs& a, int32_t* rows_lds, WorkerRows& w) {
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  w.worker = int(blockIdx.x) * kWG + wave;
  int32_t r[kItemInts];
  if constexpr (kWG == 1) {
    const const_i32_ptr wt = as_constant(a.worker_table) + size_t(w.worker) * kItemInts;
#pragma unroll
    for (int i = 0; i < kItemInts; ++i) r[i] = wt[i];
  } else {
    const int first = int(blockIdx.x) * kWG;
    const int nrows = min(kWG, a.num_workers - first);
    if (int(threadIdx.x) < nrows * kItemInts)
      rows_lds[threadIdx.x] = a.worker_table[size_t(first) * kItemInts + threadIdx.x];
    __syncthreads();
    if (w.worker >= a.num_workers) return false;
#pragma unroll
    for (int i = 0; i < kItemInts; ++i) r[i] = __builtin_amdgcn_readfirstlane(rows_lds[wave * kItemInts + i]);
  }
  w.first = r[0];
  w.count = r[1];
  w.head.seq = r[2];
  w.head.kvh = r[3];
  w.head.pb = r[4];
  w.head.pe = r[5];
  w.head.len = r[6];
  w.head.slot = r[7];
  w.v = 0;
  w.group = -1;
  w.copy_val = 0;
  return true;
}

// Requests the group of rows that holds item i (1 <= i < count), unless held.
__device__ __forceinline__ void request_rows(const AttnArgs& a, WorkerRows& w, int i) {
  if (i < 1 || i >= w.count) return;
  const int group = (i - 1) / kRowsPerLoad;
  if (group == w.group) return;
  const int b = 1 + group * kRowsPerLoad;
  const int n = min(w.count - b, kRowsPerLoad);
  const int32_t* rows = a.items + size_t(w.first + b) * kItemInts;
  const int lane = lane_id();
  w.v = lane < n * kItemInts ? rows[lane] : 0;
  w.group = group;
}

// Item i of the worker (0: the head; else its group must have been requested).
__device__ __forceinline__ Segment worker_item(const WorkerRows& w, int i) {
  return i == 0 ? w.head : segment_at(w.v, (i - 1) % kRowsPerLoad);
}

// Address context of a segment. When appending, the segment that ends the
// sequence leaves the newest token (index len - 1, not yet in the pool) out:
// its pages hold tokens [0, len_pages), and the merge launch that follows
// adds the newest one (its page may be new in this step: the merge launch
// takes it from new_pages and stores the token there).
template <int D, bool kAppend>
__device__ __forceinline__ ChunkCtx<D> segment_ctx(const AttnArgs& a, const Segment& sg, int& len_pages) {
  const int lane = lane_id();
  const int col = lane & 15;
  const int grp = lane >> 4;
  ChunkCtx<D> c;
  c.k_pool = a.k_pool;
  c.v_pool = a.v_pool;
  c.bt = as_constant(a.block_table) + size_t(sg.seq) * a.bt_stride;
  c.num_kv_heads = a.num_kv_heads;
  c.kvh = sg.kvh;
  c.pe = sg.pe;
  // K operand: A-row = token slot col, k-group grp = dims 8*grp .. +8 (+32*kb).
  c.k_off = k_elem(col, 8 * grp, D);
  // V operand: A-row = dim col (+16*jb), k-group grp = slots 4*grp .. +3.
  c.v_off = v_elem(4 * grp, col);
  c.empty_idx = -1;
  len_pages = sg.len;
  if constexpr (kAppend) {
    if (sg.len > 0 && sg.pe == (sg.len + kPage - 1) / kPage) {
      if ((sg.len - 1) % kPage == 0) c.empty_idx = (sg.len - 1) / kPage;
      len_pages = sg.len - 1;
    }
  }
  return c;
}

// Registers a worker's segments share: the two halves that blocks alternate
// between, and the query operand.
template <int D>
struct SegmentRegs {
  KHalf<D> k[2];
  VHalf<D> v[2];
  u32x4 qf[Shape<D>::KB];   // Q as the B operand of S^T = K Q^T: column = head, k = 8 dims per group
};

// First block (into half 0) and query of a segment.
template <int D, bool kAppend>
__device__ __forceinline__ void fetch_segment_start(const AttnArgs& a, const Segment& sg, const ChunkCtx<D>& c,
                                                    SegmentRegs<D>& r) {
  const int lane = lane_id();
  const int col = lane & 15;
  const int grp = lane >> 4;
  const int g = a.group;
  const bool head_ok = col < g;
  if (sg.pb < sg.pe) {
    const PagePair pp = block_pages<D, kAppend>(c, sg.pb);
    load_k(c, pp, r.k[0]);
    load_v(c, pp, r.v[0]);
  }
  const uint16_t* qrow =
      a.q + (size_t(sg.seq) * a.num_q_heads + (head_ok ? sg.kvh * g + col : sg.kvh * g)) * D + grp * 8;
#pragma unroll
  for (int kb = 0; kb < Shape<D>::KB; ++kb) {
    const u32x4 v = load16(qrow + kb * 32);
    r.qf[kb] = head_ok ? v : u32x4{0u, 0u, 0u, 0u};
  }
}

// Stores a segment's result: its normalized output rows o (this lane: head
// col, dims 16*jb + 4*grp .. +3) and l, the lse (natural log) of a pair
// finished here or the log2-unit partial lse of a cut pair's segment.
template <int D>
__device__ __forceinline__ void write_result(const AttnArgs& a, const Segment& sg, const f32x4* o, float l) {
  constexpr int JB = Shape<D>::JB;
  const int lane = lane_id();
  const int col = lane & 15;
  const int grp = lane >> 4;
  const int g = a.group;
  if (col >= g) return;
  if (sg.slot < 0) {
    const int head = sg.kvh * g + col;
    float* dst = a.out + (size_t(sg.seq) * a.num_q_heads + head) * D + 4 * grp;
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) *reinterpret_cast<f32x4*>(dst + 16 * jb) = o[jb];
    if (a.lse && grp == 0) a.lse[size_t(sg.seq) * a.num_q_heads + head] = l;
    return;
  }
  float* dst = a.part_o + (size_t(sg.slot) * g + col) * D + 4 * grp;
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) *reinterpret_cast<f32x4*>(dst + 16 * jb) = o[jb];
  if (grp == 0) a.part_lse[size_t(sg.slot) * g + col] = l;
}

// Stores the result a worker kept in LDS (this lane's values at
// [j * 64 + lane], j < 4 * JB for the output rows, 4 * JB for l).
template <int D>
__device__ __forceinline__ void flush_stash(const AttnArgs& a, const Segment& sg, const float* stash) {
  constexpr int JB = Shape<D>::JB;
  const int lane = lane_id();
  f32x4 o[JB];
#pragma unroll
  for (int jb = 0; jb < JB; ++jb)
#pragma unroll
    for (int i = 0; i < 4; ++i) o[jb][i] = stash[(4 * jb + i) * 64 + lane];
  write_result<D>(a, sg, o, stash[4 * JB * 64 + lane]);
}

// One segment, item `index` of the worker: pages [page_begin, page_end) of
// one (sequence, KV head) pair. primed: its first block and query are already
// in flight (fetched by the previous segment). Once its first loads are out
// it requests the row of the next item; once its last block is done, it
// fetches the next item's first block and query before it stores its own
// result: vector memory operations complete in issue order, so loads issued
// after the stores would wait for the stores' completion too. stash (LDS, or
// NULL): keep the result there instead of storing it (the worker stores it
// last).
template <int D, bool kAppend>
__device__ __forceinline__ void attend_segment(const AttnArgs& a, const Segment& item, WorkerRows& w, int index,
                                               SegmentRegs<D>& r, bool& primed, float* stash) {
  constexpr int JB = Shape<D>::JB;
  const int lane = lane_id();
  const int grp = lane >> 4;   // MFMA k-group

  const int pb = item.pb;
  const int pe = item.pe;
  const int slot = item.slot;

  int len_pages;
  const ChunkCtx<D> c = segment_ctx<D, kAppend>(a, item, len_pages);
  if (!primed) fetch_segment_start<D, kAppend>(a, item, c, r);
  request_rows(a, w, index + 1);
  if (index == 0) row_copy_load(a, w);
  KHalf<D>* kb_ = r.k;
  VHalf<D>* vb_ = r.v;
  const u32x4* qf = r.qf;

  SoftmaxState<D> st;
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) st.o[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -__builtin_inff();
  st.lsum = 0.f;

  // Register halves alternate between even and odd blocks.
  auto step = [&](int pg, KHalf<D>& kc, VHalf<D>& vc, KHalf<D>& kn, VHalf<D>& vn) {
    const bool more = pg + 2 < pe;
    PagePair nxt = {0, 0};
    if (more) {
      nxt = block_pages<D, kAppend>(c, pg + 2);
      load_k(c, nxt, kn);
    }
    // (appending: a last page that holds only the newest token has none,
    // nvalid <= 0, and leaves the state as it was)
    const int nvalid = min(len_pages - pg * kPage, pg + 1 < pe ? 2 * kPage : kPage);
    const BlockWeights w = score_block<D, kAppend>(kc, qf, nvalid, grp, a.scale_log2, st);
    if (more) load_v(c, nxt, vn);
    accumulate_block(vc, w, nvalid, grp, st);
  };
  for (int pg = pb; pg < pe; pg += 4) {
    step(pg, kb_[0], vb_[0], kb_[1], vb_[1]);
    if (pg + 2 >= pe) break;
    step(pg + 2, kb_[1], vb_[1], kb_[0], vb_[0]);
  }

  const bool has_next = index + 1 < w.count;
  const Segment next = worker_item(w, has_next ? index + 1 : index);
  primed = has_next && next.pb < next.pe;
  if (primed) {
    int unused;
    fetch_segment_start<D, kAppend>(a, next, segment_ctx<D, kAppend>(a, next, unused), r);
  }

  float lt = st.lsum + __shfl_xor(st.lsum, 16);
  lt += __shfl_xor(lt, 32);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  // Lane holds O[head col][16*jb + 4*grp + i], i = 0..3.
  f32x4 o[JB];
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) o[jb] = st.o[jb] * inv;
  const float l = slot < 0 ? (lt > 0.f ? (st.m + __log2f(lt)) * kLn2 : -__builtin_inff()) : st.m + __log2f(lt);
  if (stash) {
#pragma unroll
    for (int jb = 0; jb < JB; ++jb)
#pragma unroll
      for (int i = 0; i < 4; ++i) stash[(4 * jb + i) * 64 + lane] = o[jb][i];
    stash[4 * JB * 64 + lane] = l;
    return;
  }
  write_result<D>(a, item, o, l);
}

// One wave per worker: its segments are consecutive in the work list and
// together cover the same number of KV pages as every other worker's.
// Two waves per SIMD (at most 256 registers) keep 2048 workers resident.
// The appending variant reads the newest tokens from k_new / v_new and
// stores nothing: the stores come in the merge launch that follows.
template <int D, bool kAppend, int kWG>
__global__ __launch_bounds__(64 * kWG) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_worker_kernel(AttnArgs a) {
  // A worker's first segment is usually the tail of a pair cut by the
  // previous worker, and short: its result would be written early, into the
  // middle of the launch's read stream, which costs more than its bytes.
  // It waits in LDS and is stored after the worker's last segment.
  __shared__ float stash_all[kWG][(4 * Shape<D>::JB + 1) * 64];
  __shared__ int32_t rows_lds[kWG * kItemInts];
  WorkerRows w;
  if (!worker_rows<kWG>(a, rows_lds, w)) return;
  float* stash = stash_all[w.worker - int(blockIdx.x) * kWG];
  SegmentRegs<D> regs;
  bool primed = false;
  Segment sg = w.head;
  for (int i = 0; i < w.count; ++i) {
    attend_segment<D, kAppend>(a, sg, w, i, regs, primed, i == 0 && w.count > 1 ? stash : nullptr);
    if (i + 1 < w.count) sg = worker_item(w, i + 1);
  }
  if (w.count > 1) flush_stash<D>(a, w.head, stash);
  row_copy_store(a, w);
}

// ---------------------------------------------------------------------------
// attention over an fp8 (OCP E4M3) cache with per-(page, KV head) scales
// ---------------------------------------------------------------------------
// The pools hold one-byte codes in tile layouts made for 16-byte loads (a
// tile is 16*D bytes; byte of slot t, dim d):
//   K: ((d/64 * 4 + (d%32)/8) * 16 + t) * 16 + (d/32 % 2) * 8 + d%8
//   V: ((d/64 * 4 + t/4) * 16 + d%16) * 16 + (d/16 % 4) * 4 + t%4
// so a lane's K operands of two 32-dim steps, and its V operands of four
// 16-dim blocks, are one 16-byte piece, and each wave load is a contiguous
// 1 KiB: a block moves half the bytes of bf16 in a third of the loads. The
// codes are widened to bf16 in registers just before use; every E4M3 value is
// a bf16 value, so this is exact and the MFMAs are the bf16 path's. The page's
// K scale joins the score scale, its V scale the P.V operand: no per-element
// scaling.
template <int D>
struct Shape8 {
  static constexpr int KP = D / 64;   // 16-byte K pieces per page (two MFMA steps each)
  static constexpr int JQ = D / 64;   // 16-byte V pieces per page (four 16-dim blocks each)
};

template <int D>
struct KHalf8 {
  u32x4 k[2][Shape8<D>::KP];   // [page][kp]: codes of dims 64*kp + 8*grp (+32) .. +7 of slot col
  float ks[2];
};

template <int D>
struct VHalf8 {
  u32x4 v[2][Shape8<D>::JQ];   // [page][jq]: word jr = codes of slots 4*grp .. +3, dim 64*jq + 16*jr + col
  float vs[2];
};

// Codes 0, 1 (kHigh false) or 2, 3 (kHigh true) of four packed codes as two bf16.
template <bool kHigh>
__device__ __forceinline__ uint32_t widen2(uint32_t codes4) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(codes4, 1.0f, kHigh));
}

template <int D>
struct ChunkCtx8 {
  const uint8_t* k_pool;
  const uint8_t* v_pool;
  const float* k_scale;
  const float* v_scale;
  const_i32_ptr bt;
  int num_kv_heads;
  int kvh;
  int pe;
  int lane_off;   // byte offset of this lane's 16-byte piece inside a 1 KiB run
};

template <int D>
__device__ __forceinline__ PagePair block_pages8(const ChunkCtx8<D>& c, int pg) {
  PagePair pp;
  pp.p0 = c.bt[pg];
  pp.p1 = pg + 1 < c.pe ? c.bt[pg + 1] : pp.p0;
  return pp;
}

// The scales are never written while a kernel runs: scalar loads.
__device__ __forceinline__ float scale_of(const float* base, int page, int num_kv_heads, int kvh) {
  typedef __attribute__((address_space(4))) const float* const_f32_ptr;
  return ((const_f32_ptr)base)[size_t(page) * num_kv_heads + kvh];
}

template <int D>
__device__ __forceinline__ void load_k8(const ChunkCtx8<D>& c, PagePair pp, KHalf8<D>& b) {
  const uint8_t* k0 = c.k_pool + tile_offset(pp.p0, c.num_kv_heads, c.kvh, D) + c.lane_off;
  const uint8_t* k1 = c.k_pool + tile_offset(pp.p1, c.num_kv_heads, c.kvh, D) + c.lane_off;
#pragma unroll
  for (int kp = 0; kp < Shape8<D>::KP; ++kp) {
    b.k[0][kp] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(k0 + 1024 * kp));
    b.k[1][kp] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(k1 + 1024 * kp));
  }
  b.ks[0] = scale_of(c.k_scale, pp.p0, c.num_kv_heads, c.kvh);
  b.ks[1] = scale_of(c.k_scale, pp.p1, c.num_kv_heads, c.kvh);
}

template <int D>
__device__ __forceinline__ void load_v8(const ChunkCtx8<D>& c, PagePair pp, VHalf8<D>& b) {
  const uint8_t* v0 = c.v_pool + tile_offset(pp.p0, c.num_kv_heads, c.kvh, D) + c.lane_off;
  const uint8_t* v1 = c.v_pool + tile_offset(pp.p1, c.num_kv_heads, c.kvh, D) + c.lane_off;
#pragma unroll
  for (int jq = 0; jq < Shape8<D>::JQ; ++jq) {
    b.v[0][jq] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(v0 + 1024 * jq));
    b.v[1][jq] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(v1 + 1024 * jq));
  }
  b.vs[0] = scale_of(c.v_scale, pp.p0, c.num_kv_heads, c.kvh);
  b.vs[1] = scale_of(c.v_scale, pp.p1, c.num_kv_heads, c.kvh);
}

template <int D>
__device__ __forceinline__ void widen_k(const KHalf8<D>& r, KHalf<D>& b) {
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int kb = 0; kb < Shape<D>::KB; ++kb) {
      const u32x4 w = r.k[h][kb / 2];
      const uint32_t lo = w[2 * (kb % 2)], hi = w[2 * (kb % 2) + 1];
      b.k[h][kb] = u32x4{widen2<false>(lo), widen2<true>(lo), widen2<false>(hi), widen2<true>(hi)};
    }
}

template <int D>
__device__ __forceinline__ void widen_v(const VHalf8<D>& r, VHalf<D>& b) {
#pragma unroll
  for (int jb = 0; jb < Shape<D>::JB; ++jb) {
    const uint32_t p0 = r.v[0][jb / 4][jb % 4], p1 = r.v[1][jb / 4][jb % 4];
    b.v[jb] = u32x4{widen2<false>(p0), widen2<true>(p0), widen2<false>(p1), widen2<true>(p1)};
  }
}

// One segment over an fp8 cache; otherwise as attend_segment.
template <int D, int R>
__device__ __forceinline__ void attend_segment_fp8(const AttnArgs& a, const Segment& item, WorkerRows& w, int index,
                                                   float* stash) {
  constexpr int KB = Shape<D>::KB;
  constexpr int JB = Shape<D>::JB;
  const int lane = lane_id();
  const int col = lane & 15;
  const int grp = lane >> 4;
  const int seq = item.seq;
  const int kvh = item.kvh;
  const int pb = item.pb;
  const int pe = item.pe;
  const int len = item.len;
  const int slot = item.slot;
  const int g = a.group;
  const bool head_ok = col < g;
  const int head = kvh * g + col;

  ChunkCtx8<D> c;
  c.k_pool = reinterpret_cast<const uint8_t*>(a.k_pool);
  c.v_pool = reinterpret_cast<const uint8_t*>(a.v_pool);
  c.k_scale = a.k_scale;
  c.v_scale = a.v_scale;
  c.bt = as_constant(a.block_table) + size_t(seq) * a.bt_stride;
  c.num_kv_heads = a.num_kv_heads;
  c.kvh = kvh;
  c.pe = pe;
  c.lane_off = (grp * kPage + col) * 16;

  // Codes are half the bytes of bf16, so the raw buffers go R blocks deep
  // (R - 1 blocks of loads in flight behind the one being computed).
  KHalf8<D> kr[R];
  VHalf8<D> vr[R];
#pragma unroll
  for (int j = 0; j < R - 1; ++j) {
    if (pb + 2 * j >= pe) break;
    const PagePair pp = block_pages8(c, pb + 2 * j);
    load_k8(c, pp, kr[j]);
    load_v8(c, pp, vr[j]);
  }
  u32x4 qf[KB];
  {
    const uint16_t* qrow = a.q + (size_t(seq) * a.num_q_heads + (head_ok ? head : kvh * g)) * D + grp * 8;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      u32x4 v = load16(qrow + kb * 32);
      qf[kb] = head_ok ? v : u32x4{0u, 0u, 0u, 0u};
    }
  }
  // the next item's row (and the side job), behind this segment's first loads
  request_rows(a, w, index + 1);
  if (index == 0) row_copy_load(a, w);
  SoftmaxState<D> st;
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) st.o[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -__builtin_inff();
  st.lsum = 0.f;

  // Block at pg from (kc, vc); the block R - 1 ahead loads into (kn, vn).
  auto step = [&](int pg, KHalf8<D>& kc, VHalf8<D>& vc, KHalf8<D>& kn, VHalf8<D>& vn) {
    const bool more = pg + 2 * (R - 1) < pe;
    PagePair nxt = {0, 0};
    if (more) {
      nxt = block_pages8(c, pg + 2 * (R - 1));
      load_k8(c, nxt, kn);
    }
    const int nvalid = min(len - pg * kPage, pg + 1 < pe ? 2 * kPage : kPage);
    KHalf<D> kw;
    widen_k(kc, kw);
    const PageScales scl{a.scale_log2 * kc.ks[0], a.scale_log2 * kc.ks[1], vc.vs[0], vc.vs[1]};
    const BlockWeights w = score_block<D, false, true>(kw, qf, nvalid, grp, a.scale_log2, st, scl);
    if (more) load_v8(c, nxt, vn);
    VHalf<D> vw;
    widen_v(vc, vw);
    accumulate_block(vw, w, nvalid, grp, st);
  };
  for (int pg = pb; pg < pe; pg += 2 * R) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (pg + 2 * r >= pe) break;
      step(pg + 2 * r, kr[r], vr[r], kr[(r + R - 1) % R], vr[(r + R - 1) % R]);
    }
  }

  float lt = st.lsum + __shfl_xor(st.lsum, 16);
  lt += __shfl_xor(lt, 32);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  f32x4 o[JB];
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) o[jb] = st.o[jb] * inv;
  const float l = slot < 0 ? (lt > 0.f ? (st.m + __log2f(lt)) * kLn2 : -__builtin_inff()) : st.m + __log2f(lt);
  if (stash) {
#pragma unroll
    for (int jb = 0; jb < JB; ++jb)
#pragma unroll
      for (int i = 0; i < 4; ++i) stash[(4 * jb + i) * 64 + lane] = o[jb][i];
    stash[4 * JB * 64 + lane] = l;
    return;
  }
  write_result<D>(a, item, o, l);
}

template <int D, int kWG>
__global__ __launch_bounds__(64 * kWG) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_worker_fp8_kernel(AttnArgs a) {
  // The worker's first result waits in LDS, as in attn_worker_kernel.
  __shared__ float stash_all[kWG][(4 * Shape<D>::JB + 1) * 64];
  __shared__ int32_t rows_lds[kWG * kItemInts];
  WorkerRows w;
  if (!worker_rows<kWG>(a, rows_lds, w)) return;
  float* stash = stash_all[w.worker - int(blockIdx.x) * kWG];
  Segment sg = w.head;
  for (int i = 0; i < w.count; ++i) {
    attend_segment_fp8<D, 3>(a, sg, w, i, i == 0 && w.count > 1 ? stash : nullptr);
    if (i + 1 < w.count) sg = worker_item(w, i + 1);
  }
  if (w.count > 1) flush_stash<D>(a, w.head, stash);
  row_copy_store(a, w);
}

// ---------------------------------------------------------------------------
// per-page fp8 quantizer
// ---------------------------------------------------------------------------
// One block per listed page: for every KV head, the K tile and then the V
// tile (16 * D bf16 values each) become E4M3 codes with one scale per tile:
//   amax = max |x| over the valid slots;  scale = amax / 448, inv = 448 / amax
//   (correctly rounded; 1 and 1 for an all-zero tile);
//   code = round-to-nearest-even(x * inv), 0 for slots past the valid count.
template <int D>
__global__ __launch_bounds__(256) void quantize_fp8_kernel(QuantArgs a) {
  __shared__ float red[4];
  const int page = as_constant(a.pages)[blockIdx.x];
  const int valid = as_constant(a.valid)[blockIdx.x];
  constexpr int kPieces = kPage * D / 8;   // 8 values per piece
  for (int kvh = 0; kvh < a.num_kv_heads; ++kvh) {
#pragma unroll
    for (int which = 0; which < 2; ++which) {
      const uint16_t* src = (which == 0 ? a.k_src : a.v_src) + tile_offset(page, a.num_kv_heads, kvh, D);
      uint8_t* dst = (which == 0 ? a.k_dst : a.v_dst) + tile_offset(page, a.num_kv_heads, kvh, D);
      float* scale_out = which == 0 ? a.k_scale : a.v_scale;
      // Slot of value e of piece i: K tiles hold 8 dims of one slot per
      // piece; V tiles 8 consecutive slots of one dim.
      auto slot_of = [&](int piece, int e) { return which == 0 ? piece % kPage : (piece * 8 + e) % kPage; };
      float amax = 0.f;
      for (int i = threadIdx.x; i < kPieces; i += 256) {
        const u32x4 x = load16(src + 8 * i);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float v = bf16_value((x[e / 2] >> (16 * (e & 1))) & 0xFFFFu);
          if (slot_of(i, e) < valid) amax = fmaxf(amax, fabsf(v));
        }
      }
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
      if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
      __syncthreads();
      amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
      __syncthreads();
      const float inv = amax > 0.f ? __fdiv_rn(448.f, amax) : 1.f;
      if (threadIdx.x == 0) scale_out[size_t(page) * a.num_kv_heads + kvh] = amax > 0.f ? __fdiv_rn(amax, 448.f) : 1.f;
      for (int i = threadIdx.x; i < kPieces; i += 256) {
        const u32x4 x = load16(src + 8 * i);
        uint32_t w[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          float f[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int idx = 4 * q + e;
            const float v = bf16_value((x[idx / 2] >> (16 * (idx & 1))) & 0xFFFFu);
            f[e] = slot_of(i, idx) < valid ? v * inv : 0.f;
          }
          int packed = __builtin_amdgcn_cvt_pk_fp8_f32(f[0], f[1], 0, false);
          packed = __builtin_amdgcn_cvt_pk_fp8_f32(f[2], f[3], packed, true);
          w[q] = uint32_t(packed);
        }
        if (which == 0) {
          // K piece i: dims d0 .. d0 + 7 of slot t, contiguous in the fp8 layout
          const int t = i % kPage, d0 = 8 * (i / kPage);
          const int off = (((d0 / 64) * 4 + (d0 % 32) / 8) * kPage + t) * 16 + ((d0 / 32) % 2) * 8;
          *reinterpret_cast<u32x2*>(dst + off) = u32x2{w[0], w[1]};
        } else {
          // V piece i: slots t0 .. t0 + 7 of dim d, two runs of four slots
          const int d = i / 2, t0 = 8 * (i % 2);
          const int off = (((d / 64) * 4 + t0 / 4) * kPage + d % 16) * 16 + ((d / 16) % 4) * 4;
          *reinterpret_cast<uint32_t*>(dst + off) = w[0];
          *reinterpret_cast<uint32_t*>(dst + off + kPage * 16) = w[1];
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// log-sum-exp merge of the chunks of split (sequence, KV head) pairs
// ---------------------------------------------------------------------------
// Merges the n partial results of a split pair for head h, dims 4*d4 .. +3:
// one pass in chunk order with a running maximum (log2 units); the loads of
// several chunks are independent and issue together. Returns the maximum,
// the weight sum relative to it and the weighted sum of the partial outputs.
__device__ __forceinline__ void merge_partials(const CombineArgs& a, int base, int n, int h, int d4, float& mx,
                                               float& wsum, f32x4& acc) {
  const int g = a.group;
  const float* lse_h = a.part_lse + size_t(base) * g + h;           // stride g per chunk
  const float* o_h = a.part_o + (size_t(base) * g + h) * a.head_dim + 4 * d4;
  const size_t o_stride = size_t(g) * a.head_dim;
  mx = -__builtin_inff();
  wsum = 0.f;
  acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int c = 0; c < n; ++c) {
    const float l = lse_h[size_t(c) * g];
    const f32x4 o = *reinterpret_cast<const f32x4*>(o_h + c * o_stride);
    const float mnew = fmaxf(mx, l);
    const float keep = fast_exp2(mx - mnew);
    const float w = fast_exp2(l - mnew);
    acc = acc * keep + o * w;
    wsum = wsum * keep + w;
    mx = mnew;
  }
}

__device__ __forceinline__ void merge_row(const CombineArgs& a, int row) {
  const_i32_ptr it = as_constant(a.items) + size_t(row) * kItemInts;
  const int seq = it[0];
  const int kvh = it[1];
  const int base = it[2];
  const int n = it[3];
  const int g = a.group;
  const int d4n = a.head_dim / 4;
  for (int idx = threadIdx.x; idx < g * d4n; idx += blockDim.x) {
    const int h = idx / d4n;
    const int d4 = idx - h * d4n;
    float mx, wsum;
    f32x4 acc;
    merge_partials(a, base, n, h, d4, mx, wsum, acc);
    const int head = kvh * g + h;
    *reinterpret_cast<f32x4*>(a.out + (size_t(seq) * a.num_q_heads + head) * a.head_dim + 4 * d4) =
        acc * (1.f / wsum);
    if (a.lse && d4 == 0) a.lse[size_t(seq) * a.num_q_heads + head] = (mx + __log2f(wsum)) * kLn2;
  }
}

__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) { merge_row(a, blockIdx.x); }

// The merge launch of an appending step. The attention pass left each
// sequence's newest token (index len - 1, not yet in the pool) out; here it
// joins every (sequence, KV head) pair as one more term of the softmax:
//   z = scale * q . k_new (log2 units), and with the pages' result (o, l)
//   M = max(l, z); out = (o 2^(l-M) W + v_new 2^(z-M)) / (W 2^(l-M) + 2^(z-M))
//   lse = M + log2(W 2^(l-M) + 2^(z-M))
// where (o, l, W) is the merged partial sum of a split pair (its weight sum
// W relative to l = its maximum), or out, lse and W = 1 of a pair the
// attention pass finished. Then the token is stored into its page slot, and
// a page newly given to it is recorded in the block table (KV head 0).
// Blocks [0, num_items) take the split pairs' merge rows; the rest take one
// work item each (or one of single_rows, when given), acting on the
// single-segment pairs.
template <int D>
__global__ __launch_bounds__(256) void merge_append_kernel(CombineArgs a) {
  constexpr int kPerThread = (kMaxGroup * (D / 4) + 255) / 256;   // (head, 4 dims) items per thread, at most
  __shared__ float z_new[kMaxGroup];
  const bool split = int(blockIdx.x) < a.num_items;
  const const_i32_ptr rest = a.single_rows ? as_constant(a.single_rows) : as_constant(a.work_items);
  const_i32_ptr row = split ? as_constant(a.items) + size_t(blockIdx.x) * kItemInts
                            : rest + size_t(int(blockIdx.x) - a.num_items) * kItemInts;
  const int seq = row[0];
  const int kvh = row[1];
  const int base = row[2];
  const int n = row[3];
  const int len = row[4];
  if (!split && (row[7] != 1 || len <= 0)) return;   // split pairs come through their merge row
  const int g = a.group;
  const size_t new_row = (size_t(seq) * a.num_kv_heads + kvh) * D;
  const int d4n = D / 4;

  // Everything that depends on the row alone is requested first: the token's
  // page (wave 0 stores the token), and this thread's first-pass result and
  // new value; the score of the newest token and the block barrier follow.
  const int t = len - 1;
  const size_t entry = size_t(seq) * a.bt_stride + t / kPage;
  const int fresh = a.new_pages ? as_constant(a.new_pages)[seq] : -1;
  const int page = fresh >= 0 ? fresh : as_constant(a.block_table)[entry];
  f32x4 acc0[kPerThread];
  float l0[kPerThread];
  u32x2 vv[kPerThread];
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int idx = int(threadIdx.x) + 256 * i;
    acc0[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    l0[i] = 0.f;
    vv[i] = u32x2{0u, 0u};
    if (idx < g * d4n) {
      const int h = idx / d4n;
      const int d4 = idx - h * d4n;
      const size_t orow = size_t(seq) * a.num_q_heads + kvh * g + h;
      if (!split) {
        acc0[i] = *reinterpret_cast<const f32x4*>(a.out + orow * D + 4 * d4);
        l0[i] = a.lse[orow];
      }
      vv[i] = *reinterpret_cast<const u32x2*>(a.v_new + new_row + 4 * d4);
    }
  }

  // z for each query head of the group: 16 lanes per head, 8 dims each.
  {
    const int h = threadIdx.x >> 4;
    const int part = threadIdx.x & 15;
    float acc = 0.f;
    if (h < g && part < D / 8) {
      const u32x4 qv = load16(a.q + (size_t(seq) * a.num_q_heads + kvh * g + h) * D + 8 * part);
      const u32x4 kv = load16(a.k_new + new_row + 8 * part);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc += bf16_value(qv[e] & 0xFFFFu) * bf16_value(kv[e] & 0xFFFFu);
        acc += bf16_value(qv[e] >> 16) * bf16_value(kv[e] >> 16);
      }
    }
    acc += __shfl_xor(acc, 8);
    acc += __shfl_xor(acc, 4);
    acc += __shfl_xor(acc, 2);
    acc += __shfl_xor(acc, 1);
    if (part == 0 && h < g) z_new[h] = acc * a.scale_log2;
  }
  __syncthreads();

#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int idx = int(threadIdx.x) + 256 * i;
    if (idx >= g * d4n) break;
    const int h = idx / d4n;
    const int d4 = idx - h * d4n;
    const int head = kvh * g + h;
    float* out = a.out + (size_t(seq) * a.num_q_heads + head) * D + 4 * d4;
    float mx, wsum;
    f32x4 acc;
    if (split) {
      merge_partials(a, base, n, h, d4, mx, wsum, acc);
    } else {
      acc = acc0[i];
      mx = l0[i] * kLog2e;   // -inf if the pages held no token
      wsum = 1.f;
    }
    const f32x4 v = {bf16_value(vv[i][0] & 0xFFFFu), bf16_value(vv[i][0] >> 16), bf16_value(vv[i][1] & 0xFFFFu),
                     bf16_value(vv[i][1] >> 16)};
    const float z = z_new[h];
    const float m = fmaxf(mx, z);
    const float a1 = fast_exp2(mx - m);
    const float a2 = fast_exp2(z - m);
    const float den = wsum * a1 + a2;
    *reinterpret_cast<f32x4*>(out) = (acc * a1 + v * a2) * (1.f / den);
    if (d4 == 0) a.lse[size_t(seq) * a.num_q_heads + head] = (m + __log2f(den)) * kLn2;
  }

  if (threadIdx.x < 64) {
    const int lane = lane_id();
    store_token<D>(a.k_dst, a.v_dst, a.k_new, a.v_new, a.num_kv_heads, seq, kvh, page, t % kPage, lane);
    if (fresh >= 0 && kvh == 0 && lane == 0) a.bt_dst[entry] = fresh;
  }
}

// ---------------------------------------------------------------------------
// test support: dense copy of one (sequence, KV head) through the same translation
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gather_kernel(GatherArgs a) {
  const int d = a.head_dim;
  const int chunks = d / 8;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= a.len * chunks) return;
  const int t = idx / chunks;
  const int c = idx - t * chunks;
  const int32_t page = a.block_table[size_t(a.seq) * a.bt_stride + t / kPage];
  const int s = t % kPage;
  const uint16_t* kt = a.k_pool + tile_offset(page, a.num_kv_heads, a.kv_head, d);
  const uint16_t* vt = a.v_pool + tile_offset(page, a.num_kv_heads, a.kv_head, d);
  *reinterpret_cast<u32x4*>(a.k_dense + size_t(t) * d + c * 8) = load16(kt + k_elem(s, c * 8, d));
#pragma unroll
  for (int e = 0; e < 8; ++e) a.v_dense[size_t(t) * d + c * 8 + e] = vt[v_elem(s, c * 8 + e)];
}

}  // namespace

// Waves (workers) per workgroup, as the plan chose it: the kernels run two
// waves per SIMD at most, so a plan with 8, 4 or 2 workers per CU (or a
// multiple) packs that many into each workgroup, which then share one read
// of their table rows; other plans keep one worker per workgroup, spread
// over every CU. Workgroup b holds workers G b .. G b + G - 1 and runs on
// XCD b mod 8.
template <int kWG>
void (*pick_attention(const AttnArgs& a))(AttnArgs) {
  if (a.k_scale) return a.head_dim == 128 ? attn_worker_fp8_kernel<128, kWG> : attn_worker_fp8_kernel<64, kWG>;
  if (a.k_new) return a.head_dim == 128 ? attn_worker_kernel<128, true, kWG> : attn_worker_kernel<64, true, kWG>;
  return a.head_dim == 128 ? attn_worker_kernel<128, false, kWG> : attn_worker_kernel<64, false, kWG>;
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
  if (a.num_workers == 0) return hipSuccess;
  const int per_group = a.workers_per_group;   // 1, 2, 4 or 8 (checked with the plan)
  const dim3 grid((a.num_workers + per_group - 1) / per_group), block(64 * per_group);
  void (*kernel)(AttnArgs) = per_group == 8   ? pick_attention<8>(a)
                             : per_group == 4 ? pick_attention<4>(a)
                             : per_group == 2 ? pick_attention<2>(a)
                                              : pick_attention<1>(a);
  if (start || stop)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, start, stop, 0, a);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t stream) {
  if (a.k_new) {
    const int blocks = a.num_items + (a.single_rows ? a.num_single : a.num_work);
    if (blocks == 0) return hipSuccess;
    if (a.head_dim == 128)
      hipLaunchKernelGGL(merge_append_kernel<128>, dim3(blocks), dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL(merge_append_kernel<64>, dim3(blocks), dim3(256), 0, stream, a);
    return hipGetLastError();
  }
  if (a.num_items == 0) return hipSuccess;
  hipLaunchKernelGGL(combine_kernel, dim3(a.num_items), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_quantize_fp8(const QuantArgs& a, hipStream_t stream) {
  if (a.num_pages == 0) return hipSuccess;
  if (a.head_dim == 128)
    hipLaunchKernelGGL(quantize_fp8_kernel<128>, dim3(a.num_pages), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(quantize_fp8_kernel<64>, dim3(a.num_pages), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs& a, hipStream_t stream) {
  const int total = a.len * (a.head_dim / 8);
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(gather_kernel, dim3((total + 255) / 256), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace sf
