// gfx950 kernels of the paged decode-attention library.
//
// One decode step lets each running trajectory's new query attend over its
// whole cached K/V (App. B.1 of the paper, attention-latency term); the step is
// bound by reading that cache from HBM. A work item is one page-aligned chunk
// of one (sequence, KV head) pair; one wave64 owns one item and walks it two
// pages (32 tokens) at a time:
//
//   S^T[32 tok][16 heads] = K_blk Q^T      2 x (D/32) v_mfma_f32_16x16x32_bf16
//   online softmax in base 2 (wave64 max across the four 16-lane groups)
//   O^T[D][16 heads]     += V_blk^T P^T    (D/16) x 2 MFMAs, P split bf16 hi + lo
//
// The GQA group's g <= 16 query heads fill the 16 MFMA columns (zero padded),
// so K and V bytes are read exactly once per KV head. K page tiles are
// token-major and V page tiles dim-major, so both MFMA A operands are single
// 128-bit global loads straight into registers: no LDS staging is needed.
// The contraction index order inside an MFMA is free as long as both operands
// agree; the kernel assigns tokens to MFMA rows so that each lane's eight
// score values are tokens 8*grp .. 8*grp+7 of the block, which are exactly the
// eight P^T values its PV operand needs and the eight V^T values of one
// contiguous 16-byte load.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sf_internal.h"

namespace sf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994530942f;

// ---------------------------------------------------------------------------
// Block-table address translation, shared by the attention and gather kernels.
// Logical token t of sequence s lives in physical page bt[s][t / 16], slot t % 16.
// ---------------------------------------------------------------------------
__device__ __forceinline__ size_t tile_offset(int32_t page, int32_t num_kv_heads, int32_t kv_head,
                                              int32_t d) {
  return (size_t(page) * num_kv_heads + kv_head) * size_t(kPage * d);
}
__device__ __forceinline__ int k_elem(int slot, int dim, int d) { return slot * d + dim; }
__device__ __forceinline__ int v_elem(int slot, int dim) { return dim * kPage + slot; }

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
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
// nontemporal loads; the next two-page block is fetched while the current one
// is multiplied, which keeps 32 KiB in flight per wave.
__device__ __forceinline__ u32x4 stream16(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

template <int D>
struct KvBlock {
  static constexpr int KB = D / 32;  // QK MFMA steps over the head dimension
  static constexpr int JB = D / 16;  // PV output blocks of 16 dims
  u32x4 k[2][KB];
  u32x4 v[JB];
};

template <int D>
struct ChunkCtx {
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* bt;  // this sequence's block-table row
  int num_kv_heads;
  int kvh;
  int pe;             // end of this chunk (pages)
  int k_page_sel;     // which page of the block this lane's K rows come from
  int k_off;          // element offset of this lane's K row piece inside a tile
  int v_page_sel;
  int v_off;
};

// Loads the two-page block that starts at logical page pg (a single page if
// pg + 1 == pe; the missing page then aliases the first and is masked later).
template <int D>
__device__ __forceinline__ void load_block(const ChunkCtx<D>& c, int pg, KvBlock<D>& b) {
  const int pid0 = c.bt[pg];
  int pid1 = pid0;
  if (pg + 1 < c.pe) pid1 = c.bt[pg + 1];
  const uint16_t* kp = c.k_pool + tile_offset(c.k_page_sel ? pid1 : pid0, c.num_kv_heads, c.kvh, D) + c.k_off;
  const uint16_t* vp = c.v_pool + tile_offset(c.v_page_sel ? pid1 : pid0, c.num_kv_heads, c.kvh, D) + c.v_off;
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int kb = 0; kb < KvBlock<D>::KB; ++kb) b.k[h][kb] = stream16(kp + k_elem(4 * h, kb * 32, D));
#pragma unroll
  for (int jb = 0; jb < KvBlock<D>::JB; ++jb) b.v[jb] = stream16(vp + v_elem(0, 16 * jb));
}

template <int D>
struct SoftmaxState {
  f32x4 o[KvBlock<D>::JB];  // O^T block jb: O[head col][16*jb + 4*grp + i]
  float m;                  // running max of this lane's head, log2 units
  float lsum;               // this lane's share of sum_t 2^(z_t - m)
};

// Scores, online-softmax update and P.V accumulation for one block.
// nvalid = tokens of the block (from its first token) inside the sequence.
template <int D>
__device__ __forceinline__ void consume_block(KvBlock<D>& b, const u32x4* qf, int nvalid, int grp,
                                              float scale_log2, SoftmaxState<D>& st) {
  constexpr int KB = KvBlock<D>::KB;
  constexpr int JB = KvBlock<D>::JB;
  f32x4 s0 = {0.f, 0.f, 0.f, 0.f};
  f32x4 s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) {
    s0 = mfma_bf16(b.k[0][kb], qf[kb], s0);
    s1 = mfma_bf16(b.k[1][kb], qf[kb], s1);
  }
  // This lane now holds head `col`, block tokens 8*grp + e (e < 4 from s0).
  const int tok0 = 8 * grp;
  float sc[8];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    sc[e] = (tok0 + e < nvalid) ? s0[e] * scale_log2 : -__builtin_inff();
    sc[4 + e] = (tok0 + 4 + e < nvalid) ? s1[e] * scale_log2 : -__builtin_inff();
  }
  float mx = fmaxf(fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3])),
                   fmaxf(fmaxf(sc[4], sc[5]), fmaxf(sc[6], sc[7])));
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float mnew = fmaxf(st.m, mx);
  const float alpha = fast_exp2(st.m - mnew);
  st.m = mnew;

  // P^T operand: the lane's eight weights as bf16 hi + lo parts, so the
  // PV product keeps about 16 bits of each weight.
  float ps = 0.f;
  uint32_t hi[4], lo[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float p0 = fast_exp2(sc[2 * w] - mnew);
    const float p1 = fast_exp2(sc[2 * w + 1] - mnew);
    ps += p0 + p1;
    const uint32_t h0 = bf16_bits(p0), h1 = bf16_bits(p1);
    const uint32_t l0 = bf16_bits(p0 - bf16_value(h0)), l1 = bf16_bits(p1 - bf16_value(h1));
    hi[w] = h0 | (h1 << 16);
    lo[w] = l0 | (l1 << 16);
  }
  st.lsum = st.lsum * alpha + ps;
  const u32x4 phi = {hi[0], hi[1], hi[2], hi[3]};
  const u32x4 plo = {lo[0], lo[1], lo[2], lo[3]};

  if (nvalid < 2 * kPage) {
    // Slots past the sequence end may hold anything (even NaN): zero them,
    // since a zero weight times NaN would still be NaN.
    u32x4 mask;
#pragma unroll
    for (int w = 0; w < 4; ++w)
      mask[w] = (tok0 + 2 * w < nvalid ? 0x0000FFFFu : 0u) | (tok0 + 2 * w + 1 < nvalid ? 0xFFFF0000u : 0u);
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) b.v[jb] &= mask;
  }
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) {
    st.o[jb] *= alpha;
    st.o[jb] = mfma_bf16(b.v[jb], phi, st.o[jb]);
    st.o[jb] = mfma_bf16(b.v[jb], plo, st.o[jb]);
  }
}

template <int D>
__global__ __launch_bounds__(64) void attn_chunk_kernel(AttnArgs a) {
  constexpr int KB = KvBlock<D>::KB;
  constexpr int JB = KvBlock<D>::JB;
  const int lane = threadIdx.x;
  const int col = lane & 15;   // MFMA column (query head in group) and A-operand row
  const int grp = lane >> 4;   // MFMA k-group

  const int32_t* item = a.work + size_t(blockIdx.x) * kItemInts;
  const int seq = item[0];
  const int kvh = item[1];
  const int pb = item[2];
  const int pe = item[3];
  const int len = item[4];
  const int slot = item[5];
  const int g = a.group;
  const bool head_ok = col < g;
  const int head = kvh * g + col;

  ChunkCtx<D> c;
  c.k_pool = a.k_pool;
  c.v_pool = a.v_pool;
  c.bt = a.block_table + size_t(seq) * a.bt_stride;
  c.num_kv_heads = a.num_kv_heads;
  c.kvh = kvh;
  c.pe = pe;
  // K operand: A-row r = col holds block token 8*(r/4) + r%4 (+4 for the
  // second MFMA): page r/8 of the block, slot 8*((r/4)%2) + r%4.
  c.k_page_sel = col >> 3;
  c.k_off = k_elem(8 * ((col >> 2) & 1) + (col & 3), grp * 8, D);
  // V operand: A-row = dim 16*jb + col, k-group grp = block tokens 8*grp .. +7.
  c.v_page_sel = grp >> 1;
  c.v_off = v_elem(8 * (grp & 1), col);

  KvBlock<D> blk[2];
  if (pb < pe) load_block(c, pb, blk[0]);

  // Q as the B operand of S^T = K Q^T: column = head, k = 8 dims per group.
  u32x4 qf[KB];
  {
    const uint16_t* qrow = a.q + (size_t(seq) * a.num_q_heads + (head_ok ? head : kvh * g)) * D + grp * 8;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      u32x4 v = load16(qrow + kb * 32);
      qf[kb] = head_ok ? v : u32x4{0u, 0u, 0u, 0u};
    }
  }

  SoftmaxState<D> st;
#pragma unroll
  for (int jb = 0; jb < JB; ++jb) st.o[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -__builtin_inff();
  st.lsum = 0.f;

  // Two register blocks alternate: block i+1 is in flight while block i is used.
  for (int pg = pb; pg < pe; pg += 4) {
    if (pg + 2 < pe) load_block(c, pg + 2, blk[1]);
    consume_block(blk[0], qf, min(len - pg * kPage, pg + 1 < pe ? 2 * kPage : kPage), grp, a.scale_log2, st);
    if (pg + 2 >= pe) break;
    if (pg + 4 < pe) load_block(c, pg + 4, blk[0]);
    consume_block(blk[1], qf, min(len - (pg + 2) * kPage, pg + 3 < pe ? 2 * kPage : kPage), grp,
                  a.scale_log2, st);
  }

  float lt = st.lsum + __shfl_xor(st.lsum, 16);
  lt += __shfl_xor(lt, 32);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  // Lane holds O[head col][16*jb + 4*grp + i], i = 0..3.
  if (slot < 0) {
    if (!head_ok) return;
    float* dst = a.out + (size_t(seq) * a.num_q_heads + head) * D + 4 * grp;
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) *reinterpret_cast<f32x4*>(dst + 16 * jb) = st.o[jb] * inv;
    if (a.lse && grp == 0)
      a.lse[size_t(seq) * a.num_q_heads + head] = lt > 0.f ? (st.m + __log2f(lt)) * kLn2 : -__builtin_inff();
    return;
  }
  if (head_ok) {
    float* dst = a.part_o + (size_t(slot) * g + col) * D + 4 * grp;
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) *reinterpret_cast<f32x4*>(dst + 16 * jb) = st.o[jb] * inv;
    if (grp == 0) a.part_lse[size_t(slot) * g + col] = st.m + __log2f(lt);
  }
}

// ---------------------------------------------------------------------------
// log-sum-exp merge of the chunks of split (sequence, KV head) pairs
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
  const int32_t* it = a.items + size_t(blockIdx.x) * kItemInts;
  const int seq = it[0];
  const int kvh = it[1];
  const int base = it[2];
  const int n = it[3];
  const int g = a.group;
  const int d4n = a.head_dim / 4;
  for (int idx = threadIdx.x; idx < g * d4n; idx += blockDim.x) {
    const int h = idx / d4n;
    const int d4 = idx - h * d4n;
    const float* lse_h = a.part_lse + size_t(base) * g + h;           // stride g per chunk
    const float* o_h = a.part_o + (size_t(base) * g + h) * a.head_dim + 4 * d4;
    const size_t o_stride = size_t(g) * a.head_dim;
    float mx = -__builtin_inff();
#pragma unroll 8
    for (int c = 0; c < n; ++c) mx = fmaxf(mx, lse_h[size_t(c) * g]);
    float wsum = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int c = 0; c < n; ++c) {
      const float w = fast_exp2(lse_h[size_t(c) * g] - mx);
      wsum += w;
      acc += w * *reinterpret_cast<const f32x4*>(o_h + c * o_stride);
    }
    const int head = kvh * g + h;
    *reinterpret_cast<f32x4*>(a.out + (size_t(seq) * a.num_q_heads + head) * a.head_dim + 4 * d4) =
        acc * (1.f / wsum);
    if (a.lse && d4 == 0) a.lse[size_t(seq) * a.num_q_heads + head] = (mx + __log2f(wsum)) * kLn2;
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

hipError_t launch_attention(const AttnArgs& a, hipStream_t stream) {
  if (a.num_work == 0) return hipSuccess;
  const dim3 grid(a.num_work), block(64);
  if (a.head_dim == 128)
    hipLaunchKernelGGL(attn_chunk_kernel<128>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(attn_chunk_kernel<64>, grid, block, 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t stream) {
  if (a.num_items == 0) return hipSuccess;
  hipLaunchKernelGGL(combine_kernel, dim3(a.num_items), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs& a, hipStream_t stream) {
  const int total = a.len * (a.head_dim / 8);
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(gather_kernel, dim3((total + 255) / 256), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace sf
