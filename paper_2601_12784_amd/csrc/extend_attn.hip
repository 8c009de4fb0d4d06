// gfx950 kernels for extend (re-prefill) attention over the paged KV cache.
//
// A trajectory resumed on an instance after an interrupt or a migration has
// its KV cache recomputed before decoding goes on (partial rollout and
// migration, Sec. 2.3; the prefill share of rollout time is in Table
// "time_breakdown"). Such a pass appends E new tokens to a sequence whose
// cache already holds P tokens (P = 0 for a full re-prefill); new token j, at
// position P + j, attends causally to positions 0 .. P + j.
//
// Unlike a decode step this is a dense contraction: every key tile is used by
// all new tokens after it, so the work runs on the matrix cores. A work item
// is one (sequence, KV head, block of new tokens); its rows are the block's
// tokens times the g query heads of the group (token-major), at most 384 rows,
// 32 per wave (12 waves, three per SIMD). The item walks the keys in steps of
// 32 (two pages), one step per barrier: eight of the waves stage the K and V
// tiles of the next step (16 KiB at D = 128) through LDS, double buffered, and
// each wave computes, per step and 16-row tile,
//
//   S^T[32 keys][16 rows] = K Q^T        2 x (D/32) v_mfma_f32_16x16x32_bf16
//   online softmax in base 2             (row = lane column; lazily moved reference)
//   O^T[D][16 rows]      += V^T P^T      (D/16) v_mfma_f32_16x16x32_f16
//
// with each K and V operand read from LDS once per wave, just before the
// MFMAs of both row tiles that use it. Three waves per SIMD (168 registers
// each) hide the latencies that a wave's own schedule would otherwise have
// to: with two waves per SIMD and the row tiles software-pipelined inside
// each wave the same work took 17 % longer. The operand mapping is the
// decode kernel's: each lane's eight scores are keys 4*grp .. 4*grp+3 of
// both pages, the eight P^T values its P.V operand needs.
//
// The P.V product runs on fp16 operands. The weights P are rounded to fp16
// (relative error 2^-11) instead of bf16 (2^-8): with bf16 weights a row
// with a few comparable keys and values of opposite sign can miss the
// 2e-3 + 1e-2 |ref| acceptance bound, with fp16 weights it stays an order
// of magnitude inside it. V is widened from bf16 to fp16 once, while it is
// staged into LDS; that is exact for every bf16 value of magnitude in
// [2^-17, 65280], rounds smaller ones by at most 2^-25, and turns values of
// magnitude 65536 and above into infinities (fp16's range; the header
// states the limit).
//
// Measured alternatives (full re-prefill of 32 long-tail trajectories):
// 64 rows per wave (4 waves, one per SIMD) halves the LDS operand reads but
// leaves no second wave per SIMD to overlap with, and is 1.5x slower; items
// of 128 rows double the K/V staging per row and are 2x slower; 16 rows per
// wave (16 waves, four per SIMD) doubles the LDS operand reads per row and
// is 12 % slower than three waves of 32 rows.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "sf_internal.h"

namespace sf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(4))) const int32_t* const_i32_ptr;

constexpr float kLn2 = 0.69314718055994530942f;
constexpr int kWaves = 12;
constexpr int kStageWaves = 8;    // waves that stage K and V (the other four only compute)
constexpr int kThreads = 64 * kWaves;
constexpr int kRowTiles = 2;      // 16-row MFMA tiles per wave
constexpr int kStepKeys = 2 * kPage;   // keys per step (two pages)
constexpr int kSub = 1;                // steps per barrier interval
constexpr float kRescaleMax = 32768.f; // headroom of the lazily moved softmax reference, 2^15 (fp16 weights)
static_assert(kWaves * kRowTiles * 16 == kExtendRows, "rows per item");

__device__ __forceinline__ const_i32_ptr as_constant(const int32_t* p) { return (const_i32_ptr)(p); }

__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma_f16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                0, 0);
}

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
// Two floats to two fp16 (round to nearest even) in one conversion.
__device__ __forceinline__ uint32_t pack_f16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, f16x2));
}
// Two bf16 (one 32-bit word) to two fp16: widen to fp32 (exact), then round.
__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t w) {
  return pack_f16(__builtin_bit_cast(float, w << 16), __builtin_bit_cast(float, w & 0xFFFF0000u));
}

// Element offset of a (page, KV head) tile in either pool.
__device__ __forceinline__ size_t tile_base(int32_t page, int32_t num_kv_heads, int32_t kvh, int d) {
  return (size_t(page) * num_kv_heads + kvh) * size_t(kPage * d);
}

// V in LDS, both pages of a step interleaved: dim d owns 64 bytes, four
// 16-byte slots, and slot g ^ v_swizzle(d) holds [page 0 quad g | page 1
// quad g] (quad g = tokens 4g .. 4g+3 of the page). That is exactly the P.V
// operand of lane (col, grp) for dim 16*jb + col and quad grp, one 16-byte
// read; the swizzle makes every 8 lanes of such a read (128 bytes) hit 8
// distinct 16-byte bank groups.
__device__ __forceinline__ int v_swizzle(int d) { return (d >> 1) & 3; }

template <int D>
struct Tiles {
  static constexpr int kElems = kPage * D;            // bf16 per (page, KV head) tile
  static constexpr int kChunks = kElems / 8;          // 16-byte pieces per tile
  // A step stages four tiles (K and V of two pages); each is moved by
  // kStageWaves / 4 waves, kWaveChunks wave-wide 1 KiB chunks (64 pieces) each.
  static constexpr int kWaveChunks = kChunks / 64 / (kStageWaves / 4);
  static_assert(kWaveChunks * 64 * kStageWaves == 4 * kChunks, "staging split");
};

// Sum of a lane's eight weights of a step.
__device__ __forceinline__ float weight_sum(const float* p) {
  return ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
}

// Online-softmax update of one 16-row tile for one step of 32 keys, in two
// parts so that each can be interleaved with matrix-core work.
//
// Lazy reference: each row keeps a reference max m (log2 units) and the
// weights are p = 2^(z - m). m moves only when, in some lane of the wave, the
// sum of the lane's eight weights of the step exceeds kRescaleMax. That
// sum is needed for the row sum anyway, and it bounds each of its weights,
// so the check costs one compare. Until it fires the lanes of a row need not
// agree on the row's max at all, so the common step has no cross-lane
// reduction. Weights up to kRescaleMax = 2^15 stay finite in fp16 (largest
// finite value 65504) with fp16's relative precision, and O and l share the
// reference, so O / l does not change. When the check fires, each row of the
// tile whose max has risen moves m to it (the max over all four lane groups)
// and O and l are rescaled; every weight is then at most 1, so the check
// stays quiet until a row's scores rise more than 12 (log2 units) above its
// reference. Key 0 is in every row's first step, so m is finite after it.
struct TileWeights {
  float sc[8];   // raw scores of this lane (masked ones -inf)
  float p[8];    // 2^(sc * c - m)
  bool ok[8];    // key inside the row's causal limit (masked steps)
  float part;    // sum of the eight weights
  bool need;     // the sum exceeds the headroom (or is inf / NaN)
};

// Part 1: exponentiate against the current reference. s0 / s1: this lane's
// scores for keys key0 + 4*grp + e of the step's two pages.
template <bool kMasked>
__device__ __forceinline__ TileWeights exponentiate(const f32x4& s0, const f32x4& s1, int key0, int grp, int limit,
                                                    float c, float m) {
  TileWeights t;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    t.sc[e] = s0[e];
    t.sc[4 + e] = s1[e];
  }
  if constexpr (kMasked) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      t.ok[e] = key0 + (e < 4 ? 0 : kPage) + 4 * grp + (e & 3) <= limit;
      t.sc[e] = t.ok[e] ? t.sc[e] : -__builtin_inff();
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) t.p[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(t.sc[e], c, -m));
  t.part = weight_sum(t.p);
  // Also true for inf (the first step, m = -inf) and NaN (-inf * 0 for a
  // zero scale), which settle() sorts out.
  t.need = !(t.part <= kRescaleMax);
  return t;
}

// Part 2: move the reference if needed (rare), then add the sum and pack the
// weights as the P^T operand.
template <int D, bool kMasked>
__device__ __forceinline__ u32x4 settle(TileWeights& t, float c, float& m, float& lsum, f32x4* o) {
  if (__any(t.need)) {
    // The scale c is >= 0 (the host flips the query's sign for a negative
    // one), so the row max of the raw scores gives the max of the scaled ones.
    float mx = fmaxf(fmaxf(fmaxf(t.sc[0], t.sc[1]), fmaxf(t.sc[2], t.sc[3])),
                     fmaxf(fmaxf(t.sc[4], t.sc[5]), fmaxf(t.sc[6], t.sc[7])));
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mx_s = mx * c;
    const bool grow = mx_s > m;   // NaN (fully masked, zero scale) compares false
    const float mnew = grow ? mx_s : m;
    const float alpha = __builtin_amdgcn_exp2f(m - mnew);
    m = mnew;
    lsum *= alpha;
#pragma unroll
    for (int jb = 0; jb < D / 16; ++jb) o[jb] *= alpha;
#pragma unroll
    for (int e = 0; e < 8; ++e) t.p[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(t.sc[e], c, -m));
    t.part = weight_sum(t.p);
  }
  if constexpr (kMasked) {
#pragma unroll
    for (int e = 0; e < 8; ++e) t.p[e] = t.ok[e] ? t.p[e] : 0.f;
    t.part = weight_sum(t.p);
  }
  lsum += t.part;
  return u32x4{pack_f16(t.p[0], t.p[1]), pack_f16(t.p[2], t.p[3]), pack_f16(t.p[4], t.p[5]),
               pack_f16(t.p[6], t.p[7])};
}

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3, 3))) void extend_attn_kernel(ExtendArgs a) {
  constexpr int KB = D / 32;
  constexpr int JB = D / 16;
  constexpr int TE = Tiles<D>::kElems;
  constexpr int NC = Tiles<D>::kWaveChunks;
  constexpr int kWaveRows = 16 * kRowTiles;
  // [buffer][step of the interval][K page 0 | K page 1 | V of both pages, interleaved]
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][kSub][4 * TE];

  const const_i32_ptr item = as_constant(a.items) + size_t(blockIdx.x) * kItemInts;
  const int seq = item[0];
  const int kvh = item[1];
  const int t0 = item[2];
  const int nt = item[3];
  const int prefix = item[4];
  const int qrow0 = item[5];
  const int nsteps = item[6];
  const int g = a.group;
  const int rows = nt * g;
  const int kend = prefix + t0 + nt;          // keys [0, kend) are read
  const int npages = (kend + kPage - 1) / kPage;
  const const_i32_ptr bt = as_constant(a.block_table) + size_t(seq) * a.bt_stride;
  const float c = a.scale_log2;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int col = lane & 15;
  const int grp = lane >> 4;

  // Rows of this lane (one per row tile): token-major over (token, head).
  int limit[kRowTiles];
  u32x4 qf[kRowTiles][KB];
#pragma unroll
  for (int rt = 0; rt < kRowTiles; ++rt) {
    const int r = wave * kWaveRows + rt * 16 + col;
    const bool valid = r < rows;
    const int tok = valid ? r / g : 0;
    const int hh = valid ? r - tok * g : 0;
    // Padding rows see every key with a zero query: finite, never stored.
    limit[rt] = valid ? prefix + t0 + tok : kend - 1;
    const uint16_t* qrow = a.q + (size_t(qrow0 + t0 + tok) * a.num_q_heads + kvh * g + hh) * D + 8 * grp;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(qrow + 32 * kb) ^ a.q_sign;
      qf[rt][kb] = valid ? v : u32x4{0u, 0u, 0u, 0u};
    }
  }
  const int wrow0 = wave * kWaveRows;
  const int wrow1 = min(rows, wrow0 + kWaveRows) - 1;   // last valid row of the wave
  const int wave_kmin = prefix + t0 + wrow0 / g;        // every row of the wave sees keys <= this
  const int wave_kmax = wrow1 >= wrow0 ? prefix + t0 + wrow1 / g : -1;

  f32x4 o[kRowTiles][JB];
  float m[kRowTiles], lsum[kRowTiles];
#pragma unroll
  for (int rt = 0; rt < kRowTiles; ++rt) {
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) o[rt][jb] = f32x4{0.f, 0.f, 0.f, 0.f};
    m[rt] = -__builtin_inff();
    lsum[rt] = 0.f;
  }

  // Staging: wave w < 8 moves tile w / 2 of each step (0: K of the step's
  // first page, 1: K of its second, 2 and 3: V of the two pages), in 1 KiB
  // chunks (w % 2) * NC .. + NC - 1; waves 8 .. 11 stage nothing. The tile and
  // its page are wave-uniform, so the global address is a scalar base plus a
  // fixed per-lane offset, and every LDS address is fixed per lane: no
  // per-step address arithmetic. A page past the item's last is replaced by
  // its first page (always in range); its keys lie past kend and are masked.
  // The keys are walked in intervals of kSub steps with one barrier each (one
  // step: two would need prefetch registers that the three-waves-per-SIMD
  // budget does not have).
  const bool stager = wave < kStageWaves;
  const int stile = (stager ? wave : 0) >> 1;
  const uint16_t* const spool = stile < 2 ? a.k_pool : a.v_pool;
  int soff[NC];    // element offset of this lane's piece in the tile
  int sdst0[NC];   // LDS element offset of the piece (K) or of its first 8-byte half (V)
  int sdst1[NC];   // V: LDS element offset of the second half
  int skey[NC];    // V: first token of the piece within the step's 32 keys
#pragma unroll
  for (int q = 0; q < NC; ++q) {
    soff[q] = (((wave & 1) * NC + q) * 64 + lane) * 8;
    if (stile < 2) {
      sdst0[q] = stile * TE + soff[q];
      sdst1[q] = 0;
      skey[q] = 0;
    } else {
      // V pool tile [D][16 tokens]: the piece holds tokens 8c .. 8c+7 of dim d.
      const int pg = stile - 2;
      const int d = soff[q] >> 4;
      const int c = (soff[q] >> 3) & 1;
      const int row = 2 * TE + d * 32 + pg * 4;
      sdst0[q] = row + ((2 * c) ^ v_swizzle(d)) * 8;
      sdst1[q] = row + ((2 * c + 1) ^ v_swizzle(d)) * 8;
      skey[q] = pg * kPage + 8 * c;
    }
  }
  u32x4 pre[kSub][NC];
  auto fetch = [&](int j) {
#pragma unroll
    for (int u = 0; u < kSub; ++u) {
      const int js = kSub * j + u;
      if (js >= nsteps) break;
      const int pg0 = 2 * js;
      const int p0 = bt[pg0];
      const int page = (stile & 1) && pg0 + 1 < npages ? bt[pg0 + 1] : p0;
      const uint16_t* src = spool + tile_base(page, a.num_kv_heads, kvh, D);
#pragma unroll
      for (int q = 0; q < NC; ++q) pre[u][q] = *reinterpret_cast<const u32x4*>(src + soff[q]);
    }
  };
  // Writes the fetched pieces of interval j into LDS buffer `base` (one per
  // step of the interval). V pieces are widened to fp16 and split into their
  // two token quads (8 bytes each) at their interleaved slots; in the step
  // that reaches kend, V tokens at or past it are zeroed first (they may be
  // stale or NaN, and a zero weight times NaN is still NaN).
  auto stage = [&](uint16_t (*base)[4 * TE], int j) {
#pragma unroll
    for (int u = 0; u < kSub; ++u) {
      const int js = kSub * j + u;
      if (js >= nsteps) break;
      uint16_t* L = base[u];
      if (stile < 2) {
#pragma unroll
        for (int q = 0; q < NC; ++q) *reinterpret_cast<u32x4*>(L + sdst0[q]) = pre[u][q];
      } else {
        const int key0 = js * kStepKeys;
        const bool tail = key0 + kStepKeys > kend;
#pragma unroll
        for (int q = 0; q < NC; ++q) {
          u32x4 x = pre[u][q];
          if (tail) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              const int key = key0 + skey[q] + 2 * w;
              x[w] &= (key < kend ? 0x0000FFFFu : 0u) | (key + 1 < kend ? 0xFFFF0000u : 0u);
            }
          }
#pragma unroll
          for (int w = 0; w < 4; ++w) x[w] = bf16x2_to_f16x2(x[w]);
          *reinterpret_cast<u32x2*>(L + sdst0[q]) = u32x2{x[0], x[1]};
          *reinterpret_cast<u32x2*>(L + sdst1[q]) = u32x2{x[2], x[3]};
        }
      }
    }
  };

  // One step, operands read from LDS just before use: the scores of both
  // row tiles per 32 dims of K, then the softmax of both, then P.V per
  // 16 dims of V (the third wave on each SIMD hides the latencies).
  auto compute = [&](const uint16_t* L, int key0) {
    f32x4 s0[kRowTiles], s1[kRowTiles];
#pragma unroll
    for (int rt = 0; rt < kRowTiles; ++rt) {
      s0[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
      s1[rt] = s0[rt];
    }
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const int ko = ((4 * kb + grp) * kPage + col) * 8;
      const u32x4 k0 = *reinterpret_cast<const u32x4*>(L + ko);
      const u32x4 k1 = *reinterpret_cast<const u32x4*>(L + TE + ko);
#pragma unroll
      for (int rt = 0; rt < kRowTiles; ++rt) {
        s0[rt] = mfma_bf16(k0, qf[rt][kb], s0[rt]);
        s1[rt] = mfma_bf16(k1, qf[rt][kb], s1[rt]);
      }
    }
    const int vo = 2 * TE + col * 32 + (grp ^ v_swizzle(col)) * 8;
    auto tail = [&](auto masked_tag) {
      constexpr bool kMasked = decltype(masked_tag)::value;
      u32x4 pf[kRowTiles];
#pragma unroll
      for (int rt = 0; rt < kRowTiles; ++rt) {
        TileWeights t = exponentiate<kMasked>(s0[rt], s1[rt], key0, grp, limit[rt], c, m[rt]);
        pf[rt] = settle<D, kMasked>(t, c, m[rt], lsum[rt], o[rt]);
      }
#pragma unroll
      for (int jb = 0; jb < JB; ++jb) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(L + vo + jb * 16 * 32);
#pragma unroll
        for (int rt = 0; rt < kRowTiles; ++rt) o[rt][jb] = mfma_f16(v, pf[rt], o[rt][jb]);
      }
    };
    if (key0 + kStepKeys - 1 > wave_kmin)
      tail(std::true_type{});
    else
      tail(std::false_type{});
  };

  const int nint = (nsteps + kSub - 1) / kSub;
  if (stager) {
    fetch(0);
    stage(lds[0], 0);
  }
  __syncthreads();

  // One interval from buffer `cur` while the next is staged into `nxt`; the
  // loop is unrolled by two so that both buffers' addresses are constants.
  auto interval = [&](int j, uint16_t (*cur)[4 * TE], uint16_t (*nxt)[4 * TE]) {
    if (stager && j + 1 < nint) fetch(j + 1);
#pragma unroll
    for (int u = 0; u < kSub; ++u) {
      const int js = kSub * j + u;
      const int key0 = js * kStepKeys;
      if (js < nsteps && key0 <= wave_kmax) compute(cur[u], key0);
    }
    if (stager && j + 1 < nint) stage(nxt, j + 1);
    __syncthreads();
  };
  for (int j = 0; j < nint; j += 2) {
    interval(j, lds[0], lds[1]);
    if (j + 1 < nint) interval(j + 1, lds[1], lds[0]);
  }

  // Lane holds O[row col][16*jb + 4*grp + i] of each row tile.
#pragma unroll
  for (int rt = 0; rt < kRowTiles; ++rt) {
    float lt = lsum[rt] + __shfl_xor(lsum[rt], 16);
    lt += __shfl_xor(lt, 32);
    const int r = wave * kWaveRows + rt * 16 + col;
    if (r >= rows) continue;
    const int tok = r / g;
    const int head = kvh * g + (r - tok * g);
    const size_t orow = size_t(qrow0 + t0 + tok) * a.num_q_heads + head;
    const float inv = 1.f / lt;
    float* dst = a.out + orow * D + 4 * grp;
#pragma unroll
    for (int jb = 0; jb < JB; ++jb) *reinterpret_cast<f32x4*>(dst + 16 * jb) = o[rt][jb] * inv;
    if (a.lse && grp == 0) a.lse[orow] = (m[rt] + __log2f(lt)) * kLn2;
  }
}

// Stores the new tokens' keys and values of one item (one sequence and KV
// head, tokens t0 .. t0 + nt - 1) into their page slots. Keys: one 16-byte
// piece per (token, 8 dims). Values: one thread per (page, dim) writes the
// 16 slots of a page it fills completely as two 16-byte stores, else slot by
// slot.
constexpr int kStoreThreads = 256;

template <int D>
__global__ __launch_bounds__(kStoreThreads) void kv_store_kernel(ExtendArgs a) {
  const const_i32_ptr item = as_constant(a.items) + size_t(blockIdx.x) * kItemInts;
  const int seq = item[0];
  const int kvh = item[1];
  const int t0 = item[2];
  const int nt = item[3];
  const int prefix = item[4];
  const int qrow0 = item[5];
  const const_i32_ptr bt = as_constant(a.block_table) + size_t(seq) * a.bt_stride;
  const int first = prefix + t0;   // position of the item's first token
  const size_t row_stride = size_t(a.num_kv_heads) * D;
  const uint16_t* kn = a.k_new + size_t(qrow0 + t0) * row_stride + size_t(kvh) * D;
  const uint16_t* vn = a.v_new + size_t(qrow0 + t0) * row_stride + size_t(kvh) * D;

  for (int i = threadIdx.x; i < nt * (D / 8); i += kStoreThreads) {
    const int t = i / (D / 8);
    const int c = i - t * (D / 8);
    const int pos = first + t;
    const int page = bt[pos / kPage];
    uint16_t* dst = a.k_dst + tile_base(page, a.num_kv_heads, kvh, D) + ((c * kPage) + pos % kPage) * 8;
    *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(kn + size_t(t) * row_stride + 8 * c);
  }

  const int pg_a = first / kPage;
  const int pg_b = (first + nt - 1) / kPage;
  for (int i = threadIdx.x; i < (pg_b - pg_a + 1) * D; i += kStoreThreads) {
    const int pg = pg_a + i / D;
    const int dim = i % D;
    const int lo = max(first, pg * kPage);
    const int hi = min(first + nt, (pg + 1) * kPage);
    uint16_t* dst = a.v_dst + tile_base(bt[pg], a.num_kv_heads, kvh, D) + dim * kPage;
    if (hi - lo == kPage) {
      uint32_t w[8];
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const uint32_t x = vn[size_t(lo + 2 * s - first) * row_stride + dim];
        const uint32_t y = vn[size_t(lo + 2 * s + 1 - first) * row_stride + dim];
        w[s] = x | (y << 16);
      }
      reinterpret_cast<u32x4*>(dst)[0] = u32x4{w[0], w[1], w[2], w[3]};
      reinterpret_cast<u32x4*>(dst)[1] = u32x4{w[4], w[5], w[6], w[7]};
    } else {
      for (int pos = lo; pos < hi; ++pos) dst[pos % kPage] = vn[size_t(pos - first) * row_stride + dim];
    }
  }
}

}  // namespace

hipError_t launch_extend(const ExtendArgs& a, hipStream_t stream) {
  if (a.num_items == 0) return hipSuccess;
  const dim3 grid(a.num_items), block(kThreads);
  if (a.k_new) {
    if (a.head_dim == 128)
      hipLaunchKernelGGL(kv_store_kernel<128>, grid, dim3(kStoreThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(kv_store_kernel<64>, grid, dim3(kStoreThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.head_dim == 128)
    hipLaunchKernelGGL(extend_attn_kernel<128>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(extend_attn_kernel<64>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace sf
