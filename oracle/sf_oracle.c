/*
 * sf_oracle.c -- slow, plain fp64 reference for batched decode attention over
 * a paged KV cache.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library. It shares no code,
 * header or constant with the HIP library; it reads the same documented
 * memory layouts with its own indexing.
 *
 * What it computes (App. B.1 of the paper: one decode step lets every running
 * trajectory's single new query token attend over that trajectory's whole
 * cached keys/values; the cost grows linearly with the cache it reads):
 *
 *   for sequence s with L = seq_lens[s] cached tokens and query head h,
 *   with g = Hq / Hkv query heads sharing KV head kvh = h / g:
 *     K_s[t][d] = k_pool[bt[s][t / P]][kvh][d / 8][t % P][d % 8]   t = 0 .. L-1
 *     V_s[t][d] = v_pool[bt[s][t / P]][kvh][d][t % P]
 *     z_t    = scale * sum_d q[s,h,d] * K_s[t][d]
 *     m      = max_t z_t,  w_t = exp(z_t - m)
 *     out    = sum_t w_t V_s[t] / sum_t w_t
 *     lse    = m + log(sum_t w_t)
 *   L = 0 gives out = 0 and lse = -inf.
 *
 * Everything is widened exactly from the stored bf16 bits to double and
 * accumulated in double, in token order. There is no blocking, no online
 * rescaling and no split: subtracting the max is the textbook way to keep
 * exp() in range and does not change the mathematical value.
 *
 * Layouts: q [B][Hq][D]; k_pool [N][Hkv][D/8][P][8]; v_pool [N][Hkv][D][P];
 * bt [B][stride] int32; all bf16 stored as uint16 bit patterns.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Element offsets of key and value (page pg, KV head kvh, slot, dim d). */
static int64_t k_index(int64_t pg, int Hkv, int kvh, int D, int P, int slot, int d) {
  return ((((pg * Hkv + kvh) * (D / 8) + d / 8) * P) + slot) * 8 + d % 8;
}
static int64_t v_index(int64_t pg, int Hkv, int kvh, int D, int P, int slot, int d) {
  return ((pg * Hkv + kvh) * D + d) * P + slot;
}

/* bf16 is the upper half of an IEEE binary32; widening is exact. */
static double bf16_to_double(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

int sf_oracle_version(void) { return 3; }

int sf_oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Checks every block-table entry the computation will touch.
 * Returns 0 if all lie in [0, num_pages), else 1 + the first bad sequence. */
static int check_pages(int B, int P, int stride, int num_pages,
                       const int32_t* bt, const int32_t* lens) {
  for (int s = 0; s < B; ++s) {
    int L = lens[s];
    if (L < 0) return 1 + s;
    int npg = (L + P - 1) / P;
    if (npg > stride) return 1 + s;
    for (int j = 0; j < npg; ++j) {
      int32_t pg = bt[(int64_t)s * stride + j];
      if (pg < 0 || pg >= num_pages) return 1 + s;
    }
  }
  return 0;
}

/* Dense copy of the cached keys and values of (seq, kvh): k_out and v_out are
 * [L][D] uint16, token-major. Returns 0, or nonzero on a bad page id. */
int sf_oracle_gather(int Hkv, int D, int P, int stride, int num_pages,
                     const uint16_t* k_pool, const uint16_t* v_pool,
                     const int32_t* bt, int seq, int kvh, int L,
                     uint16_t* k_out, uint16_t* v_out) {
  for (int t = 0; t < L; ++t) {
    int32_t pg = bt[(int64_t)seq * stride + t / P];
    if (pg < 0 || pg >= num_pages) return 1;
    int slot = t % P;
    for (int d = 0; d < D; ++d) {
      k_out[(int64_t)t * D + d] = k_pool[k_index(pg, Hkv, kvh, D, P, slot, d)];
      v_out[(int64_t)t * D + d] = v_pool[v_index(pg, Hkv, kvh, D, P, slot, d)];
    }
  }
  return 0;
}

/*
 * Full reference. out is [B][Hq][D] double, lse [B][Hq] double (may be NULL).
 * nthreads <= 0 uses the OpenMP default. Returns 0 on success, -1 on a bad
 * shape, or 1 + s for the first sequence s with an invalid block-table entry.
 */
int sf_oracle_decode_attn(int B, int Hq, int Hkv, int D, int P, int stride, int num_pages,
                          const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool,
                          const int32_t* bt, const int32_t* lens, double scale,
                          double* out, double* lse, int nthreads) {
  if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || D <= 0 || P <= 0) return -1;
  int bad = check_pages(B, P, stride, num_pages, bt, lens);
  if (bad) return bad;
  const int g = Hq / Hkv;
  const int64_t pairs = (int64_t)B * Hq;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#endif
#pragma omp parallel
  {
    double* z = NULL;
    double* acc = (double*)malloc(sizeof(double) * (size_t)D);
    int zcap = 0;
#pragma omp for schedule(dynamic, 1)
    for (int64_t sh = 0; sh < pairs; ++sh) {
      const int s = (int)(sh / Hq);
      const int h = (int)(sh % Hq);
      const int kvh = h / g;
      const int L = lens[s];
      double* o = out + sh * D;
      if (L == 0) {
        for (int d = 0; d < D; ++d) o[d] = 0.0;
        if (lse) lse[sh] = -INFINITY;
        continue;
      }
      if (L > zcap) {
        free(z);
        z = (double*)malloc(sizeof(double) * (size_t)L);
        zcap = L;
      }
      const uint16_t* qv = q + sh * D;
      /* scores */
      double m = -INFINITY;
      for (int t = 0; t < L; ++t) {
        int32_t pg = bt[(int64_t)s * stride + t / P];
        int slot = t % P;
        double dot = 0.0;
        for (int d = 0; d < D; ++d)
          dot += bf16_to_double(qv[d]) * bf16_to_double(k_pool[k_index(pg, Hkv, kvh, D, P, slot, d)]);
        z[t] = scale * dot;
        if (z[t] > m) m = z[t];
      }
      /* softmax weights and weighted sum of values */
      double wsum = 0.0;
      for (int d = 0; d < D; ++d) acc[d] = 0.0;
      for (int t = 0; t < L; ++t) {
        int32_t pg = bt[(int64_t)s * stride + t / P];
        int slot = t % P;
        double w = exp(z[t] - m);
        wsum += w;
        for (int d = 0; d < D; ++d) acc[d] += w * bf16_to_double(v_pool[v_index(pg, Hkv, kvh, D, P, slot, d)]);
      }
      for (int d = 0; d < D; ++d) o[d] = acc[d] / wsum;
      if (lse) lse[sh] = m + log(wsum);
    }
    free(z);
    free(acc);
  }
  return 0;
}

/*
 * fp8 KV cache (next to the bf16 one): keys and values stored as OCP FP8
 * E4M3 codes, one fp32 scale per (page, KV head) tile for K and one for V.
 * A code (sign s, exponent e, mantissa m) is
 *   (-1)^s * m/8 * 2^-6            if e = 0
 *   (-1)^s * (1 + m/8) * 2^(e - 7) otherwise, NaN for e = 15, m = 7,
 * and the cached key of slot t, dim d is that value times k_scale[page][kvh]
 * (values likewise with v_scale). Pools k8 and v8 are [N][Hkv][16*D] bytes,
 * scales [N][Hkv]; inside a tile the byte of (slot t, dim d) is at
 *   K: ((d/64 * 4 + (d%32)/8) * 16 + t) * 16 + (d/32 % 2) * 8 + d%8
 *   V: ((d/64 * 4 + t/4) * 16 + d%16) * 16 + (d/16 % 4) * 4 + t%4
 * The attention itself is the bf16 oracle's: widen exactly, fp64 throughout.
 */
static int64_t k8_index(int64_t pg, int Hkv, int kvh, int D, int t, int d) {
  return (pg * Hkv + kvh) * 16 * D + (((d / 64) * 4 + (d % 32) / 8) * 16 + t) * 16 + ((d / 32) % 2) * 8 + d % 8;
}
static int64_t v8_index(int64_t pg, int Hkv, int kvh, int D, int t, int d) {
  return (pg * Hkv + kvh) * 16 * D + (((d / 64) * 4 + t / 4) * 16 + d % 16) * 16 + ((d / 16) % 4) * 4 + t % 4;
}

double sf_oracle_e4m3_value(int code) {
  const int s = (code >> 7) & 1, e = (code >> 3) & 15, m = code & 7;
  double v;
  if (e == 15 && m == 7) return NAN;
  if (e == 0) v = ldexp((double)m / 8.0, -6);
  else v = ldexp(1.0 + (double)m / 8.0, e - 7);
  return s ? -v : v;
}

int sf_oracle_decode_attn_fp8(int B, int Hq, int Hkv, int D, int P, int stride, int num_pages,
                              const uint16_t* q, const uint8_t* k8, const uint8_t* v8,
                              const float* k_scale, const float* v_scale,
                              const int32_t* bt, const int32_t* lens, double scale,
                              double* out, double* lse, int nthreads) {
  if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || D <= 0 || D % 64 != 0 || P != 16) return -1;
  int bad = check_pages(B, P, stride, num_pages, bt, lens);
  if (bad) return bad;
  double table[256];
  for (int c = 0; c < 256; ++c) table[c] = sf_oracle_e4m3_value(c);
  const int g = Hq / Hkv;
  const int64_t pairs = (int64_t)B * Hq;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#endif
#pragma omp parallel
  {
    double* z = NULL;
    double* acc = (double*)malloc(sizeof(double) * (size_t)D);
    int zcap = 0;
#pragma omp for schedule(dynamic, 1)
    for (int64_t sh = 0; sh < pairs; ++sh) {
      const int s = (int)(sh / Hq);
      const int h = (int)(sh % Hq);
      const int kvh = h / g;
      const int L = lens[s];
      double* o = out + sh * D;
      if (L == 0) {
        for (int d = 0; d < D; ++d) o[d] = 0.0;
        if (lse) lse[sh] = -INFINITY;
        continue;
      }
      if (L > zcap) {
        free(z);
        z = (double*)malloc(sizeof(double) * (size_t)L);
        zcap = L;
      }
      const uint16_t* qv = q + sh * D;
      double m = -INFINITY;
      for (int t = 0; t < L; ++t) {
        int32_t pg = bt[(int64_t)s * stride + t / P];
        int slot = t % P;
        double ks = (double)k_scale[(int64_t)pg * Hkv + kvh];
        double dot = 0.0;
        for (int d = 0; d < D; ++d)
          dot += bf16_to_double(qv[d]) * (table[k8[k8_index(pg, Hkv, kvh, D, slot, d)]] * ks);
        z[t] = scale * dot;
        if (z[t] > m) m = z[t];
      }
      double wsum = 0.0;
      for (int d = 0; d < D; ++d) acc[d] = 0.0;
      for (int t = 0; t < L; ++t) {
        int32_t pg = bt[(int64_t)s * stride + t / P];
        int slot = t % P;
        double vs = (double)v_scale[(int64_t)pg * Hkv + kvh];
        double w = exp(z[t] - m);
        wsum += w;
        for (int d = 0; d < D; ++d) acc[d] += w * (table[v8[v8_index(pg, Hkv, kvh, D, slot, d)]] * vs);
      }
      for (int d = 0; d < D; ++d) o[d] = acc[d] / wsum;
      if (lse) lse[sh] = m + log(wsum);
    }
    free(z);
    free(acc);
  }
  return 0;
}
