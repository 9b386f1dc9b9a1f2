/*
 * fp64 CPU oracle for the prefill/decode attention hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the HIP library and includes no HIP header.
 *
 * Every function is the plain definition, with no tiling, no online softmax
 * and no split of the key range:
 *
 *   attention (Eq. 1 of the paper, with the softmax scale as an argument):
 *     o_i = sum_j p_j v_j / sum_j p_j,  p_j = exp(sc_j - m),
 *     sc_j = sigma * <q_i, k_j>,  m = max_j sc_j,  lse_i = m + ln sum_j p_j,
 *   taken over j <= i inside one request for prefill (causal, no prefix) and
 *   over the j < ctx cached tokens of a request for decode.
 *
 *   The K/V cache lives in fixed-size blocks addressed per request (the
 *   paper's KV-cache blocks moved between instances, Sec. I and Sec. V-C).
 *   Layouts: k_pool[page][Hkv][16][d], v_pool[page][Hkv][d][16];
 *   page_table[r][i] = physical page of logical page i of request r.
 *
 *   GQA: query head h reads KV head h / (Hq/Hkv).
 *
 * Inputs are bf16 bit patterns (uint16) or fp32, widened exactly to double.
 * sigma is the float scale widened to double.  Outputs are double.
 *
 * FP8 KV pages (a storage format the paper's FP8 models imply, Sec. VI-A;
 * the paper gives no scaling rule): OCP 8-bit floating point E4M3 -- 1 sign,
 * 4 exponent (bias 7) and 3 mantissa bits, no infinities, S.1111.111 is NaN,
 * largest finite value 448.  One scale per KV head and pool (K and V
 * separately): the stored code of element x of head h is
 *   code = E4M3_rne(sat(float(x) * float(1 / scale[h])))
 * where 1/scale and the product are fp32 operations rounded to nearest even,
 * sat() clamps to [-448, 448] (NaN stays NaN) and E4M3_rne rounds to the
 * nearest code, ties to the even code.  The cached value is value(code) *
 * scale[h], exactly, in double.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_BF16 0
#define OR_FP32 1
#define OR_E4M3 2
#define OR_PAGE 16

/* Value of an E4M3 code: (-1)^s 2^(E-7) (1 + M/8) for E >= 1, (-1)^s 2^-6 M/8
 * for E = 0. */
double oracle_e4m3_value(uint8_t c) {
  const int s = c >> 7, e = (c >> 3) & 15, m = c & 7;
  if (e == 15 && m == 7) return NAN;
  const double v = e == 0 ? ldexp((double)m, -9) : ldexp((double)(8 + m), e - 10);
  return s ? -v : v;
}

/* Nearest E4M3 code of y (ties to even), saturating at +-448. */
uint8_t oracle_e4m3_encode(float y) {
  const uint8_t s = signbit(y) ? 0x80 : 0;
  if (isnan(y)) return s | 0x7F;
  const double a = fabs((double)y);
  if (a >= 448.0) return s | 0x7E;
  if (a < ldexp(1.0, -6)) /* subnormal step 2^-9; 8 steps is the code of 2^-6 */
    return s | (uint8_t)nearbyint(a * 512.0);
  int ex;
  frexp(a, &ex); /* a in [2^(ex-1), 2^ex) */
  int E = ex - 1; /* -6 .. 8 */
  int m = (int)nearbyint(ldexp(a, 3 - E)); /* 8 .. 16 */
  if (m == 16) {
    m = 8;
    E += 1;
  }
  return s | (uint8_t)((E + 7) << 3) | (uint8_t)(m - 8);
}

/* Codes of x[n][hkv][d] (bf16 bits or fp32) with one scale per head. */
int oracle_e4m3_quantize(int dtype, int64_t n, int hkv, int d, const void *x,
                         const float *scale, uint8_t *out) {
  for (int h = 0; h < hkv; ++h)
    if (!(scale[h] > 0.0f)) return 1;
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < n; ++t)
    for (int h = 0; h < hkv; ++h) {
      const float inv = 1.0f / scale[h];
      for (int e = 0; e < d; ++e) {
        const int64_t i = (t * hkv + h) * d + e;
        float xf;
        if (dtype == OR_BF16) {
          uint32_t u = (uint32_t)((const uint16_t *)x)[i] << 16;
          memcpy(&xf, &u, 4);
        } else {
          xf = ((const float *)x)[i];
        }
        out[i] = oracle_e4m3_encode(xf * inv);
      }
    }
  return 0;
}

static inline double ld(const void *base, int dtype, int64_t i) {
  if (dtype == OR_E4M3) return oracle_e4m3_value(((const uint8_t *)base)[i]);
  if (dtype == OR_BF16) {
    uint32_t u = (uint32_t)((const uint16_t *)base)[i] << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
  }
  return (double)((const float *)base)[i];
}

/* One query row against n keys given by explicit element offsets.
 * koff[j] / voff[j] are the element offsets of key/value j; element e of
 * key j is at koff[j] + e*kstride_e, of value j at voff[j] + e*vstride_e. */
static void attend_row_kv(int qdt, int kvdt, double kscale, double vscale, int d,
                          double sigma, const void *q, int64_t qoff, const void *kb,
                          const int64_t *koff, int64_t kse, const void *vb,
                          const int64_t *voff, int64_t vse, int n, double *sc, double *out,
                          double *lse) {
  double m = -INFINITY;
  for (int j = 0; j < n; ++j) {
    double s = 0.0;
    for (int e = 0; e < d; ++e)
      s += ld(q, qdt, qoff + e) * (ld(kb, kvdt, koff[j] + e * kse) * kscale);
    sc[j] = sigma * s;
    if (sc[j] > m) m = sc[j];
  }
  double l = 0.0;
  for (int j = 0; j < n; ++j) {
    sc[j] = exp(sc[j] - m);
    l += sc[j];
  }
  for (int e = 0; e < d; ++e) {
    double acc = 0.0;
    for (int j = 0; j < n; ++j) acc += sc[j] * (ld(vb, kvdt, voff[j] + e * vse) * vscale);
    out[e] = acc / l;
  }
  if (lse) *lse = m + log(l);
}

/* Q, K and V of one element type, unscaled. */
static void attend_row(int dtype, int d, double sigma, const void *q, int64_t qoff,
                       const void *kb, const int64_t *koff, int64_t kse,
                       const void *vb, const int64_t *voff, int64_t vse, int n,
                       double *sc, double *out, double *lse) {
  attend_row_kv(dtype, dtype, 1.0, 1.0, d, sigma, q, qoff, kb, koff, kse, vb, voff, vse, n, sc,
                out, lse);
}

/* Varlen causal prefill over contiguous token-major Q[T][Hq][d], K/V[T][Hkv][d].
 * out[T][Hq][d], lse[T][Hq] (lse may be NULL). */
int oracle_prefill(int dtype, int hq, int hkv, int d, float scale, const void *q,
                   const void *k, const void *v, const int32_t *cu, int nreq,
                   double *out, double *lse) {
  if (hkv <= 0 || hq % hkv) return 1;
  const int g = hq / hkv;
  const double sigma = (double)scale;
  int maxlen = 0;
  for (int r = 0; r < nreq; ++r)
    if (cu[r + 1] - cu[r] > maxlen) maxlen = cu[r + 1] - cu[r];
  const int64_t npairs = (int64_t)nreq * hq;
#pragma omp parallel
  {
    double *sc = (double *)malloc(sizeof(double) * (maxlen + 1));
    int64_t *koff = (int64_t *)malloc(sizeof(int64_t) * (maxlen + 1));
    int64_t *voff = (int64_t *)malloc(sizeof(int64_t) * (maxlen + 1));
#pragma omp for schedule(dynamic, 1)
    for (int64_t p = 0; p < npairs; ++p) {
      const int r = (int)(p / hq), h = (int)(p % hq), c = h / g;
      const int base = cu[r], len = cu[r + 1] - cu[r];
      for (int j = 0; j < len; ++j) {
        koff[j] = ((int64_t)(base + j) * hkv + c) * d;
        voff[j] = koff[j];
      }
      for (int i = 0; i < len; ++i) {
        const int64_t row = (int64_t)(base + i) * hq + h;
        attend_row(dtype, d, sigma, q, row * d, k, koff, 1, v, voff, 1, i + 1, sc,
                   out + row * d, lse ? lse + row : NULL);
      }
    }
    free(sc);
    free(koff);
    free(voff);
  }
  return 0;
}

/* Same definition for a list of (token, head) rows only: out[n][d], lse[n]. */
int oracle_prefill_rows(int dtype, int hq, int hkv, int d, float scale, const void *q,
                        const void *k, const void *v, const int32_t *cu, int nreq,
                        const int32_t *tok, const int32_t *head, int nrows, double *out,
                        double *lse) {
  if (hkv <= 0 || hq % hkv) return 1;
  const int g = hq / hkv;
  const double sigma = (double)scale;
  int maxlen = 0;
  for (int r = 0; r < nreq; ++r)
    if (cu[r + 1] - cu[r] > maxlen) maxlen = cu[r + 1] - cu[r];
  int bad = 0;
#pragma omp parallel
  {
    double *sc = (double *)malloc(sizeof(double) * (maxlen + 1));
    int64_t *koff = (int64_t *)malloc(sizeof(int64_t) * (maxlen + 1));
#pragma omp for schedule(dynamic, 1)
    for (int n = 0; n < nrows; ++n) {
      const int t = tok[n], h = head[n], c = h / g;
      int r = 0;
      while (r < nreq && cu[r + 1] <= t) ++r;
      if (r == nreq || h < 0 || h >= hq) {
#pragma omp atomic write
        bad = 1;
        continue;
      }
      const int base = cu[r], i = t - base;
      for (int j = 0; j <= i; ++j) koff[j] = ((int64_t)(base + j) * hkv + c) * d;
      attend_row(dtype, d, sigma, q, ((int64_t)t * hq + h) * d, k, koff, 1, v, koff, 1,
                 i + 1, sc, out + (int64_t)n * d, lse ? lse + n : NULL);
    }
    free(sc);
    free(koff);
  }
  return bad ? 2 : 0;
}

/* Single-query decode over the paged cache.
 * q[B][Hq][d]; context_lens[B] counts the current token; out[B][Hq][d]; lse[B][Hq]. */
static int decode_impl(int qdt, int kvdt, const float *k_scale, const float *v_scale, int hq,
                       int hkv, int d, float scale, const void *q, const void *k_pool,
                       const void *v_pool, const int32_t *page_table, int pt_stride,
                       const int32_t *ctx, int nreq, double *out, double *lse) {
  if (hkv <= 0 || hq % hkv) return 1;
  const int g = hq / hkv;
  const double sigma = (double)scale;
  int maxlen = 0;
  for (int r = 0; r < nreq; ++r)
    if (ctx[r] > maxlen) maxlen = ctx[r];
  const int64_t npairs = (int64_t)nreq * hq;
#pragma omp parallel
  {
    double *sc = (double *)malloc(sizeof(double) * (maxlen + 1));
    int64_t *koff = (int64_t *)malloc(sizeof(int64_t) * (maxlen + 1));
    int64_t *voff = (int64_t *)malloc(sizeof(int64_t) * (maxlen + 1));
#pragma omp for schedule(dynamic, 1)
    for (int64_t p = 0; p < npairs; ++p) {
      const int r = (int)(p / hq), h = (int)(p % hq), c = h / g;
      for (int j = 0; j < ctx[r]; ++j) {
        const int64_t page = page_table[(int64_t)r * pt_stride + j / OR_PAGE];
        const int slot = j % OR_PAGE;
        koff[j] = ((page * hkv + c) * OR_PAGE + slot) * d;   /* element e at +e   */
        voff[j] = (page * hkv + c) * (int64_t)d * OR_PAGE + slot; /* element e at +16e */
      }
      attend_row_kv(qdt, kvdt, k_scale ? (double)k_scale[c] : 1.0,
                    v_scale ? (double)v_scale[c] : 1.0, d, sigma, q, p * d, k_pool, koff, 1,
                    v_pool, voff, OR_PAGE, ctx[r], sc, out + p * d, lse ? lse + p : NULL);
    }
    free(sc);
    free(koff);
    free(voff);
  }
  return 0;
}

int oracle_decode(int dtype, int hq, int hkv, int d, float scale, const void *q,
                  const void *k_pool, const void *v_pool, const int32_t *page_table,
                  int pt_stride, const int32_t *ctx, int nreq, double *out, double *lse) {
  return decode_impl(dtype, dtype, NULL, NULL, hq, hkv, d, scale, q, k_pool, v_pool, page_table,
                     pt_stride, ctx, nreq, out, lse);
}

/* Decode over E4M3 pools (codes, same page layouts) with per-KV-head scales:
 * key j of head c is value(code) * k_scale[c], value j is value(code) *
 * v_scale[c].  q (bf16 or fp32 by qdtype) [B][Hq][d]. */
int oracle_decode_e4m3(int qdtype, int hq, int hkv, int d, float scale, const void *q,
                       const uint8_t *k_pool, const uint8_t *v_pool, const float *k_scale,
                       const float *v_scale, const int32_t *page_table, int pt_stride,
                       const int32_t *ctx, int nreq, double *out, double *lse) {
  return decode_impl(qdtype, OR_E4M3, k_scale, v_scale, hq, hkv, d, scale, q, k_pool, v_pool,
                     page_table, pt_stride, ctx, nreq, out, lse);
}

/* Prefill of a chunk over the paged cache (a prompt processed in chunks, or a
 * request that already holds a cached prefix): request r has prefix_lens[r]
 * cached tokens and a chunk of n_r = cu_q[r+1] - cu_q[r] new tokens whose K/V
 * are already written at positions prefix_lens[r] .. + n_r - 1.  Chunk token i
 * (query row cu_q[r] + i, position prefix_lens[r] + i) attends to the cached
 * positions 0 .. prefix_lens[r] + i: causal with the chunk aligned to the end
 * of the cache.  q/out [T][Hq][d], lse [T][Hq].  With rows != NULL only the
 * nrows (token, head) pairs tok[n], head[n] are computed, into out[n][d] and
 * lse[n]. */
static int prefill_paged_impl(int qdt, int kvdt, const float *k_scale, const float *v_scale,
                              int hq, int hkv, int d, float scale, const void *q,
                              const void *k_pool, const void *v_pool, const int32_t *page_table,
                              int pt_stride, const int32_t *cu_q, const int32_t *prefix_lens,
                              int nreq, const int32_t *tok, const int32_t *head, int nrows,
                              double *out, double *lse) {
  if (hkv <= 0 || hq % hkv) return 1;
  const int g = hq / hkv;
  const double sigma = (double)scale;
  int maxlen = 0;
  for (int r = 0; r < nreq; ++r) {
    const int len = prefix_lens[r] + cu_q[r + 1] - cu_q[r];
    if (len > maxlen) maxlen = len;
  }
  const int64_t T = cu_q[nreq];
  const int64_t total = tok ? nrows : T * hq;
  int bad = 0;
#pragma omp parallel
  {
    double *sc = (double *)malloc(sizeof(double) * (maxlen + 1));
    int64_t *koff = (int64_t *)malloc(sizeof(int64_t) * (maxlen + 1));
    int64_t *voff = (int64_t *)malloc(sizeof(int64_t) * (maxlen + 1));
#pragma omp for schedule(dynamic, 1)
    for (int64_t n = 0; n < total; ++n) {
      const int64_t t = tok ? tok[n] : n / hq;
      const int h = tok ? head[n] : (int)(n % hq);
      int r = 0;
      while (r < nreq && cu_q[r + 1] <= t) ++r;
      if (t < 0 || r == nreq || h < 0 || h >= hq) {
#pragma omp atomic write
        bad = 1;
        continue;
      }
      const int c = h / g;
      const int nkeys = prefix_lens[r] + (int)(t - cu_q[r]) + 1;
      for (int j = 0; j < nkeys; ++j) {
        const int64_t page = page_table[(int64_t)r * pt_stride + j / OR_PAGE];
        const int slot = j % OR_PAGE;
        koff[j] = ((page * hkv + c) * OR_PAGE + slot) * d;
        voff[j] = (page * hkv + c) * (int64_t)d * OR_PAGE + slot;
      }
      const int64_t orow = tok ? n : t * hq + h;
      attend_row_kv(qdt, kvdt, k_scale ? (double)k_scale[c] : 1.0,
                    v_scale ? (double)v_scale[c] : 1.0, d, sigma, q, (t * hq + h) * d, k_pool,
                    koff, 1, v_pool, voff, OR_PAGE, nkeys, sc, out + orow * d,
                    lse ? lse + orow : NULL);
    }
    free(sc);
    free(koff);
    free(voff);
  }
  return bad ? 2 : 0;
}

int oracle_prefill_paged(int dtype, int hq, int hkv, int d, float scale, const void *q,
                         const void *k_pool, const void *v_pool, const int32_t *page_table,
                         int pt_stride, const int32_t *cu_q, const int32_t *prefix_lens,
                         int nreq, const int32_t *tok, const int32_t *head, int nrows,
                         double *out, double *lse) {
  return prefill_paged_impl(dtype, dtype, NULL, NULL, hq, hkv, d, scale, q, k_pool, v_pool,
                            page_table, pt_stride, cu_q, prefix_lens, nreq, tok, head, nrows,
                            out, lse);
}

/* The same chunk prefill over E4M3 pools (codes, same page layouts) with
 * per-KV-head scales: key j of head c is value(code) * k_scale[c], value j is
 * value(code) * v_scale[c], in double (the FP8 cache of the paper's FP8
 * models, Sec. VI-A, read by Eq. 1).  q (bf16 or fp32 by qdtype) [T][Hq][d];
 * tok/head/nrows select rows as in oracle_prefill_paged. */
int oracle_prefill_paged_e4m3(int qdtype, int hq, int hkv, int d, float scale, const void *q,
                              const uint8_t *k_pool, const uint8_t *v_pool, const float *k_scale,
                              const float *v_scale, const int32_t *page_table, int pt_stride,
                              const int32_t *cu_q, const int32_t *prefix_lens, int nreq,
                              const int32_t *tok, const int32_t *head, int nrows, double *out,
                              double *lse) {
  return prefill_paged_impl(qdtype, OR_E4M3, k_scale, v_scale, hq, hkv, d, scale, q, k_pool,
                            v_pool, page_table, pt_stride, cu_q, prefix_lens, nreq, tok, head,
                            nrows, out, lse);
}

/* Paged write: for request r, new tokens at logical positions
 * p in [start[r], start[r] + n_r) with n_r = cu_new[r+1]-cu_new[r] come from
 * rows cu_new[r] + (p - start[r]) of k_new/v_new[T][Hkv][d].  Bit copy. */
int oracle_kv_write(int esize, int hkv, int d, const void *k_new, const void *v_new,
                    void *k_pool, void *v_pool, const int32_t *page_table, int pt_stride,
                    const int32_t *cu_new, const int32_t *start, int nreq) {
  for (int r = 0; r < nreq; ++r) {
    const int n = cu_new[r + 1] - cu_new[r];
    for (int i = 0; i < n; ++i) {
      const int p = start[r] + i;
      const int64_t page = page_table[(int64_t)r * pt_stride + p / OR_PAGE];
      const int slot = p % OR_PAGE;
      const int64_t tok = cu_new[r] + i;
      for (int h = 0; h < hkv; ++h)
        for (int e = 0; e < d; ++e) {
          const int64_t src = (tok * hkv + h) * d + e;
          const int64_t kd = ((page * hkv + h) * OR_PAGE + slot) * d + e;
          const int64_t vd = ((page * hkv + h) * d + e) * OR_PAGE + slot;
          memcpy((char *)k_pool + kd * esize, (const char *)k_new + src * esize, esize);
          memcpy((char *)v_pool + vd * esize, (const char *)v_new + src * esize, esize);
        }
    }
  }
  return 0;
}

/* Handoff pack: request req_ids[n] with seq_lens[n] tokens goes to
 * out[off[n] + (((layer*2 + c)*Hkv + h)*len + t)*d + e], c = 0 for K, 1 for V.
 * Pools carry a leading layer dimension of num_pages pages each.  Bit copy. */
int oracle_pack(int esize, int hkv, int d, int num_layers, const void *k_pool,
                const void *v_pool, int num_pages, const int32_t *page_table, int pt_stride,
                const int32_t *req_ids, const int32_t *seq_lens, const int64_t *off, int nh,
                void *out) {
  for (int n = 0; n < nh; ++n) {
    const int r = req_ids[n], len = seq_lens[n];
    for (int layer = 0; layer < num_layers; ++layer)
      for (int c = 0; c < 2; ++c)
        for (int h = 0; h < hkv; ++h)
          for (int t = 0; t < len; ++t) {
            const int64_t page = page_table[(int64_t)r * pt_stride + t / OR_PAGE];
            const int slot = t % OR_PAGE;
            const int64_t lp = (int64_t)layer * num_pages + page;
            for (int e = 0; e < d; ++e) {
              const int64_t dst = off[n] + ((((int64_t)layer * 2 + c) * hkv + h) * len + t) * d + e;
              int64_t src;
              const void *pool;
              if (c == 0) {
                src = ((lp * hkv + h) * OR_PAGE + slot) * d + e;
                pool = k_pool;
              } else {
                src = ((lp * hkv + h) * d + e) * OR_PAGE + slot;
                pool = v_pool;
              }
              memcpy((char *)out + dst * esize, (const char *)pool + src * esize, esize);
            }
          }
  }
  return 0;
}

/* Handoff unpack on the receiving instance: the inverse index map of
 * oracle_pack.  Element (layer, c, h, t, e) of handoff n, read from
 * in[off[n] + (((layer*2 + c)*Hkv + h)*len + t)*d + e], goes to page
 * page_table[r*stride + t/16], slot t % 16 of request r = req_ids[n] in the
 * destination pools.  Slots past len are left untouched.  Bit copy. */
int oracle_unpack(int esize, int hkv, int d, int num_layers, const void *in,
                  const int64_t *off, const int32_t *req_ids, const int32_t *seq_lens, int nh,
                  void *k_pool, void *v_pool, int num_pages, const int32_t *page_table,
                  int pt_stride) {
  for (int n = 0; n < nh; ++n) {
    const int r = req_ids[n], len = seq_lens[n];
    for (int layer = 0; layer < num_layers; ++layer)
      for (int c = 0; c < 2; ++c)
        for (int h = 0; h < hkv; ++h)
          for (int t = 0; t < len; ++t) {
            const int64_t page = page_table[(int64_t)r * pt_stride + t / OR_PAGE];
            const int slot = t % OR_PAGE;
            const int64_t lp = (int64_t)layer * num_pages + page;
            for (int e = 0; e < d; ++e) {
              const int64_t src = off[n] + ((((int64_t)layer * 2 + c) * hkv + h) * len + t) * d + e;
              int64_t dst;
              void *pool;
              if (c == 0) {
                dst = ((lp * hkv + h) * OR_PAGE + slot) * d + e;
                pool = k_pool;
              } else {
                dst = ((lp * hkv + h) * d + e) * OR_PAGE + slot;
                pool = v_pool;
              }
              memcpy((char *)pool + dst * esize, (const char *)in + src * esize, esize);
            }
          }
  }
  return 0;
}
