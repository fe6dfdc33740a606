/*
 * GVA decode-step oracle: a plain, slow, fp64 CPU implementation of one
 * decode step of Grouped Value Attention with decoupled RoPE.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header, table or constant with the
 * HIP library.
 *
 * Everything here follows the paper "Grouped Value Attention: Efficient KV
 * Caching via On-Demand Key Reconstruction":
 *   - Algorithm 1 (one decode step of GVA with decoupled RoPE): append the new
 *     value rows and the rotated positional key, rotate the query's positional
 *     slice, absorb M_h into the query, score every cached position, apply the
 *     scaled softmax and weight the values;
 *   - eq. (absorb), Section 3.2: the content score q_h (v_j M_h)^T equals
 *     (q_h M_h^T) v_j^T, so the absorbed query is q~_h = q_h M_h^T;
 *   - eq. (knope)/(krope) and the decoupled score, Section 3.3: the score is
 *     the absorbed content term plus q^rope . k^rope_j with one shared,
 *     already-rotated positional key per position; scores are scaled by
 *     1/sqrt(d_qk), d_qk = d_n + d_r.
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - RoPE acts on interleaved pairs (2i, 2i+1) with frequency
 *     theta_i = base^(-2i/d_r), counter-clockwise, row-vector form x R_p^T;
 *     the angle p*theta_i is formed in fp64;
 *   - positions are 0-based; the query of a sequence with L cached rows sits at
 *     position L-1 (Algorithm 1 appends the current token before attending);
 *   - head h reads value group g(h) = h / (H/G) (contiguous GQA grouping);
 *   - the query row is [content slice (d_c) | positional slice (d_r)];
 *   - M is stored [H][d_v][d_c]: M_h maps a d_v-wide value to a d_c-wide key;
 *   - an empty row range gives o = 0 and lse = -inf.
 *
 * All arithmetic is fp64 on values upcast exactly from their storage type.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* storage type codes understood by every entry point */
#define ORC_F64 0
#define ORC_F32 1
#define ORC_BF16 2

static double ld(const void* base, int64_t i, int dt) {
  if (dt == ORC_F64) return ((const double*)base)[i];
  if (dt == ORC_F32) return (double)((const float*)base)[i];
  /* bf16: the 16 high bits of an IEEE binary32 */
  uint32_t bits = (uint32_t)((const uint16_t*)base)[i] << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

/* Round a double to the nearest bfloat16 (8 significant bits, binary32
 * exponent range), ties to even, in ONE rounding step.  Returns the bits. */
uint16_t gva_oracle_round_bf16(double x) {
  if (isnan(x)) return (uint16_t)0x7FC0;
  double ax = fabs(x);
  double r;
  if (ax == 0.0 || isinf(x)) {
    r = x;
  } else {
    int e;
    frexp(ax, &e);                       /* ax = f * 2^e, 0.5 <= f < 1 */
    int qexp = e - 8;                    /* quantum of an 8-bit significand */
    if (qexp < -133) qexp = -133;        /* bf16 subnormal quantum 2^-133 */
    double scaled = ldexp(x, -qexp);     /* exact: power-of-two scaling */
    double n = nearbyint(scaled);        /* default mode: ties to even */
    r = ldexp(n, qexp);
    if (fabs(r) >= ldexp(1.0, 128)) r = copysign(INFINITY, x);
  }
  float f = (float)r;                    /* exact: r has <= 8 significant bits */
  uint32_t bits;
  memcpy(&bits, &f, sizeof bits);
  return (uint16_t)(bits >> 16);
}

static void st(void* base, int64_t i, int dt, double x) {
  if (dt == ORC_F64) ((double*)base)[i] = x;
  else if (dt == ORC_F32) ((float*)base)[i] = (float)x; /* C cast: nearest-even */
  else ((uint16_t*)base)[i] = gva_oracle_round_bf16(x);
}

/* RoPE of one d_r-wide row at position pos (row-vector form y = x R_pos^T). */
void gva_oracle_rope(const double* x, int d_r, int64_t pos, double base, double* y) {
  for (int i = 0; i < d_r / 2; ++i) {
    double theta = pow(base, -2.0 * (double)i / (double)d_r);
    double a = (double)pos * theta;
    double c = cos(a), s = sin(a);
    double x0 = x[2 * i], x1 = x[2 * i + 1];
    y[2 * i] = x0 * c - x1 * s;
    y[2 * i + 1] = x0 * s + x1 * c;
  }
}

/* Algorithm 1, the cache-append steps: for each new row r,
 *   V[seq_r, g, pos_r, :] <- v_new[r, g, :]           for every group g
 *   kr[seq_r, pos_r, :]   <- RoPE(kr_new[r, :], pos_r)  (eq. krope)
 * Rows whose seq/pos fall outside the cache are skipped; returns how many. */
int gva_oracle_append(int B, int G, int T_max, int d_v, int d_r,
                      void* v_cache, void* kr_cache, int dt_cache,
                      const void* v_new, const void* kr_new, int dt_new,
                      const int32_t* seq, const int32_t* pos, int n_rows,
                      double rope_base) {
  int skipped = 0;
  double* raw = (double*)malloc(sizeof(double) * (size_t)(d_r > 0 ? d_r : 1));
  double* rot = (double*)malloc(sizeof(double) * (size_t)(d_r > 0 ? d_r : 1));
  for (int r = 0; r < n_rows; ++r) {
    int b = seq[r], p = pos[r];
    if (b < 0 || b >= B || p < 0 || p >= T_max) { ++skipped; continue; }
    for (int g = 0; g < G; ++g)
      for (int i = 0; i < d_v; ++i) {
        double x = ld(v_new, ((int64_t)r * G + g) * d_v + i, dt_new);
        st(v_cache, (((int64_t)b * G + g) * T_max + p) * d_v + i, dt_cache, x);
      }
    for (int j = 0; j < d_r; ++j) raw[j] = ld(kr_new, (int64_t)r * d_r + j, dt_new);
    gva_oracle_rope(raw, d_r, p, rope_base, rot);
    for (int j = 0; j < d_r; ++j)
      st(kr_cache, ((int64_t)b * T_max + p) * d_r + j, dt_cache, rot[j]);
  }
  free(raw);
  free(rot);
  return skipped;
}

/* Algorithm 1, the query steps for one (b, h):
 *   q^rope <- q^rope R_p^T  at p = L-1;
 *   q~     <- q^nope M_h^T  (eq. absorb), i.e. q~[i] = sum_k q^nope[k] M_h[i][k]. */
static void absorb_one(int H, int d_v, int d_c, int d_r, const void* q, int dt_q,
                       const void* m, int dt_m, int b, int h, int64_t pos,
                       double rope_base, double* q_abs, double* q_rot) {
  const int64_t qrow = ((int64_t)b * H + h) * (d_c + d_r);
  for (int i = 0; i < d_v; ++i) {
    double acc = 0.0;
    for (int k = 0; k < d_c; ++k)
      acc += ld(q, qrow + k, dt_q) * ld(m, ((int64_t)h * d_v + i) * d_c + k, dt_m);
    q_abs[i] = acc;
  }
  if (d_r > 0) {
    double* raw = (double*)malloc(sizeof(double) * (size_t)d_r);
    for (int j = 0; j < d_r; ++j) raw[j] = ld(q, qrow + d_c + j, dt_q);
    gva_oracle_rope(raw, d_r, pos, rope_base, q_rot);
    free(raw);
  }
}

void gva_oracle_absorb(int B, int H, int d_v, int d_c, int d_r,
                       const void* q, int dt_q, const void* m, int dt_m,
                       const int32_t* lens, double rope_base,
                       double* q_abs /* [B][H][d_v] */, double* q_rot /* [B][H][d_r] */) {
  for (int b = 0; b < B; ++b)
    for (int h = 0; h < H; ++h) {
      int64_t p = lens[b] > 0 ? lens[b] - 1 : 0;
      absorb_one(H, d_v, d_c, d_r, q, dt_q, m, dt_m, b, h, p, rope_base,
                 q_abs + ((int64_t)b * H + h) * d_v,
                 q_rot + ((int64_t)b * H + h) * (d_r > 0 ? d_r : 0));
    }
}

/* Algorithm 1, the attention steps, for every (b, h), over cached rows
 * t in [t_begin[b], t_end[b]) (default [0, lens[b])):
 *   s[t] = scale * ( q~ . V[b, g(h), t, :] + q^rope . kr[b, t, :] )
 *   o    = sum_t softmax(s)[t] V[b, g(h), t, :],   lse = log sum_t exp(s[t]).
 * scale <= 0 selects 1/sqrt(d_c + d_r).  Writes o [B][H][d_v], lse [B][H];
 * optionally the absorbed query q_abs [B][H][d_v] and q_rot [B][H][d_r]. */
void gva_oracle_decode(int B, int H, int G, int T_max, int d_v, int d_c, int d_r,
                       const void* q, int dt_q, const void* m, int dt_m,
                       const void* v_cache, const void* kr_cache, int dt_cache,
                       const int32_t* lens, const int32_t* t_begin, const int32_t* t_end,
                       double scale, double rope_base, int n_threads,
                       double* o, double* lse, double* q_abs_out, double* q_rot_out) {
  if (scale <= 0.0) scale = 1.0 / sqrt((double)(d_c + d_r));
  const int hpg = H / G;
  const int n_pairs = B * H;
#ifdef _OPENMP
  if (n_threads > 0) omp_set_num_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int bh = 0; bh < n_pairs; ++bh) {
    const int b = bh / H, h = bh % H, g = h / hpg;
    int L = lens[b];
    if (L < 0) L = 0;
    if (L > T_max) L = T_max;
    int t0 = t_begin ? t_begin[b] : 0;
    int t1 = t_end ? t_end[b] : L;
    if (t0 < 0) t0 = 0;
    if (t1 > L) t1 = L;
    double* qa = (double*)malloc(sizeof(double) * (size_t)d_v);
    double* qr = (double*)malloc(sizeof(double) * (size_t)(d_r > 0 ? d_r : 1));
    const int64_t p = L > 0 ? L - 1 : 0;
    absorb_one(H, d_v, d_c, d_r, q, dt_q, m, dt_m, b, h, p, rope_base, qa, qr);
    if (q_abs_out) memcpy(q_abs_out + (int64_t)bh * d_v, qa, sizeof(double) * (size_t)d_v);
    if (q_rot_out && d_r > 0) memcpy(q_rot_out + (int64_t)bh * d_r, qr, sizeof(double) * (size_t)d_r);

    double* out = o + (int64_t)bh * d_v;
    for (int i = 0; i < d_v; ++i) out[i] = 0.0;
    if (t1 <= t0) {
      lse[bh] = -INFINITY;
      free(qa);
      free(qr);
      continue;
    }
    const int n = t1 - t0;
    double* s = (double*)malloc(sizeof(double) * (size_t)n);
    const int64_t vbase = ((int64_t)b * G + g) * T_max;
    for (int t = 0; t < n; ++t) {
      const int64_t row = vbase + t0 + t;
      double content = 0.0, positional = 0.0;
      for (int i = 0; i < d_v; ++i) content += qa[i] * ld(v_cache, row * d_v + i, dt_cache);
      for (int j = 0; j < d_r; ++j)
        positional += qr[j] * ld(kr_cache, ((int64_t)b * T_max + t0 + t) * d_r + j, dt_cache);
      s[t] = scale * (content + positional);
    }
    double mx = -INFINITY;
    for (int t = 0; t < n; ++t) mx = s[t] > mx ? s[t] : mx;
    double z = 0.0;
    for (int t = 0; t < n; ++t) {
      double w = exp(s[t] - mx);
      z += w;
      const int64_t row = vbase + t0 + t;
      for (int i = 0; i < d_v; ++i) out[i] += w * ld(v_cache, row * d_v + i, dt_cache);
    }
    for (int i = 0; i < d_v; ++i) out[i] /= z;
    lse[bh] = mx + log(z);
    free(s);
    free(qa);
    free(qr);
  }
}

/* Prefill: Algorithm 1's loop run for every prompt position at once, with
 * causal attention (training uses the same content-position split with
 * standard causal attention, Section 3.3).  Each sequence's N query rows
 * are the last N of its L cached rows, so query i sits at position
 * p = L - N + i and sees rows 0..p.  For every (b, i, h) with p >= 0:
 *   q~ = q^nope M_h^T,  q^ = RoPE(q^rope, p)
 *   s[t] = scale * ( q~ . V[b, g(h), t, :] + q^ . kr[b, t, :] ),  t <= p
 *   o = sum_t softmax(s)[t] V[b, g(h), t, :],  lse = log sum_t exp(s[t]);
 * rows with p < 0 give o = 0, lse = -inf.  scale <= 0 selects
 * 1/sqrt(d_c + d_r).  q [B][N][H][d_c+d_r], o [B][N][H][d_v], lse [B][N][H]. */
void gva_oracle_prefill(int B, int N, int H, int G, int T_max, int d_v, int d_c, int d_r,
                        const void* q, int dt_q, const void* m, int dt_m,
                        const void* v_cache, const void* kr_cache, int dt_cache,
                        const int32_t* lens, double scale, double rope_base, int n_threads,
                        double* o, double* lse) {
  if (scale <= 0.0) scale = 1.0 / sqrt((double)(d_c + d_r));
  const int hpg = H / G;
  const int64_t n_rows = (int64_t)B * N * H;
#ifdef _OPENMP
  if (n_threads > 0) omp_set_num_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int64_t r = 0; r < n_rows; ++r) {
    const int h = (int)(r % H);
    const int i = (int)((r / H) % N);
    const int b = (int)(r / ((int64_t)H * N));
    const int g = h / hpg;
    int L = lens[b];
    if (L < 0) L = 0;
    if (L > T_max) L = T_max;
    const int64_t p = (int64_t)L - N + i;
    double* out = o + r * d_v;
    for (int k = 0; k < d_v; ++k) out[k] = 0.0;
    if (p < 0) {
      lse[r] = -INFINITY;
      continue;
    }
    double* qa = (double*)malloc(sizeof(double) * (size_t)d_v);
    double* qr = (double*)malloc(sizeof(double) * (size_t)(d_r > 0 ? d_r : 1));
    double* s = (double*)malloc(sizeof(double) * (size_t)(p + 1));
    /* q is [B*N][H][W]: row (b*N + i) */
    absorb_one(H, d_v, d_c, d_r, q, dt_q, m, dt_m, b * N + i, h, p, rope_base, qa, qr);
    const int64_t vbase = ((int64_t)b * G + g) * T_max;
    for (int64_t t = 0; t <= p; ++t) {
      double content = 0.0, positional = 0.0;
      for (int k = 0; k < d_v; ++k) content += qa[k] * ld(v_cache, (vbase + t) * d_v + k, dt_cache);
      for (int j = 0; j < d_r; ++j)
        positional += qr[j] * ld(kr_cache, ((int64_t)b * T_max + t) * d_r + j, dt_cache);
      s[t] = scale * (content + positional);
    }
    double mx = -INFINITY;
    for (int64_t t = 0; t <= p; ++t) mx = s[t] > mx ? s[t] : mx;
    double z = 0.0;
    for (int64_t t = 0; t <= p; ++t) {
      double w = exp(s[t] - mx);
      z += w;
      for (int k = 0; k < d_v; ++k) out[k] += w * ld(v_cache, (vbase + t) * d_v + k, dt_cache);
    }
    for (int k = 0; k < d_v; ++k) out[k] /= z;
    lse[r] = mx + log(z);
    free(qa);
    free(qr);
    free(s);
  }
}

/* GVA without decoupled RoPE (Section 3.2: the ordinary-RoPE variants the
 * paper evaluates, which cannot absorb M_h at decode), for every (b, h):
 *   k_t = RoPE(V[b, g(h), t, :] M_h, t + shift)        (key reconstructed,
 *                                                        rotated over d_c)
 *   q'  = RoPE(q[b, h, :], L-1 + shift)
 *   s[t] = scale * q' . k_t,   o = sum_t softmax(s)[t] V[b, g(h), t, :]
 * RoPE here acts on the whole d_c-wide key (theta_i = base^(-2i/d_c)).
 * scale <= 0 selects 1/sqrt(d_c).  q is [B][H][d_c].  shift moves every
 * position by the same amount (the scores depend only on differences). */
void gva_oracle_rope_decode(int B, int H, int G, int T_max, int d_v, int d_c,
                            const void* q, int dt_q, const void* m, int dt_m,
                            const void* v_cache, int dt_cache, const int32_t* lens,
                            double scale, double rope_base, int64_t shift, int n_threads,
                            double* o, double* lse) {
  if (scale <= 0.0) scale = 1.0 / sqrt((double)d_c);
  const int hpg = H / G;
  const int n_pairs = B * H;
#ifdef _OPENMP
  if (n_threads > 0) omp_set_num_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int bh = 0; bh < n_pairs; ++bh) {
    const int b = bh / H, h = bh % H, g = h / hpg;
    int L = lens[b];
    if (L < 0) L = 0;
    if (L > T_max) L = T_max;
    double* out = o + (int64_t)bh * d_v;
    for (int i = 0; i < d_v; ++i) out[i] = 0.0;
    if (L == 0) { lse[bh] = -INFINITY; continue; }
    double* qraw = (double*)malloc(sizeof(double) * (size_t)d_c);
    double* qrot = (double*)malloc(sizeof(double) * (size_t)d_c);
    double* k = (double*)malloc(sizeof(double) * (size_t)d_c);
    double* krot = (double*)malloc(sizeof(double) * (size_t)d_c);
    double* s = (double*)malloc(sizeof(double) * (size_t)L);
    for (int c = 0; c < d_c; ++c) qraw[c] = ld(q, (int64_t)bh * d_c + c, dt_q);
    gva_oracle_rope(qraw, d_c, (int64_t)(L - 1) + shift, rope_base, qrot);
    const int64_t vbase = ((int64_t)b * G + g) * T_max;
    for (int t = 0; t < L; ++t) {
      for (int c = 0; c < d_c; ++c) {         /* k = v M_h: k[c] = sum_i v[i] M_h[i][c] */
        double acc = 0.0;
        for (int i = 0; i < d_v; ++i)
          acc += ld(v_cache, (vbase + t) * d_v + i, dt_cache) * ld(m, ((int64_t)h * d_v + i) * d_c + c, dt_m);
        k[c] = acc;
      }
      gva_oracle_rope(k, d_c, (int64_t)t + shift, rope_base, krot);
      double dot = 0.0;
      for (int c = 0; c < d_c; ++c) dot += qrot[c] * krot[c];
      s[t] = scale * dot;
    }
    double mx = -INFINITY;
    for (int t = 0; t < L; ++t) mx = s[t] > mx ? s[t] : mx;
    double z = 0.0;
    for (int t = 0; t < L; ++t) {
      double w = exp(s[t] - mx);
      z += w;
      for (int i = 0; i < d_v; ++i) out[i] += w * ld(v_cache, (vbase + t) * d_v + i, dt_cache);
    }
    for (int i = 0; i < d_v; ++i) out[i] /= z;
    lse[bh] = mx + log(z);
    free(qraw); free(qrot); free(k); free(krot); free(s);
  }
}

/* Log-sum-exp merge of partial results over disjoint row ranges:
 *   LSE = log sum_s exp(lse_s),  o = sum_s exp(lse_s - LSE) o_s.
 * Partials with lse_s = -inf carry no rows and are skipped; if all are, the
 * result is o = 0, LSE = -inf.  o_part is [rows][S][d_v], lse_part [rows][S]. */
void gva_oracle_combine(int rows, int S, int d_v, const double* o_part,
                        const double* lse_part, double* o, double* lse) {
  for (int r = 0; r < rows; ++r) {
    double mx = -INFINITY;
    for (int s = 0; s < S; ++s) {
      double x = lse_part[(int64_t)r * S + s];
      if (x > mx) mx = x;
    }
    double* out = o + (int64_t)r * d_v;
    for (int i = 0; i < d_v; ++i) out[i] = 0.0;
    if (mx == -INFINITY) { lse[r] = -INFINITY; continue; }
    double z = 0.0;
    for (int s = 0; s < S; ++s) {
      double x = lse_part[(int64_t)r * S + s];
      if (x == -INFINITY) continue;
      z += exp(x - mx);
    }
    double big = mx + log(z);
    for (int s = 0; s < S; ++s) {
      double x = lse_part[(int64_t)r * S + s];
      if (x == -INFINITY) continue;
      double w = exp(x - big);
      for (int i = 0; i < d_v; ++i) out[i] += w * o_part[((int64_t)r * S + s) * d_v + i];
    }
    lse[r] = big;
  }
}

/* Matched grouped-query attention decode (the GQA baseline of Section 2):
 * explicit key cache K [B][G][T_max][d_k], the query's first d_k entries,
 *   o = softmax(q K^T * scale) V,  scale <= 0 selects 1/sqrt(d_k).
 * K is taken as stored (already rotated), as a standard GQA cache is. */
void gva_oracle_gqa_decode(int B, int H, int G, int T_max, int d_v, int d_k, int q_stride,
                           const void* q, int dt_q, const void* k_cache, const void* v_cache,
                           int dt_cache, const int32_t* lens, double scale, int n_threads,
                           double* o, double* lse) {
  if (scale <= 0.0) scale = 1.0 / sqrt((double)d_k);
  const int hpg = H / G;
  const int n_pairs = B * H;
#ifdef _OPENMP
  if (n_threads > 0) omp_set_num_threads(n_threads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int bh = 0; bh < n_pairs; ++bh) {
    const int b = bh / H, h = bh % H, g = h / hpg;
    int L = lens[b];
    if (L < 0) L = 0;
    if (L > T_max) L = T_max;
    double* out = o + (int64_t)bh * d_v;
    for (int i = 0; i < d_v; ++i) out[i] = 0.0;
    if (L == 0) { lse[bh] = -INFINITY; continue; }
    double* s = (double*)malloc(sizeof(double) * (size_t)L);
    const int64_t base = ((int64_t)b * G + g) * T_max;
    for (int t = 0; t < L; ++t) {
      double acc = 0.0;
      for (int i = 0; i < d_k; ++i)
        acc += ld(q, (int64_t)bh * q_stride + i, dt_q) * ld(k_cache, (base + t) * d_k + i, dt_cache);
      s[t] = scale * acc;
    }
    double mx = -INFINITY;
    for (int t = 0; t < L; ++t) mx = s[t] > mx ? s[t] : mx;
    double z = 0.0;
    for (int t = 0; t < L; ++t) {
      double w = exp(s[t] - mx);
      z += w;
      for (int i = 0; i < d_v; ++i) out[i] += w * ld(v_cache, (base + t) * d_v + i, dt_cache);
    }
    for (int i = 0; i < d_v; ++i) out[i] /= z;
    lse[bh] = mx + log(z);
    free(s);
  }
}

int gva_oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
