/*
 * AECCT inference oracle -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg use it.
 *
 * Plain scalar loops over one word at a time; OpenMP only splits independent
 * words across threads.  Build with -ffp-contract=off and no fast-math: every
 * fused multiply-add below is written as fmaf and nothing else is fused.
 *
 * Canonical fp32 evaluation order (chosen where the paper fixes none):
 *   TREE(v, w)  pairwise sum: v[t] += v[t + w/2] for t < w/2, then recurse on
 *               the first half (w a power of two);
 *   SEQ         left-to-right from 0 in ascending index;
 *   DOT         q.k as a multiply followed by fused multiply-adds in ascending
 *               index order; a head of 16 dimensions forms its two 8-dimension
 *               halves that way and adds them (low half + high half);
 *   EXP2        oracle_exp2 below (2^x, floor split, minimax degree-5 polynomial);
 *   RSQRT       oracle_rsqrt below (three Newton steps from a bit-level seed).
 */
#include "aecct_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_MAX_TREE 8192

static int64_t lin_in(const oracle_model *M, int kind) {
  return kind == ORC_FF2 ? M->d_ff : M->d;
}
static int64_t lin_out(const oracle_model *M, int kind) {
  return kind == ORC_FF1 ? M->d_ff : M->d;
}

/* Pairwise summation of w values, w a power of two (canonical order TREE). */
float oracle_tree_sum(const float *v, int32_t w) {
  float buf[ORC_MAX_TREE];
  memcpy(buf, v, sizeof(float) * (size_t)w);
  while (w > 1) {
    int32_t h = w / 2;
    for (int32_t t = 0; t < h; ++t) buf[t] = buf[t] + buf[t + h];
    w = h;
  }
  return buf[0];
}

/*
 * 2^x, the exponential of the attention softmax (Section 3, CASA; Section 4.2,
 * HPSA) taken in base 2: softmax(s) = 2^(s log2 e) / sum, with log2 e folded
 * into the scores.  x is clamped to [-125, 128] (the result stays a normal
 * number or becomes +inf from 2^128 on, and k below fits an int), split into
 * k = floor(x) and r = min(x - k, 1 - 2^-24) in [0, 1) (x - k is exact except
 * for x in (-1, 0), where it is rounded once and can round up to 1; the min
 * keeps r below 1 then), and 2^x = 2^k p(r) with
 *   p(r) = 1 + a1 r + a2 r^2 + a3 r^3 + a4 r^4 + a5 r^5,
 * the degree-5 polynomial with constant term 1 (so that 2^x is exact at
 * integers) whose maximum relative error against 2^r on [0, 1] is least
 * (5.2e-8, found by linear programming over 20000 points of the interval),
 * coefficients rounded to fp32.  Horner with fmaf, then the exact scaling by
 * 2^k.
 * Pin: relative error below 3e-7 over [-125, 64]; exact at integers; +inf
 * from 128.
 */
static const float exp2_coef[6] = {1.0f,           0x1.62e4f0p-1f, 0x1.ebd24ep-3f,
                                   0x1.c98e60p-5f, 0x1.2552ccp-7f, 0x1.f08ff4p-10f};

float oracle_exp2(float x) {
  if (x < -125.0f) x = -125.0f;
  if (x > 128.0f) x = 128.0f;
  const float k = floorf(x);
  float r = x - k;
  if (r > 0x1.fffffep-1f) r = 0x1.fffffep-1f;
  float p = exp2_coef[5];
  for (int j = 4; j >= 0; --j) p = fmaf(p, r, exp2_coef[j]);
  return ldexpf(p, (int)k);
}

/*
 * 1/sqrt(v) for v > 0, the normaliser of LayerNorm: the bit-level seed
 * 0x5F3759DF - (bits(v) >> 1) (Lomont, "Fast inverse square root", 2003),
 * then three Newton steps y <- y (3/2 - (v/2) y^2).
 * Pin: within 4 ulp of 1/sqrt(v) in double over the LayerNorm range.
 */
float oracle_rsqrt(float v) {
  const float h = 0.5f * v;
  uint32_t bits;
  memcpy(&bits, &v, sizeof bits);
  bits = 0x5F3759DFu - (bits >> 1);
  float y;
  memcpy(&y, &bits, sizeof y);
  for (int it = 0; it < 3; ++it) {
    float t = y * y;
    t = fmaf(-h, t, 1.5f);
    y = y * t;
  }
  return y;
}

/* Score scale of the scaled queries: fp32(log2(e) / sqrt(d_h)). */
float oracle_query_scale(int32_t dh) {
  return (float)(1.4426950408889634074 / sqrt((double)dh));
}

/*
 * HPSA masks (Section 4.2, Fig. 2-3).  Tokens 0..n-1 are variable nodes and
 * n..n+m-1 check nodes (Section 3: h(y) = [|y|, 1-2s(y)]).  A is the Tanner
 * graph adjacency; M1 (first ring, c->v and v->c) = A != 0, M2 (second ring,
 * v->v and c->c) = A.A != 0, which keeps the diagonal so that M1 and M2 split
 * the ECCT mask of Section 3 (distance <= 2) exactly.
 * Pin: symmetric, disjoint, union = BFS distance <= 2, closed-form counts.
 */
void oracle_masks(const uint8_t *H, int32_t m, int32_t n, uint8_t *M1, uint8_t *M2) {
  const int32_t L = n + m;
  memset(M1, 0, (size_t)L * L);
  memset(M2, 0, (size_t)L * L);
  for (int32_t j = 0; j < m; ++j)
    for (int32_t i = 0; i < n; ++i)
      if (H[(int64_t)j * n + i]) {
        M1[(int64_t)i * L + n + j] = 1;
        M1[(int64_t)(n + j) * L + i] = 1;
      }
  for (int32_t a = 0; a < L; ++a)
    for (int32_t k = 0; k < L; ++k)
      if (M1[(int64_t)a * L + k])
        for (int32_t b = 0; b < L; ++b)
          if (M1[(int64_t)k * L + b]) M2[(int64_t)a * L + b] = 1;
}

/*
 * Pre-processing h(y) of Section 3: bin(y) = 0.5(1 - sign(y)), i.e. bit 1 iff
 * y < 0; syndrome s = H bin(y) over GF(2); tokens [|y|, 1 - 2s].
 * Pin: every noiseless codeword gives s = 0; a single flipped bit gives the
 * matching column of H.
 */
void oracle_preprocess(const uint8_t *H, int32_t m, int32_t n, const float *y, float *t) {
  for (int32_t i = 0; i < n; ++i) t[i] = fabsf(y[i]);
  for (int32_t j = 0; j < m; ++j) {
    int s = 0;
    for (int32_t i = 0; i < n; ++i)
      if (H[(int64_t)j * n + i] && y[i] < 0.0f) s ^= 1;
    t[n + j] = s ? -1.0f : 1.0f;
  }
}

/*
 * Absmax int8 activation quantisation, Eq. 2 with Q_b = 127, applied per token
 * row: alpha = max|x|, q = RoundClip(x * (Q_b / alpha), -Q_b, Q_b) with
 * Q_b / alpha rounded to fp32 and the product x * (Q_b / alpha) rounded once,
 * half to even, straight to an integer (the product of two floats is exact in
 * double).  An all-zero row gives q = 0 and alpha = 0.
 * Pin: |q| <= 127, the argmax maps to +-127, sign kept, monotone, error bound.
 */
void oracle_quant_rows(const float *x, int64_t rows, int32_t K, int8_t *q, float *r) {
  for (int64_t i = 0; i < rows; ++i) {
    const float *xi = x + i * K;
    int8_t *qi = q + i * K;
    float a = 0.0f;
    for (int32_t c = 0; c < K; ++c) {
      float v = fabsf(xi[c]);
      if (v > a) a = v;
    }
    if (a == 0.0f) {
      memset(qi, 0, (size_t)K);
      r[i] = 0.0f;
      continue;
    }
    float inv = 127.0f / a;
    for (int32_t c = 0; c < K; ++c) {
      double v = rint((double)xi[c] * (double)inv);
      if (v > 127.0) v = 127.0;
      if (v < -127.0) v = -127.0;
      qi[c] = (int8_t)v;
    }
    r[i] = a;
  }
}

/*
 * The same quantiser with one alpha per word (Section 4.1 states alpha = ||x||_inf of the layer
 * input x and calls every scaling factor a scalar): alpha = max |x| over all rows*K values of the
 * word, every row's codes x * fp32(Q_b / alpha) rounded half to even, and every row's r set to
 * that alpha (so the dequantisation of Eq. 3 is unchanged).  An all-zero word gives q = 0, r = 0.
 * Pin: alpha equals the library maximum of |x| over the word; on a word whose rows share one
 * maximum it equals the per-token form bit for bit; |q| <= 127, the argmax maps to +-127, the
 * error bound of Eq. 2 with alpha of the word.
 */
void oracle_quant_word(const float *x, int64_t rows, int32_t K, int8_t *q, float *r) {
  float a = 0.0f;
  for (int64_t e = 0; e < rows * K; ++e) {
    float v = fabsf(x[e]);
    if (v > a) a = v;
  }
  for (int64_t i = 0; i < rows; ++i) r[i] = a;
  if (a == 0.0f) {
    memset(q, 0, (size_t)(rows * K));
    return;
  }
  const float inv = 127.0f / a;
  for (int64_t e = 0; e < rows * K; ++e) {
    double v = rint((double)x[e] * (double)inv);
    if (v > 127.0) v = 127.0;
    if (v < -127.0) v = -127.0;
    q[e] = (int8_t)v;
  }
}

/* Eq. 2 at one quantisation point of a word: per token or per word, as the model says. */
static void quant_act(const oracle_model *M, const float *x, int64_t rows, int32_t K, int8_t *q, float *r) {
  if (M->act_scale_mode == 1)
    oracle_quant_word(x, rows, K, q, r);
  else
    oracle_quant_rows(x, rows, K, q, r);
}

/*
 * AAPLinear at inference, Eq. 3: integer product of the int8 activations and
 * the ternary weights (additions and subtractions only), dequantised by
 * gamma*delta*alpha/Q_b before the bias is added (Section 4.1).  With
 * sq = s / 127 (s = gamma*delta, the caller rounds it to fp32) the scale is
 * alpha * sq and dequant plus bias is one fused multiply-add:
 * out = fma(acc, alpha * sq, b).
 * Pin: accumulators equal an int64 library matmul; zero weights give the bias.
 */
void oracle_linear_rows(const int8_t *q, const float *r, int64_t rows, const int8_t *T, int32_t K,
                        int32_t n_out, float sq, const float *b, float *out, int32_t *acc) {
  for (int64_t i = 0; i < rows; ++i) {
    const int8_t *qi = q + i * K;
    float sc = r[i] * sq;
    for (int32_t o = 0; o < n_out; ++o) {
      int32_t a = 0;
      for (int32_t c = 0; c < K; ++c) a += (int32_t)qi[c] * (int32_t)T[(int64_t)c * n_out + o];
      if (acc) acc[i * n_out + o] = a;
      out[i * n_out + o] = fmaf((float)a, sc, b[o]);
    }
  }
}

/*
 * LayerNorm of the Post-LN block (Section 6): mean and biased variance over
 * the d features (TREE sums), out = (x - mean) / sqrt(var + eps) * g + b,
 * evaluated as fma((x - mean) * RSQRT(var + eps), g, b).
 * Pin: within 1e-5 of the fp64 library layer_norm.
 */
void oracle_layernorm_rows(const float *R, int64_t rows, int32_t d, const float *g, const float *b,
                           float eps, float *out) {
  float e[ORC_MAX_TREE], sq[ORC_MAX_TREE];
  for (int64_t i = 0; i < rows; ++i) {
    const float *ri = R + i * d;
    float mean = oracle_tree_sum(ri, d) / (float)d;
    for (int32_t c = 0; c < d; ++c) {
      e[c] = ri[c] - mean;
      sq[c] = e[c] * e[c];
    }
    float var = oracle_tree_sum(sq, d) / (float)d;
    float rho = oracle_rsqrt(var + eps);
    for (int32_t c = 0; c < d; ++c) out[i * d + c] = fmaf(e[c] * rho, g[c], b[c]);
  }
}

/* Whether key j is allowed for row i of head h: HPSA (Section 4.2) gives heads below h_f the
 * first-ring mask and the others the second-ring mask; CASA (Section 3, the ECCT mask) gives
 * every head their union, the nodes at most two steps away including the node itself. */
static int key_allowed(const oracle_model *M, const uint8_t *M1, const uint8_t *M2, int32_t h, int32_t i,
                       int32_t j) {
  const int64_t e = (int64_t)i * (M->n + M->m) + j;
  if (M->attention == 1) return M1[e] || M2[e];
  return h < M->first_ring_heads ? M1[e] : M2[e];
}

/* DOT of the scaled query of row i with the key of token j, head h (d_h dims): a multiply then
 * fused multiply-adds in ascending dims; with d_h = 16 the two 8-dim halves separately, then
 * their sum. */
static float dot_seq(const float *q, const float *k, int32_t w) {
  float s = q[0] * k[0];
  for (int32_t t = 1; t < w; ++t) s = fmaf(q[t], k[t], s);
  return s;
}
static float score_f32(const float *qkv, int32_t d, int32_t i, int32_t j, int32_t h, int32_t dh) {
  const float *qi = qkv + (int64_t)i * 3 * d + h * dh;
  const float *kj = qkv + (int64_t)j * 3 * d + d + h * dh;
  if (dh == 16) return dot_seq(qi, kj, 8) + dot_seq(qi + 8, kj + 8, 8);
  return dot_seq(qi, kj, dh);
}

/*
 * Head-partitioned self-attention (Section 4.2): heads 0..h_f-1 attend over
 * the first-ring mask M1, the others over the second-ring mask M2 (with
 * attention = 1, the CASA variant of Section 3: every head over M1 | M2).  Per row i
 * and head h the softmax of the scaled dot products over the allowed keys j
 * (ascending) weighs the value rows; the scale is 1/sqrt(d_h) per head.  The
 * query rows arrive already multiplied by log2(e)/sqrt(d_h) (folded into the
 * query map, see oracle_query_scale), so the softmax is taken in base 2:
 * s_j = DOT(q', k_j); the weights are the plain definition e_j = EXP2(s_j)
 * with S = SEQ sum e_j and acc = SEQ fma(e_j, v_j, acc), kept when
 * 2^-64 <= S <= 2^64 (no overflow; every weight clamped at 2^-125 then lies
 * below 2^-61 S); otherwise the row is redone with the usual stabilising
 * shift, e_j = EXP2(s_j - mu), mu = max s_j.  o = acc * (1 / S).  Both forms
 * are the same softmax up to rounding.  Returns 0, or -1 for a row with no
 * allowed key.
 * Pin: within 1e-6 relative of the fp64 dense (-inf)-masked softmax, on rows
 * of either form; a row with one allowed key returns that value row to 3 ulp.
 */
int oracle_attention_word(const oracle_model *M, const uint8_t *M1, const uint8_t *M2,
                          const float *qkv, float *o) {
  const int32_t L = M->n + M->m, d = M->d, dh = M->d / M->heads;
  for (int32_t i = 0; i < L; ++i)
    for (int32_t h = 0; h < M->heads; ++h) {
      float mu = -INFINITY;
      int cnt = 0;
      for (int32_t j = 0; j < L; ++j)
        if (key_allowed(M, M1, M2, h, i, j)) {
          float s = score_f32(qkv, d, i, j, h, dh);
          if (s > mu) mu = s;
          ++cnt;
        }
      if (cnt == 0) return -1;
      float S = 0.0f, acc[ORC_MAX_TREE];
      for (int pass = 0; pass < 2; ++pass) {
        const float shift = pass == 0 ? 0.0f : mu;
        S = 0.0f;
        for (int32_t t = 0; t < dh; ++t) acc[t] = 0.0f;
        for (int32_t j = 0; j < L; ++j)
          if (key_allowed(M, M1, M2, h, i, j)) {
            float s = score_f32(qkv, d, i, j, h, dh);
            float e = oracle_exp2(pass == 0 ? s : s - shift);
            S = S + e;
            const float *vj = qkv + (int64_t)j * 3 * d + 2 * d + h * dh;
            for (int32_t t = 0; t < dh; ++t) acc[t] = fmaf(e, vj[t], acc[t]);
          }
        if (S >= 0x1p-64f && S <= 0x1p64f) break;
      }
      const float rS = 1.0f / S;
      for (int32_t t = 0; t < dh; ++t) o[(int64_t)i * d + h * dh + t] = acc[t] * rS;
    }
  return 0;
}

/*
 * Output head and hard decision (Section 3): per token z_i = W_{d->1} x_i + b1
 * (TREE over d), noise estimate f_o = sum_i z_i W_o[i][o] + b_o (SEQ over the
 * L tokens), soft codeword y * f and bit = bin(y * f) = [y < 0] xor [f < 0].
 * Pin: codeword invariance decode(x_s + e) xor x == decode(1 + x_s e).
 */
void oracle_head_word(const oracle_model *M, const float *X, const float *y, float *f, uint8_t *bits,
                      float *z) {
  const int32_t L = M->n + M->m, d = M->d, n = M->n;
  float zz[ORC_MAX_TREE], p[ORC_MAX_TREE];
  for (int32_t i = 0; i < L; ++i) {
    for (int32_t c = 0; c < d; ++c) p[c] = X[(int64_t)i * d + c] * M->head_w1[c];
    zz[i] = oracle_tree_sum(p, d) + M->head_b1;
    if (z) z[i] = zz[i];
  }
  for (int32_t o = 0; o < n; ++o) {
    float acc = 0.0f;
    for (int32_t i = 0; i < L; ++i) acc = fmaf(zz[i], M->head_wo[(int64_t)i * n + o], acc);
    float fo = acc + M->head_bo[o];
    f[o] = fo;
    bits[o] = (uint8_t)((y[o] < 0.0f) ^ (fo < 0.0f));
  }
}

/* ------------------------------------------------------------------ AAP import */

static int cmp_float(const void *a, const void *b) {
  const float x = *(const float *)a, y = *(const float *)b;
  return (x > y) - (x < y);
}

/*
 * Adaptive Absolute Percentile ternarisation of one weight matrix (Section 4.1,
 * Eq. 1): gamma = Percentile(Abs(W), p) with the paper's p = 0.5; the scale of
 * Eq. 3 is gamma * delta; Ternary(W) = RoundClip(W / (gamma delta + eps), -1, 1)
 * with RoundClip(x, a, b) = max(a, min(b, round(x))).
 * Readings: the percentile is the p-quantile with linear interpolation between
 * the order statistics around p (count - 1) (zero based), computed in double
 * and rounded once to fp32; round is to nearest, ties to even; the quotient is
 * the correctly rounded fp32 division by fp32(fp32(gamma delta) + eps); when
 * that denominator is 0, nonzero weights map to their sign.
 * Pin: gamma equals numpy's median of |W| (p = 0.5) and its linear-method
 * quantile otherwise; the ternary entries equal numpy's float32 division
 * rounded half to even and clipped; zeros / signs / clipping invariants.
 */
int oracle_aap_ternarize(const float *w, int64_t count, float p, float delta, float eps, int8_t *t,
                         float *scale) {
  if (count < 1 || !(p >= 0.0f && p <= 1.0f) || !(delta > 0.0f) || !(eps >= 0.0f)) return -1;
  float *a = (float *)malloc(sizeof(float) * (size_t)count);
  if (!a) return -1;
  for (int64_t i = 0; i < count; ++i) a[i] = fabsf(w[i]);
  qsort(a, (size_t)count, sizeof(float), cmp_float);
  const double pos = (double)p * (double)(count - 1);
  int64_t lo = (int64_t)floor(pos);
  if (lo > count - 1) lo = count - 1;
  const int64_t hi = lo + 1 < count ? lo + 1 : lo;
  const double frac = pos - (double)lo;
  const float gamma = (float)((double)a[lo] + frac * ((double)a[hi] - (double)a[lo]));
  free(a);
  const float s = gamma * delta;
  const float den = s + eps;
  for (int64_t i = 0; i < count; ++i) {
    float r;
    if (den == 0.0f)
      r = w[i] > 0.0f ? 1.0f : (w[i] < 0.0f ? -1.0f : 0.0f);
    else
      r = rintf(w[i] / den);
    if (r > 1.0f) r = 1.0f;
    if (r < -1.0f) r = -1.0f;
    t[i] = (int8_t)r;
  }
  *scale = s;
  return 0;
}

/* ------------------------------------------------------------------ whole decode */

typedef struct {
  float *t, *X, *qkv, *O, *X1, *F, *Y, *R, *bq;
  int8_t *q, *gq;
  float *r, *rg;
  int32_t *acc, *accf;
} word_buf;

static int alloc_buf(const oracle_model *M, word_buf *w) {
  const int64_t L = M->n + M->m, d = M->d, dff = M->d_ff;
  w->t = malloc(sizeof(float) * L);
  w->X = malloc(sizeof(float) * L * d);
  w->qkv = malloc(sizeof(float) * L * 3 * d);
  w->O = malloc(sizeof(float) * L * d);
  w->X1 = malloc(sizeof(float) * L * d);
  w->F = malloc(sizeof(float) * L * dff);
  w->Y = malloc(sizeof(float) * L * (dff > 3 * d ? dff : 3 * d));
  w->R = malloc(sizeof(float) * L * d);
  w->bq = malloc(sizeof(float) * d);
  w->q = malloc((size_t)(L * (dff > d ? dff : d)));
  w->gq = malloc((size_t)(L * dff));
  w->r = malloc(sizeof(float) * L);
  w->rg = malloc(sizeof(float) * L);
  w->acc = malloc(sizeof(int32_t) * L * d);
  w->accf = malloc(sizeof(int32_t) * L * dff);
  return (w->t && w->X && w->qkv && w->O && w->X1 && w->F && w->Y && w->R && w->bq && w->q && w->gq &&
          w->r && w->rg && w->acc && w->accf) ? 0 : -1;
}

static void free_buf(word_buf *w) {
  free(w->t); free(w->X); free(w->qkv); free(w->O); free(w->X1); free(w->F); free(w->Y);
  free(w->R); free(w->bq); free(w->q); free(w->gq); free(w->r); free(w->rg); free(w->acc); free(w->accf);
}

static const int8_t *wmat(const oracle_model *M, int kind, int layer) {
  return M->w[kind] + (int64_t)layer * lin_in(M, kind) * lin_out(M, kind);
}
static const float *bvec(const oracle_model *M, int kind, int layer) {
  return M->bias[kind] + (int64_t)layer * lin_out(M, kind);
}

/* One word through embedding, N encoder blocks and the head (Sections 3, 4, 6). */
static int decode_word(const oracle_model *M, const uint8_t *M1, const uint8_t *M2, const float *y,
                       uint8_t *bits, float *f, word_buf *w, const oracle_taps *tp) {
  const int64_t L = M->n + M->m, d = M->d, dff = M->d_ff;
  /* embedding of the 2n-k input scalars: X_i = t_i * E_i (+ fixed positional row) */
  oracle_preprocess(M->H, M->m, M->n, y, w->t);
  for (int64_t i = 0; i < L; ++i)
    for (int64_t c = 0; c < d; ++c)
      w->X[i * d + c] = fmaf(w->t[i], M->embed[i * d + c], M->pos ? M->pos[i * d + c] : 0.0f);

  const float kq = oracle_query_scale(M->d / M->heads);
  for (int32_t l = 0; l < M->n_layers; ++l) {
    const float *sc = M->scale + (int64_t)l * 6;
    float sq[6];
    for (int k = 0; k < 6; ++k) sq[k] = sc[k] / 127.0f;
    const int64_t LD = L * d;
    if (tp && tp->x_in) memcpy(tp->x_in + l * LD, w->X, sizeof(float) * LD);
    /* a. Q, K, V from the int8 input */
    quant_act(M, w->X, L, (int32_t)d, w->q, w->r);
    if (tp && tp->xq) memcpy(tp->xq + l * LD, w->q, (size_t)LD);
    if (tp && tp->ax) memcpy(tp->ax + l * L, w->r, sizeof(float) * L);
    /* the query map carries the score scale log2(e)/sqrt(d_h) in its dequant scale and bias */
    for (int64_t c = 0; c < d; ++c) w->bq[c] = bvec(M, ORC_Q, l)[c] * kq;
    for (int kind = ORC_Q; kind <= ORC_V; ++kind) {
      oracle_linear_rows(w->q, w->r, L, wmat(M, kind, l), (int32_t)d, (int32_t)d,
                         kind == ORC_Q ? sq[kind] * kq : sq[kind], kind == ORC_Q ? w->bq : bvec(M, kind, l),
                         w->Y, NULL);
      for (int64_t i = 0; i < L; ++i)
        memcpy(w->qkv + i * 3 * d + kind * d, w->Y + i * d, sizeof(float) * d);
    }
    if (tp && tp->qkv) memcpy(tp->qkv + l * 3 * LD, w->qkv, sizeof(float) * 3 * LD);
    /* b. head-partitioned attention */
    if (oracle_attention_word(M, M1, M2, w->qkv, w->O)) return -1;
    if (tp && tp->o) memcpy(tp->o + l * LD, w->O, sizeof(float) * LD);
    /* c. output projection, residual, LN1 */
    quant_act(M, w->O, L, (int32_t)d, w->q, w->r);
    if (tp && tp->oq) memcpy(tp->oq + l * LD, w->q, (size_t)LD);
    if (tp && tp->ao) memcpy(tp->ao + l * L, w->r, sizeof(float) * L);
    oracle_linear_rows(w->q, w->r, L, wmat(M, ORC_O, l), (int32_t)d, (int32_t)d, sq[ORC_O],
                       bvec(M, ORC_O, l), w->Y, w->acc);
    if (tp && tp->acc_o) memcpy(tp->acc_o + l * LD, w->acc, sizeof(int32_t) * LD);
    for (int64_t e = 0; e < LD; ++e) w->R[e] = w->X[e] + w->Y[e];
    oracle_layernorm_rows(w->R, L, (int32_t)d, M->ln1_g + l * d, M->ln1_b + l * d, M->ln_eps, w->X1);
    if (tp && tp->x1) memcpy(tp->x1 + l * LD, w->X1, sizeof(float) * LD);
    /* d. FFN with ReLU, residual, LN2 */
    quant_act(M, w->X1, L, (int32_t)d, w->q, w->r);
    if (tp && tp->x1q) memcpy(tp->x1q + l * LD, w->q, (size_t)LD);
    if (tp && tp->a1) memcpy(tp->a1 + l * L, w->r, sizeof(float) * L);
    oracle_linear_rows(w->q, w->r, L, wmat(M, ORC_FF1, l), (int32_t)d, (int32_t)dff, sq[ORC_FF1],
                       bvec(M, ORC_FF1, l), w->F, w->accf);
    if (tp && tp->acc_ff1) memcpy(tp->acc_ff1 + l * L * dff, w->accf, sizeof(int32_t) * L * dff);
    for (int64_t e = 0; e < L * dff; ++e) w->F[e] = w->F[e] > 0.0f ? w->F[e] : 0.0f;
    quant_act(M, w->F, L, (int32_t)dff, w->gq, w->rg);
    if (tp && tp->gq) memcpy(tp->gq + l * L * dff, w->gq, (size_t)(L * dff));
    if (tp && tp->ag) memcpy(tp->ag + l * L, w->rg, sizeof(float) * L);
    oracle_linear_rows(w->gq, w->rg, L, wmat(M, ORC_FF2, l), (int32_t)dff, (int32_t)d, sq[ORC_FF2],
                       bvec(M, ORC_FF2, l), w->Y, w->acc);
    if (tp && tp->acc_ff2) memcpy(tp->acc_ff2 + l * LD, w->acc, sizeof(int32_t) * LD);
    for (int64_t e = 0; e < LD; ++e) w->R[e] = w->X1[e] + w->Y[e];
    oracle_layernorm_rows(w->R, L, (int32_t)d, M->ln2_g + l * d, M->ln2_b + l * d, M->ln_eps, w->X);
    if (tp && tp->x_out) memcpy(tp->x_out + l * LD, w->X, sizeof(float) * LD);
  }
  oracle_head_word(M, w->X, y, f, bits, tp ? tp->z : NULL);
  return 0;
}

static int check_model(const oracle_model *M) {
  if (M->d <= 0 || M->heads <= 0 || M->d % M->heads) return -1;
  int32_t dh = M->d / M->heads;
  if ((M->d & (M->d - 1)) || (dh & (dh - 1))) return -1;
  if (M->d > ORC_MAX_TREE || M->d_ff > ORC_MAX_TREE || M->n + M->m > ORC_MAX_TREE) return -1;
  if (M->act_scale_mode != 0 && M->act_scale_mode != 1) return -1;
  return 0;
}

int oracle_decode(const oracle_model *M, const float *y, int64_t batch, uint8_t *bits, float *f,
                  int32_t n_threads) {
  if (check_model(M)) return -1;
  const int64_t L = M->n + M->m;
  uint8_t *M1 = malloc((size_t)(L * L)), *M2 = malloc((size_t)(L * L));
  if (!M1 || !M2) { free(M1); free(M2); return -1; }
  oracle_masks(M->H, M->m, M->n, M1, M2);
  int err = 0;
#ifdef _OPENMP
  if (n_threads < 1) n_threads = 1;
#pragma omp parallel num_threads(n_threads) reduction(| : err)
#endif
  {
    word_buf w;
    if (alloc_buf(M, &w)) {
      err |= 1;
    } else {
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
      for (int64_t b = 0; b < batch; ++b)
        if (decode_word(M, M1, M2, y + b * M->n, bits + b * M->n, f + b * M->n, &w, NULL)) err |= 1;
    }
    free_buf(&w);
  }
  free(M1);
  free(M2);
  return err ? -1 : 0;
}

int oracle_decode_taps(const oracle_model *M, const float *y, uint8_t *bits, float *f,
                       const oracle_taps *taps) {
  if (check_model(M)) return -1;
  const int64_t L = M->n + M->m;
  uint8_t *M1 = malloc((size_t)(L * L)), *M2 = malloc((size_t)(L * L));
  word_buf w;
  int err = (!M1 || !M2 || alloc_buf(M, &w)) ? -1 : 0;
  if (!err) {
    oracle_masks(M->H, M->m, M->n, M1, M2);
    err = decode_word(M, M1, M2, y, bits, f, &w, taps);
    free_buf(&w);
  }
  free(M1);
  free(M2);
  return err;
}

/* ------------------------------------------------------------------ fp64 reference mode */

/* Decisions of near-tie codes (test support): where x * 127 / alpha lies within `margin` of a
 * rounding tie k + 1/2 the fp64 decision and a fp32 one may both be right, so the code is taken
 * from `force` (a code list of the same layout, e.g. the canonical mode's) when that code is one
 * of the two neighbours of the tie; stats[0] counts such codes that differ from the fp64
 * decision, stats[1] codes of `force` that differ from it anywhere else. */
typedef struct {
  const int8_t *force;
  double margin;
  int64_t stats[2];
} tie_rule;

/* Eq. 2 in fp64: alpha per row (act_scale_mode 0) or one alpha over all rows (1); codes as
 * rint(x * 127 / alpha) clipped to +-127.  When codes is not NULL the int8 codes are also
 * copied there; when ties is not NULL, near-tie codes follow it (see tie_rule). */
static void quant_rows_f64(const double *x, int64_t rows, int32_t K, int per_word, int32_t *q, double *r,
                           int8_t *codes, tie_rule *ties, int64_t tie_off) {
  double aw = 0.0;
  if (per_word)
    for (int64_t e = 0; e < rows * K; ++e) aw = fmax(aw, fabs(x[e]));
  for (int64_t i = 0; i < rows; ++i) {
    double a = aw;
    if (!per_word)
      for (int32_t c = 0; c < K; ++c) a = fmax(a, fabs(x[i * K + c]));
    r[i] = a;
    for (int32_t c = 0; c < K; ++c) {
      const double u = a == 0.0 ? 0.0 : x[i * K + c] * (127.0 / a);
      double v = fmin(127.0, fmax(-127.0, rint(u)));
      if (ties && ties->force) {
        const double fv = (double)ties->force[tie_off + i * K + c];
        if (fv != v) {
          const double lo = floor(u);
          if (fabs(u - (lo + 0.5)) <= ties->margin && (fv == lo || fv == lo + 1.0)) {
            ++ties->stats[0];
            v = fv;
          } else {
            ++ties->stats[1];
          }
        }
      }
      q[i * K + c] = (int32_t)v;
      if (codes) codes[i * K + c] = (int8_t)v;
    }
  }
}

static void linear_rows_f64(const int32_t *q, const double *r, int64_t rows, const int8_t *T,
                            int32_t K, int32_t n_out, double s, const float *b, double *out) {
  for (int64_t i = 0; i < rows; ++i)
    for (int32_t o = 0; o < n_out; ++o) {
      int64_t a = 0;
      for (int32_t c = 0; c < K; ++c) a += (int64_t)q[i * K + c] * T[(int64_t)c * n_out + o];
      out[i * n_out + o] = (double)a * (s * r[i] / 127.0) + (double)b[o];
    }
}

static void layernorm_f64(double *R, int64_t rows, int32_t d, const float *g, const float *b,
                          double eps) {
  for (int64_t i = 0; i < rows; ++i) {
    double *ri = R + i * d, mean = 0.0, var = 0.0;
    for (int32_t c = 0; c < d; ++c) mean += ri[c];
    mean /= d;
    for (int32_t c = 0; c < d; ++c) var += (ri[c] - mean) * (ri[c] - mean);
    var /= d;
    for (int32_t c = 0; c < d; ++c) ri[c] = (ri[c] - mean) / sqrt(var + eps) * g[c] + b[c];
  }
}

/* Dense attention: softmax(score_scale * q.k) over all L keys with the masked
 * scores set to -inf, libm exp. */
int oracle_attention_dense_f64(const oracle_model *M, const uint8_t *M1, const uint8_t *M2,
                               const double *qkv, double score_scale, double *o) {
  const int32_t L = M->n + M->m, d = M->d, dh = M->d / M->heads;
  double *s = malloc(sizeof(double) * L);
  if (!s) return -1;
  for (int32_t i = 0; i < L; ++i)
    for (int32_t h = 0; h < M->heads; ++h) {
      double mx = -INFINITY;
      for (int32_t j = 0; j < L; ++j) {
        double dot = 0.0;
        for (int32_t t = 0; t < dh; ++t)
          dot += qkv[(int64_t)i * 3 * d + h * dh + t] * qkv[(int64_t)j * 3 * d + d + h * dh + t];
        s[j] = key_allowed(M, M1, M2, h, i, j) ? dot * score_scale : -INFINITY;
        if (s[j] > mx) mx = s[j];
      }
      if (mx == -INFINITY) { free(s); return -1; }
      double S = 0.0;
      for (int32_t j = 0; j < L; ++j) { s[j] = exp(s[j] - mx); S += s[j]; }
      for (int32_t t = 0; t < dh; ++t) {
        double acc = 0.0;
        for (int32_t j = 0; j < L; ++j) acc += s[j] / S * qkv[(int64_t)j * 3 * d + 2 * d + h * dh + t];
        o[(int64_t)i * d + h * dh + t] = acc;
      }
    }
  free(s);
  return 0;
}

/* One word of the fp64 reference decode (embedding, N Post-LN blocks with dense masked
 * attention, head); codes as described in the header, or NULL. */
static int ref64_word(const oracle_model *M, const uint8_t *M1, const uint8_t *M2, const float *yb,
                      uint8_t *bits, double *f, int8_t *codes, tie_rule *ties) {
  const int64_t L = M->n + M->m, d = M->d, dff = M->d_ff, n = M->n;
  const int pw = M->act_scale_mode == 1;
  int err = 0;
  double *X = malloc(sizeof(double) * L * d), *qkv = malloc(sizeof(double) * L * 3 * d);
  double *O = malloc(sizeof(double) * L * d), *Y = malloc(sizeof(double) * L * dff);
  double *X1 = malloc(sizeof(double) * L * d), *r = malloc(sizeof(double) * L);
  int32_t *q = malloc(sizeof(int32_t) * L * dff);
  float *t = malloc(sizeof(float) * L);
  if (!X || !qkv || !O || !Y || !X1 || !r || !q || !t) {
    err = -1;
  } else {
    oracle_preprocess(M->H, M->m, M->n, yb, t);
    for (int64_t i = 0; i < L; ++i)
      for (int64_t c = 0; c < d; ++c)
        X[i * d + c] = (double)t[i] * M->embed[i * d + c] + (M->pos ? M->pos[i * d + c] : 0.0);
    for (int32_t l = 0; l < M->n_layers && !err; ++l) {
      const float *sc = M->scale + (int64_t)l * 6;
      const int64_t lo = (int64_t)l * L * (3 * d + dff);
      int8_t *cl = codes ? codes + lo : NULL;
      quant_rows_f64(X, L, (int32_t)d, pw, q, r, cl, ties, lo);
      for (int kind = ORC_Q; kind <= ORC_V; ++kind) {
        linear_rows_f64(q, r, L, wmat(M, kind, l), (int32_t)d, (int32_t)d, sc[kind], bvec(M, kind, l), Y);
        for (int64_t i = 0; i < L; ++i)
          for (int64_t c = 0; c < d; ++c) qkv[i * 3 * d + kind * d + c] = Y[i * d + c];
      }
      if (oracle_attention_dense_f64(M, M1, M2, qkv, 1.0 / sqrt((double)(d / M->heads)), O)) { err = -1; break; }
      quant_rows_f64(O, L, (int32_t)d, pw, q, r, cl ? cl + L * d : NULL, ties, lo + L * d);
      linear_rows_f64(q, r, L, wmat(M, ORC_O, l), (int32_t)d, (int32_t)d, sc[ORC_O], bvec(M, ORC_O, l), Y);
      for (int64_t e = 0; e < L * d; ++e) X1[e] = X[e] + Y[e];
      layernorm_f64(X1, L, (int32_t)d, M->ln1_g + l * d, M->ln1_b + l * d, M->ln_eps);
      quant_rows_f64(X1, L, (int32_t)d, pw, q, r, cl ? cl + 2 * L * d : NULL, ties, lo + 2 * L * d);
      linear_rows_f64(q, r, L, wmat(M, ORC_FF1, l), (int32_t)d, (int32_t)dff, sc[ORC_FF1], bvec(M, ORC_FF1, l), Y);
      for (int64_t e = 0; e < L * dff; ++e) Y[e] = Y[e] > 0.0 ? Y[e] : 0.0;
      quant_rows_f64(Y, L, (int32_t)dff, pw, q, r, cl ? cl + 3 * L * d : NULL, ties, lo + 3 * L * d);
      linear_rows_f64(q, r, L, wmat(M, ORC_FF2, l), (int32_t)dff, (int32_t)d, sc[ORC_FF2], bvec(M, ORC_FF2, l), X);
      for (int64_t e = 0; e < L * d; ++e) X[e] = X1[e] + X[e];
      layernorm_f64(X, L, (int32_t)d, M->ln2_g + l * d, M->ln2_b + l * d, M->ln_eps);
    }
    if (!err) {
      for (int64_t i = 0; i < L; ++i) {          /* z_i = W_{d->1} x_i + b1, kept in r */
        double z = M->head_b1;
        for (int64_t c = 0; c < d; ++c) z += X[i * d + c] * M->head_w1[c];
        r[i] = z;
      }
      for (int64_t o = 0; o < n; ++o) {
        double acc = M->head_bo[o];
        for (int64_t i = 0; i < L; ++i) acc += r[i] * M->head_wo[i * n + o];
        f[o] = acc;
        bits[o] = (uint8_t)((yb[o] < 0.0f) ^ (acc < 0.0));
      }
    }
  }
  free(X); free(qkv); free(O); free(Y); free(X1); free(r); free(q); free(t);
  return err;
}

int oracle_decode_ref64(const oracle_model *M, const float *y, int64_t batch, uint8_t *bits,
                        double *f, int32_t n_threads) {
  if (check_model(M)) return -1;
  const int64_t L = M->n + M->m, n = M->n;
  uint8_t *M1 = malloc((size_t)(L * L)), *M2 = malloc((size_t)(L * L));
  if (!M1 || !M2) { free(M1); free(M2); return -1; }
  oracle_masks(M->H, M->m, M->n, M1, M2);
  int err = 0;
#ifdef _OPENMP
  if (n_threads < 1) n_threads = 1;
#pragma omp parallel for num_threads(n_threads) schedule(dynamic, 1) reduction(| : err)
#endif
  for (int64_t b = 0; b < batch; ++b)
    if (ref64_word(M, M1, M2, y + b * n, bits + b * n, f + b * n, NULL, NULL)) err |= 1;
  free(M1);
  free(M2);
  return err ? -1 : 0;
}

int oracle_decode_ref64_word(const oracle_model *M, const float *y, uint8_t *bits, double *f,
                             int8_t *codes, const int8_t *force, double margin, int64_t *stats) {
  if (check_model(M) || (force && !(margin >= 0.0))) return -1;
  const int64_t L = M->n + M->m;
  uint8_t *M1 = malloc((size_t)(L * L)), *M2 = malloc((size_t)(L * L));
  int err = (!M1 || !M2) ? -1 : 0;
  tie_rule ties = {force, margin, {0, 0}};
  if (!err) {
    oracle_masks(M->H, M->m, M->n, M1, M2);
    err = ref64_word(M, M1, M2, y, bits, f, codes, force ? &ties : NULL);
  }
  if (stats) {
    stats[0] = ties.stats[0];
    stats[1] = ties.stats[1];
  }
  free(M1);
  free(M2);
  return err;
}
