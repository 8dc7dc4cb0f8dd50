/*
 * AECCT inference oracle -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.
 *
 * A plain, slow CPU implementation of the AECCT inference forward pass
 * (Levy, Choukroun, Wolf, "Accelerating Error Correction Code Transformers").
 * Only the test suite, the package smoke check and the CPU-baseline leg of the
 * benchmark may load it.  It shares no code with the GPU library and includes
 * none of its headers.
 *
 * Two modes:
 *   canonical fp32 -- the paper's arithmetic in IEEE binary32 (activations,
 *                     biases and scales are fp32 in Section 4.1), in a fixed,
 *                     stated evaluation order so that any correct
 *                     implementation that keeps the same order reproduces
 *                     every value bit for bit (the qkv tap holds the query
 *                     rows scaled by log2(e)/sqrt(d_h), see oracle_query_scale);
 *   reference fp64 -- the same model in double precision with dense
 *                     (-inf)-masked softmax attention and libm exp; the
 *                     semantic check of the canonical mode.
 *
 * Parity status: every function is pinned by the CPU test suite (see the
 * comments of each function for its pin), except that decoding quality
 * (bit error rate against the paper's Table 1) is parity unpinned: it needs
 * trained weights and the paper's parity-check files.
 */
#ifndef AECCT_ORACLE_H
#define AECCT_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Order of the six in-block linear maps. */
enum { ORC_Q = 0, ORC_K = 1, ORC_V = 2, ORC_O = 3, ORC_FF1 = 4, ORC_FF2 = 5 };

typedef struct oracle_model {
  int32_t n, m;               /* code length, parity checks; L = n + m tokens */
  int32_t d, n_layers, heads, first_ring_heads, d_ff;
  float ln_eps;
  const uint8_t *H;           /* [m][n] 0/1 */
  const float *embed;         /* [L][d] */
  const float *pos;           /* [L][d] or NULL */
  const int8_t *w[6];         /* q,k,v,o: [N][d][d]; ff1: [N][d][d_ff]; ff2: [N][d_ff][d]; [in][out] */
  const float *scale;         /* [N][6] weight scale gamma*delta per matrix */
  const float *bias[6];       /* [N][out] */
  const float *ln1_g, *ln1_b, *ln2_g, *ln2_b;   /* [N][d] */
  const float *head_w1;       /* [d]  (W_{d->1}) */
  float head_b1;
  const float *head_wo;       /* [L][n] (W_o) */
  const float *head_bo;       /* [n] */
  int32_t attention;          /* 0: HPSA head partitioning (Section 4.2); 1: CASA, every head
                                 over the ECCT mask M1 | M2 (Section 3) */
  int32_t act_scale_mode;     /* Eq. 2 scale alpha: 0 = per token (max over the row's features),
                                 1 = per word (max over all of the word's tokens and features) */
} oracle_model;

/* Per-layer intermediate values of one word (each pointer may be NULL). */
typedef struct oracle_taps {
  float *x_in;     int8_t *xq;  float *ax;      /* [N][L][d], [N][L][d], [N][L] */
  float *qkv;                                   /* [N][L][3d]: Q | K | V per row */
  float *o;        int8_t *oq;  float *ao;      /* attention output and its quantisation */
  int32_t *acc_o;                               /* [N][L][d] */
  float *x1;       int8_t *x1q; float *a1;      /* after LN1 */
  int32_t *acc_ff1;                             /* [N][L][d_ff] */
  int8_t *gq;      float *ag;                   /* [N][L][d_ff], [N][L] */
  int32_t *acc_ff2;                             /* [N][L][d] */
  float *x_out;                                 /* [N][L][d] after LN2 */
  float *z;                                     /* [L] per-token head value */
} oracle_taps;

/* ---- building blocks (canonical fp32) ---- */
float oracle_tree_sum(const float *v, int32_t w);
float oracle_exp2(float x);
float oracle_rsqrt(float v);
float oracle_query_scale(int32_t dh);
void oracle_masks(const uint8_t *H, int32_t m, int32_t n, uint8_t *M1, uint8_t *M2);
void oracle_preprocess(const uint8_t *H, int32_t m, int32_t n, const float *y, float *t);
void oracle_quant_rows(const float *x, int64_t rows, int32_t K, int8_t *q, float *r);
void oracle_quant_word(const float *x, int64_t rows, int32_t K, int8_t *q, float *r);
void oracle_linear_rows(const int8_t *q, const float *r, int64_t rows, const int8_t *T, int32_t K,
                        int32_t n_out, float sq, const float *b, float *out, int32_t *acc);
void oracle_layernorm_rows(const float *R, int64_t rows, int32_t d, const float *g, const float *b,
                           float eps, float *out);
int oracle_attention_word(const oracle_model *M, const uint8_t *M1, const uint8_t *M2,
                          const float *qkv, float *o);
void oracle_head_word(const oracle_model *M, const float *X, const float *y, float *f, uint8_t *bits,
                      float *z);

/* ---- whole decode ---- */
int oracle_decode(const oracle_model *M, const float *y, int64_t batch, uint8_t *bits, float *f,
                  int32_t n_threads);
int oracle_decode_taps(const oracle_model *M, const float *y, uint8_t *bits, float *f,
                       const oracle_taps *taps);
int oracle_decode_ref64(const oracle_model *M, const float *y, int64_t batch, uint8_t *bits,
                        double *f, int32_t n_threads);
/* One word in the fp64 reference mode; codes (may be NULL) receives every int8 activation code
 * the word's layers form, per layer l in the order Q/K/V input [L][d], attention output [L][d],
 * LN1 output [L][d], hidden [L][d_ff] (N (3d + d_ff) L bytes in all).  With force (same layout,
 * may be NULL): a code whose fp64 value x 127 / alpha lies within margin of a rounding tie takes
 * force's code when that is one of the tie's two neighbours; stats[0] counts codes so taken that
 * differ from the fp64 decision, stats[1] codes of force that differ from it elsewhere. */
int oracle_decode_ref64_word(const oracle_model *M, const float *y, uint8_t *bits, double *f,
                             int8_t *codes, const int8_t *force, double margin, int64_t *stats);
/* AAP weight import (Section 4.1, Eq. 1): gamma = p-quantile of |w| (linear interpolation,
 * double, rounded to fp32), *scale = fp32(gamma * delta), t = RoundClip(w / fp32(scale + eps)).
 * Returns 0, or -1 for invalid arguments. */
int oracle_aap_ternarize(const float *w, int64_t count, float p, float delta, float eps, int8_t *t,
                         float *scale);
/* fp64 dense masked softmax attention of one word (reference for the sparse canonical one). */
int oracle_attention_dense_f64(const oracle_model *M, const uint8_t *M1, const uint8_t *M2,
                               const double *qkv, double score_scale, double *o);

#ifdef __cplusplus
}
#endif
#endif
