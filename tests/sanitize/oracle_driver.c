/* Drives the CPU oracle for the sanitizer build (test infrastructure).  argv: files of parity-
 * check matrices, each "m n" then m*n bytes 0/1; the model and the channel words are drawn here
 * (ternary weights, finite parameters), since only their shapes matter to memory and UB checks. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "aecct_oracle.h"

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static double urand(void) {
  rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
  return (double)(rng >> 11) * 0x1.0p-53;
}
static float *fvec(size_t k, double sd, double mean) {
  float *v = malloc(sizeof(float) * (k ? k : 1));
  for (size_t i = 0; i < k; ++i) v[i] = (float)(mean + sd * (urand() * 2 - 1));
  return v;
}

static int run(const uint8_t *H, int m, int n, int d, int N, int act_word, int casa) {
  const int L = n + m, dff = 4 * d;
  oracle_model M;
  memset(&M, 0, sizeof M);
  M.n = n; M.m = m; M.d = d; M.n_layers = N; M.heads = 8; M.first_ring_heads = 4; M.d_ff = dff;
  M.ln_eps = 1e-5f; M.H = H; M.attention = casa; M.act_scale_mode = act_word;
  float *embed = fvec((size_t)L * d, 1, 0), *pos = fvec((size_t)L * d, 0.5, 0);
  M.embed = embed; M.pos = pos;
  const size_t in[6] = {d, d, d, d, d, dff}, out[6] = {d, d, d, d, dff, d};
  int8_t *w[6];
  float *b[6];
  for (int k = 0; k < 6; ++k) {
    const size_t cnt = (size_t)N * in[k] * out[k];
    w[k] = malloc(cnt);
    for (size_t i = 0; i < cnt; ++i) w[k][i] = (int8_t)((int)(urand() * 3) - 1);
    b[k] = fvec((size_t)N * out[k], 0.1, 0);
    M.w[k] = w[k]; M.bias[k] = b[k];
  }
  float *scale = fvec((size_t)N * 6, 0.01, 1.0 / sqrt(d));
  float *ln[4];
  for (int k = 0; k < 4; ++k) ln[k] = fvec((size_t)N * d, 0.1, k % 2 ? 0.0 : 1.0);
  M.scale = scale; M.ln1_g = ln[0]; M.ln1_b = ln[1]; M.ln2_g = ln[2]; M.ln2_b = ln[3];
  float *w1 = fvec(d, 0.2, 0), *wo = fvec((size_t)L * n, 0.1, 0), *bo = fvec(n, 0.1, 0);
  M.head_w1 = w1; M.head_b1 = 0.05f; M.head_wo = wo; M.head_bo = bo;
  const int B = 3;
  float *y = fvec((size_t)B * n, 2, 0);
  uint8_t *bits = malloc((size_t)B * n);
  float *f = malloc(sizeof(float) * B * n);
  double *f64 = malloc(sizeof(double) * B * n);
  int rc = oracle_decode(&M, y, B, bits, f, 2);
  rc |= oracle_decode_ref64(&M, y, B, bits, f64, 2);
  /* taps of one word, and the fp64 word decode forced to its codes */
  const size_t LD = (size_t)N * L * d, LF = (size_t)N * L * dff;
  oracle_taps T;
  memset(&T, 0, sizeof T);
  T.x_in = malloc(4 * LD); T.xq = malloc(LD); T.ax = malloc(4 * (size_t)N * L); T.qkv = malloc(12 * LD);
  T.o = malloc(4 * LD); T.oq = malloc(LD); T.ao = malloc(4 * (size_t)N * L); T.acc_o = malloc(4 * LD);
  T.x1 = malloc(4 * LD); T.x1q = malloc(LD); T.a1 = malloc(4 * (size_t)N * L); T.acc_ff1 = malloc(4 * LF);
  T.gq = malloc(LF); T.ag = malloc(4 * (size_t)N * L); T.acc_ff2 = malloc(4 * LD); T.x_out = malloc(4 * LD);
  T.z = malloc(4 * (size_t)L);
  rc |= oracle_decode_taps(&M, y, bits, f, &T);
  int8_t *codes = malloc((size_t)N * L * (3 * d + dff)), *force = malloc((size_t)N * L * (3 * d + dff));
  for (int l = 0; l < N; ++l) {
    int8_t *c = force + (size_t)l * L * (3 * d + dff);
    memcpy(c, T.xq + (size_t)l * L * d, (size_t)L * d);
    memcpy(c + (size_t)L * d, T.oq + (size_t)l * L * d, (size_t)L * d);
    memcpy(c + 2 * (size_t)L * d, T.x1q + (size_t)l * L * d, (size_t)L * d);
    memcpy(c + 3 * (size_t)L * d, T.gq + (size_t)l * L * dff, (size_t)L * dff);
  }
  int64_t stats[2];
  rc |= oracle_decode_ref64_word(&M, y, bits, f64, codes, force, 1e-3, stats);
  /* building blocks */
  uint8_t *M1 = malloc((size_t)L * L), *M2 = malloc((size_t)L * L);
  oracle_masks(H, m, n, M1, M2);
  double *q64 = malloc(sizeof(double) * 3 * L * d), *o64 = malloc(sizeof(double) * L * d);
  for (size_t i = 0; i < (size_t)3 * L * d; ++i) q64[i] = urand() - 0.5;
  rc |= oracle_attention_dense_f64(&M, M1, M2, q64, 0.5, o64);
  float *xr = fvec((size_t)L * d, 3, 0);
  int8_t *qq = malloc((size_t)L * d);
  float *rr = malloc(4 * (size_t)L);
  oracle_quant_rows(xr, L, d, qq, rr);
  oracle_quant_word(xr, L, d, qq, rr);
  float *wm = fvec(4096, 1, 0);
  int8_t *tm = malloc(4096);
  float sc;
  rc |= oracle_aap_ternarize(wm, 4096, 0.5f, 1.0f, 1e-8f, tm, &sc);
  /* release */
  free(embed); free(pos); for (int k = 0; k < 6; ++k) { free(w[k]); free(b[k]); }
  free(scale); for (int k = 0; k < 4; ++k) free(ln[k]);
  free(w1); free(wo); free(bo); free(y); free(bits); free(f); free(f64);
  free(T.x_in); free(T.xq); free(T.ax); free(T.qkv); free(T.o); free(T.oq); free(T.ao); free(T.acc_o);
  free(T.x1); free(T.x1q); free(T.a1); free(T.acc_ff1); free(T.gq); free(T.ag); free(T.acc_ff2); free(T.x_out);
  free(T.z); free(codes); free(force); free(M1); free(M2); free(q64); free(o64); free(xr); free(qq); free(rr);
  free(wm); free(tm);
  return rc;
}

int main(int argc, char **argv) {
  for (int a = 1; a < argc; ++a) {
    FILE *fp = fopen(argv[a], "rb");
    if (!fp) return 1;
    int mn[2];
    if (fread(mn, sizeof(int), 2, fp) != 2) { fclose(fp); return 1; }
    uint8_t *H = malloc((size_t)mn[0] * mn[1]);
    const size_t got = fread(H, 1, (size_t)mn[0] * mn[1], fp);
    fclose(fp);
    if (got != (size_t)mn[0] * mn[1]) return 1;
    const int L = mn[0] + mn[1];
    const int ds[2] = {32, 128};
    for (int k = 0; k < 2; ++k) {
      if (ds[k] == 128 && L > 400) continue;
      for (int casa = 0; casa < 2; ++casa)
        for (int act = 0; act < 2; ++act)
          if (run(H, mn[0], mn[1], ds[k], 2, act, casa)) { printf("FAIL %s d %d casa %d act %d\n", argv[a], ds[k], casa, act); return 1; }
    }
    printf("code %s ok\n", argv[a]);
    fflush(stdout);
    free(H);
  }
  printf("oracle driver ok\n");
  return 0;
}
