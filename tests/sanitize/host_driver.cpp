// Drives the library's host code through its C ABI for the sanitizer build (test infrastructure).
// argv: files of parity-check matrices, each "m n" then m*n bytes 0/1.  Weights are drawn here
// (ternary, finite), since only their shapes and validity matter to the host code.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "aecct.h"

static uint64_t rng = 0x243F6A8885A308D3ull;
static double urand() {
  rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
  return (double)(rng >> 11) * 0x1.0p-53;
}

#define CHECK(x) do { aecct_status s_ = (x); if (s_ != AECCT_OK) { std::printf("FAIL %s:%d %s -> %d\n", __FILE__, __LINE__, #x, (int)s_); return 1; } } while (0)
#define EXPECT(x, st) do { aecct_status s_ = (x); if (s_ != (st)) { std::printf("FAIL %s:%d %s -> %d, expected %d\n", __FILE__, __LINE__, #x, (int)s_, (int)(st)); return 1; } } while (0)

struct Weights {
  std::vector<float> embed, pos, scale, b[6], ln[4], w1, wo, bo;
  std::vector<int8_t> w[6];
  aecct_weights view{};
};

static void make_weights(Weights &W, int n, int m, int d, int N, bool with_pos) {
  const int L = n + m, dff = 4 * d;
  auto f = [](std::vector<float> &v, size_t k, double sd, double mean) {
    v.resize(k);
    for (auto &x : v) x = (float)(mean + sd * (urand() * 2 - 1));
  };
  f(W.embed, (size_t)L * d, 1.0, 0.0);
  if (with_pos) f(W.pos, (size_t)L * d, 0.5, 0.0);
  const size_t in[6] = {(size_t)d, (size_t)d, (size_t)d, (size_t)d, (size_t)d, (size_t)dff};
  const size_t out[6] = {(size_t)d, (size_t)d, (size_t)d, (size_t)d, (size_t)dff, (size_t)d};
  for (int k = 0; k < 6; ++k) {
    W.w[k].resize((size_t)N * in[k] * out[k]);
    for (auto &x : W.w[k]) x = (int8_t)((int)(urand() * 3) - 1);
    f(W.b[k], (size_t)N * out[k], 0.1, 0.0);
  }
  f(W.scale, (size_t)N * 6, 0.01, 1.0 / std::sqrt((double)d));
  for (int k = 0; k < 4; ++k) f(W.ln[k], (size_t)N * d, 0.1, k % 2 ? 0.0 : 1.0);
  f(W.w1, d, 0.2, 0.0);
  f(W.wo, (size_t)L * n, 0.1, 0.0);
  f(W.bo, n, 0.1, 0.0);
  aecct_weights &v = W.view;
  v.embed = W.embed.data();
  v.pos = with_pos ? W.pos.data() : nullptr;
  v.w_q = W.w[0].data(); v.w_k = W.w[1].data(); v.w_v = W.w[2].data(); v.w_o = W.w[3].data();
  v.w_ff1 = W.w[4].data(); v.w_ff2 = W.w[5].data();
  v.scale = W.scale.data();
  v.b_q = W.b[0].data(); v.b_k = W.b[1].data(); v.b_v = W.b[2].data(); v.b_o = W.b[3].data();
  v.b_ff1 = W.b[4].data(); v.b_ff2 = W.b[5].data();
  v.ln1_g = W.ln[0].data(); v.ln1_b = W.ln[1].data(); v.ln2_g = W.ln[2].data(); v.ln2_b = W.ln[3].data();
  v.head_w1 = W.w1.data(); v.head_b1 = 0.05f; v.head_wo = W.wo.data(); v.head_bo = W.bo.data();
}

static int run_code(const std::vector<uint8_t> &H, int m, int n) {
  const int L = n + m;
  const int dims[3] = {32, 64, 128};
  for (int d : dims) {
    if (L > 4096) continue;
    const int N = 2;
    Weights W;
    make_weights(W, n, m, d, N, d == 32);
    for (int att = 0; att < 2; ++att)
      for (int act = 0; act < 2; ++act)
        for (int lattn = -1; lattn <= 3; ++lattn) {
          aecct_options o{-1, -1, 0.0f, AECCT_PATH_AUTO, att, lattn, act};
          aecct_model *M = nullptr;
          aecct_status st = aecct_create(H.data(), m, n, &W.view, d, N, 8, &o, &M);
          if (st == AECCT_ERR_UNSUPPORTED) continue;      // a form this shape does not allow
          CHECK(st);
          aecct_model_info info;
          CHECK(aecct_get_info(M, &info));
          for (int64_t B : {(int64_t)1, (int64_t)37, (int64_t)(L <= 64 ? 5000 : 2)}) {
            size_t ws = 0;
            CHECK(aecct_workspace_size(M, B, &ws));
            std::vector<float> y((size_t)B * n);
            for (auto &v : y) v = (float)(urand() * 4 - 2);
            std::vector<uint8_t> bits((size_t)B * n);
            std::vector<float> logits((size_t)B * n);
            std::vector<unsigned char> wsb(ws ? ws : 1);
            CHECK(aecct_decode(M, y.data(), B, bits.data(), logits.data(), ws ? wsb.data() : nullptr, ws, nullptr));
            if (ws) EXPECT(aecct_decode(M, y.data(), B, bits.data(), nullptr, wsb.data(), ws - 1, nullptr),
                           AECCT_ERR_WORKSPACE_TOO_SMALL);
            CHECK(aecct_decode_static(M, y.data(), B, bits.data(), logits.data(), nullptr));
          }
          aecct_destroy(M);
        }
    // the training step's host side
    aecct_trainer *T = nullptr;
    aecct_options o{-1, -1, 0.0f, AECCT_PATH_AUTO, AECCT_ATTN_HPSA, -1, AECCT_ACT_SCALE_TOKEN};
    CHECK(aecct_train_create(H.data(), m, n, d, N, 8, &o, 1e-8f, &T));
    size_t tws = 0;
    CHECK(aecct_train_workspace_size(T, 3, &tws));
    std::vector<float> pbuf((size_t)4 << 20), gbuf((size_t)4 << 20), wsf(tws / 4 + 64);
    aecct_train_params P;
    aecct_train_grads G;
    float *pp = pbuf.data(), *gg = gbuf.data();
    const float **pf = (const float **)&P;
    float **gf = (float **)&G;
    for (size_t k = 0; k < sizeof(P) / sizeof(void *); ++k) pf[k] = pp;
    for (size_t k = 0; k < sizeof(G) / sizeof(void *); ++k) gf[k] = gg;
    P.pos = nullptr;
    std::vector<float> y((size_t)3 * n, 0.5f);
    CHECK(aecct_train_grad(T, &P, y.data(), nullptr, 3, &G, gg, wsf.data(), tws, nullptr));
    aecct_train_destroy(T);
  }
  // spectrum of small graphs (host float64)
  if (L <= 200) {
    std::vector<double> lam(L), vec((size_t)L * L);
    CHECK(aecct_tanner_spectrum(H.data(), m, n, lam.data(), vec.data()));
  }
  return 0;
}

int main(int argc, char **argv) {
  // argument errors before any device call
  aecct_model *M = nullptr;
  EXPECT(aecct_create(nullptr, 3, 7, nullptr, 32, 2, 8, nullptr, &M), AECCT_ERR_INVALID_ARG);
  std::vector<float> wf(4096);
  for (auto &x : wf) x = (float)(urand() - 0.5);
  std::vector<int8_t> t(wf.size());
  float sc = 0;
  for (float p : {0.0f, 0.25f, 0.5f, 1.0f}) CHECK(aecct_aap_ternarize(wf.data(), (int64_t)wf.size(), p, 1.0f, 1e-8f, t.data(), &sc));
  EXPECT(aecct_aap_ternarize(wf.data(), 0, 0.5f, 1.0f, 1e-8f, t.data(), &sc), AECCT_ERR_INVALID_ARG);
  for (int a = 1; a < argc; ++a) {
    FILE *fp = std::fopen(argv[a], "rb");
    if (!fp) { std::printf("FAIL cannot open %s\n", argv[a]); return 1; }
    int mn[2];
    if (std::fread(mn, sizeof(int), 2, fp) != 2) { std::fclose(fp); return 1; }
    std::vector<uint8_t> H((size_t)mn[0] * mn[1]);
    const size_t got = std::fread(H.data(), 1, H.size(), fp);
    std::fclose(fp);
    if (got != H.size()) return 1;
    std::printf("code %s: m %d n %d\n", argv[a], mn[0], mn[1]);
    std::fflush(stdout);
    if (run_code(H, mn[0], mn[1])) return 1;
  }
  std::printf("host driver ok\n");
  return 0;
}
