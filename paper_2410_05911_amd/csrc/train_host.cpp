// Host side of the quantisation-aware training step (Section 6, second phase): validation, the
// Tanner-graph lists on the device, the workspace layout and the launch sequence of one forward
// and backward pass.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <vector>

#include <hip/hip_runtime.h>

#include "../../include/aecct.h"
#include "aecct_internal.h"

struct aecct_trainer {
  int n, m, L, d, N, heads, hf, dff, dh;
  float ln_eps, aap_eps;
  int device, cu_count;
  void *blk;
  const int32_t *chk_ptr, *chk_idx, *m1_ptr, *m1_idx, *m2_ptr, *m2_idx;
};

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Workspace regions (float offsets) for `batch` words.
struct TrainWs {
  struct Layer { size_t xh, qkv, lse, o, oh, xn1, rho1, x1h, f, gh, xn2, rho2; };
  std::vector<Layer> layer;
  size_t t, x, x1, y, z, fo, df, dz, tw, tb16, gam, sc, lpart, dx, dr, dx1, dg, dO, dqkv, dv, part;
  size_t part_floats, total_bytes;
};

size_t weight_floats(const aecct_trainer &T) {
  return (size_t)T.N * (4 * (size_t)T.d * T.d + 2 * (size_t)T.d * T.dff);
}

TrainWs train_ws(const aecct_trainer &T, int64_t batch) {
  const size_t R = (size_t)batch * T.L, d = T.d, dff = T.dff, h = T.heads;
  TrainWs w{};
  size_t off = 0;   // bytes
  auto take = [&](size_t floats) { size_t o = off; off = align_up(off + 4 * floats); return o / 4; };
  w.layer.resize(T.N);
  for (auto &q : w.layer) {
    q.xh = take(R * d);
    q.qkv = take(R * 3 * d);
    q.lse = take(R * h);
    q.o = take(R * d);
    q.oh = take(R * d);
    q.xn1 = take(R * d);
    q.rho1 = take(R);
    q.x1h = take(R * d);
    q.f = take(R * dff);
    q.gh = take(R * dff);
    q.xn2 = take(R * d);
    q.rho2 = take(R);
  }
  w.t = take(R);
  w.x = take(R * d);
  w.x1 = take(R * d);
  w.y = take(R * d);
  w.z = take(R);
  w.fo = take((size_t)batch * T.n);
  w.df = take((size_t)batch * T.n);
  w.dz = take(R);
  w.tw = take(weight_floats(T));
  w.tb16 = take(weight_floats(T));   // every ternary matrix as bf16 B fragments, T and T^T
  w.gam = take((size_t)T.N * 6);
  w.sc = take((size_t)T.N * 6);
  w.lpart = take(((size_t)batch * T.n + 255) / 256 + 1);
  w.dx = take(R * d);
  w.dr = take(R * d);
  w.dx1 = take(R * d);
  w.dg = take(R * dff);
  w.dO = take(R * d);
  w.dqkv = take(R * 3 * d);
  w.dv = take(R * h);
  w.part_floats = std::max<size_t>(size_t(1) << 22, 4 * std::max<size_t>((size_t)T.L * T.n, d * dff));
  w.part = take(w.part_floats);
  w.total_bytes = off;
  return w;
}

inline aecct_status st(hipError_t e) { return e == hipSuccess ? AECCT_OK : AECCT_ERR_DEVICE; }

}  // namespace

extern "C" {

aecct_status aecct_train_create(const uint8_t *H, int32_t m, int32_t n, int32_t d, int32_t n_layers, int32_t heads,
                                const aecct_options *opt, float aap_eps, aecct_trainer **out) {
  if (!out) return AECCT_ERR_INVALID_ARG;
  *out = nullptr;
  if (!H || m <= 0 || n <= 0 || d <= 0 || n_layers <= 0 || heads <= 0 || d % heads) return AECCT_ERR_INVALID_ARG;
  if (!std::isfinite(aap_eps) || aap_eps < 0.0f) return AECCT_ERR_INVALID_ARG;
  const int hf = (opt && opt->first_ring_heads >= 0) ? opt->first_ring_heads : heads / 2;
  if ((opt && opt->first_ring_heads < -1) || hf > heads) return AECCT_ERR_INVALID_ARG;
  const int dff = (opt && opt->d_ff > 0) ? opt->d_ff : 4 * d;
  if (opt && (opt->d_ff < -1 || !std::isfinite(opt->ln_eps))) return AECCT_ERR_INVALID_ARG;
  const float eps = (opt && opt->ln_eps > 0.0f) ? opt->ln_eps : 1e-5f;
  const int attention = opt ? opt->attention : AECCT_ATTN_HPSA;
  if (attention != AECCT_ATTN_HPSA && attention != AECCT_ATTN_CASA) return AECCT_ERR_INVALID_ARG;
  const int act_mode = opt ? opt->act_scale_mode : AECCT_ACT_SCALE_TOKEN;
  if (act_mode != AECCT_ACT_SCALE_TOKEN && act_mode != AECCT_ACT_SCALE_WORD) return AECCT_ERR_INVALID_ARG;
  const int64_t L64 = (int64_t)n + m;
  std::vector<int> rowdeg(m, 0), coldeg(n, 0);
  for (int j = 0; j < m; ++j)
    for (int i = 0; i < n; ++i) {
      const uint8_t v = H[(size_t)j * n + i];
      if (v > 1) return AECCT_ERR_INVALID_ARG;
      if (v) { ++rowdeg[j]; ++coldeg[i]; }
    }
  for (int j = 0; j < m; ++j) if (!rowdeg[j]) return AECCT_ERR_INVALID_ARG;
  for (int i = 0; i < n; ++i) if (!coldeg[i]) return AECCT_ERR_INVALID_ARG;
  const int dh = d / heads;
  if (!(d == 32 || d == 64 || d == 128) || !(dh == 4 || dh == 8 || dh == 16) || dff != 4 * d || L64 > 4096 ||
      n_layers > aecct::kMaxLayers || act_mode != AECCT_ACT_SCALE_TOKEN)
    return AECCT_ERR_UNSUPPORTED;
  const int L = (int)L64;

  aecct::TannerLists TL = aecct::tanner_lists(H, m, n);
  int hf_eff = hf;
  if (attention == AECCT_ATTN_CASA) {
    aecct::casa_union(TL);
    hf_eff = 0;
  }
  const std::vector<int32_t> *parts[6] = {&TL.chk_ptr, &TL.chk_idx, &TL.m1_ptr, &TL.m1_idx, &TL.m2_ptr, &TL.m2_idx};
  size_t offs[6], total = 0;
  for (int k = 0; k < 6; ++k) {
    offs[k] = total;
    total = align_up(total + 4 * std::max<size_t>(1, parts[k]->size()));
  }
  std::vector<unsigned char> img(total, 0);
  for (int k = 0; k < 6; ++k)
    if (!parts[k]->empty()) std::memcpy(img.data() + offs[k], parts[k]->data(), 4 * parts[k]->size());

  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return AECCT_ERR_DEVICE;
  void *blk = nullptr;
  hipError_t e = hipMalloc(&blk, total);
  if (e != hipSuccess) return e == hipErrorOutOfMemory ? AECCT_ERR_OUT_OF_MEMORY : AECCT_ERR_DEVICE;
  if (hipMemcpy(blk, img.data(), total, hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipFree(blk);
    return AECCT_ERR_DEVICE;
  }
  aecct_trainer *tr = new (std::nothrow) aecct_trainer;
  if (!tr) {
    (void)hipFree(blk);
    return AECCT_ERR_OUT_OF_MEMORY;
  }
  unsigned char *b = (unsigned char *)blk;
  *tr = aecct_trainer{n, m, L, d, n_layers, heads, hf_eff, dff, dh, eps, aap_eps, dev, cus, blk,
                      (const int32_t *)(b + offs[0]), (const int32_t *)(b + offs[1]), (const int32_t *)(b + offs[2]),
                      (const int32_t *)(b + offs[3]), (const int32_t *)(b + offs[4]), (const int32_t *)(b + offs[5])};
  *out = tr;
  return AECCT_OK;
}

void aecct_train_destroy(aecct_trainer *tr) {
  if (!tr) return;
  if (tr->blk) (void)hipFree(tr->blk);
  delete tr;
}

aecct_status aecct_train_workspace_size(const aecct_trainer *tr, int64_t batch, size_t *bytes) {
  if (!tr || !bytes || batch < 0) return AECCT_ERR_INVALID_ARG;
  *bytes = batch == 0 ? 0 : train_ws(*tr, batch).total_bytes;
  return AECCT_OK;
}

aecct_status aecct_train_grad(const aecct_trainer *tr, const aecct_train_params *p, const float *y, const float *xs,
                              int64_t batch, const aecct_train_grads *g, float *loss, void *workspace,
                              size_t workspace_bytes, void *stream) {
  using namespace aecct;
  if (!tr || !p || !g || !loss || batch <= 0 || !y) return AECCT_ERR_INVALID_ARG;
  const float *pw[6] = {p->w_q, p->w_k, p->w_v, p->w_o, p->w_ff1, p->w_ff2};
  const float *pb[6] = {p->b_q, p->b_k, p->b_v, p->b_o, p->b_ff1, p->b_ff2};
  float *gw[6] = {g->w_q, g->w_k, g->w_v, g->w_o, g->w_ff1, g->w_ff2};
  float *gb[6] = {g->b_q, g->b_k, g->b_v, g->b_o, g->b_ff1, g->b_ff2};
  for (int k = 0; k < 6; ++k)
    if (!pw[k] || !pb[k] || !gw[k] || !gb[k]) return AECCT_ERR_INVALID_ARG;
  if (!p->embed || !p->delta || !p->ln1_g || !p->ln1_b || !p->ln2_g || !p->ln2_b || !p->head_w1 || !p->head_b1 ||
      !p->head_wo || !p->head_bo || !g->embed || !g->delta || !g->ln1_g || !g->ln1_b || !g->ln2_g || !g->ln2_b ||
      !g->head_w1 || !g->head_b1 || !g->head_wo || !g->head_bo)
    return AECCT_ERR_INVALID_ARG;
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return AECCT_ERR_DEVICE;
  if (cur != tr->device) return AECCT_ERR_INVALID_ARG;
  const TrainWs W = train_ws(*tr, batch);
  if (workspace_bytes < W.total_bytes) return AECCT_ERR_WORKSPACE_TOO_SMALL;
  if (!workspace) return AECCT_ERR_INVALID_ARG;

  const aecct_trainer &T = *tr;
  hipStream_t s = (hipStream_t)stream;
  float *ws = (float *)workspace;
  const int64_t R = batch * T.L, B = batch;
  const int d = T.d, dff = T.dff, N = T.N;
  const int64_t K_in[6] = {d, d, d, d, d, dff}, K_out[6] = {d, d, d, d, dff, d};
  const size_t PF = W.part_floats;
  float *part = ws + W.part;
  auto wofs = [&](int l, int k) {   // float offset of matrix k of layer l inside a [N][in][out] tensor
    return (size_t)l * K_in[k] * K_out[k];
  };
  // the ternary copies: per layer the six maps back to back
  auto tmat = [&](int l, int k) {
    size_t o = W.tw;
    for (int ll = 0; ll < l; ++ll)
      for (int kk = 0; kk < 6; ++kk) o += K_in[kk] * K_out[kk];
    for (int kk = 0; kk < k; ++kk) o += K_in[kk] * K_out[kk];
    return ws + o;
  };
  float *gam = ws + W.gam, *sc = ws + W.sc;
  // the ternary matrices as bf16 fragments of B = T (the forward products) and B = T^T (the input
  // gradients): at d, d_ff multiples of 64 every product with a ternary operand runs on
  // train_gemm_tern, else on the fp32 kernels
  const bool tern = d % 64 == 0 && dff % 64 == 0;
  auto tfrag = [&](int l, int k, bool trans) {
    size_t o = 0;   // in uint16 units
    for (int ll = 0; ll < l; ++ll)
      for (int kk = 0; kk < 6; ++kk) o += 2 * (size_t)K_in[kk] * K_out[kk];
    for (int kk = 0; kk < k; ++kk) o += 2 * (size_t)K_in[kk] * K_out[kk];
    if (trans) o += (size_t)K_in[k] * K_out[k];
    return (void *)((uint16_t *)(ws + W.tb16) + o);
  };
  hipError_t e = hipSuccess;
#define AECCT_TRY(call)              \
  do {                               \
    e = (call);                      \
    if (e != hipSuccess) return st(e); \
  } while (0)

  // ---- forward -------------------------------------------------------------------------------
  // Eq. 1 of every layer's six matrices first (they depend on the weights only), a launch per
  // eight layers
  for (int l0 = 0; l0 < N; l0 += kTrainJobsPerLaunch / 6) {
    TrainAapJobs jobs{};
    for (int l = l0; l < std::min(N, l0 + kTrainJobsPerLaunch / 6); ++l)
      for (int k = 0; k < 6; ++k)
        jobs.j[jobs.n++] = TrainAapJob{pw[k] + wofs(l, k), tmat(l, k), K_in[k] * K_out[k], p->delta + 6 * l + k,
                                       gam + 6 * l + k, sc + 6 * l + k};
    AECCT_TRY(train_aap(jobs, T.aap_eps, s));
  }
  if (tern)   // both layouts of every matrix, a launch per four layers
    for (int l0 = 0; l0 < N; l0 += kTrainJobsPerLaunch / 12) {
      TernPackJobs pj{};
      for (int l = l0; l < std::min(N, l0 + kTrainJobsPerLaunch / 12); ++l)
        for (int k = 0; k < 6; ++k)
          for (int tr = 0; tr < 2; ++tr)
            pj.j[pj.n++] = TernPackJob{tmat(l, k), (int)K_in[k], (int)K_out[k], tr, tfrag(l, k, tr != 0)};
      AECCT_TRY(train_pack_tern(pj, s));
    }
  float *X = ws + W.x, *X1 = ws + W.x1, *Y = ws + W.y, *tv = ws + W.t;
  AECCT_TRY(train_embed(y, R, T.n, T.L, d, T.chk_ptr, T.chk_idx, p->embed, p->pos, X, tv, s));
  auto gemm = [&](bool ta, bool tb, const float *A, int64_t lda, const float *Bm, int64_t ldb, float *C, int64_t ldc,
                  int64_t M, int64_t Nn, int64_t K, const float *scale, const float *bias, bool acc) {
    return train_gemm(ta, tb, A, lda, Bm, ldb, C, ldc, M, Nn, K, scale, bias, acc, part, (int64_t)PF, T.cu_count, s);
  };
  // C = scale (A op(T)) + bias (+ C) for ternary matrix k of layer l, op(T) = T or (trans) T^T
  auto tgemm = [&](bool trans, int l, int k, const float *A, int64_t lda, float *C, int64_t ldc, int64_t M, int64_t Nn,
                   int64_t K, const float *scale, const float *bias, bool acc) {
    if (tern && train_tern_operands_ok(A, lda, C, ldc, bias, Nn, K))
      return train_gemm_tern(A, lda, tfrag(l, k, trans), C, ldc, M, Nn, K, scale, bias, acc, s);
    return gemm(false, trans, A, lda, tmat(l, k), trans ? K : Nn, C, ldc, M, Nn, K, scale, bias, acc);
  };
  for (int l = 0; l < N; ++l) {
    const TrainWs::Layer &q = W.layer[l];
    float *Xh = ws + q.xh, *QKV = ws + q.qkv;
    if (l == 0) AECCT_TRY(train_quant(X, R, d, false, Xh, s));   // later layers: from the previous LN2
    {
      // the query, key and value maps as one product over one read of Xh where the ternary path applies
      const float *bq[3] = {pb[0] + (size_t)l * d, pb[1] + (size_t)l * d, pb[2] + (size_t)l * d};
      const float *sq[3] = {sc + 6 * l, sc + 6 * l + 1, sc + 6 * l + 2};
      bool fused = tern;
      for (int k = 0; k < 3; ++k) fused = fused && train_tern_operands_ok(Xh, d, QKV + k * d, 3 * d, bq[k], d, d);
      if (fused) {
        const void *fq[3] = {tfrag(l, 0, false), tfrag(l, 1, false), tfrag(l, 2, false)};
        AECCT_TRY(train_gemm_tern_seg(Xh, d, fq, QKV, 3 * d, R, d, 3, d, sq, bq, false, s));
      } else {
        for (int k = 0; k < 3; ++k) AECCT_TRY(tgemm(false, l, k, Xh, d, QKV + k * d, 3 * d, R, d, d, sq[k], bq[k], false));
      }
    }
    TrainAttn at{QKV, R, T.L, d, T.heads, T.hf, T.m1_ptr, T.m1_idx, T.m2_ptr, T.m2_idx, ws + q.o, ws + q.lse,
                 nullptr, nullptr, nullptr};
    AECCT_TRY(train_attention(0, T.dh, at, s));
    AECCT_TRY(train_quant(ws + q.o, R, d, false, ws + q.oh, s));
    AECCT_TRY(tgemm(false, l, 3, ws + q.oh, d, Y, d, R, d, d, sc + 6 * l + 3, pb[3] + (size_t)l * d, false));
    AECCT_TRY(train_ln_fwd(X, Y, R, d, p->ln1_g + (size_t)l * d, p->ln1_b + (size_t)l * d, T.ln_eps, X1, ws + q.xn1,
                           ws + q.rho1, ws + q.x1h, s));
    AECCT_TRY(tgemm(false, l, 4, ws + q.x1h, d, ws + q.f, dff, R, dff, d, sc + 6 * l + 4, pb[4] + (size_t)l * dff, false));
    AECCT_TRY(train_quant(ws + q.f, R, dff, true, ws + q.gh, s));
    AECCT_TRY(tgemm(false, l, 5, ws + q.gh, dff, Y, d, R, d, dff, sc + 6 * l + 5, pb[5] + (size_t)l * d, false));
    AECCT_TRY(train_ln_fwd(X1, Y, R, d, p->ln2_g + (size_t)l * d, p->ln2_b + (size_t)l * d, T.ln_eps, X, ws + q.xn2,
                           ws + q.rho2, l + 1 < N ? ws + W.layer[l + 1].xh : nullptr, s));
  }
  // head and loss (Section 3, Section 6)
  float *z = ws + W.z, *fo = ws + W.fo, *df = ws + W.df, *dz = ws + W.dz;
  AECCT_TRY(train_rowdot(X, R, d, p->head_w1, p->head_b1, z, s));
  AECCT_TRY(gemm(false, false, z, T.L, p->head_wo, T.n, fo, T.n, B, T.n, T.L, nullptr, p->head_bo, false));
  AECCT_TRY(train_loss(fo, y, xs, B * T.n, df, ws + W.lpart, loss, s));

  // ---- backward ------------------------------------------------------------------------------
  auto colsum = [&](const float *A, int64_t lda, const float *Bm, const float *wr, int64_t rows, int C, float *o) {
    return train_colsum(A, lda, Bm, wr, rows, C, o, false, part, (int64_t)PF, s);
  };
  AECCT_TRY(colsum(df, T.n, nullptr, nullptr, B, T.n, g->head_bo));
  AECCT_TRY(gemm(true, false, z, T.L, df, T.n, g->head_wo, T.n, T.L, T.n, B, nullptr, nullptr, false));
  AECCT_TRY(gemm(false, true, df, T.n, p->head_wo, T.n, dz, T.L, B, T.L, T.n, nullptr, nullptr, false));
  AECCT_TRY(colsum(dz, 1, nullptr, nullptr, R, 1, g->head_b1));
  AECCT_TRY(colsum(X, d, nullptr, dz, R, d, g->head_w1));
  float *dX = ws + W.dx, *dR = ws + W.dr, *dX1 = ws + W.dx1, *dG = ws + W.dg, *dO = ws + W.dO, *dQKV = ws + W.dqkv;
  AECCT_TRY(train_outer(dz, R, p->head_w1, d, dX, s));
  for (int l = N - 1; l >= 0; --l) {
    const TrainWs::Layer &q = W.layer[l];
    const size_t ld_ = (size_t)l * d;
    // LN2, second feed-forward map, ReLU, first map
    AECCT_TRY(train_ln_bwd(dX, p->ln2_g + ld_, ws + q.xn2, ws + q.rho2, R, d, dR, s));
    AECCT_TRY(train_colsum_dual(dX, d, ws + q.xn2, R, d, g->ln2_g + ld_, g->ln2_b + ld_, part, (int64_t)PF, s));
    AECCT_TRY(gemm(true, false, ws + q.gh, dff, dR, d, gw[5] + wofs(l, 5), d, dff, d, R, nullptr, nullptr, false));
    AECCT_TRY(colsum(dR, d, nullptr, nullptr, R, d, gb[5] + ld_));
    AECCT_TRY(tgemm(true, l, 5, dR, d, dG, dff, R, dff, d, sc + 6 * l + 5, nullptr, false));
    AECCT_TRY(train_relu_bwd(dG, ws + q.f, R * dff, s));
    AECCT_TRY(gemm(true, false, ws + q.x1h, d, dG, dff, gw[4] + wofs(l, 4), dff, d, dff, R, nullptr, nullptr, false));
    AECCT_TRY(colsum(dG, dff, nullptr, nullptr, R, dff, gb[4] + (size_t)l * dff));
    // dX1 = dR + dG T4^T: on the ternary path with dR as the product's addend, else a copy and an
    // accumulating product
    if (tern && train_tern_operands_ok(dG, dff, dX1, d, nullptr, d, dff) && ((uintptr_t)dR & 15u) == 0) {
      const void *f4 = tfrag(l, 4, true);
      const float *s4 = sc + 6 * l + 4;
      AECCT_TRY(train_gemm_tern_ksum(dG, dff, &f4, 1, dff, &s4, dR, dX1, d, R, d, s));
    } else {
      AECCT_TRY(hipMemcpyAsync(dX1, dR, sizeof(float) * R * d, hipMemcpyDeviceToDevice, s));
      AECCT_TRY(tgemm(true, l, 4, dG, dff, dX1, d, R, d, dff, sc + 6 * l + 4, nullptr, true));
    }
    // LN1, output map
    AECCT_TRY(train_ln_bwd(dX1, p->ln1_g + ld_, ws + q.xn1, ws + q.rho1, R, d, dR, s));
    AECCT_TRY(train_colsum_dual(dX1, d, ws + q.xn1, R, d, g->ln1_g + ld_, g->ln1_b + ld_, part, (int64_t)PF, s));
    // dX = dR + sum_k dQKV_k T_k^T below: one product over the packed gradient with dR as its addend
    // on the ternary path, else a copy now and three accumulating products
    const bool qkv_sum = tern && train_tern_operands_ok(dQKV, 3 * d, dX, d, nullptr, d, 3 * d) &&
                         ((uintptr_t)dR & 15u) == 0;
    if (!qkv_sum) AECCT_TRY(hipMemcpyAsync(dX, dR, sizeof(float) * R * d, hipMemcpyDeviceToDevice, s));
    AECCT_TRY(gemm(true, false, ws + q.oh, d, dR, d, gw[3] + wofs(l, 3), d, d, d, R, nullptr, nullptr, false));
    AECCT_TRY(colsum(dR, d, nullptr, nullptr, R, d, gb[3] + ld_));
    AECCT_TRY(tgemm(true, l, 3, dR, d, dO, d, R, d, d, sc + 6 * l + 3, nullptr, false));
    // attention, then the query, key and value maps
    TrainAttn at{ws + q.qkv, R, T.L, d, T.heads, T.hf, T.m1_ptr, T.m1_idx, T.m2_ptr, T.m2_idx, ws + q.o, ws + q.lse,
                 dO, dQKV, ws + W.dv};
    AECCT_TRY(train_attention(1, T.dh, at, s));
    AECCT_TRY(train_attention(2, T.dh, at, s));
    float *const gbq[3] = {gb[0] + ld_, gb[1] + ld_, gb[2] + ld_};
    AECCT_TRY(train_colsum_split(dQKV, 3 * d, R, d, 3, gbq, part, (int64_t)PF, s));
    for (int k = 0; k < 3; ++k) {
      AECCT_TRY(gemm(true, false, ws + q.xh, d, dQKV + k * d, 3 * d, gw[k] + wofs(l, k), d, d, d, R, nullptr, nullptr,
                     false));
      if (!qkv_sum) AECCT_TRY(tgemm(true, l, k, dQKV + k * d, 3 * d, dX, d, R, d, d, sc + 6 * l + k, nullptr, true));
    }
    if (qkv_sum) {
      const void *fq[3] = {tfrag(l, 0, true), tfrag(l, 1, true), tfrag(l, 2, true)};
      const float *sq[3] = {sc + 6 * l, sc + 6 * l + 1, sc + 6 * l + 2};
      AECCT_TRY(train_gemm_tern_ksum(dQKV, 3 * d, fq, 3, d, sq, dR, dX, d, R, d, s));
    }
  }
  // the straight-through Eq. 1 gradients of every matrix from its G = Xh^T dY (nothing in the
  // backward reads G once it is formed), a launch per eight layers
  for (int l0 = 0; l0 < N; l0 += kTrainJobsPerLaunch / 6) {
    TrainDeltaJobs dj{};
    for (int l = l0; l < std::min(N, l0 + kTrainJobsPerLaunch / 6); ++l)
      for (int k = 0; k < 6; ++k)
        dj.j[dj.n++] = TrainDeltaJob{gw[k] + wofs(l, k), pw[k] + wofs(l, k), tmat(l, k), K_in[k] * K_out[k],
                                     gam + 6 * l + k, sc + 6 * l + k, g->delta + 6 * l + k};
    AECCT_TRY(train_delta_grad(dj, T.aap_eps, s));
  }
  AECCT_TRY(train_embed_grad(tv, dX, B, T.L, d, g->embed, s));
#undef AECCT_TRY
  return AECCT_OK;
}

}  // extern "C"
