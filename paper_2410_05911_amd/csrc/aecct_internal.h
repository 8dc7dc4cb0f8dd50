// Internal model representation shared by the host library and the kernels.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include <hip/hip_runtime.h>

#include "fused_layout.h"

namespace aecct {

constexpr int kMaxLayers = 64;
constexpr int kWave = 64;

// Packed ternary weights of one layer: for every linear map, 16x32 MFMA B-operand
// blocks (16 output columns x 32 inputs), each block 64 lanes x 16 bits (8 codes of
// 2 bits: 00 -> 0, 01 -> +1, 11 -> -1).  Block (t, s) of a map with S = in/32 input
// steps sits at block index t * S + s; the query, key and value maps are packed as
// one [d][3d] map.
struct LayerWeights {
  const uint16_t *qkv;   // blocks of the [d][3d] map
  const uint16_t *qkv_tb;  // the same map reading its inputs in lane order (d = 64, 128), or null
  const uint16_t *o;     // [d][d]
  const uint16_t *ff1;   // [d][d_ff]
  const uint16_t *ff2;   // [d_ff][d]
  // token block (d = 64, 128): O, FF1, FF2 as permuted int8 A fragments and six d-vectors
  // (b_o, ln1_g, ln1_b, b_ff2, ln2_g, ln2_b) in lane order; null otherwise
  const uint64_t *tb_o, *tb_1, *tb_2;
  const float *tb_vec;
  const float *b_qkv;    // [3d]; the query third pre-multiplied by the score scale (see Model::kq)
  const float *b_o, *b_ff1, *b_ff2;
  const float *ln1_g, *ln1_b, *ln2_g, *ln2_b;
  float sq[6];           // fp32(scale / 127) per map, aecct_linear order
  float sq_qs;           // fp32(sq[0] * kq): dequant scale of the scaled queries
};

struct Model {
  int n, m, L, d, n_layers, heads, hf, dff, dh;
  float eps;
  float kq;              // fp32(log2(e) / sqrt(d_h)): score scale folded into the query map
  int path;              // resolved aecct_path
  int attention;         // aecct_attention; under CASA the second-ring lists hold the union, hf = 0
  int lattn;             // resolved aecct_layered_attention: the layered decode's Q/K/V + attention form
  int act_word;          // 1: Eq. 2 takes one alpha per word (aecct_act_scale WORD), else per token
  int device;            // HIP device the model's memory lives on
  int cu_count;          // compute units of that device (persistent grids)
  size_t lds_max;        // LDS bytes one workgroup may use on it
  int64_t nnz1, nnz2;
  size_t device_bytes;
  void *dev_block;       // single device allocation holding everything below
  unsigned char *static_scratch;  // the device's address of the library's static scratch array

  // Tanner graph: check j's variables chk_idx[chk_ptr[j] .. chk_ptr[j+1]) ascending
  const int32_t *chk_ptr, *chk_idx;
  // attention neighbour lists per token, ascending: first ring (M1) and second ring (M2, or
  // M1 | M2 under CASA)
  const int32_t *m1_ptr, *m1_idx, *m2_ptr, *m2_idx;
  // the same lists in groups of four 16-bit token indices (built when L < 2^16): token a's list
  // starts at group meta[2a] and has meta[2a + 1] entries, followed by at least one more group
  bool grouped;
  const int32_t *g1_meta, *g2_meta;
  const uint16_t *g1_tab, *g2_tab;
  // with head partitioning every list holds one node type: the same lists with entries counted
  // from the first token of that type (variables from 0, checks from n), or null
  const uint16_t *g1s_tab, *g2s_tab;
  int32_t g1_groups, g2_groups;      // groups of four entries in g1_tab, g2_tab
  const float *embed, *pos;   // pos may be null
  const float *head_w1, *head_wo, *head_bo;
  const float *head_w1_lo;    // W_{d->1} in the token block's lane order ([4][d/4], d = 64, 128), or null
  const float *embed_lo, *pos_lo;   // embedding / positional rows in that lane order ([L][4][d/4]), or null
  float head_b1;
  LayerWeights layer[kMaxLayers];
  FusedTables fused;
};

// Tanner graph lists (host.cpp): check j's variables chk_idx[chk_ptr[j] .. chk_ptr[j+1]); per token
// its first-ring (M1) and second-ring (M2, self included) neighbours, ascending.
struct TannerLists {
  std::vector<int32_t> chk_ptr, chk_idx, m1_ptr, m1_idx, m2_ptr, m2_idx;
};
TannerLists tanner_lists(const uint8_t *H, int m, int n);
void casa_union(TannerLists &T);   // M2 lists := M1 | M2 (every head on the ECCT mask)

// ---- launchers (kernels_layered.hip) ---------------------------------------------------
// Activation layouts.  Natural: X [rows][d] fp32 and its codes Xq [rows][d] by feature.  Lane
// order (the decode with the token block, d = 64, 128): the token block holds feature 4 v + g
// of a token in register v of lane group g, so X stores feature f at (f % 4) (d / 4) + f / 4
// (a lane's d / 4 values contiguous) and Xq stores feature 32 s + 4 k + g (k < 8, g < 4) at
// byte 32 s + 8 g + k (a lane's eight codes of step s as one 8-byte word); the Q/K/V map is
// packed a second time to read its inputs in that byte order.
hipError_t launch_embed(const Model &M, const float *y, int64_t words, float *x, int8_t *xq, float *ax,
                        bool lane_order, hipStream_t s, float *t = nullptr);
hipError_t launch_qkv(const Model &M, int layer, const int8_t *xq, const float *ax, int64_t rows, float *qkv,
                      bool lane_order, hipStream_t s);
hipError_t launch_attention(const Model &M, const float *qkv, int64_t words, float *o, int8_t *oq, float *ao,
                            hipStream_t s);
// Q/K/V projection and attention fused per word, one 16-dimension head group at a time, into
// fp32 O, then (when oq is not null) Eq. 2 per token of O: the layered decode's path for
// d = 64, 128 when L tokens' Q, K, V of a group fit LDS.  Where the lane-pair form holds a row's
// outputs of every group in registers (qkv_attention_pair_quantises: d = 128, 16-dimension heads,
// at most 384 tokens) and oq is given, the kernel writes only the codes and scales (o unused).
bool qkv_attention_supported(const Model &M);
bool qkv_attention_pair_quantises(const Model &M);
hipError_t launch_qkv_attention(const Model &M, int layer, const int8_t *xq, const float *ax, int64_t words,
                                float *o, int8_t *oq, float *ao, bool lane_order, hipStream_t s);
// The same with keys and values kept in LDS as int16 accumulators (words too long for the fp32
// form, up to about 1800 tokens): writes O in fp32 only.
bool qkv_attention_i16_supported(const Model &M);
// Rows one node type at a time with the other type's keys and values in LDS as fp32 (d = 128,
// 16-dimension heads, head partitioning): writes O in fp32 only.
bool qkv_attention_split_supported(const Model &M);
hipError_t launch_qkv_attention_split(const Model &M, int layer, const int8_t *xq, const float *ax, int64_t words,
                                      float *o, bool lane_order, hipStream_t s);
hipError_t launch_qkv_attention_i16(const Model &M, int layer, const int8_t *xq, const float *ax, int64_t words,
                                    float *o, bool lane_order, hipStream_t s);
// Eq. 2 of the attention output (given as fp32 o, or already as codes oq with scales ao: exactly
// one of o and oq is not null; natural layout), O-projection, residual, LN1, FFN with ReLU,
// residual, LN2 and Eq. 2 of the next layer's input in one kernel (d = 64, 128): one wavefront
// per 16-token strip, activations between the maps only in registers; X and Xq in lane order.
bool token_block_supported(const Model &M);
// words processed at once by the layered attention form `form` (aecct_layered_attention)
int64_t attention_word_slots(const Model &M, int form);
// With z (the last layer): the head's z_i = W_{d->1} x_i + b1 of every output row to z [rows], and
// neither x nor xq nor ax written.
// With t (the first layer): x is not read; X is rebuilt from each token's t_i and the embedding.
hipError_t launch_token_block(const Model &M, int layer, const float *o, const int8_t *oq, const float *ao,
                              float *x, int64_t rows, int8_t *xq, float *ax, hipStream_t s, float *z = nullptr,
                              const float *t = nullptr);
hipError_t launch_oproj_ln(const Model &M, int layer, const int8_t *oq, const float *ao, const float *x,
                           int64_t rows, float *x1, int8_t *x1q, float *a1, hipStream_t s);
hipError_t launch_ffn1(const Model &M, int layer, const int8_t *x1q, const float *a1, int64_t rows, int8_t *gq,
                      float *ag, hipStream_t s);
hipError_t launch_ffn2_ln(const Model &M, int layer, const int8_t *gq, const float *ag, const float *x1,
                          int64_t rows, float *x, int8_t *xq, float *ax, hipStream_t s);
// The head of a decode: z per token into zbuf (words * L floats), then the word-tiled product.
hipError_t launch_head_tiled(const Model &M, const float *x, const float *y, int64_t words, uint8_t *bits,
                             float *logits, bool lane_order, float *zbuf, hipStream_t s, bool z_ready = false);
hipError_t launch_head(const Model &M, const float *x, const float *y, int64_t words, uint8_t *bits,
                       float *logits, bool lane_order, hipStream_t s);
hipError_t launch_ternary_gemm(const Model &M, int layer, int kind, const int8_t *a, int64_t rows, int32_t *acc,
                               hipStream_t s);
// Eq. 2 with one alpha per word over x [words][L][K] fp32 (of max(x, 0) when relu), natural
// layout: codes q [words][L][K], a[row] = the word's alpha for each of its L rows.
hipError_t launch_word_quant(const Model &M, const float *x, int64_t words, int K, bool relu, int8_t *q, float *a,
                             hipStream_t s);
// First feed-forward map (Eq. 3) to fp32, before the ReLU: h [rows][d_ff].
hipError_t launch_ffn1_f32(const Model &M, int layer, const int8_t *x1q, const float *a1, int64_t rows, float *h,
                           hipStream_t s);
// Dynamic-LDS limits of the kernels, set for the current device at create time.
hipError_t set_layered_kernel_attributes(const Model &M);
hipError_t set_fused_kernel_attributes(const Model &M);
// ---- fused path (kernel_fused.hip) -----------------------------------------------------
bool fused_supported(const Model &M);                 // shape check
bool fused_fits(const Model &M, int nbr_words);       // LDS check with the built neighbour table
hipError_t launch_fused(const Model &M, const float *y, int64_t words, uint8_t *bits, float *logits,
                        hipStream_t s);

// ---- quantisation-aware training step (train.hip) ------------------------------------------
// Eq. 1 of one latent matrix: gamma, scale = fp32(gamma * delta) and its ternary copy t (fp32).
struct TrainAapJob {
  const float *w;
  float *t;
  int64_t count;
  const float *delta;
  float *gamma, *scale;
};
// The straight-through Eq. 1 gradients of one matrix from G = Xh^T dY held in dw.
struct TrainDeltaJob {
  float *dw;
  const float *w, *t;
  int64_t count;
  const float *gamma, *scale;
  float *ddelta;
};
struct TrainAttn {
  const float *qkv;     // [rows][3d] Q | K | V (queries unscaled)
  int64_t rows;
  int L, d, heads, hf;
  const int32_t *m1_ptr, *m1_idx, *m2_ptr, *m2_idx;
  float *o, *lse;       // [rows][d] output, [rows][heads] log-sum-exp of the scores
  const float *dout;    // [rows][d] gradient of O (backward)
  float *dqkv;          // [rows][3d] gradients of Q | K | V (backward)
  float *Dv;            // [rows][heads] dO . O (backward)
};
// the six maps of up to eight layers per launch (one block per matrix), passed by value
constexpr int kTrainJobsPerLaunch = 48;
struct TrainAapJobs { TrainAapJob j[kTrainJobsPerLaunch]; int n; };
struct TrainDeltaJobs { TrainDeltaJob j[kTrainJobsPerLaunch]; int n; };
hipError_t train_aap(const TrainAapJobs &jobs, float eps, hipStream_t s);
hipError_t train_delta_grad(const TrainDeltaJobs &jobs, float eps, hipStream_t s);
hipError_t train_embed(const float *y, int64_t rows, int n, int L, int d, const int32_t *chk_ptr,
                       const int32_t *chk_idx, const float *E, const float *P, float *x, float *t, hipStream_t s);
hipError_t train_quant(const float *x, int64_t rows, int K, bool relu, float *xh, hipStream_t s);
// C[M][N] = (accumulate ? C : 0) + scale (op(A) op(B)) + bias; ta: A stored [K][M]; tb: B stored [N][K].
// part: scratch of part_floats floats for split reductions over K.
// Products with a ternary right operand on the bf16 matrix cores (fp32 A split exactly into three
// bf16 parts): train_pack_tern lays each job's T [R][C] (or its transpose) out as B fragments in
// out (2 R C bytes), train_gemm_tern forms C = beta C + scale (A B) + bias; N a multiple of 64, K
// of 32, A, C and the bias 16-byte aligned with lda and ldc multiples of 4 (train_tern_operands_ok).
bool train_tern_shape_ok(int64_t N, int64_t K);
bool train_tern_operands_ok(const float *A, int64_t lda, const float *C, int64_t ldc, const float *bias, int64_t N,
                            int64_t K);
struct TernPackJob {
  const float *T;
  int R, C, trans;
  void *out;
};
struct TernPackJobs { TernPackJob j[kTrainJobsPerLaunch]; int n; };
hipError_t train_pack_tern(const TernPackJobs &jobs, hipStream_t s);
hipError_t train_gemm_tern(const float *A, int64_t lda, const void *frag, float *C, int64_t ldc, int64_t M, int64_t N,
                           int64_t K, const float *scale, const float *bias, bool accumulate, hipStream_t s);
// nseg (<= 3) ternary matrices side by side: C[:, k seg_n .. (k + 1) seg_n) = beta C + scale[k] (A T_k) +
// bias[k] for each k, over one read of A
hipError_t train_gemm_tern_seg(const float *A, int64_t lda, const void *const *frag, float *C, int64_t ldc, int64_t M,
                               int64_t seg_n, int nseg, int64_t K, const float *const *scale, const float *const *bias,
                               bool accumulate, hipStream_t s);
// C = D + sum_k scale[k] (A[:, k kseg .. (k + 1) kseg) T_k) over nseg (<= 3) ternary matrices along A's
// row, D (optional, laid out like C, may be C) an addend: the input gradient summed over the query,
// key and value maps from their packed gradient
hipError_t train_gemm_tern_ksum(const float *A, int64_t lda, const void *const *frag, int nseg, int64_t kseg,
                                const float *const *scale, const float *D, float *C, int64_t ldc, int64_t M, int64_t N,
                                hipStream_t s);
hipError_t train_gemm(bool ta, bool tb, const float *A, int64_t lda, const float *B, int64_t ldb, float *C, int64_t ldc,
                      int64_t M, int64_t N, int64_t K, const float *scale, const float *bias, bool accumulate,
                      float *part, int64_t part_floats, int cu_count, hipStream_t s);
// which: 0 forward (o, lse), 1 query gradients (dqkv's Q third, Dv), 2 key and value gradients
hipError_t train_attention(int which, int dh, const TrainAttn &a, hipStream_t s);
// out = LN(a + b), xn the normalised row, rho its 1 / sigma; xh (if given) the Eq. 2 codes of out and
// their values, as train_quant forms them
hipError_t train_ln_fwd(const float *a, const float *b, int64_t rows, int d, const float *g, const float *beta, float eps,
                        float *out, float *xn, float *rho, float *xh, hipStream_t s);
hipError_t train_ln_bwd(const float *dy, const float *g, const float *xn, const float *rho, int64_t rows, int d,
                        float *dR, hipStream_t s);
// out[c] (+)= sum_r A[r][c] (B[r][c] if B) (w[r] if w), rows of A lda apart, B dense [rows][C]
hipError_t train_colsum(const float *A, int64_t lda, const float *Bm, const float *w, int64_t rows, int C, float *out,
                        bool accumulate, float *part, int64_t part_floats, hipStream_t s);
// out_ab[c] = sum_r A[r][c] B[r][c] and out_a[c] = sum_r A[r][c] in one pass (a LayerNorm's gain and
// shift gradients)
hipError_t train_colsum_dual(const float *A, int64_t lda, const float *Bm, int64_t rows, int C, float *out_ab,
                             float *out_a, float *part, int64_t part_floats, hipStream_t s);
// the column sums of A's nseg * seg columns, segment k to outs[k] (nseg <= 3: the query, key and value
// bias gradients from one pass over the packed [rows][3 d] gradient)
hipError_t train_colsum_split(const float *A, int64_t lda, int64_t rows, int seg, int nseg, float *const *outs,
                              float *part, int64_t part_floats, hipStream_t s);
hipError_t train_relu_bwd(float *dg, const float *f, int64_t count, hipStream_t s);
hipError_t train_rowdot(const float *x, int64_t rows, int d, const float *w1, const float *b1, float *z, hipStream_t s);
hipError_t train_outer(const float *dz, int64_t rows, const float *w1, int d, float *dx, hipStream_t s);
hipError_t train_loss(const float *f, const float *y, const float *xs, int64_t count, float *df, float *part,
                      float *loss, hipStream_t s);
hipError_t train_embed_grad(const float *t, const float *dx, int64_t words, int L, int d, float *de, hipStream_t s);

}  // namespace aecct
