// Internal model representation shared by the host library and the kernels.
#pragma once

#include <cstddef>
#include <cstdint>

#include <hip/hip_runtime.h>

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
  const uint16_t *o;     // [d][d]
  const uint16_t *ff1;   // [d][d_ff]
  const uint16_t *ff2;   // [d_ff][d]
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
  int device;
  int64_t nnz1, nnz2;
  size_t device_bytes;
  void *dev_block;       // single device allocation holding everything below

  // Tanner graph: check j's variables chk_idx[chk_ptr[j] .. chk_ptr[j+1]) ascending
  const int32_t *chk_ptr, *chk_idx;
  // attention neighbour lists per token, ascending: first ring (M1) and second ring (M2)
  const int32_t *m1_ptr, *m1_idx, *m2_ptr, *m2_idx;
  const float *embed, *pos;   // pos may be null
  const float *head_w1, *head_wo, *head_bo;
  float head_b1;
  LayerWeights layer[kMaxLayers];
};

// ---- launchers (kernels_layered.hip) ---------------------------------------------------
hipError_t launch_embed(const Model &M, const float *y, int64_t words, float *x, int8_t *xq, float *ax,
                        hipStream_t s);
hipError_t launch_qkv(const Model &M, int layer, const int8_t *xq, const float *ax, int64_t rows, float *qkv,
                      hipStream_t s);
hipError_t launch_attention(const Model &M, const float *qkv, int64_t words, float *o, int8_t *oq, float *ao,
                            hipStream_t s);
hipError_t launch_oproj_ln(const Model &M, int layer, const int8_t *oq, const float *ao, const float *x,
                           int64_t rows, float *x1, int8_t *x1q, float *a1, hipStream_t s);
hipError_t launch_ffn1(const Model &M, int layer, const int8_t *x1q, const float *a1, int64_t rows, int8_t *gq,
                      float *ag, hipStream_t s);
hipError_t launch_ffn2_ln(const Model &M, int layer, const int8_t *gq, const float *ag, const float *x1,
                          int64_t rows, float *x, int8_t *xq, float *ax, hipStream_t s);
hipError_t launch_head(const Model &M, const float *x, const float *y, int64_t words, uint8_t *bits,
                       float *logits, hipStream_t s);
hipError_t launch_ternary_gemm(const Model &M, int layer, int kind, const int8_t *a, int64_t rows, int32_t *acc,
                               hipStream_t s);
// ---- fused path (kernel_fused.hip) -----------------------------------------------------
bool fused_supported(const Model &M);
hipError_t launch_fused(const Model &M, const float *y, int64_t words, uint8_t *bits, float *logits,
                        hipStream_t s);

}  // namespace aecct
