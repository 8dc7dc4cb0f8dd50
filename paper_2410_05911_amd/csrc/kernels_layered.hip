// Layered path: one kernel per stage of the AECCT forward pass, activations in
// device memory between stages.  Used for any code length; the fused path covers
// short codes in a single launch.
//
// Row layout of every activation: row b * L + r for token r of word b, features
// contiguous.  Tokens 0..n-1 are variable nodes, n..n+m-1 check nodes (Section 3).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "aecct_internal.h"
#include "device_common.h"

namespace aecct {

// Positions of feature f of a d-wide row in the lane-order layouts (the token block's register
// layout): X (fp32) and Xq (codes).
template <int D>
__device__ __forceinline__ int lane_order_x(int f) { return (f & 3) * (D / 4) + (f >> 2); }
__device__ __forceinline__ int lane_order_q(int f) { return (f & ~31) + 8 * (f & 3) + ((f >> 2) & 7); }

// The two values of lanes l and l ^ M (M = 16 or 32) with the gfx950 lane swaps: a swap of v
// with itself returns, in some order, the lane's own v and its partner's, so their sum or
// maximum is a butterfly step's (both operations commute).  The swap's two results are taken
// out of its vector as integers: __builtin_bit_cast applied directly to an element of a vector
// reads element 0 with this compiler.
template <int M>
__device__ __forceinline__ void lane_swap_pair(uint32_t v, uint32_t &a, uint32_t &b) {
  if constexpr (M == 32) {
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    a = r[0];
    b = r[1];
  } else {
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    a = r[0];
    b = r[1];
  }
}
// v of this lane plus v of lane l ^ M (the same bits in both lanes)
template <int M>
__device__ __forceinline__ float lane_xor_add(float t) {
  uint32_t a, b;
  lane_swap_pair<M>(__builtin_bit_cast(uint32_t, t), a, b);
  return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
}

// Byte 0 of eight Eq. 2 code patterns into one 64-bit B operand (byte e from b[e]).
__device__ __forceinline__ long tb_pack8(const uint32_t (&b)[8]) {
  const uint32_t lo = __builtin_amdgcn_perm(__builtin_amdgcn_perm(b[3], b[2], 0x0c0c0400u),
                                            __builtin_amdgcn_perm(b[1], b[0], 0x0c0c0400u), 0x05040100u);
  const uint32_t hi = __builtin_amdgcn_perm(__builtin_amdgcn_perm(b[7], b[6], 0x0c0c0400u),
                                            __builtin_amdgcn_perm(b[5], b[4], 0x0c0c0400u), 0x05040100u);
  return (long)(((uint64_t)hi << 32) | lo);
}

// ------------------------------------------------------------------------------------------
// Embedding: pre-processing h(y) (Section 3), X = t * E (+ P), and the Eq. 2 code of X.
// 16 lanes per row.  Natural layout: lane c holds features c + 16 t, t < D / 16.  LO: X and Xq in
// lane order, lane c holding the D / 16 consecutive lane-order positions from c D / 16 on (of
// Xq, position 32 s + 8 g + e holds feature 32 s + 4 e + g; of X and of the lane-order
// embedding rows, position g D / 4 + v holds feature 4 v + g, the same features), so that its
// reads and writes are contiguous.
// ------------------------------------------------------------------------------------------
struct EmbedArgs {
  const float *y;
  int64_t rows;
  int n, L;
  const int32_t *chk_ptr, *chk_idx;
  const float *embed, *pos;
  float *x;
  int8_t *xq;
  float *ax;
  float *t;   // with x null: each token's t_i (|y_i| or the syndrome sign), from which the first
              // token block rebuilds X
  const float *elo, *plo;   // LO: embedding and positional rows in lane order (plo may be null)
};

// Row g (token i of its word, t = t_i) in lane order, lane c of the row's 16: positions F c ..
// F c + F - 1 of Xq (F = D / 16): s = F c / 32, g = (F c / 8) mod 4, e from F c mod 8, whose
// features 32 s + 4 e + g sit at lane-order position g D / 4 + 8 s + e of X and of the
// lane-order embedding rows.
template <int D>
__device__ __forceinline__ void embed_row_lo(const EmbedArgs &p, int64_t g, int i, float t, int c) {
  constexpr int F = D / 16;
  const int q0 = F * c, sx = q0 >> 5, gx = (q0 >> 3) & 3, e0 = q0 & 7;
  const int xo = gx * (D / 4) + 8 * sx + e0;
  float v[F];
  float amax = 0.0f;
#pragma unroll
  for (int u = 0; u < F; u += 4) {
    const float4 e = *(const float4 *)(p.elo + (int64_t)i * D + xo + u);
    const float4 q = p.plo ? *(const float4 *)(p.plo + (int64_t)i * D + xo + u) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    v[u] = __builtin_fmaf(t, e.x, q.x);
    v[u + 1] = __builtin_fmaf(t, e.y, q.y);
    v[u + 2] = __builtin_fmaf(t, e.z, q.z);
    v[u + 3] = __builtin_fmaf(t, e.w, q.w);
    if (p.x) *(float4 *)(p.x + g * D + xo + u) = make_float4(v[u], v[u + 1], v[u + 2], v[u + 3]);
  }
#pragma unroll
  for (int u = 0; u < F; ++u) amax = fmaxf(amax, fabsf(v[u]));
  amax = row16_max(amax);
  const float inv = inv127(amax);
  uint32_t b[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) b[u] = quant_bits(v[u < F ? u : 0], inv);
  if constexpr (F == 8) {
    *(long *)(p.xq + g * D + q0) = tb_pack8(b);
  } else {
    *(uint32_t *)(p.xq + g * D + q0) = (uint32_t)tb_pack8(b);
  }
  if (c == 0) p.ax[g] = amax;
  if (c == 0 && p.t) p.t[g] = t;
}

// Lane order, one word per block (persistent over the words): the word's y in LDS, every
// token's t_i from it (the checks' lists from the L2), then the rows, 16 lanes each.
constexpr int kEwThreads = 256;
template <int D>
__global__ __launch_bounds__(kEwThreads) void k_embed_words(EmbedArgs p, int64_t words) {
  extern __shared__ float esm[];   // [n] the word's y, [L] its t
  float *ys = esm, *ts = esm + p.n;
  const int tid = threadIdx.x, c = tid & 15;
  for (int64_t w = blockIdx.x; w < words; w += gridDim.x) {
    const float *yw = p.y + w * p.n;
    for (int i = tid; i < p.n; i += kEwThreads) ys[i] = yw[i];
    __syncthreads();
    for (int i = tid; i < p.L; i += kEwThreads) {
      float t;
      if (i < p.n) {
        t = fabsf(ys[i]);
      } else {
        int s = 0;
        for (int e = p.chk_ptr[i - p.n]; e < p.chk_ptr[i - p.n + 1]; ++e) s ^= (ys[p.chk_idx[e]] < 0.0f) ? 1 : 0;
        t = s ? -1.0f : 1.0f;
      }
      ts[i] = t;
    }
    __syncthreads();
    for (int i = tid >> 4; i < p.L; i += kEwThreads / 16) embed_row_lo<D>(p, w * p.L + i, i, ts[i], c);
    __syncthreads();   // the next word overwrites y and t
  }
}

// 16 lanes per row, one row per 16 lanes of the grid: the natural layout, or (LO) the lane order
// for words whose y and t do not fit LDS.
template <int D, bool LO>
__global__ __launch_bounds__(256) void k_embed(EmbedArgs p) {
  constexpr int T = D / 16;
  const int c = threadIdx.x & 15;
  const int64_t g = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
  if (g >= p.rows) return;  // uniform over the 16 lanes of a row
  const int64_t w = g / p.L;
  const int i = (int)(g - w * p.L);
  const float *yw = p.y + w * p.n;
  float t;
  if (i < p.n) {
    t = fabsf(yw[i]);
  } else {
    int s = 0;
    for (int e = p.chk_ptr[i - p.n]; e < p.chk_ptr[i - p.n + 1]; ++e) s ^= (yw[p.chk_idx[e]] < 0.0f) ? 1 : 0;
    t = s ? -1.0f : 1.0f;
  }
  if constexpr (LO) {
    embed_row_lo<D>(p, g, i, t, c);
    return;
  }
  float v[T];
  float amax = 0.0f;
#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    const int col = 16 * tt + c;
    v[tt] = __builtin_fmaf(t, p.embed[(int64_t)i * D + col], p.pos ? p.pos[(int64_t)i * D + col] : 0.0f);
    if (p.x) p.x[g * D + col] = v[tt];
    amax = fmaxf(amax, fabsf(v[tt]));
  }
  amax = row16_max(amax);
  const float inv = inv127(amax);
#pragma unroll
  for (int tt = 0; tt < T; ++tt) p.xq[g * D + 16 * tt + c] = quant_code(v[tt], inv);
  if (c == 0) p.ax[g] = amax;
}

// ------------------------------------------------------------------------------------------
// Ternary x int8 GEMM on int8 MFMA (Eq. 3) with fused epilogues.
// A block stages its packed weights once into LDS as int8 B fragments, then its four
// waves walk 16-row strips: one wave owns all output columns of its 16 rows, so the
// row-wise LayerNorm and absmax reductions stay inside the wave (intra-lane over the
// column tiles, then a 16-lane DPP reduction).
// ------------------------------------------------------------------------------------------
// EPI_QKV_MAP: one of the three maps of EPI_QKV per launch (out_f and bias pointing at the map's
// columns, rows 3 NOUT apart, scale sq[0]), a third of the accumulators of the fused launch.
// Orders this wavefront's LDS writes before its following LDS reads (and the reverse).
__device__ __forceinline__ void wave_barrier_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// EPI_F32: plain fp32 output fma(acc, alpha sq[0], bias) of every column (the feed-forward hidden
// row before its ReLU, when Eq. 2 of the hidden row takes one alpha per word).
enum Epi { EPI_RAW = 0, EPI_QKV = 1, EPI_LN = 2, EPI_RELU_QUANT = 3, EPI_QKV_MAP = 4, EPI_F32 = 5 };

struct GemmArgs {
  const int8_t *a;        // [rows][K]
  const float *alpha;     // [rows] Eq. 2 scale of each A row
  const uint16_t *bpack;  // packed B blocks of the whole map
  int tile0;              // first 16-column tile of the map this launch computes
  int64_t rows;
  float sq[3];            // per 1/3 of the columns (QKV) or sq[0] for all: fp32(scale / 127)
  const float *bias;      // [NOUT] (QKV: the query third already scaled like sq[0])
  const float *resid;     // [rows][NOUT] (LN)
  const float *ln_g, *ln_b;
  float eps;
  float *out_f;           // fp32 output (QKV, LN)
  int8_t *out_q;          // int8 output (LN, RELU_QUANT)
  float *out_a;           // [rows] scale of out_q rows
  int32_t *out_acc;       // raw accumulators (RAW)
};

constexpr int kGemmWaves = 8;

template <int K, int NOUT, int EPI>
__global__ __launch_bounds__(kGemmWaves * 64) void k_gemm(GemmArgs p) {
  constexpr int S = K / 32;
  constexpr int T = NOUT / 16;
  constexpr bool kQuantOut = (EPI == EPI_LN || EPI == EPI_RELU_QUANT);
  __shared__ uint64_t bsm[T * S * 64];
  __shared__ __attribute__((aligned(16))) int8_t qstage[kQuantOut ? kGemmWaves : 1][kQuantOut ? 16 * NOUT : 16];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  {
    const uint16_t *src = p.bpack + (size_t)p.tile0 * S * 64;
    for (int u = tid; u < T * S * 64; u += kGemmWaves * 64) bsm[u] = unpack_ternary8(src[u]);
  }
  __syncthreads();

  const int64_t nstrips = (p.rows + 15) / 16;
  const int64_t ngroups = (nstrips + kGemmWaves - 1) / kGemmWaves;
  const int col = lane & 15, rg = lane >> 4;
  for (int64_t grp = blockIdx.x; grp < ngroups; grp += gridDim.x) {
    const int64_t row0 = (grp * kGemmWaves + wave) * 16;
    long afr[S];
    {
      const int64_t ar = row0 + col;
#pragma unroll
      for (int s = 0; s < S; ++s)
        afr[s] = ar < p.rows ? *(const long *)(p.a + ar * K + 32 * s + 8 * rg) : 0;
    }
    v4i acc[T];
#pragma unroll
    for (int t = 0; t < T; ++t) {
      acc[t] = v4i{0, 0, 0, 0};
      acc[t] = mfma_i8_steps<S>([&](int s) { return afr[s]; }, [&](int s) { return (long)bsm[(t * S + s) * 64 + lane]; },
                                acc[t]);
    }

    int64_t r[4];
    bool ok[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      r[i] = row0 + 4 * rg + i;
      ok[i] = r[i] < p.rows;
    }

    if constexpr (EPI == EPI_RAW) {
#pragma unroll
      for (int t = 0; t < T; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (ok[i]) p.out_acc[r[i] * NOUT + 16 * t + col] = acc[t][i];
    } else {
      float al[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) al[i] = ok[i] ? p.alpha[r[i]] : 0.0f;
      if constexpr (EPI == EPI_F32) {
#pragma unroll
        for (int t = 0; t < T; ++t) {
          const int j = 16 * t + col;
          const float b = p.bias[j];
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (ok[i]) p.out_f[r[i] * NOUT + j] = __builtin_fmaf((float)acc[t][i], al[i] * p.sq[0], b);
        }
      } else if constexpr (EPI == EPI_QKV_MAP) {
#pragma unroll
        for (int t = 0; t < T; ++t) {
          const int j = 16 * t + col;
          const float b = p.bias[j];
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (ok[i]) p.out_f[r[i] * (3 * NOUT) + j] = __builtin_fmaf((float)acc[t][i], al[i] * p.sq[0], b);
        }
      } else if constexpr (EPI == EPI_QKV) {
        constexpr int TB = T / 3;  // tiles per map
#pragma unroll
        for (int t = 0; t < T; ++t) {
          const int j = 16 * t + col;
          const float sq = p.sq[t / TB];
          const float b = p.bias[j];
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (ok[i]) p.out_f[r[i] * NOUT + j] = __builtin_fmaf((float)acc[t][i], al[i] * sq, b);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float sc = al[i] * p.sq[0];
          float v[T];
          if constexpr (EPI == EPI_LN) {
            // residual + LayerNorm over the NOUT (= d) features of row r[i]
            float e[T], sq[T], tmp[T];
#pragma unroll
            for (int t = 0; t < T; ++t) {
              const int j = 16 * t + col;
              const float y = __builtin_fmaf((float)acc[t][i], sc, p.bias[j]);
              const float res = ok[i] ? p.resid[r[i] * NOUT + j] : 0.0f;
              v[t] = res + y;
              tmp[t] = v[t];
            }
            const float mean = row16_sum(lane_tree<T>(tmp)) / (float)NOUT;
#pragma unroll
            for (int t = 0; t < T; ++t) {
              e[t] = v[t] - mean;
              sq[t] = e[t] * e[t];
            }
            const float var = row16_sum(lane_tree<T>(sq)) / (float)NOUT;
            const float rho = ln_rsqrt(var + p.eps);
#pragma unroll
            for (int t = 0; t < T; ++t) {
              const int j = 16 * t + col;
              v[t] = __builtin_fmaf(e[t] * rho, p.ln_g[j], p.ln_b[j]);
              if (ok[i]) p.out_f[r[i] * NOUT + j] = v[t];
            }
          } else {  // EPI_RELU_QUANT
#pragma unroll
            for (int t = 0; t < T; ++t) {
              const float f = __builtin_fmaf((float)acc[t][i], sc, p.bias[16 * t + col]);
              v[t] = f > 0.0f ? f : 0.0f;
            }
          }
          // Eq. 2 on the finished row
          float amax = 0.0f;
#pragma unroll
          for (int t = 0; t < T; ++t) amax = fmaxf(amax, fabsf(v[t]));
          amax = row16_max(amax);
          const float inv = inv127(amax);
#pragma unroll
          for (int t = 0; t < T; ++t) qstage[wave][(4 * rg + i) * NOUT + 16 * t + col] = quant_code(v[t], inv);
          if (col == 0 && ok[i]) p.out_a[r[i]] = amax;
        }
      }
    }
    if constexpr (kQuantOut) {
      __syncthreads();
      const int64_t valid = p.rows - row0 < 16 ? (p.rows - row0 > 0 ? p.rows - row0 : 0) : 16;
      const int chunks = (int)(valid * NOUT / 16);
      const uint4 *src = (const uint4 *)qstage[wave];
      uint4 *dst = (uint4 *)(p.out_q + row0 * NOUT);
      for (int cidx = lane; cidx < chunks; cidx += 64) dst[cidx] = src[cidx];
      __syncthreads();
    }
  }
}

// ------------------------------------------------------------------------------------------
// Head-partitioned attention (Section 4.2): one lane per (row, head); heads 0..hf-1 read
// the first-ring neighbour list of the row, the others the second-ring list.  One pass over
// the neighbours (ascending) sums the base-2 exponentials of the scores (query rows arrive
// scaled by log2(e)/sqrt(d_h)) and the weighted values; a row whose sum falls outside
// [2^-64, 2^64] is redone with the scores shifted by their maximum.  The heads of a row sit
// in adjacent lanes, so the row's Eq. 2 scale is a shuffle reduction.
// ------------------------------------------------------------------------------------------
struct AttnArgs {
  const float *qkv;
  int64_t rows;
  int L, d, heads, hf;
  const int32_t *m1_ptr, *m1_idx, *m2_ptr, *m2_idx;
  float *o;
  int8_t *oq;
  float *ao;
};

template <int DH>
__global__ __launch_bounds__(256) void k_attention(AttnArgs p) {
  const int heads = p.heads;
  const int rpb = 256 / heads;
  const int h = threadIdx.x % heads;
  const int64_t g = (int64_t)blockIdx.x * rpb + threadIdx.x / heads;
  const bool valid = g < p.rows;
  const int d = p.d, d3 = 3 * p.d;
  const int64_t w = valid ? g / p.L : 0;
  const int i = valid ? (int)(g - w * p.L) : 0;
  const int32_t *ptr = h < p.hf ? p.m1_ptr : p.m2_ptr;
  const int32_t *idx = h < p.hf ? p.m1_idx : p.m2_idx;
  const int beg = valid ? ptr[i] : 0, end = valid ? ptr[i + 1] : 0;
  const float *base = p.qkv + w * p.L * d3;
  float q[DH];
#pragma unroll
  for (int t = 0; t < DH; ++t) q[t] = valid ? base[(int64_t)i * d3 + h * DH + t] : 0.0f;

  // weights 2^s unshifted; rows whose sum leaves [2^-64, 2^64] are redone shifted by max s
  float S = 0.0f, acc[DH];
#pragma unroll
  for (int t = 0; t < DH; ++t) acc[t] = 0.0f;
  for (int e = beg; e < end; ++e) {
    const float *kr = base + (int64_t)idx[e] * d3 + d + h * DH;
    const float ex = softmax_exp2(head_dot<DH>(q, kr));
    S = S + ex;
    const float *vr = kr + d;
#pragma unroll
    for (int t = 0; t < DH; ++t) acc[t] = __builtin_fmaf(ex, vr[t], acc[t]);
  }
  if (end > beg && !(S >= 0x1p-64f && S <= 0x1p64f)) {
    float mu = -INFINITY;
    for (int e = beg; e < end; ++e) {
      const float *kr = base + (int64_t)idx[e] * d3 + d + h * DH;
      mu = fmaxf(mu, head_dot<DH>(q, kr));
    }
    S = 0.0f;
#pragma unroll
    for (int t = 0; t < DH; ++t) acc[t] = 0.0f;
    for (int e = beg; e < end; ++e) {
      const float *kr = base + (int64_t)idx[e] * d3 + d + h * DH;
      const float ex = softmax_exp2(head_dot<DH>(q, kr) - mu);
      S = S + ex;
      const float *vr = kr + d;
#pragma unroll
      for (int t = 0; t < DH; ++t) acc[t] = __builtin_fmaf(ex, vr[t], acc[t]);
    }
  }
  const float rS = valid ? recip_softmax_sum(S) : 0.0f;
  float amax = 0.0f;
#pragma unroll
  for (int t = 0; t < DH; ++t) {
    acc[t] = acc[t] * rS;
    amax = fmaxf(amax, fabsf(acc[t]));
  }
  for (int off = 1; off < heads; off <<= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  if (!valid) return;
  const float inv = inv127(amax);
  int8_t qv[DH];
#pragma unroll
  for (int t = 0; t < DH; ++t) qv[t] = quant_code(acc[t], inv);
  int8_t *dq = p.oq + g * d + h * DH;
#pragma unroll
  for (int t = 0; t < DH; ++t) dq[t] = qv[t];
  if (p.o) {
#pragma unroll
    for (int t = 0; t < DH; ++t) p.o[g * d + h * DH + t] = acc[t];
  }
  if (h == 0) p.ao[g] = amax;
}

// ------------------------------------------------------------------------------------------
// Query/key/value projection and attention of one word, one 16-dimension head group at a time
// (d = 64 or 128).  The group's three 16-column tiles of the packed QKV map (Eq. 3) are
// multiplied for all L tokens on v_mfma_i32_16x16x32_i8 and dequantised into LDS (fp32: Q as
// [L][16], K and V of a token side by side in one 144-byte row), then the group's attention
// rows (Section 4.2, the same single-pass base-2 softmax and the same evaluation order as
// k_attention) gather their neighbours' keys and values from LDS.  A row's neighbour indices
// come four to an 8-byte group, the next group read while the current one's rows are gathered.
// Blocks are persistent over the words and take every head group of a word in turn, so
// first-ring groups (short neighbour lists) and second-ring groups (long ones) share each
// block's time; the next group's weight tiles are loaded while the current group's rows run.
// Writes the attention output O (fp32 [rows][d]); Eq. 2 of O runs in the token block (or in
// k_quant_rows).  A head's keys are gathered by neighbour index: the 144-byte row stride puts
// rows on 16 different 16-byte bank groups (at 128 bytes random gathers collide far more, and
// the kernel ran about 30 % slower).
// ------------------------------------------------------------------------------------------
struct QkvAttnArgs {
  const int8_t *xq;       // [rows][d] Eq. 2 codes of the layer input
  const float *ax;        // [rows] their scales
  const uint16_t *bpack;  // packed QKV map ([d][3d])
  const float *bias;      // [3d]; the query third pre-scaled like sq[0]
  float sq[3];            // dequant scale of Q (with log2(e)/sqrt(d_h)), K, V
  int64_t words;
  int L, hf;
  const int2 *meta1, *meta2;   // per token: first group, entry count (first ring, second ring)
  const uint2 *tab1, *tab2;    // four 16-bit token indices per group
  float *o;                    // [rows][d]
  // k_qkv_attention_pair with the quantised output: Eq. 2 codes [rows][d] and scales [rows] of
  // O instead of o
  int8_t *oq;
  float *ao;
  int resident;                // k_qkv_attention: every head group's weight tiles stay in LDS
  // k_qkv_attention_split: the same lists with every entry counted from the first token of its
  // node type (variables from 0, checks from n), the variable count n, and the LDS capacity in
  // tokens of the larger node type
  const uint2 *tab1s, *tab2s;
  int n_var, kv_cap;
  int tab1_n, tab2_n;          // groups in tab1, tab2 (k_qkv_attention_pair with the lists in LDS)
};

constexpr int kQaThreads = 512;
// K (16 floats) and V (16 floats) of a token in one row of kQaRow floats: 144 bytes apart, rows
// start on 16 different 16-byte bank groups, so random neighbour gathers collide less, and a
// value sits at a fixed 64-byte offset from its key.
constexpr int kQaRow = 36;

// Block barrier that orders LDS accesses only: waits for this wave's LDS operations, not for
// its global stores or loads in flight (the attention outputs and the next weight tiles).
__device__ __forceinline__ void block_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <int D>
constexpr size_t qa_frag_bytes() { return (size_t)3 * (D / 32) * 64 * 8; }
// Token tiles a wavefront keeps in registers across a word's head groups (L <= 16 x 8 x 4).
constexpr int kQaTilesPerWave = 4;

// Head group hg's three weight tiles, 2-bit codes from HBM: the loads are issued early (into
// registers) and unpacked into int8 fragments in LDS later, so their latency overlaps the rows.
template <int D, int NT = kQaThreads>
struct QaStage {
  static constexpr int kWords = 3 * (D / 32) * 64, kPer = (kWords + NT - 1) / NT;
  uint32_t pk[kPer];
  __device__ __forceinline__ void load(const uint16_t *bpack, int hg, int tid) {
    constexpr int S = D / 32, G = D / 16;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int u = tid + k * NT;
      const int m = u / (S * 64), rest = u - m * (S * 64);
      pk[k] = u < kWords ? bpack[(size_t)(m * G + hg) * S * 64 + rest] : 0u;
    }
  }
  __device__ __forceinline__ void store(uint64_t *bf, int tid) const {
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int u = tid + k * NT;
      if (u < kWords) bf[u] = unpack_ternary8(pk[k]);
    }
  }
  // only the query map's fragments (Q) or only the key and value maps' (!Q)
  template <bool Q>
  __device__ __forceinline__ void store_part(uint64_t *bf, int tid) const {
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int u = tid + k * NT;
      if (u < kWords && (u < (D / 32) * 64) == Q) bf[u] = unpack_ternary8(pk[k]);
    }
  }
};

// d_h consecutive floats of LDS (16-byte aligned) into registers.
template <int DH>
__device__ __forceinline__ void qa_load(float (&x)[DH], const float *p) {
#pragma unroll
  for (int t = 0; t < DH; t += 4) {
    const float4 a = *(const float4 *)(p + t);
    x[t] = a.x; x[t + 1] = a.y; x[t + 2] = a.z; x[t + 3] = a.w;
  }
}

// One neighbour of the base-2 softmax: score DOT(q', k), weight 2^(s - shift), and the running
// sums S and acc (ascending neighbours).
template <int DH>
__device__ __forceinline__ void qa_step(const float (&q)[DH], const float (&k)[DH], const float (&v)[DH], float shift,
                                        float &S, float (&acc)[DH]) {
  const float ex = softmax_exp2(head_dot<DH>(q, k) - shift);
  S = S + ex;
#pragma unroll
  for (int t = 0; t < DH; ++t) acc[t] = __builtin_fmaf(ex, v[t], acc[t]);
}
// kr points at the neighbour's key, its value 16 floats further.
template <int DH>
__device__ __forceinline__ void qa_step(const float (&q)[DH], const float *kr, float shift, float &S,
                                        float (&acc)[DH]) {
  float k[DH], v[DH];
#pragma unroll
  for (int t = 0; t < DH; t += 4) {
    const float4 a = *(const float4 *)(kr + t), b = *(const float4 *)(kr + 16 + t);
    k[t] = a.x; k[t + 1] = a.y; k[t + 2] = a.z; k[t + 3] = a.w;
    v[t] = b.x; v[t + 1] = b.y; v[t + 2] = b.z; v[t + 3] = b.w;
  }
  qa_step<DH>(q, k, v, shift, S, acc);
}

__device__ __forceinline__ uint32_t qa_entry(const uint2 *eg, int e) {
  const uint2 gq = eg[e >> 2];
  const uint32_t w = (e & 2) ? gq.y : gq.x;
  return (e & 1) ? w >> 16 : w & 0xffffu;
}

// Attention of one (token, head) row over its cnt neighbours (ascending), entries from eg with
// the first group already in g0; writes the row's d_h outputs.
template <int DH, bool PIPE>
__device__ __forceinline__ void qa_row(const float *qrow, const float *kb, const uint2 *eg, uint2 g0, int cnt,
                                       float *orow) {
  constexpr int R = kQaRow;
  float q[DH];
#pragma unroll
  for (int t = 0; t < DH; t += 4) {
    const float4 a = *(const float4 *)(qrow + t);
    q[t] = a.x; q[t + 1] = a.y; q[t + 2] = a.z; q[t + 3] = a.w;
  }
  float S_ = 0.0f, acc[DH];
#pragma unroll
  for (int t = 0; t < DH; ++t) acc[t] = 0.0f;
  // Software pipelined (PIPE): a neighbour's value and the next neighbour's key are read
  // before the neighbour's score is computed.  Every list stores a group after its last full
  // one (unused slots hold token 0), so each look-ahead read stays within the word's rows.
  // The scheduling barriers keep the compiler from hoisting further reads (their registers
  // would spill).
  if constexpr (PIPE) {
    uint2 gc = g0;
    float ka[DH], kb_[DH], v[DH];
    qa_load<DH>(ka, kb + (gc.x & 0xffffu) * R);
    auto stage = [&](uint32_t cur, uint32_t nxt, float (&kc)[DH], float (&kn)[DH]) {
      qa_load<DH>(v, kb + cur * R + 16);
      qa_load<DH>(kn, kb + nxt * R);
      qa_step<DH>(q, kc, v, 0.0f, S_, acc);
      __builtin_amdgcn_sched_barrier(0);
    };
    for (int u = 0; u < (cnt >> 2); ++u) {
      const uint2 gn = eg[u + 1];
      stage(gc.x & 0xffffu, gc.x >> 16, ka, kb_);
      stage(gc.x >> 16, gc.y & 0xffffu, kb_, ka);
      stage(gc.y & 0xffffu, gc.y >> 16, ka, kb_);
      stage(gc.y >> 16, gn.x & 0xffffu, kb_, ka);
      gc = gn;
    }
    const int rem = cnt & 3;    // the last, partial group is in gc, its first key in ka
    if (rem > 0) stage(gc.x & 0xffffu, gc.x >> 16, ka, kb_);
    if (rem > 1) stage(gc.x >> 16, gc.y & 0xffffu, kb_, ka);
    if (rem > 2) stage(gc.y & 0xffffu, gc.y >> 16, ka, kb_);
  } else {
    uint2 nx = g0;
    for (int u = 0; u < (cnt >> 2); ++u) {
      const uint32_t e0 = nx.x & 0xffffu, e1 = nx.x >> 16, e2 = nx.y & 0xffffu, e3 = nx.y >> 16;
      nx = eg[u + 1];           // stored: every list has a group after its last full one
      qa_step<DH>(q, kb + e0 * R, 0.0f, S_, acc);
      qa_step<DH>(q, kb + e1 * R, 0.0f, S_, acc);
      qa_step<DH>(q, kb + e2 * R, 0.0f, S_, acc);
      qa_step<DH>(q, kb + e3 * R, 0.0f, S_, acc);
    }
    const int rem = cnt & 3;    // the last, partial group is already in nx
    if (rem > 0) qa_step<DH>(q, kb + (nx.x & 0xffffu) * R, 0.0f, S_, acc);
    if (rem > 1) qa_step<DH>(q, kb + (nx.x >> 16) * R, 0.0f, S_, acc);
    if (rem > 2) qa_step<DH>(q, kb + (nx.y & 0xffffu) * R, 0.0f, S_, acc);
  }
  if (cnt > 0 && !(S_ >= 0x1p-64f && S_ <= 0x1p64f)) {
    float mu = -INFINITY;
    for (int e = 0; e < cnt; ++e) {
      const float *kr = kb + qa_entry(eg, e) * R;
      float k[DH];
#pragma unroll
      for (int t = 0; t < DH; ++t) k[t] = kr[t];
      mu = fmaxf(mu, head_dot<DH>(q, k));
    }
    S_ = 0.0f;
#pragma unroll
    for (int t = 0; t < DH; ++t) acc[t] = 0.0f;
    for (int e = 0; e < cnt; ++e) qa_step<DH>(q, kb + qa_entry(eg, e) * R, mu, S_, acc);
  }
  const float rS = cnt > 0 ? recip_softmax_sum(S_) : 0.0f;
#pragma unroll
  for (int t = 0; t < DH; ++t) orow[t] = acc[t] * rS;
}

// The word's token tiles stay in registers across its head groups (d = 128: one block per CU,
// 2 wavefronts per SIMD; d = 64 with 8-dimension heads: at most two tiles per wave, and a
// register budget of 4 wavefronts per SIMD, two blocks per CU: at 6 the loop-invariant values
// spill, and every reload from scratch waits for the outputs in flight); d = 64 with
// 16-dimension heads reloads them per group (up to four tiles per wave would not fit the
// registers of 4 wavefronts per SIMD).
template <int D, int DH>
constexpr bool qa_keep_tiles() { return D == 128 || DH == 8; }
template <int D, int DH>
constexpr int qa_waves_per_simd() { return D == 128 ? 2 : 4; }

// Q, K, V of token tile tt (16 tokens) for the head group whose fragments are bf: the A
// fragments a (the tile's Eq. 2 codes) and the four token scales al of this lane's outputs.
template <int D>
__device__ __forceinline__ void qa_project(const uint64_t *bf, const long (&a)[D / 32], const float (&al)[4],
                                           int tt, int L, int lane, float bq, float bk, float bv, const float (&sq)[3],
                                           float *qs, float *kv) {
  constexpr int S = D / 32, R = kQaRow;
  const int col = lane & 15, rg = lane >> 4;
  v4i aq = v4i{0, 0, 0, 0}, ak = v4i{0, 0, 0, 0}, av = v4i{0, 0, 0, 0};
  const auto fa = [&](int s) { return a[s]; };
  aq = mfma_i8_steps<S>(fa, [&](int s) { return (long)bf[(0 * S + s) * 64 + lane]; }, aq);
  ak = mfma_i8_steps<S>(fa, [&](int s) { return (long)bf[(1 * S + s) * 64 + lane]; }, ak);
  av = mfma_i8_steps<S>(fa, [&](int s) { return (long)bf[(2 * S + s) * 64 + lane]; }, av);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tok = 16 * tt + 4 * rg + i;
    if (tok < L) {
      qs[tok * 16 + col] = __builtin_fmaf((float)aq[i], al[i] * sq[0], bq);
      kv[tok * R + col] = __builtin_fmaf((float)ak[i], al[i] * sq[1], bk);
      kv[tok * R + 16 + col] = __builtin_fmaf((float)av[i], al[i] * sq[2], bv);
    }
  }
}

template <int D>
__device__ __forceinline__ void qa_load_tile(const int8_t *xw, const float *aw, int tt, int L, int lane,
                                             long (&a)[D / 32], float (&al)[4]) {
  const int col = lane & 15, rg = lane >> 4, ra = 16 * tt + col;
#pragma unroll
  for (int s = 0; s < D / 32; ++s) a[s] = ra < L ? *(const long *)(xw + (size_t)ra * D + 32 * s + 8 * rg) : 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tok = 16 * tt + 4 * rg + i;
    al[i] = tok < L ? aw[tok] : 0.0f;
  }
}

// LT (every group's weights resident, the word's tiles kept in registers): the neighbour lists and
// their metadata staged in LDS once per block, so the rows issue no global loads, and the next
// word's token tiles read right after the last group's projection, while its rows run.
template <int D, int DH, bool LT = false>
__global__ __launch_bounds__(kQaThreads, (qa_waves_per_simd<D, DH>())) void k_qkv_attention(QkvAttnArgs p) {
  constexpr int NWV = kQaThreads / 64;
  // at most kQaThreads rows of L tokens x 16 / d_h heads: a wave holds up to TW of the L / 16 tiles
  constexpr int S = D / 32, G = D / 16, HPG = 16 / DH, TW = qa_keep_tiles<D, DH>() ? (kQaThreads / HPG / 16 + NWV - 1) / NWV : 1;
  static_assert(TW <= kQaTilesPerWave, "token tiles per wave");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int L = p.L, ntiles = (L + 15) / 16;
  // weight fragments: [G][3][S][64] when resident (staged once per block), else one group's
  // [3][S][64], restaged per group
  constexpr int FW = 3 * S * 64;
  const bool resident = p.resident != 0;
  uint64_t *bfa = (uint64_t *)smem;
  float *qs = (float *)(smem + (resident ? G : 1) * qa_frag_bytes<D>()), *kv = qs + (size_t)L * 16;
  float *bl = kv + (size_t)L * kQaRow;                               // [3][D] Q, K, V biases
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, col = lane & 15;
  if (blockIdx.x >= p.words) return;
  for (int hg = 0; hg < (resident ? G : 1); ++hg) {
    QaStage<D> st;
    st.load(p.bpack, hg, tid);
    st.store(bfa + hg * FW, tid);
  }
  for (int u = tid; u < 3 * D; u += kQaThreads) bl[u] = p.bias[u];
  static_assert(!LT || qa_keep_tiles<D, DH>(), "lists in LDS with the tiles kept in registers");
  // LT: [L] metadata of both masks, then both lists, after the biases
  int2 *ml1 = (int2 *)(bl + 3 * D), *ml2 = ml1 + L;
  uint2 *tl1 = (uint2 *)(ml2 + L), *tl2 = tl1 + p.tab1_n;
  if constexpr (LT) {
    for (int u = tid; u < L; u += kQaThreads) {
      ml1[u] = p.meta1[u];
      ml2[u] = p.meta2[u];
    }
    for (int u = tid; u < p.tab1_n; u += kQaThreads) tl1[u] = p.tab1[u];
    for (int u = tid; u < p.tab2_n; u += kQaThreads) tl2[u] = p.tab2[u];
    __syncthreads();
  }
  const uint2 *tab1 = LT ? tl1 : p.tab1, *tab2 = LT ? tl2 : p.tab2;
  // the thread's row (token i0, head hh0 of the group; L d / (16 d_h) <= kQaThreads rows): its
  // list metadata and first entry group for both masks stay in registers for the whole kernel
  const bool row0 = tid < L * HPG;
  const int hh0 = row0 ? tid / L : 0, i0 = row0 ? tid - hh0 * L : 0;
  const int2 mt1 = LT ? ml1[i0] : p.meta1[i0], mt2 = LT ? ml2[i0] : p.meta2[i0];
  const uint2 g01 = tab1[mt1.x], g02 = tab2[mt2.x];
  __syncthreads();
  const float sq[3] = {p.sq[0], p.sq[1], p.sq[2]};
  long afr[TW][S];
  float alw[TW][4];
  auto load_tiles = [&](int64_t w) {
    int wv = wave;
    __asm__ volatile("" : "+v"(wv));   // per-tile addresses are not hoisted out of the loops
#pragma unroll
    for (int k = 0; k < TW; ++k) qa_load_tile<D>(p.xq + w * L * D, p.ax + w * L, wv + NWV * k, L, lane, afr[k], alw[k]);
  };
  if constexpr (LT) load_tiles(blockIdx.x);
  for (int64_t w = blockIdx.x; w < p.words; w += gridDim.x) {
    const int8_t *xw = p.xq + w * L * D;
    const float *aw = p.ax + w * L;
    if constexpr (qa_keep_tiles<D, DH>()) {
      // the wave's token tiles of the word, used by all its head groups and waited for here: no
      // global load is then outstanding inside the group loop, where a wait would also wait for
      // the row outputs being written (vmcnt counts stores too; LT: read during the previous
      // word's last rows)
      if constexpr (!LT) load_tiles(w);
#pragma unroll
      for (int k = 0; k < TW; ++k) {
#pragma unroll
        for (int s2 = 0; s2 < S; ++s2) __asm__ volatile("" : "+v"(afr[k][s2]));
        __asm__ volatile("" : "+v"(alw[k][0]), "+v"(alw[k][1]), "+v"(alw[k][2]), "+v"(alw[k][3]));
      }
    }
    for (int hg = 0; hg < G; ++hg) {
      const uint64_t *bf = resident ? bfa + hg * FW : bfa;
      const float bq = bl[16 * hg + col], bk = bl[D + 16 * hg + col], bv = bl[2 * D + 16 * hg + col];
      if constexpr (qa_keep_tiles<D, DH>()) {
        int wg = wave;
        __asm__ volatile("" : "+v"(wg));
#pragma unroll
        for (int k = 0; k < TW; ++k) {
          const int tt = wg + NWV * k;
          if (tt < ntiles) qa_project<D>(bf, afr[k], alw[k], tt, L, lane, bq, bk, bv, sq, qs, kv);
        }
      } else {
        for (int tt = wave; tt < ntiles; tt += NWV) {
          qa_load_tile<D>(xw, aw, tt, L, lane, afr[0], alw[0]);
          qa_project<D>(bf, afr[0], alw[0], tt, L, lane, bq, bk, bv, sq, qs, kv);
        }
      }
      block_sync_lds();
      // LT: the projection of the word's last group has read its tiles: the next word's now
      if constexpr (LT)
        if (hg == G - 1 && w + gridDim.x < p.words) load_tiles(w + gridDim.x);
      // not resident: the fragments were last read before the barrier above, so the next group's
      // weights are loaded now and written after the rows
      const bool more = !LT && !resident && (hg + 1 < G || w + gridDim.x < p.words);
      QaStage<D> st;
      if (more) st.load(p.bpack, hg + 1 < G ? hg + 1 : 0, tid);
      if (row0) {
        const int h = hg * HPG + hh0;
        const bool first = h < p.hf;
        const int2 mt = first ? mt1 : mt2;
        qa_row<DH, D == 128>(qs + i0 * 16 + hh0 * DH, kv + hh0 * DH, (first ? tab1 : tab2) + mt.x, first ? g01 : g02,
                   mt.y, p.o + (w * L + i0) * D + h * DH);
      }
      if (more) st.store(bfa, tid);
      block_sync_lds();
    }
  }
}

// ------------------------------------------------------------------------------------------
// The same projection and attention for 16-dimension heads (d = 128) with every attention row
// split over a lane pair: lane 2 r + h of the block takes dimensions 8 h .. 8 h + 7 of row r (its
// query, key, value halves), forms its half of the score, and the pair adds the two halves with
// one DPP exchange (the canonical order: low half + high half, so both lanes hold the same
// bits); both lanes then compute the same weight and sums, each for its own 8 output
// dimensions.  Blocks of 12 wavefronts, so that a word of up to 384 tokens fills every lane
// and three wavefronts per SIMD have rows in flight; every head group's weight tiles resident in
// LDS.
// ------------------------------------------------------------------------------------------
constexpr int kQpThreads = 768;
constexpr int kQpTilesPerWave = 3;


// the partner lane's value (lane ^ 1) within the quad
__device__ __forceinline__ float pair_other(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xf, 0xf, true));
}

// One neighbour of a half row: kr points at the neighbour's key half (8 floats), its value half
// 16 floats further.
__device__ __forceinline__ void qp_step(const float (&q)[8], const float (&k)[8], const float (&v)[8], float shift,
                                        float &S, float (&acc)[8]) {
  const float h = dot_seq<8>(q, k);
  const float ex = softmax_exp2(h + pair_other(h) - shift);
  S = S + ex;
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = __builtin_fmaf(ex, v[t], acc[t]);
}

// Attention of one half row whose query half is q: kb and orow already offset to this lane's
// half; entries as in qa_row, the first group in g0.  Both lanes of a pair run it with the same
// row.
__device__ __forceinline__ void qp_row_q(const float (&q)[8], const float *kb, const uint2 *eg, uint2 g0, int cnt,
                                         float (&out)[8]) {
  constexpr int R = kQaRow;
  float S_ = 0.0f, acc[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = 0.0f;
  // a neighbour's value half and the next neighbour's key half are read before the neighbour's
  // score (every list stores a group after its last full one; unused slots hold token 0)
  uint2 gc = g0;
  float ka[8], kb_[8], v[8];
  qa_load<8>(ka, kb + (gc.x & 0xffffu) * R);
  auto stage = [&](uint32_t cur, uint32_t nxt, float (&kc)[8], float (&kn)[8]) {
    qa_load<8>(v, kb + cur * R + 16);
    qa_load<8>(kn, kb + nxt * R);
    qp_step(q, kc, v, 0.0f, S_, acc);
    __builtin_amdgcn_sched_barrier(0);
  };
  for (int u = 0; u < (cnt >> 2); ++u) {
    const uint2 gn = eg[u + 1];
    stage(gc.x & 0xffffu, gc.x >> 16, ka, kb_);
    stage(gc.x >> 16, gc.y & 0xffffu, kb_, ka);
    stage(gc.y & 0xffffu, gc.y >> 16, ka, kb_);
    stage(gc.y >> 16, gn.x & 0xffffu, kb_, ka);
    gc = gn;
  }
  const int rem = cnt & 3;
  if (rem > 0) stage(gc.x & 0xffffu, gc.x >> 16, ka, kb_);
  if (rem > 1) stage(gc.x >> 16, gc.y & 0xffffu, kb_, ka);
  if (rem > 2) stage(gc.y & 0xffffu, gc.y >> 16, ka, kb_);
  if (cnt > 0 && !(S_ >= 0x1p-64f && S_ <= 0x1p64f)) {     // the same decision in both lanes
    float mu = -INFINITY;
    for (int e = 0; e < cnt; ++e) {
      float k[8];
      qa_load<8>(k, kb + qa_entry(eg, e) * R);
      const float h = dot_seq<8>(q, k);
      mu = fmaxf(mu, h + pair_other(h));
    }
    S_ = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[t] = 0.0f;
    for (int e = 0; e < cnt; ++e) {
      const float *kr = kb + qa_entry(eg, e) * R;
      float k[8], vv[8];
      qa_load<8>(k, kr);
      qa_load<8>(vv, kr + 16);
      qp_step(q, k, vv, mu, S_, acc);
    }
  }
  const float rS = cnt > 0 ? recip_softmax_sum(S_) : 0.0f;
#pragma unroll
  for (int t = 0; t < 8; ++t) out[t] = acc[t] * rS;
}

// The same with the query half read from qrow first and the outputs stored to orow.
__device__ __forceinline__ void qp_row(const float *qrow, const float *kb, const uint2 *eg, uint2 g0, int cnt,
                                       float *orow) {
  float q[8], out[8];
  qa_load<8>(q, qrow);
  qp_row_q(q, kb, eg, g0, cnt, out);
  *(float4 *)orow = make_float4(out[0], out[1], out[2], out[3]);
  *(float4 *)(orow + 4) = make_float4(out[4], out[5], out[6], out[7]);
}

// OQ: a word of at most 384 tokens (one row per lane pair) keeps each row's outputs of all head
// groups in registers (64 per lane) and writes the row's Eq. 2 codes and scale once the last
// group is done, so the token block reads a quarter of the bytes; else fp32 rows per group.
// LT (with OQ): the neighbour lists and their per-token metadata are staged in LDS once per block,
// so the rows issue no global loads, and the next word's token tiles are read into registers
// right after the last group's projection, while its rows run (a wait for any global load would
// also wait for every earlier one).
template <int D, bool OQ, bool LT = false>
__global__ __launch_bounds__(kQpThreads, 1) void k_qkv_attention_pair(QkvAttnArgs p) {
  // token tiles per wave: 384 tokens take two of the 12 waves' tiles
  constexpr int S = D / 32, G = D / 16, TW = OQ ? 2 : kQpTilesPerWave, NWV = kQpThreads / 64, FW = 3 * S * 64;
  static_assert(D == 128, "16-dimension heads, one per head group");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int L = p.L, ntiles = (L + 15) / 16;
  uint64_t *bfa = (uint64_t *)smem;                                  // [G][3][S][64] weight fragments
  float *qs = (float *)(smem + G * qa_frag_bytes<D>()), *kv = qs + (size_t)L * 16;
  float *bl = kv + (size_t)L * kQaRow;                               // [3][D] Q, K, V biases
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, col = lane & 15, half = tid & 1;
  if (blockIdx.x >= p.words) return;
  for (int hg = 0; hg < G; ++hg) {
    QaStage<D, kQpThreads> st;
    st.load(p.bpack, hg, tid);
    st.store(bfa + hg * FW, tid);
  }
  for (int u = tid; u < 3 * D; u += kQpThreads) bl[u] = p.bias[u];
  static_assert(!LT || OQ, "lists in LDS with the quantised output");
  // LT: [L] metadata of both masks, then both lists, after the biases
  int2 *ml1 = (int2 *)(bl + 3 * D), *ml2 = ml1 + L;
  uint2 *tl1 = (uint2 *)(ml2 + L), *tl2 = tl1 + p.tab1_n;
  if constexpr (LT) {
    for (int u = tid; u < L; u += kQpThreads) {
      ml1[u] = p.meta1[u];
      ml2[u] = p.meta2[u];
    }
    for (int u = tid; u < p.tab1_n; u += kQpThreads) tl1[u] = p.tab1[u];
    for (int u = tid; u < p.tab2_n; u += kQpThreads) tl2[u] = p.tab2[u];
  }
  // this pair's first row (token tid / 2): list metadata of both masks held for the kernel, in
  // registers, or with the quantised output (whose row outputs take 64 registers) in LDS
  const int r0 = tid >> 1, i0 = r0 < L ? r0 : 0;
  int2 mt1 = make_int2(0, 0), mt2 = make_int2(0, 0);
  uint2 g01 = make_uint2(0, 0), g02 = make_uint2(0, 0);
  uint4 *mdl = (uint4 *)(bl + 3 * D) + 2 * tid;
  if constexpr (!LT) {
    mt1 = p.meta1[i0];
    mt2 = p.meta2[i0];
    g01 = p.tab1[mt1.x];
    g02 = p.tab2[mt2.x];
    if constexpr (OQ) {
      mdl[0] = make_uint4((uint32_t)mt1.x, (uint32_t)mt1.y, (uint32_t)mt2.x, (uint32_t)mt2.y);
      mdl[1] = make_uint4(g01.x, g01.y, g02.x, g02.y);
    }
  }
  __syncthreads();
  const float sq[3] = {p.sq[0], p.sq[1], p.sq[2]};
  long afr[TW][S];
  float alw[TW][4];
  auto load_tiles = [&](int64_t w) {
    int wv = wave;
    __asm__ volatile("" : "+v"(wv));
#pragma unroll
    for (int k = 0; k < TW; ++k) qa_load_tile<D>(p.xq + w * L * D, p.ax + w * L, wv + NWV * k, L, lane, afr[k], alw[k]);
  };
  if constexpr (LT) load_tiles(blockIdx.x);
  for (int64_t w = blockIdx.x; w < p.words; w += gridDim.x) {
    // the word's token tiles, waited for here: no global load is then outstanding inside the
    // group loop, where a wait would also wait for the row outputs being written (LT: read
    // during the previous word's last rows)
    if constexpr (!LT) load_tiles(w);
#pragma unroll
    for (int k = 0; k < TW; ++k) {
#pragma unroll
      for (int s2 = 0; s2 < S; ++s2) __asm__ volatile("" : "+v"(afr[k][s2]));
      __asm__ volatile("" : "+v"(alw[k][0]), "+v"(alw[k][1]), "+v"(alw[k][2]), "+v"(alw[k][3]));
    }
    // head group hg: its Q, K, V into LDS, then its rows; row r0's outputs to out
    auto group = [&](int hg, float (&out)[8]) {
      const uint64_t *bf = bfa + hg * FW;
      const float bq = bl[16 * hg + col], bk = bl[D + 16 * hg + col], bv = bl[2 * D + 16 * hg + col];
      int wg = wave;
      __asm__ volatile("" : "+v"(wg));
#pragma unroll
      for (int k = 0; k < TW; ++k) {
        if (wg + NWV * k < ntiles) qa_project<D>(bf, afr[k], alw[k], wg + NWV * k, L, lane, bq, bk, bv, sq, qs, kv);
      }
      block_sync_lds();
      const bool first = hg < p.hf;
      if constexpr (LT) {
        // the projection of the word's last group has read its tiles: the next word's now
        if (hg == G - 1 && w + gridDim.x < p.words) load_tiles(w + gridDim.x);
        mt1 = ml1[i0];
        mt2 = ml2[i0];
      } else if constexpr (OQ) {
        uint32_t *mdp = (uint32_t *)mdl;
        __asm__ volatile("" : "+v"(mdp));   // read here, not kept from the kernel's start
        const uint4 m0 = *(const uint4 *)mdp, m1 = *(const uint4 *)(mdp + 4);
        mt1 = make_int2((int)m0.x, (int)m0.y);
        mt2 = make_int2((int)m0.z, (int)m0.w);
        g01 = make_uint2(m1.x, m1.y);
        g02 = make_uint2(m1.z, m1.w);
      }
      if (r0 < L) {
        float q[8];
        qa_load<8>(q, qs + r0 * 16 + 8 * half);
        if constexpr (LT) {
          const uint2 *eg = first ? tl1 + mt1.x : tl2 + mt2.x;
          qp_row_q(q, kv + 8 * half, eg, eg[0], first ? mt1.y : mt2.y, out);
        } else {
          qp_row_q(q, kv + 8 * half, (first ? p.tab1 : p.tab2) + (first ? mt1.x : mt2.x), first ? g01 : g02,
                   first ? mt1.y : mt2.y, out);
        }
      }
      if constexpr (!OQ) {
        float *ow = p.o + w * L * D + hg * 16 + 8 * half;
        if (r0 < L) {
          *(float4 *)(ow + (size_t)r0 * D) = make_float4(out[0], out[1], out[2], out[3]);
          *(float4 *)(ow + (size_t)r0 * D + 4) = make_float4(out[4], out[5], out[6], out[7]);
        }
        for (int r = r0 + kQpThreads / 2; r < L; r += kQpThreads / 2) {   // words of more than 384 tokens
          const int2 mt = (first ? p.meta1 : p.meta2)[r];
          const uint2 *eg = (first ? p.tab1 : p.tab2) + mt.x;
          qp_row(qs + r * 16 + 8 * half, kv + 8 * half, eg, eg[0], mt.y, ow + (size_t)r * D);
        }
      }
      block_sync_lds();
    };
    if constexpr (OQ) {
      float ko[G][8];
#pragma unroll
      for (int hg = 0; hg < G; ++hg) group(hg, ko[hg]);
      if (r0 < L) {
        // Eq. 2 of the row: alpha = max |O| over the pair's 2 x 64 features (the same value in
        // both lanes), the codes of this lane's features 16 hg + 8 half + t
        float om = 0.0f;
#pragma unroll
        for (int hg = 0; hg < G; ++hg)
#pragma unroll
          for (int t = 0; t < 8; ++t) om = fmaxf(om, fabsf(ko[hg][t]));
        om = fmaxf(om, pair_other(om));
        const float inv = inv127(om);
        int8_t *orow = p.oq + (w * L + r0) * D + 8 * half;
#pragma unroll
        for (int hg = 0; hg < G; ++hg) {
          uint32_t b[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) b[t] = quant_bits(ko[hg][t], inv);
          *(long *)(orow + 16 * hg) = tb_pack8(b);
        }
        if (half == 0) p.ao[w * L + r0] = om;
      }
    } else {
      for (int hg = 0; hg < G; ++hg) {
        float out[8];
        group(hg, out);
      }
    }
  }
}

// ------------------------------------------------------------------------------------------
// The same projection and attention for words whose keys and values of a head group do not fit
// LDS in fp32 (d = 64, 128 with up to about 1800 tokens).  Keys and values stay in LDS as their
// exact int32 accumulators, which fit int16 (|acc| <= 127 d < 2^15), with each token's two
// dequantisation scales (alpha * s_k / 127, alpha * s_v / 127); every gather rebuilds the fp32
// key and value with the same fma(acc, scale, bias) the projection would have applied, so the
// results are those of k_attention bit for bit.  Queries go through the output rows in memory:
// the projection writes the group's queries where the group's attention outputs will go, and
// each row's thread reads its query there before overwriting it with the output.
// ------------------------------------------------------------------------------------------
constexpr int kQwRow = 40;   // int16 per token: key (16), value (16), pad; 80 bytes apart

template <int D>
size_t qkv_attention_i16_lds_bytes(int L) {
  return qa_frag_bytes<D>() + (size_t)L * (kQwRow * 2 + 8);
}

// One neighbour: kw points at the neighbour's key accumulators (d_h int16, 16-byte aligned), its
// value accumulators 16 int16 further; c = its (key, value) scales; bk, bv the head's biases.
template <int DH>
__device__ __forceinline__ void qw_step(const float (&q)[DH], const int16_t *kw, float2 c, const float (&bk)[DH],
                                        const float (&bv)[DH], float shift, float &S, float (&acc)[DH]) {
  float k[DH], v[DH];
#pragma unroll
  for (int t = 0; t < DH; t += 8) {
    const uint4 a = *(const uint4 *)(kw + t), b = *(const uint4 *)(kw + 16 + t);
    const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, bw[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      k[t + 2 * u] = __builtin_fmaf((float)(int)(short)(aw[u] & 0xffffu), c.x, bk[t + 2 * u]);
      k[t + 2 * u + 1] = __builtin_fmaf((float)((int)aw[u] >> 16), c.x, bk[t + 2 * u + 1]);
      v[t + 2 * u] = __builtin_fmaf((float)(int)(short)(bw[u] & 0xffffu), c.y, bv[t + 2 * u]);
      v[t + 2 * u + 1] = __builtin_fmaf((float)((int)bw[u] >> 16), c.y, bv[t + 2 * u + 1]);
    }
  }
  const float ex = softmax_exp2(head_dot<DH>(q, k) - shift);
  S = S + ex;
#pragma unroll
  for (int t = 0; t < DH; ++t) acc[t] = __builtin_fmaf(ex, v[t], acc[t]);
}

template <int D, int DH>
__global__ __launch_bounds__(kQaThreads) void k_qkv_attention_i16(QkvAttnArgs p) {
  constexpr int S = D / 32, G = D / 16, HPG = 16 / DH, R = kQwRow, NWV = kQaThreads / 64;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int L = p.L, ntiles = (L + 15) / 16;
  uint64_t *bf = (uint64_t *)smem;                                   // [3][S][64] weight fragments
  int16_t *kvw = (int16_t *)(smem + qa_frag_bytes<D>());             // [L][R] key, value accumulators
  float2 *cs = (float2 *)(kvw + (size_t)L * R);                      // [L] key, value scales
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, col = lane & 15, rg = lane >> 4;
  if (blockIdx.x >= p.words) return;
  {
    QaStage<D> st;
    st.load(p.bpack, 0, tid);
    st.store(bf, tid);
  }
  __syncthreads();
  for (int64_t w = blockIdx.x; w < p.words; w += gridDim.x) {
    const int8_t *xw = p.xq + w * L * D;
    const float *aw = p.ax + w * L;
    float *ow = p.o + w * L * D;
    for (int hg = 0; hg < G; ++hg) {
      const float bq = p.bias[16 * hg + col];
      // the wave's next tile is read while the current one is projected
      long a[S], an[S];
      float al[4], aln[4];
      if (wave < ntiles) qa_load_tile<D>(xw, aw, wave, L, lane, a, al);
      for (int tt = wave; tt < ntiles; tt += NWV) {
        if (tt + NWV < ntiles) qa_load_tile<D>(xw, aw, tt + NWV, L, lane, an, aln);
        v4i aq = v4i{0, 0, 0, 0}, ak = v4i{0, 0, 0, 0}, av = v4i{0, 0, 0, 0};
        const auto fa = [&](int s) { return a[s]; };
        aq = mfma_i8_steps<S>(fa, [&](int s) { return (long)bf[(0 * S + s) * 64 + lane]; }, aq);
        ak = mfma_i8_steps<S>(fa, [&](int s) { return (long)bf[(1 * S + s) * 64 + lane]; }, ak);
        av = mfma_i8_steps<S>(fa, [&](int s) { return (long)bf[(2 * S + s) * 64 + lane]; }, av);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tok = 16 * tt + 4 * rg + i;
          if (tok < L) {
            ow[(size_t)tok * D + 16 * hg + col] = __builtin_fmaf((float)aq[i], al[i] * p.sq[0], bq);
            kvw[tok * R + col] = (int16_t)ak[i];
            kvw[tok * R + 16 + col] = (int16_t)av[i];
            if (hg == 0 && col == 0) cs[tok] = make_float2(al[i] * p.sq[1], al[i] * p.sq[2]);
          }
        }
#pragma unroll
        for (int u = 0; u < S; ++u) a[u] = an[u];
#pragma unroll
        for (int u = 0; u < 4; ++u) al[u] = aln[u];
      }
      __syncthreads();   // also orders the queries written to memory before their rows read them
      const bool more = hg + 1 < G || w + gridDim.x < p.words;
      QaStage<D> st;
      if (more) st.load(p.bpack, hg + 1 < G ? hg + 1 : 0, tid);
      for (int r = tid; r < L * HPG; r += kQaThreads) {
        const int hh = r / L, i = r - hh * L, h = hg * HPG + hh;
        const bool first = h < p.hf;
        const int2 mt = (first ? p.meta1 : p.meta2)[i];
        const uint2 *eg = (first ? p.tab1 : p.tab2) + mt.x;
        const int cnt = mt.y;
        float *orow = ow + (size_t)i * D + h * DH;
        float q[DH], bk[DH], bv[DH];
#pragma unroll
        for (int t = 0; t < DH; t += 4) {
          const float4 a = *(const float4 *)(orow + t);
          const float4 b = *(const float4 *)(p.bias + D + h * DH + t);
          const float4 c = *(const float4 *)(p.bias + 2 * D + h * DH + t);
          q[t] = a.x; q[t + 1] = a.y; q[t + 2] = a.z; q[t + 3] = a.w;
          bk[t] = b.x; bk[t + 1] = b.y; bk[t + 2] = b.z; bk[t + 3] = b.w;
          bv[t] = c.x; bv[t + 1] = c.y; bv[t + 2] = c.z; bv[t + 3] = c.w;
        }
        const int16_t *kb = kvw + hh * DH;
        float S_ = 0.0f, acc[DH];
#pragma unroll
        for (int t = 0; t < DH; ++t) acc[t] = 0.0f;
        uint2 nx = eg[0];
        for (int u = 0; u < (cnt >> 2); ++u) {
          const uint32_t e0 = nx.x & 0xffffu, e1 = nx.x >> 16, e2 = nx.y & 0xffffu, e3 = nx.y >> 16;
          nx = eg[u + 1];             // stored: every list has a group after its last full one
          qw_step<DH>(q, kb + e0 * R, cs[e0], bk, bv, 0.0f, S_, acc);
          qw_step<DH>(q, kb + e1 * R, cs[e1], bk, bv, 0.0f, S_, acc);
          qw_step<DH>(q, kb + e2 * R, cs[e2], bk, bv, 0.0f, S_, acc);
          qw_step<DH>(q, kb + e3 * R, cs[e3], bk, bv, 0.0f, S_, acc);
        }
        const int rem = cnt & 3;
        if (rem > 0) { const uint32_t e = nx.x & 0xffffu; qw_step<DH>(q, kb + e * R, cs[e], bk, bv, 0.0f, S_, acc); }
        if (rem > 1) { const uint32_t e = nx.x >> 16; qw_step<DH>(q, kb + e * R, cs[e], bk, bv, 0.0f, S_, acc); }
        if (rem > 2) { const uint32_t e = nx.y & 0xffffu; qw_step<DH>(q, kb + e * R, cs[e], bk, bv, 0.0f, S_, acc); }
        if (cnt > 0 && !(S_ >= 0x1p-64f && S_ <= 0x1p64f)) {
          float mu = -INFINITY;
          for (int e = 0; e < cnt; ++e) {
            const uint32_t j = qa_entry(eg, e);
            const float cx = cs[j].x;
            float k[DH];
#pragma unroll
            for (int t = 0; t < DH; ++t) k[t] = __builtin_fmaf((float)kb[j * R + t], cx, bk[t]);
            mu = fmaxf(mu, head_dot<DH>(q, k));
          }
          S_ = 0.0f;
#pragma unroll
          for (int t = 0; t < DH; ++t) acc[t] = 0.0f;
          for (int e = 0; e < cnt; ++e) {
            const uint32_t j = qa_entry(eg, e);
            qw_step<DH>(q, kb + j * R, cs[j], bk, bv, mu, S_, acc);
          }
        }
        const float rS = cnt > 0 ? recip_softmax_sum(S_) : 0.0f;
#pragma unroll
        for (int t = 0; t < DH; t += 4)
          *(float4 *)(orow + t) = make_float4(acc[t] * rS, acc[t + 1] * rS, acc[t + 2] * rS, acc[t + 3] * rS);
      }
      if (more) st.store(bf, tid);
      block_sync_lds();            // the next group's projection overwrites keys and values
    }
  }
}

// ------------------------------------------------------------------------------------------
// Long words with 16-dimension heads (d = 128, up to 1536 tokens): keys in LDS as fp32
// (dequantised once, in the projection), values as their int16 accumulators, rebuilt by
// fma(acc, alpha s_v, bias) at every gather as in k_qkv_attention_i16.  Blocks of 12 wavefronts
// (three per SIMD with rows in flight).  Each wavefront keeps the int8 codes of its token tiles in
// registers for all head groups of a word, read at the word's start with the tokens' Eq. 2 scales
// alpha, which sit in LDS beside the keys and values.  The queries never leave registers: a
// wavefront owns pairs of adjacent token tiles and runs their rows itself, forming a pair's
// queries just before its rows with the transposed product (weights as the MFMA A operand, codes
// as B), whose result holds one token and four query dimensions per lane; one lane swap per
// dimension then leaves lane (t, r) (t = lane mod 16, r = lane / 16) with query dimensions
// 8 (r / 2) .. 8 (r / 2) + 7 of token t of the pair's tile r mod 2, the half row that lane runs;
// the two halves of a row sit in lanes l and l ^ 32 and add their score halves with a lane swap
// (the canonical order: low half + high half, commuted bit for bit).
// ------------------------------------------------------------------------------------------
constexpr int kQvThreads = 768;
constexpr int kQvTilesPerWave = 8;
constexpr int kQvRow = 24;   // floats per token: key (16 fp32), value (16 int16); 96 bytes apart

template <int D>
size_t qkv_attention_v16_lds_bytes(int L) {
  return qa_frag_bytes<D>() + (size_t)L * (kQvRow * 4 + 4);
}

// 8 int16 accumulators (raw pairs) to fp32 with the dequantisation fma(acc, c, bias).
__device__ __forceinline__ void qv_dequant(uint4 a, float c, const float (&b)[8], float (&x)[8]) {
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    x[2 * u] = __builtin_fmaf((float)(int)(short)(w[u] & 0xffffu), c, b[2 * u]);
    x[2 * u + 1] = __builtin_fmaf((float)((int)w[u] >> 16), c, b[2 * u + 1]);
  }
}

// A token's key in LDS as four 16-byte chunks holding dimensions 0-3, 8-11, 4-7, 12-15: the two
// lanes of a row then read chunks h and h + 2 (dimensions 8 h .. 8 h + 7), so that with the 96-byte
// token rows (6 bank groups of 16 bytes apart) the two halves' reads fall on bank groups of both
// parities, where chunks 2 h, 2 h + 1 put every first read on an even group.
__device__ __forceinline__ int qv_key_slot(int dim) { return (dim & 3) | ((dim & 4) << 1) | ((dim & 8) >> 1); }
// this lane's key half of a token: kh points at the token's chunk h
__device__ __forceinline__ void qv_load_key(float (&k)[8], const float *kh) {
  const float4 a = *(const float4 *)kh, b = *(const float4 *)(kh + 8);
  k[0] = a.x; k[1] = a.y; k[2] = a.z; k[3] = a.w; k[4] = b.x; k[5] = b.y; k[6] = b.z; k[7] = b.w;
}

// One neighbour of a half row: k this lane's key half, va its value accumulators, c their scale;
// the row's other half runs in lane l ^ 32.
__device__ __forceinline__ void qv_step(const float (&q)[8], const float (&k)[8], uint4 va, float c,
                                        const float (&bv)[8], float shift, float &S, float (&acc)[8]) {
  float v[8];
  qv_dequant(va, c, bv, v);
  const float h = dot_seq<8>(q, k);
  const float ex = softmax_exp2(lane_xor_add<32>(h) - shift);
  S = S + ex;
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = __builtin_fmaf(ex, v[t], acc[t]);
}

// Attention of one half row with query half q: kb (keys, at this lane's chunk h) and vb (value
// accumulators, at this lane's half) already offset, orow to its 8 outputs; a value's scale is
// alpha sv, alpha from al.
// Both lanes of a row run it with the same lists.
__device__ __forceinline__ void qv_row(const float (&q)[8], float *orow, const float *kb, const int16_t *vb,
                                       const float *al, float sv, const float (&bv)[8], const uint2 *eg, int cnt) {
  constexpr int R = kQvRow, RV = 2 * kQvRow;
  float S_ = 0.0f, acc[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = 0.0f;
  // a neighbour's value half and alpha and the next neighbour's key half are read before the
  // neighbour's score (every list stores a group after its last full one; unused slots hold
  // token 0)
  uint2 gc = eg[0];
  float ka[8], kn[8];
  qv_load_key(ka, kb + (gc.x & 0xffffu) * R);
  auto stage = [&](uint32_t cur, uint32_t nxt, float (&kc)[8], float (&kx)[8]) {
    const uint4 va = *(const uint4 *)(vb + cur * RV);
    const float c = al[cur] * sv;
    qv_load_key(kx, kb + nxt * R);
    qv_step(q, kc, va, c, bv, 0.0f, S_, acc);
    __builtin_amdgcn_sched_barrier(0);
  };
  for (int u = 0; u < (cnt >> 2); ++u) {
    const uint2 gn = eg[u + 1];
    stage(gc.x & 0xffffu, gc.x >> 16, ka, kn);
    stage(gc.x >> 16, gc.y & 0xffffu, kn, ka);
    stage(gc.y & 0xffffu, gc.y >> 16, ka, kn);
    stage(gc.y >> 16, gn.x & 0xffffu, kn, ka);
    gc = gn;
  }
  const int rem = cnt & 3;
  if (rem > 0) stage(gc.x & 0xffffu, gc.x >> 16, ka, kn);
  if (rem > 1) stage(gc.x >> 16, gc.y & 0xffffu, kn, ka);
  if (rem > 2) stage(gc.y & 0xffffu, gc.y >> 16, ka, kn);
  if (cnt > 0 && !(S_ >= 0x1p-64f && S_ <= 0x1p64f)) {     // the same decision in both lanes
    float mu = -INFINITY;
    for (int e = 0; e < cnt; ++e) {
      float k[8];
      qv_load_key(k, kb + qa_entry(eg, e) * R);
      mu = fmaxf(mu, lane_xor_add<32>(dot_seq<8>(q, k)));
    }
    S_ = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[t] = 0.0f;
    for (int e = 0; e < cnt; ++e) {
      const uint32_t j = qa_entry(eg, e);
      float k[8];
      qv_load_key(k, kb + j * R);
      qv_step(q, k, *(const uint4 *)(vb + j * RV), al[j] * sv, bv, mu, S_, acc);
    }
  }
  const float rS = cnt > 0 ? recip_softmax_sum(S_) : 0.0f;
  *(float4 *)orow = make_float4(acc[0] * rS, acc[1] * rS, acc[2] * rS, acc[3] * rS);
  *(float4 *)(orow + 4) = make_float4(acc[4] * rS, acc[5] * rS, acc[6] * rS, acc[7] * rS);
}

// The int8 codes of token tile tt of a word as the MFMA A operand (zero rows past L).
template <int D>
__device__ __forceinline__ void qa_load_codes(const int8_t *xw, int tt, int L, int lane, long (&a)[D / 32]) {
  const int ra = 16 * tt + (lane & 15);
#pragma unroll
  for (int s = 0; s < D / 32; ++s) a[s] = ra < L ? *(const long *)(xw + (size_t)ra * D + 32 * s + 8 * (lane >> 4)) : 0;
}

template <int D>
__global__ __launch_bounds__(kQvThreads) void k_qkv_attention_v16(QkvAttnArgs p) {
  constexpr int S = D / 32, G = D / 16, R = kQvRow, NT = kQvThreads, NWV = NT / 64, TW = kQvTilesPerWave;
  static_assert(TW % 2 == 0, "tiles in pairs");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int L = p.L, ntiles = (L + 15) / 16;
  uint64_t *bf = (uint64_t *)smem;                                   // [3][S][64] weight fragments
  float *kvf = (float *)(smem + qa_frag_bytes<D>());                 // [L][R] keys, value accumulators
  int16_t *kvi = (int16_t *)kvf;
  float *als = kvf + (size_t)L * R;                                  // [L] the word's alpha per token
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, col = lane & 15, rg = lane >> 4;
  // the half row this lane runs in a tile pair: tile rg & 1 of the pair, dimensions 8 hq ..
  const int hq = rg >> 1;
  if (blockIdx.x >= p.words) return;
  {
    QaStage<D, NT> st;
    st.load(p.bpack, 0, tid);
    st.store(bf, tid);
  }
  const float sq[3] = {p.sq[0], p.sq[1], p.sq[2]};
  long afr[TW][S];
  // Global loads are waited for only at the word's first barrier and after each projection:
  // vmcnt counts stores too, so any other wait would also wait for the outputs still being written.
  for (int64_t w = blockIdx.x; w < p.words; w += gridDim.x) {
    float *ow = p.o + w * L * D;
    // the word's token tiles (registers, for all head groups) and alphas (LDS); the previous word's
    // rows are done with both.  Tile k of a wavefront: 2 wave + (k mod 2) + 2 NWV (k / 2), so that
    // k = 2 j, 2 j + 1 are the adjacent tiles of the wavefront's j-th pair.
    // An opaque copy of the wave index per word and per group: the per-tile addresses derived
    // from it are not hoisted out of the loops (held for all tiles, they would not fit the
    // registers).
    int wv = wave;
    __asm__ volatile("" : "+v"(wv));
#pragma unroll
    for (int k = 0; k < TW; ++k)
      qa_load_codes<D>(p.xq + w * L * D, 2 * wv + (k & 1) + 2 * NWV * (k >> 1), L, lane, afr[k]);
    for (int t = tid; t < L; t += NT) als[t] = p.ax[w * L + t];
    __syncthreads();
    for (int hg = 0; hg < G; ++hg) {
      // the next group's weight tiles: read now; the key and value maps' written to LDS once
      // this projection is done, the query map's once this group's rows are
      const bool more = hg + 1 < G || w + gridDim.x < p.words;
      QaStage<D, NT> st;
      if (more) st.load(p.bpack, hg + 1 < G ? hg + 1 : 0, tid);
      float bkc = p.bias[D + 16 * hg + col];
      int wg = wave;
      __asm__ volatile("" : "+v"(wg), "+v"(bkc));
#pragma unroll
      for (int k = 0; k < TW; ++k) {
        const int tt = 2 * wg + (k & 1) + 2 * NWV * (k >> 1);
        if (tt >= ntiles) continue;
        float alv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tok = 16 * tt + 4 * rg + i;
          alv[i] = tok < L ? als[tok] : 0.0f;
        }
        v4i ak = v4i{0, 0, 0, 0}, av = v4i{0, 0, 0, 0};
        const auto fa = [&](int s) { return afr[k][s]; };
        ak = mfma_i8_steps<S>(fa, [&](int s) { return (long)bf[(1 * S + s) * 64 + lane]; }, ak);
        av = mfma_i8_steps<S>(fa, [&](int s) { return (long)bf[(2 * S + s) * 64 + lane]; }, av);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tok = 16 * tt + 4 * rg + i;
          if (tok < L) {
            kvf[tok * R + qv_key_slot(col)] = __builtin_fmaf((float)ak[i], alv[i] * sq[1], bkc);
            kvi[tok * 2 * R + 32 + col] = (int16_t)av[i];
          }
        }
      }
      __syncthreads();
      if (more) st.template store_part<false>(bf, tid);   // no wave reads this group's K, V fragments any more
      const bool first = hg < p.hf;
      float bv[8], bq[4];
      qa_load<8>(bv, p.bias + 2 * D + 16 * hg + 8 * hq);
#pragma unroll
      for (int i = 0; i < 4; ++i) bq[i] = p.bias[16 * hg + 4 * rg + i];
#pragma unroll
      for (int j = 0; j < TW / 2; ++j) {
        const int ta = 2 * wg + 2 * NWV * j;   // the pair's first tile
        if (ta >= ntiles) break;
        // the pair's queries, transposed: lane (t, r) gets query dimensions 4 r + i of token t
        // of each tile, dequantised as the projection defines them
        v4i qa = v4i{0, 0, 0, 0}, qb = v4i{0, 0, 0, 0};
        const auto fw = [&](int s) { return (long)bf[(0 * S + s) * 64 + lane]; };
        qa = mfma_i8_steps<S>(fw, [&](int s) { return afr[2 * j][s]; }, qa);
        qb = mfma_i8_steps<S>(fw, [&](int s) { return afr[2 * j + 1][s]; }, qb);
        const int ra = 16 * ta + col, rb = ra + 16;
        const float sa = (ra < L ? als[ra] : 0.0f) * sq[0], sb = (rb < L ? als[rb] : 0.0f) * sq[0];
        float q[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float va = __builtin_fmaf((float)qa[i], sa, bq[i]), vb = __builtin_fmaf((float)qb[i], sb, bq[i]);
          // rows 0, 1 | 2, 3 of the lanes: (a of row 2 u, b of row 2 u) | (a of row 2 u + 1, b of
          // row 2 u + 1) -> lane row 2 u + c: tile c's dimensions 8 u + i and 8 u + 4 + i
          const auto sw = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, va),
                                                           __builtin_bit_cast(uint32_t, vb), false, false);
          const uint32_t lo = sw[0], hi = sw[1];   // as integers first (see lane_swap_pair)
          q[i] = __builtin_bit_cast(float, lo);
          q[4 + i] = __builtin_bit_cast(float, hi);
        }
        const int r = 16 * (ta + (rg & 1)) + col;
        if (r < L) {
          const int2 mt = (first ? p.meta1 : p.meta2)[r];
          qv_row(q, ow + (size_t)r * D + 16 * hg + 8 * hq, kvf + 4 * hq, kvi + 32 + 8 * hq, als, sq[2], bv,
                 (first ? p.tab1 : p.tab2) + mt.x, mt.y);
        }
      }
      block_sync_lds();            // the next group's projection overwrites keys and values
      if (more) st.template store_part<true>(bf, tid);   // read only by the next group's rows
    }
  }
}

// ------------------------------------------------------------------------------------------
// Long words with 16-dimension heads (d = 128, head partitioning), rows one node type at a time
// (Section 4.2, Fig. 2): a first-ring head's variable rows read only check keys and its check
// rows only variable keys; a second-ring head's rows read keys of their own type.  Each head
// group therefore runs in two phases, variable rows then check rows; a phase projects the keys
// and values of the one node type its rows read into LDS as fp32 (144-byte rows, as in
// k_qkv_attention_pair) and the queries of its rows into the output rows in device memory.  Each
// token's query, key and value is projected in exactly one phase of a group, so the MFMA work is
// that of one projection; the larger node type (n = 1024 variables of the 1536 tokens of
// LDPC(1024,512)) bounds the LDS.  Rows split over lane pairs (qp_row); blocks of 12 wavefronts,
// each keeping its 8 token tiles' int8 codes in registers for all head groups of a word.
// ------------------------------------------------------------------------------------------
constexpr int kQsThreads = 768;
constexpr int kQsTilesPerWave = 8;

template <int D>
size_t qkv_attention_split_lds_bytes(int kv_cap, int L) {
  return qa_frag_bytes<D>() + (size_t)kv_cap * kQaRow * 4 + (size_t)L * 4;
}

template <int D>
__global__ __launch_bounds__(kQsThreads) void k_qkv_attention_split(QkvAttnArgs p) {
  constexpr int S = D / 32, G = D / 16, R = kQaRow, NT = kQsThreads, NWV = NT / 64, TW = kQsTilesPerWave;
  static_assert(D == 128, "16-dimension heads, one per head group");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int L = p.L, n = p.n_var, ntiles = (L + 15) / 16;
  uint64_t *bf = (uint64_t *)smem;                                   // [3][S][64] weight fragments
  float *kv = (float *)(smem + qa_frag_bytes<D>());                  // [kv_cap][R] keys | values
  float *als = kv + (size_t)p.kv_cap * R;                            // [L] the word's alpha per token
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, col = lane & 15, rg = lane >> 4, half = tid & 1;
  if (blockIdx.x >= p.words) return;
  {
    QaStage<D, NT> st;
    st.load(p.bpack, 0, tid);
    st.store(bf, tid);
  }
  const float sq[3] = {p.sq[0], p.sq[1], p.sq[2]};
  long afr[TW][S];
  for (int64_t w = blockIdx.x; w < p.words; w += gridDim.x) {
    float *ow = p.o + w * L * D;
    // an opaque copy of the wave index per word and per phase keeps the per-tile addresses from
    // being hoisted out of the loops (held for all tiles, they would not fit the registers)
    int wv = wave;
    __asm__ volatile("" : "+v"(wv));
#pragma unroll
    for (int k = 0; k < TW; ++k) qa_load_codes<D>(p.xq + w * L * D, wv + NWV * k, L, lane, afr[k]);
    for (int t = tid; t < L; t += NT) als[t] = p.ax[w * L + t];
    __syncthreads();
    for (int hg = 0; hg < G; ++hg) {
      const bool first = hg < p.hf;
      for (int ph = 0; ph < 2; ++ph) {
        const int rlo = ph ? n : 0, rhi = ph ? L : n;                // this phase's rows
        const bool kvar = first == (ph == 1);                        // its keys are variables
        const int klo = kvar ? 0 : n, khi = kvar ? n : L;
        // the next group's weight tiles: read in the group's last phase, written to LDS once its
        // projection is done
        const bool more = ph == 1 && (hg + 1 < G || w + gridDim.x < p.words);
        QaStage<D, NT> st;
        if (more) st.load(p.bpack, hg + 1 < G ? hg + 1 : 0, tid);
        float bq = p.bias[16 * hg + col], bkc = p.bias[D + 16 * hg + col], bvc = p.bias[2 * D + 16 * hg + col];
        int wg = wave;
        // waited for here, before the first query store (not behind it)
        __asm__ volatile("" : "+v"(wg), "+v"(bq), "+v"(bkc), "+v"(bvc));
#pragma unroll
        for (int k = 0; k < TW; ++k) {
          const int tt = wg + NWV * k;
          if (tt >= ntiles) continue;
          const int t0 = 16 * tt, t1 = t0 + 16;
          const bool needq = t0 < rhi && t1 > rlo, needkv = t0 < khi && t1 > klo;   // uniform per wave
          if (!needq && !needkv) continue;
          float alv[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int tok = t0 + 4 * rg + i;
            alv[i] = tok < L ? als[tok] : 0.0f;
          }
          const auto fa = [&](int s) { return afr[k][s]; };
          if (needq) {
            v4i aq = v4i{0, 0, 0, 0};
            aq = mfma_i8_steps<S>(fa, [&](int s) { return (long)bf[(0 * S + s) * 64 + lane]; }, aq);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int tok = t0 + 4 * rg + i;
              if (tok >= rlo && tok < rhi) ow[(size_t)tok * D + 16 * hg + col] = __builtin_fmaf((float)aq[i], alv[i] * sq[0], bq);
            }
          }
          if (needkv) {
            v4i ak = v4i{0, 0, 0, 0}, av = v4i{0, 0, 0, 0};
            ak = mfma_i8_steps<S>(fa, [&](int s) { return (long)bf[(1 * S + s) * 64 + lane]; }, ak);
            av = mfma_i8_steps<S>(fa, [&](int s) { return (long)bf[(2 * S + s) * 64 + lane]; }, av);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int tok = t0 + 4 * rg + i;
              if (tok >= klo && tok < khi) {
                kv[(tok - klo) * R + col] = __builtin_fmaf((float)ak[i], alv[i] * sq[1], bkc);
                kv[(tok - klo) * R + 16 + col] = __builtin_fmaf((float)av[i], alv[i] * sq[2], bvc);
              }
            }
          }
        }
        __syncthreads();   // also orders the queries written to memory before their rows read them
        if (more) st.store(bf, tid);   // no wave reads this group's fragments any more
        const int2 *meta = first ? p.meta1 : p.meta2;
        const uint2 *tab = first ? p.tab1s : p.tab2s;
        for (int r = rlo + (tid >> 1); r < rhi; r += NT / 2) {
          const int2 mt = meta[r];
          const uint2 *eg = tab + mt.x;
          float *orow = ow + (size_t)r * D + 16 * hg + 8 * half;
          qp_row(orow, kv + 8 * half, eg, eg[0], mt.y, orow);
        }
        block_sync_lds();            // the next phase's projection overwrites keys and values
      }
    }
  }
}

// Eq. 2 per row of an fp32 [rows][D] matrix: 16 lanes per row, lane c holding the D / 16
// consecutive features from c D / 16; alpha = max |x| (order-free), codes as everywhere.
template <int D>
__global__ __launch_bounds__(256) void k_quant_rows(const float *x, int64_t rows, int8_t *q, float *a) {
  constexpr int V = D / 16;
  const int64_t r = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
  const int c = threadIdx.x & 15;
  float v[V];
  if (r < rows) {
#pragma unroll
    for (int u = 0; u < V; u += 4) {
      const float4 f = *(const float4 *)(x + r * D + c * V + u);
      v[u] = f.x; v[u + 1] = f.y; v[u + 2] = f.z; v[u + 3] = f.w;
    }
  } else {
#pragma unroll
    for (int u = 0; u < V; ++u) v[u] = 0.0f;
  }
  float amax = 0.0f;
#pragma unroll
  for (int u = 0; u < V; ++u) amax = fmaxf(amax, fabsf(v[u]));
  amax = row16_max(amax);
  if (r >= rows) return;
  const float inv = inv127(amax);
  uint32_t pk[V / 4];
#pragma unroll
  for (int u = 0; u < V / 4; ++u)
    pk[u] = (uint32_t)(uint8_t)quant_code(v[4 * u], inv) | (uint32_t)(uint8_t)quant_code(v[4 * u + 1], inv) << 8 |
            (uint32_t)(uint8_t)quant_code(v[4 * u + 2], inv) << 16 |
            (uint32_t)(uint8_t)quant_code(v[4 * u + 3], inv) << 24;
  if constexpr (V == 8) {
    *(uint2 *)(q + r * D + c * V) = make_uint2(pk[0], pk[1]);
  } else {
    *(uint32_t *)(q + r * D + c * V) = pk[0];
  }
  if (c == 0) a[r] = amax;
}

// ------------------------------------------------------------------------------------------
// The token-local half of a layer in one kernel (d = 64, 128): output projection, residual,
// LN1 (Eq. 3, Section 6), Eq. 2, FFN1 with ReLU, Eq. 2, FFN2, residual, LN2 and Eq. 2 of the
// next layer's input.  One wavefront per 16-token strip.  The products run transposed on
// int8 MFMA (weights are the A operand, from LDS; the strip's 16 tokens are the
// columns), so lane (c, g) = (lane & 15, lane >> 4) holds, for token c, the d-wide activations
// as register v = feature 4 v + g.  The host permutes the fragments' rows and k-slots so that
// (a) the O and FF2 outputs land in that layout, (b) the 8 codes a lane quantises for k-step s
// are exactly its B-operand bytes for FF1, and (c) two FF1 output tiles give exactly the
// B-operand bytes of one FF2 k-step: no activation leaves registers between the maps.  The
// hidden row (4 d values per token) is computed once and held in registers while its ReLU maximum
// (the Eq. 2 scale of the hidden row) is formed, then quantised, each pair of tiles feeding FF2 at
// once (with kTbKeepHidden off, FF1 runs a second time instead).  LayerNorm sums are the
// pairwise order (in-lane over v, then lanes xor 32, xor 16); epilogues and evaluation order
// are those of k_gemm's EPI_LN / EPI_RELU_QUANT.  X and the next layer's codes are kept in that
// lane order in memory too, so every lane reads and writes contiguous words.  No block barrier
// after the weight staging.
// ------------------------------------------------------------------------------------------
struct TokenBlockArgs {
  const float *o;               // [rows][d] attention output (fp32), or
  const int8_t *oq;             // [rows][d] its Eq. 2 codes and
  const float *ao;              // [rows] their scales
  float *x;                     // [rows][d] layer input (residual); overwritten with the output
  const uint64_t *fo, *f1, *f2; // permuted A fragments of O, FF1, FF2
  const float *vec;             // [6][4][d/4] b_o, ln1_g, ln1_b, b_ff2, ln2_g, ln2_b in lane order
  const float *b1;              // [4d] FF1 bias
  float sq_o, sq_1, sq_2, eps;
  int64_t rows;
  int8_t *xq;                   // [rows][d] Eq. 2 codes of the output
  float *ax;                    // [rows]
  // the last layer: z_i = W_{d->1} x_i + b1 of the output rows to z [rows] instead of x, xq, ax
  float *z;
  const float *w1;              // [4][d/4] W_{d->1} in lane order (with z)
  float head_b1;
  // the first layer: x is not read; X = fma(t_i, E_i, P_i) from each token's t [rows] and the
  // embedding (and positional) rows in lane order [L][4][d/4] (pos may be null)
  const float *t, *elo, *plo;
  int L;
};

constexpr int kTbWaves = 8;
// Whether pass 1 keeps the hidden row's fp32 values in registers for pass 2 (instead of pass 2
// recomputing them).
constexpr bool kTbKeepHidden = true;

// A strip's inputs as one lane holds them: the attention output's features 32 s + 8 g + k (its
// B-operand slots) in fp32, or (OQ) their Eq. 2 codes and the token's scale, and the residual X
// in lane order (register v = feature 4 v + g).
template <int D, bool OQ>
struct TbIn {
  float o[OQ ? 1 : D / 32][8];
  long oc[OQ ? D / 32 : 1];
  float ao;
  float x[D / 4];
  // E: the first layer, whose X is rebuilt from t_i and the embedding rows (ie: the token's
  // position i in its word, or any position for a padding column)
  template <bool E>
  __device__ __forceinline__ void load(const TokenBlockArgs &p, int64_t tl, int g, uint32_t ie) {
    if constexpr (OQ) {
#pragma unroll
      for (int s = 0; s < D / 32; ++s) oc[s] = *(const long *)(p.oq + tl * D + 32 * s + 8 * g);
      ao = p.ao[tl];
    } else {
#pragma unroll
      for (int s = 0; s < D / 32; ++s)
#pragma unroll
        for (int k = 0; k < 8; k += 4) {
          const float4 f = *(const float4 *)(p.o + tl * D + 32 * s + 8 * g + k);
          o[s][k] = f.x; o[s][k + 1] = f.y; o[s][k + 2] = f.z; o[s][k + 3] = f.w;
        }
    }
    if constexpr (E) {   // X as the embedding computes it
      const float tt = p.t[tl];
      const float *er = p.elo + ie * D + g * (D / 4), *pr = p.plo ? p.plo + ie * D + g * (D / 4) : nullptr;
#pragma unroll
      for (int u = 0; u < D / 4; u += 4) {
        const float4 e = *(const float4 *)(er + u);
        const float4 q = pr ? *(const float4 *)(pr + u) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        x[u] = __builtin_fmaf(tt, e.x, q.x); x[u + 1] = __builtin_fmaf(tt, e.y, q.y);
        x[u + 2] = __builtin_fmaf(tt, e.z, q.z); x[u + 3] = __builtin_fmaf(tt, e.w, q.w);
      }
      return;
    }
#pragma unroll
    for (int u = 0; u < D / 4; u += 4) {
      const float4 r = *(const float4 *)(p.x + tl * D + g * (D / 4) + u);
      x[u] = r.x; x[u + 1] = r.y; x[u + 2] = r.z; x[u + 3] = r.w;
    }
  }
};

// LDS: the FF1, FF2 and O fragments (9 d^2 bytes), then the six d-vectors, the FF1 bias and
// W_{d->1} in lane order.
template <int D>
constexpr size_t token_block_lds() {
  return (size_t)9 * D * D + (size_t)11 * D * 4;
}

// Pairwise sum of a token's d features held as x[v] = feature 4 v + g.
template <int V>
__device__ __forceinline__ float tb_token_sum(const float (&x)[V]) {
  float u[V];
#pragma unroll
  for (int v = 0; v < V; ++v) u[v] = x[v];
  return lane_xor_add<16>(lane_xor_add<32>(lane_tree<V>(u)));
}
// Maximum over the four lanes of a token (non-negative floats order like their bit patterns).
__device__ __forceinline__ float tb_token_max(float a) {
  uint32_t u = __builtin_bit_cast(uint32_t, a), p, q;
  lane_swap_pair<32>(u, p, q);
  lane_swap_pair<16>(max(p, q), p, q);
  return __builtin_bit_cast(float, max(p, q));
}

// Z: the last layer, which leaves the head's z per token (TokenBlockArgs::z) instead of x, xq, ax.
// E: the first layer, which rebuilds its residual X from t_i and the embedding instead of reading x.
template <int D, bool OQ, bool Z, bool E>
__global__ __launch_bounds__(kTbWaves * 64) void k_token_block(TokenBlockArgs p) {
  constexpr int V = D / 4, S = D / 32, TO = D / 16, TH = D / 4, SH = D / 8;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  constexpr size_t frag_bytes = (size_t)9 * D * D;
  uint64_t *f1 = (uint64_t *)smem, *f2 = f1 + (size_t)TH * S * 64, *fo = f2 + (size_t)TO * SH * 64;
  for (int u = threadIdx.x; u < TH * S * 64; u += kTbWaves * 64) f1[u] = p.f1[u];
  for (int u = threadIdx.x; u < TO * SH * 64; u += kTbWaves * 64) f2[u] = p.f2[u];
  for (int u = threadIdx.x; u < TO * S * 64; u += kTbWaves * 64) fo[u] = p.fo[u];
  float *lv = (float *)(smem + frag_bytes);
  for (int u = threadIdx.x; u < 6 * D; u += kTbWaves * 64) lv[u] = p.vec[u];
  for (int u = threadIdx.x; u < 4 * D; u += kTbWaves * 64) lv[6 * D + u] = p.b1[u];
  if constexpr (Z)
    for (int u = threadIdx.x; u < D; u += kTbWaves * 64) lv[10 * D + u] = p.w1[u];
  const float *vec = lv;
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, c = lane & 15, g = lane >> 4;
  const float *vb_o = vec + 0 * D + g * V, *vg1 = vec + 1 * D + g * V, *vb1 = vec + 2 * D + g * V;
  const float *vb_2 = vec + 3 * D + g * V, *vg2 = vec + 4 * D + g * V, *vbb2 = vec + 5 * D + g * V;
  // Per-lane bases of the FF1 / FF2 fragments and the FF1 bias as opaque byte offsets: each loop
  // then keeps one running address per array and reaches the rest through the 16-bit immediate
  // offset of the LDS reads (rather than an add per read past the first 64 KB).
  uint32_t o_f1 = (uint32_t)lane * 8u, o_f2 = (uint32_t)(TH * S * 64 + lane) * 8u,
           o_b1 = (uint32_t)(frag_bytes + (size_t)6 * D * 4) + 16u * (uint32_t)g;
  asm volatile("" : "+v"(o_f1), "+v"(o_f2), "+v"(o_b1));
  const uint64_t *f1l = (const uint64_t *)(smem + o_f1), *f2l = (const uint64_t *)(smem + o_f2);
  const float *b1l = (const float *)(smem + o_b1);        // b1l[16 o + i] = FF1 bias 16 o + 4 g + i
  const int64_t nstrips = (p.rows + 15) / 16, sstride = (int64_t)gridDim.x * kTbWaves;
  // loads of a padding column read the last row instead: each column's results depend on
  // that column alone and padding columns are never stored
  auto load_row = [&](int64_t st) { const int64_t t = st * 16 + c; return t < p.rows ? t : p.rows - 1; };
  for (int64_t strip = (int64_t)blockIdx.x * kTbWaves + wave; strip < nstrips; strip += sstride) {
    const int64_t row0 = strip * 16, tok = row0 + c;
    const bool ok = tok < p.rows;
    TbIn<D, OQ> cur;
    uint32_t ie = 0;
    if constexpr (E) {
      // the strip's first row is wave-uniform, so its position in the word is scalar work; rows
      // < 2^31 with t (checked at launch)
      const uint32_t L = (uint32_t)p.L;
      ie = (uint32_t)row0 % L + (uint32_t)c;
      while (ie >= L) ie -= L;
    }
    cur.template load<E>(p, load_row(strip), g, ie);
    // ---- output projection, residual, LN1, Eq. 2 ----
    float x1[V];
    long xb[S];
    float a1;
    {
      // Eq. 2 of the token's attention output: the lane's B-operand features 32 s + 8 g + k,
      // alpha = max |O| over the four lanes of the token
      long bq[S];
      float sc;
      if constexpr (OQ) {
#pragma unroll
        for (int s = 0; s < S; ++s) bq[s] = cur.oc[s];
        sc = cur.ao * p.sq_o;
      } else {
        const float (&ov)[S][8] = cur.o;
        float om = 0.0f;
#pragma unroll
        for (int s = 0; s < S; ++s)
#pragma unroll
          for (int k = 0; k < 8; ++k) om = fmaxf(om, fabsf(ov[s][k]));
        om = tb_token_max(om);
        const float oinv = inv127(om);
#pragma unroll
        for (int s = 0; s < S; ++s) {
          uint32_t b[8];
#pragma unroll
          for (int k = 0; k < 8; ++k) b[k] = quant_bits(ov[s][k], oinv);
          bq[s] = tb_pack8(b);
        }
        sc = om * p.sq_o;
      }
#pragma unroll
      for (int o = 0; o < TO; ++o) {
        v4i acc = v4i{0, 0, 0, 0};
        acc = mfma_i8_steps<S>([&](int s) { return (long)fo[(o * S + s) * 64 + lane]; }, [&](int s) { return bq[s]; }, acc);
        // the residual: four consecutive values of X in lane order
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int v = 4 * o + i;
          const float y = __builtin_fmaf((float)acc[i], sc, vb_o[v]);
          x1[v] = cur.x[v] + y;
        }
      }
      const float mean = tb_token_sum<V>(x1) / (float)D;
      float e[V], sq[V];
#pragma unroll
      for (int v = 0; v < V; ++v) {
        e[v] = x1[v] - mean;
        sq[v] = e[v] * e[v];
      }
      const float var = tb_token_sum<V>(sq) / (float)D;
      const float rho = ln_rsqrt(var + p.eps);
      float amax = 0.0f;
#pragma unroll
      for (int v = 0; v < V; ++v) {
        x1[v] = __builtin_fmaf(e[v] * rho, vg1[v], vb1[v]);
        amax = fmaxf(amax, fabsf(x1[v]));
      }
      amax = tb_token_max(amax);
      const float inv = inv127(amax);
#pragma unroll
      for (int s = 0; s < S; ++s) {
        uint32_t b[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) b[k] = quant_bits(x1[8 * s + k], inv);
        xb[s] = tb_pack8(b);
      }
      a1 = amax;
    }
    // ---- FFN1 with ReLU feeding FFN2 ----
    const float sc1 = a1 * p.sq_1;
    // pass 1: the row's ReLU maximum, max(0, F_0, F_1, ...) = max over ReLU(F); adding +0
    // turns a -0 result into +0, so the cross-lane maximum may compare bit patterns
    float am = 0.0f;
    [[maybe_unused]] float hid[kTbKeepHidden ? TH : 1][4];
    if constexpr (kTbKeepHidden) {
      // software-pipelined: tile o + 2's fragments and bias are read and tile o + 1's products
      // issued before tile o's epilogue, so the LDS reads and the MFMA latency overlap the VALU
      long fq[2][S];
      float4 bq1[2];
      auto ldf = [&](int o, long (&f)[S], float4 &b) {
#pragma unroll
        for (int s2 = 0; s2 < S; ++s2) f[s2] = (long)f1l[(o * S + s2) * 64];
        b = *(const float4 *)(b1l + 16 * o);
      };
      const auto xbf = [&](int s2) { return xb[s2]; };
      ldf(0, fq[0], bq1[0]);
      ldf(1, fq[1], bq1[1]);
      v4i acc = mfma_i8_steps<S>([&](int s2) { return fq[0][s2]; }, xbf, v4i{0, 0, 0, 0});
      float4 bc = bq1[0];
#pragma unroll
      for (int o = 0; o < TH; ++o) {
        v4i acn = v4i{0, 0, 0, 0};
        float4 bn = bc;
        if (o + 1 < TH) {
          acn = mfma_i8_steps<S>([&](int s2) { return fq[(o + 1) & 1][s2]; }, xbf, acn);
          bn = bq1[(o + 1) & 1];
        }
        if (o + 2 < TH) ldf(o + 2, fq[o & 1], bq1[o & 1]);
        __builtin_amdgcn_sched_barrier(0);
        const float bb[4] = {bc.x, bc.y, bc.z, bc.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          hid[o][i] = __builtin_fmaf((float)acc[i], sc1, bb[i]);
          am = fmaxf(am, hid[o][i]);
        }
        __builtin_amdgcn_sched_barrier(0);
        acc = acn;
        bc = bn;
      }
    } else {
#pragma unroll 2
      for (int o = 0; o < TH; ++o) {
        v4i acc = v4i{0, 0, 0, 0};
        acc = mfma_i8_steps<S>([&](int s) { return (long)f1l[(o * S + s) * 64]; }, [&](int s) { return xb[s]; }, acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) am = fmaxf(am, __builtin_fmaf((float)acc[i], sc1, b1l[16 * o + i]));
      }
    }
    am = tb_token_max(am + 0.0f);
    const float inv1 = inv127(am);
    v4i acc2[TO];
#pragma unroll
    for (int o = 0; o < TO; ++o) acc2[o] = v4i{0, 0, 0, 0};
    static_assert(SH % 2 == 0, "FF2 k-steps taken in pairs");
    // pass 2: tiles 2 s2 .. 2 s2 + 3 -> FF2 steps s2, s2 + 1
    auto pass2 = [&](int s2) {
      long gb[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int t0 = 2 * (s2 + j);
        uint32_t b[8];
        if constexpr (kTbKeepHidden) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            b[i] = quant_bits(hid[t0][i], inv1);
            b[4 + i] = quant_bits(hid[t0 + 1][i], inv1);
          }
        } else {
          v4i h0 = v4i{0, 0, 0, 0}, h1 = v4i{0, 0, 0, 0};
          h0 = mfma_i8_steps<S>([&](int s) { return (long)f1l[(t0 * S + s) * 64]; }, [&](int s) { return xb[s]; }, h0);
          h1 = mfma_i8_steps<S>([&](int s) { return (long)f1l[((t0 + 1) * S + s) * 64]; }, [&](int s) { return xb[s]; },
                                h1);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            b[i] = quant_bits(__builtin_fmaf((float)h0[i], sc1, b1l[16 * t0 + i]), inv1);
            b[4 + i] = quant_bits(__builtin_fmaf((float)h1[i], sc1, b1l[16 * (t0 + 1) + i]), inv1);
          }
        }
        // ReLU on the codes: the code of max(F, 0) is max(code of F, 0)
        gb[j] = (long)(((uint64_t)pack4_relu(b[4], b[5], b[6], b[7]) << 32) | pack4_relu(b[0], b[1], b[2], b[3]));
      }
#pragma unroll
      for (int o = 0; o < TO; ++o)
        acc2[o] = mfma_i8_16x16x64((long)f2l[(o * SH + s2) * 64], (long)f2l[(o * SH + s2 + 1) * 64], gb[0], gb[1], acc2[o]);
    };
    if constexpr (kTbKeepHidden) {
#pragma unroll
      for (int s2 = 0; s2 < SH; s2 += 2) pass2(s2);
    } else {
#pragma unroll 1
      for (int s2 = 0; s2 < SH; s2 += 2) pass2(s2);
    }
    // ---- FFN2 epilogue: residual, LN2, Eq. 2 of the next layer's input ----
    {
      const float sc2 = am * p.sq_2;
      float v2[V];
#pragma unroll
      for (int o = 0; o < TO; ++o)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int v = 4 * o + i;
          v2[v] = x1[v] + __builtin_fmaf((float)acc2[o][i], sc2, vb_2[v]);
        }
      const float mean = tb_token_sum<V>(v2) / (float)D;
      float e[V], sq[V];
#pragma unroll
      for (int v = 0; v < V; ++v) {
        e[v] = v2[v] - mean;
        sq[v] = e[v] * e[v];
      }
      const float var = tb_token_sum<V>(sq) / (float)D;
      const float rho = ln_rsqrt(var + p.eps);
      float amax = 0.0f;
#pragma unroll
      for (int v = 0; v < V; ++v) {
        v2[v] = __builtin_fmaf(e[v] * rho, vg2[v], vbb2[v]);
        amax = fmaxf(amax, fabsf(v2[v]));
      }
      if constexpr (Z) {
        // the last layer: the head's z of the token, pairwise over its features like the LayerNorm
        // sums (Section 3, W_{d->1}); X itself is not needed any more
        const float *w1l = vec + 10 * D + g * V;
        float pr[V];
#pragma unroll
        for (int v = 0; v < V; ++v) pr[v] = v2[v] * w1l[v];
        const float zt = tb_token_sum<V>(pr) + p.head_b1;
        if (ok && g == 0) p.z[tok] = zt;
      } else {
        if (ok) {
#pragma unroll
          for (int u = 0; u < V; u += 4)
            *(float4 *)(p.x + tok * D + g * V + u) = make_float4(v2[u], v2[u + 1], v2[u + 2], v2[u + 3]);
        }
        amax = tb_token_max(amax);
        const float inv = inv127(amax);
        if (ok) {
          // the next layer's codes in lane order: step s's eight codes of this lane as one word
#pragma unroll
          for (int s = 0; s < S; ++s) {
            uint32_t b[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) b[k] = quant_bits(v2[8 * s + k], inv);
            *(long *)(p.xq + tok * D + 32 * s + 8 * g) = tb_pack8(b);
          }
          if (g == 0) p.ax[tok] = amax;
        }
      }
    }
    // keeps the scheduler from overlapping strips (their live ranges would not fit the registers)
    __builtin_amdgcn_sched_barrier(0);
  }
}

// ------------------------------------------------------------------------------------------
// Output head and hard decision (Section 3): one block per word.  z_i = W_{d->1} x_i + b1
// (16 lanes per token, pairwise over features), then f_o = sum_i z_i W_o[i][o] + b_o in
// ascending token order, bit = [y < 0] xor [f < 0].
// ------------------------------------------------------------------------------------------
struct HeadArgs {
  const float *x, *y;
  int n, L;
  const float *w1, *wo, *bo;
  float b1;
  uint8_t *bits;
  float *logits;
};

template <int D, bool LO>
__global__ __launch_bounds__(256) void k_head(HeadArgs p) {
  constexpr int T = D / 16;
  extern __shared__ float zs[];
  const int64_t w = blockIdx.x;
  const int c = threadIdx.x & 15;
  for (int i = threadIdx.x >> 4; i < p.L; i += 16) {
    const float *xr = p.x + (w * p.L + i) * D;
    float v[T];
#pragma unroll
    for (int t = 0; t < T; ++t) v[t] = xr[LO ? lane_order_x<D>(16 * t + c) : 16 * t + c] * p.w1[16 * t + c];
    const float z = row16_sum(lane_tree<T>(v)) + p.b1;
    if (c == 0) zs[i] = z;
  }
  __syncthreads();
  for (int o = threadIdx.x; o < p.n; o += 256) {
    float acc = 0.0f;
    for (int i = 0; i < p.L; ++i) acc = __builtin_fmaf(zs[i], p.wo[(int64_t)i * p.n + o], acc);
    const float f = acc + p.bo[o];
    const float yv = p.y[w * p.n + o];
    p.bits[w * p.n + o] = (uint8_t)((yv < 0.0f) != (f < 0.0f));
    if (p.logits) p.logits[w * p.n + o] = f;
  }
}

// The same head for a batch of words in two kernels: z per token into a buffer, then
// f = W_o^T z + b_o as a product tiled over words and outputs, so that each block reads a
// 64-output strip of W_o once for 16 words instead of once per word.  Every f_o is still the
// ascending chain acc = fma(z_i, W_o[i][o], acc) from 0 over i = 0 .. L-1, then + b_o.
template <int D, bool LO>
__global__ __launch_bounds__(256) void k_head_z(HeadArgs p, int64_t rows, float *z) {
  constexpr int T = D / 16;
  const int c = threadIdx.x & 15;
  for (int64_t r = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 4; r < rows; r += (int64_t)gridDim.x * 16) {
    const float *xr = p.x + r * D;
    float v[T];
#pragma unroll
    for (int t = 0; t < T; ++t) v[t] = xr[LO ? lane_order_x<D>(16 * t + c) : 16 * t + c] * p.w1[16 * t + c];
    const float zr = row16_sum(lane_tree<T>(v)) + p.b1;
    if (c == 0) z[r] = zr;
  }
}

constexpr int kHeadWords = 16, kHeadOuts = 64, kHeadK = 32;

// Block (word tile, output tile): thread (w = tid / 16, j = tid % 16) owns word w and outputs
// 4 j .. 4 j + 3 of the tile.  Per chunk of 32 tokens the tile's z values and W_o rows are
// staged in LDS; the chunk length is the same for every thread (the order of the chains).
__global__ __launch_bounds__(256) void k_head_gemm(HeadArgs p, int64_t words, const float *z) {
  __shared__ float zs[kHeadK][kHeadWords];
  __shared__ __attribute__((aligned(16))) float ws[kHeadK][kHeadOuts];
  const int tid = threadIdx.x, wl = tid >> 4, j = tid & 15;
  const int64_t w0 = (int64_t)blockIdx.x * kHeadWords;
  const int o0 = blockIdx.y * kHeadOuts;
  const int n = p.n, L = p.L;
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int i0 = 0; i0 < L; i0 += kHeadK) {
    const int kc = min(kHeadK, L - i0);
    for (int u = tid; u < kHeadK * kHeadWords; u += 256) {      // z of the tile's words
      const int k = u / kHeadWords, w = u % kHeadWords;
      const int64_t wg = w0 + w;
      zs[k][w] = (k < kc && wg < words) ? z[wg * L + i0 + k] : 0.0f;
    }
    for (int u = tid; u < kHeadK * kHeadOuts; u += 256) {       // rows i0 .. i0 + kc - 1 of W_o
      const int k = u / kHeadOuts, o = u % kHeadOuts;
      ws[k][o] = (k < kc && o0 + o < n) ? p.wo[(int64_t)(i0 + k) * n + o0 + o] : 0.0f;
    }
    __syncthreads();
    for (int k = 0; k < kc; ++k) {
      const float zv = zs[k][wl];
      const float4 wv = *(const float4 *)&ws[k][4 * j];
      acc[0] = __builtin_fmaf(zv, wv.x, acc[0]);
      acc[1] = __builtin_fmaf(zv, wv.y, acc[1]);
      acc[2] = __builtin_fmaf(zv, wv.z, acc[2]);
      acc[3] = __builtin_fmaf(zv, wv.w, acc[3]);
    }
    __syncthreads();
  }
  const int64_t w = w0 + wl;
  if (w >= words) return;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int o = o0 + 4 * j + u;
    if (o >= n) break;
    const float f = acc[u] + p.bo[o];
    const float yv = p.y[w * n + o];
    p.bits[w * n + o] = (uint8_t)((yv < 0.0f) != (f < 0.0f));
    if (p.logits) p.logits[w * n + o] = f;
  }
}

// ------------------------------------------------------------------------------------------
// Eq. 2 with one alpha per word (the reading of Section 4.1 in which alpha = ||x||_inf is taken
// over the whole layer input of a word): alpha = max |x| over the word's L rows of K values
// (of max(x, 0) when RELU, the feed-forward hidden row), then every value's code
// x * fp32(127 / alpha) rounded half to even, and a[row] = alpha for each of the word's rows, so
// the dequantisation of Eq. 3 reads it like a per-token scale.  One block per word (persistent
// over the words), natural layout, four values per lane and step.
// ------------------------------------------------------------------------------------------
constexpr int kWqThreads = 256;

template <bool RELU>
__global__ __launch_bounds__(kWqThreads) void k_word_quant(const float *x, int64_t words, int64_t per_word, int L,
                                                           int8_t *q, float *a) {
  __shared__ float red[kWqThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t n4 = per_word / 4;                       // per_word = L K, K a multiple of 32
  for (int64_t w = blockIdx.x; w < words; w += gridDim.x) {
    const float4 *xw = (const float4 *)(x + w * per_word);
    float m = 0.0f;
    for (int64_t e = tid; e < n4; e += kWqThreads) {
      float4 v = xw[e];
      if (RELU) {
        v.x = v.x > 0.0f ? v.x : 0.0f; v.y = v.y > 0.0f ? v.y : 0.0f;
        v.z = v.z > 0.0f ? v.z : 0.0f; v.w = v.w > 0.0f ? v.w : 0.0f;
      }
      m = fmaxf(m, fmaxf(fmaxf(fabsf(v.x), fabsf(v.y)), fmaxf(fabsf(v.z), fabsf(v.w))));
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    if (lane == 0) red[wave] = m;
    __syncthreads();
    float alpha = red[0];
#pragma unroll
    for (int k = 1; k < kWqThreads / 64; ++k) alpha = fmaxf(alpha, red[k]);
    const float inv = inv127(alpha);
    uint32_t *qw = (uint32_t *)(q + w * per_word);
    for (int64_t e = tid; e < n4; e += kWqThreads) {
      float4 v = xw[e];
      if (RELU) {
        v.x = v.x > 0.0f ? v.x : 0.0f; v.y = v.y > 0.0f ? v.y : 0.0f;
        v.z = v.z > 0.0f ? v.z : 0.0f; v.w = v.w > 0.0f ? v.w : 0.0f;
      }
      qw[e] = (quant_bits(v.x, inv) & 0xffu) | (quant_bits(v.y, inv) & 0xffu) << 8 |
              (quant_bits(v.z, inv) & 0xffu) << 16 | (quant_bits(v.w, inv) & 0xffu) << 24;
    }
    for (int r = tid; r < L; r += kWqThreads) a[w * L + r] = alpha;
    __syncthreads();                                     // red[] is rewritten for the next word
  }
}

// ------------------------------------------------------------------------------------------
// launchers
// ------------------------------------------------------------------------------------------
namespace {

// Persistent grid: as many blocks as stay resident (LDS-limited), each staging its map's
// weights once and striding over the 16-row strips.
int gemm_grid(const Model &M, int64_t rows, size_t lds_bytes) {
  const int64_t groups = ((rows + 15) / 16 + kGemmWaves - 1) / kGemmWaves;
  const int64_t per_cu = lds_bytes ? std::max<int64_t>(1, (int64_t)(M.lds_max / lds_bytes)) : 8;
  const int64_t g = std::min<int64_t>(groups, (int64_t)M.cu_count * std::min<int64_t>(per_cu, 8));
  return (int)(g > 0 ? g : 1);
}

template <int K, int NOUT, int EPI>
hipError_t run_gemm(const Model &M, const GemmArgs &a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  constexpr bool kQuantOut = (EPI == EPI_LN || EPI == EPI_RELU_QUANT);
  constexpr size_t lds = (size_t)(NOUT / 16) * (K / 32) * 64 * 8 + (kQuantOut ? (size_t)kGemmWaves * 16 * NOUT : 16);
  hipLaunchKernelGGL((k_gemm<K, NOUT, EPI>), dim3(gemm_grid(M, a.rows, lds)), dim3(kGemmWaves * 64), 0, s, a);
  return hipGetLastError();
}

GemmArgs gemm_base(const int8_t *a, const float *alpha, const uint16_t *bpack, int64_t rows) {
  GemmArgs g{};
  g.a = a;
  g.alpha = alpha;
  g.bpack = bpack;
  g.rows = rows;
  return g;
}

}  // namespace

// LDS of k_embed_words: the word's y and t.
static size_t embed_words_lds(const Model &M) { return sizeof(float) * (size_t)(M.n + M.L); }

hipError_t launch_embed(const Model &M, const float *y, int64_t words, float *x, int8_t *xq, float *ax,
                        bool lane_order, hipStream_t s, float *t) {
  EmbedArgs a{y, words * M.L, M.n, M.L, M.chk_ptr, M.chk_idx, M.embed, M.pos, x, xq, ax, t, M.embed_lo, M.pos_lo};
  if (a.rows <= 0) return hipSuccess;
  if (!x && !t) return hipErrorInvalidValue;
  if (lane_order && ((M.d != 64 && M.d != 128) || !M.embed_lo)) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((a.rows + 15) / 16));
  if (lane_order) {
    const size_t lds = embed_words_lds(M);
    if (lds <= M.lds_max) {
      const unsigned wgrid = (unsigned)std::min<int64_t>(words, (int64_t)M.cu_count * 8);
      if (M.d == 64) hipLaunchKernelGGL((k_embed_words<64>), dim3(wgrid), dim3(kEwThreads), lds, s, a, words);
      else hipLaunchKernelGGL((k_embed_words<128>), dim3(wgrid), dim3(kEwThreads), lds, s, a, words);
    } else if (M.d == 64) {
      hipLaunchKernelGGL((k_embed<64, true>), grid, dim3(256), 0, s, a);
    } else {
      hipLaunchKernelGGL((k_embed<128, true>), grid, dim3(256), 0, s, a);
    }
    return hipGetLastError();
  }
  if (t) return hipErrorInvalidValue;   // t only with the lane order (the token block's first layer)
  switch (M.d) {
    case 32: hipLaunchKernelGGL((k_embed<32, false>), grid, dim3(256), 0, s, a); break;
    case 64: hipLaunchKernelGGL((k_embed<64, false>), grid, dim3(256), 0, s, a); break;
    case 128: hipLaunchKernelGGL((k_embed<128, false>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_qkv(const Model &M, int layer, const int8_t *xq, const float *ax, int64_t rows, float *qkv,
                      bool lane_order, hipStream_t s) {
  const LayerWeights &W = M.layer[layer];
  if (lane_order && !W.qkv_tb) return hipErrorInvalidValue;
  GemmArgs a = gemm_base(xq, ax, lane_order ? W.qkv_tb : W.qkv, rows);
  a.sq[0] = W.sq_qs;
  a.sq[1] = W.sq[1];
  a.sq[2] = W.sq[2];
  a.bias = W.b_qkv;
  a.out_f = qkv;
  switch (M.d) {
    case 32: return run_gemm<32, 96, EPI_QKV>(M, a, s);
    case 64: return run_gemm<64, 192, EPI_QKV>(M, a, s);
    case 128:
      // one launch per map: 8 output tiles per wave instead of 24
      for (int m = 0; m < 3; ++m) {
        GemmArgs b = a;
        b.tile0 = 8 * m;
        b.sq[0] = a.sq[m];
        b.bias = a.bias + 128 * m;
        b.out_f = a.out_f + 128 * m;
        const hipError_t e = run_gemm<128, 128, EPI_QKV_MAP>(M, b, s);
        if (e != hipSuccess) return e;
      }
      return hipSuccess;
  }
  return hipErrorInvalidValue;
}

hipError_t launch_oproj_ln(const Model &M, int layer, const int8_t *oq, const float *ao, const float *x,
                           int64_t rows, float *x1, int8_t *x1q, float *a1, hipStream_t s) {
  const LayerWeights &W = M.layer[layer];
  GemmArgs a = gemm_base(oq, ao, W.o, rows);
  a.sq[0] = W.sq[3];
  a.bias = W.b_o;
  a.resid = x;
  a.ln_g = W.ln1_g;
  a.ln_b = W.ln1_b;
  a.eps = M.eps;
  a.out_f = x1;
  a.out_q = x1q;
  a.out_a = a1;
  switch (M.d) {
    case 32: return run_gemm<32, 32, EPI_LN>(M, a, s);
    case 64: return run_gemm<64, 64, EPI_LN>(M, a, s);
    case 128: return run_gemm<128, 128, EPI_LN>(M, a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_ffn1(const Model &M, int layer, const int8_t *x1q, const float *a1, int64_t rows, int8_t *gq,
                      float *ag, hipStream_t s) {
  const LayerWeights &W = M.layer[layer];
  GemmArgs a = gemm_base(x1q, a1, W.ff1, rows);
  a.sq[0] = W.sq[4];
  a.bias = W.b_ff1;
  a.out_q = gq;
  a.out_a = ag;
  switch (M.d) {
    case 32: return run_gemm<32, 128, EPI_RELU_QUANT>(M, a, s);
    case 64: return run_gemm<64, 256, EPI_RELU_QUANT>(M, a, s);
    case 128: return run_gemm<128, 512, EPI_RELU_QUANT>(M, a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_ffn2_ln(const Model &M, int layer, const int8_t *gq, const float *ag, const float *x1,
                          int64_t rows, float *x, int8_t *xq, float *ax, hipStream_t s) {
  const LayerWeights &W = M.layer[layer];
  GemmArgs a = gemm_base(gq, ag, W.ff2, rows);
  a.sq[0] = W.sq[5];
  a.bias = W.b_ff2;
  a.resid = x1;
  a.ln_g = W.ln2_g;
  a.ln_b = W.ln2_b;
  a.eps = M.eps;
  a.out_f = x;
  a.out_q = xq;
  a.out_a = ax;
  switch (M.d) {
    case 32: return run_gemm<128, 32, EPI_LN>(M, a, s);
    case 64: return run_gemm<256, 64, EPI_LN>(M, a, s);
    case 128: return run_gemm<512, 128, EPI_LN>(M, a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_ternary_gemm(const Model &M, int layer, int kind, const int8_t *a_in, int64_t rows,
                               int32_t *acc, hipStream_t s) {
  const LayerWeights &W = M.layer[layer];
  const uint16_t *bp = kind <= 2 ? W.qkv : kind == 3 ? W.o : kind == 4 ? W.ff1 : W.ff2;
  GemmArgs a = gemm_base(a_in, nullptr, bp, rows);
  a.tile0 = kind <= 2 ? kind * (M.d / 16) : 0;
  a.out_acc = acc;
  const int d = M.d;
  if (kind <= 3) {
    if (d == 32) return run_gemm<32, 32, EPI_RAW>(M, a, s);
    if (d == 64) return run_gemm<64, 64, EPI_RAW>(M, a, s);
    if (d == 128) return run_gemm<128, 128, EPI_RAW>(M, a, s);
  } else if (kind == 4) {
    if (d == 32) return run_gemm<32, 128, EPI_RAW>(M, a, s);
    if (d == 64) return run_gemm<64, 256, EPI_RAW>(M, a, s);
    if (d == 128) return run_gemm<128, 512, EPI_RAW>(M, a, s);
  } else {
    if (d == 32) return run_gemm<128, 32, EPI_RAW>(M, a, s);
    if (d == 64) return run_gemm<256, 64, EPI_RAW>(M, a, s);
    if (d == 128) return run_gemm<512, 128, EPI_RAW>(M, a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_attention(const Model &M, const float *qkv, int64_t words, float *o, int8_t *oq, float *ao,
                            hipStream_t s) {
  AttnArgs a{qkv, words * M.L, M.L, M.d, M.heads, M.hf, M.m1_ptr, M.m1_idx, M.m2_ptr, M.m2_idx, o, oq, ao};
  if (a.rows <= 0) return hipSuccess;
  const int rpb = 256 / M.heads;
  const dim3 grid((unsigned)((a.rows + rpb - 1) / rpb));
  switch (M.dh) {
    case 4: hipLaunchKernelGGL(k_attention<4>, grid, dim3(256), 0, s, a); break;
    case 8: hipLaunchKernelGGL(k_attention<8>, grid, dim3(256), 0, s, a); break;
    case 16: hipLaunchKernelGGL(k_attention<16>, grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

size_t qkv_attention_lds(const Model &M, bool resident = false) {
  return (size_t)(resident ? M.d / 16 : 1) * 3 * (M.d / 32) * 64 * 8 + (size_t)M.L * (16 + kQaRow) * 4 +
         (size_t)3 * M.d * 4;
}

// Blocks of k_qkv_attention resident on a CU: as many as LDS holds, at most as many as its
// register budget (qa_waves_per_simd waves per SIMD, blocks of kQaThreads / 64 waves on 4 SIMDs)
// leaves room for; a grid of more would run its last blocks in a half-empty round.
static int64_t qkv_attention_blocks_per_cu(const Model &M, size_t lds) {
  const int64_t by_lds = std::max<int64_t>(1, (int64_t)(M.lds_max / std::max<size_t>(lds, 1)));
  const int64_t by_waves = std::max<int64_t>(1, (M.d == 128 ? 2 : 4) * 4 / (kQaThreads / 64));
  return std::min(by_lds, by_waves);
}

// Keep every head group's weight tiles in LDS when that does not lower the blocks per CU.
bool qkv_attention_resident(const Model &M) {
  const size_t one = qkv_attention_lds(M, false), all = qkv_attention_lds(M, true);
  return all <= M.lds_max && qkv_attention_blocks_per_cu(M, all) >= qkv_attention_blocks_per_cu(M, one);
}

bool qkv_attention_supported(const Model &M) {
  return (M.d == 64 || M.d == 128) && (M.dh == 8 || M.dh == 16) && M.grouped &&
         M.L <= 16 * (kQaThreads / 64) * kQaTilesPerWave && M.L * (16 / M.dh) <= kQaThreads &&
         qkv_attention_lds(M) <= M.lds_max;
}


// The lists and their metadata in LDS beside the form's own use (LT).
static size_t qkv_attention_lists_lds(const Model &M) {
  return qkv_attention_lds(M, true) + (size_t)16 * M.L + (size_t)8 * (M.g1_groups + M.g2_groups);
}

template <int D, int DH>
static hipError_t run_qkv_attention(const Model &M, const QkvAttnArgs &a, size_t lds, hipStream_t s) {
  // LT where every group's weights stay resident, the tiles stay in registers and the lists fit
  // without fewer resident blocks
  if constexpr (qa_keep_tiles<D, DH>()) {
    const size_t ll = qkv_attention_lists_lds(M);
    if (a.resident && ll <= M.lds_max &&
        qkv_attention_blocks_per_cu(M, ll) >= qkv_attention_blocks_per_cu(M, lds)) {
      QkvAttnArgs b = a;
      b.tab1_n = M.g1_groups;
      b.tab2_n = M.g2_groups;
      const int64_t blocks = std::min<int64_t>(a.words, (int64_t)M.cu_count * qkv_attention_blocks_per_cu(M, ll));
      hipLaunchKernelGGL((k_qkv_attention<D, DH, true>), dim3((unsigned)blocks), dim3(kQaThreads), ll, s, b);
      return hipGetLastError();
    }
  }
  const int64_t blocks = std::min<int64_t>(a.words, (int64_t)M.cu_count * qkv_attention_blocks_per_cu(M, lds));
  hipLaunchKernelGGL((k_qkv_attention<D, DH>), dim3((unsigned)blocks), dim3(kQaThreads), lds, s, a);
  return hipGetLastError();
}

// The lane-pair form (16-dimension heads): every group's weights resident, up to 36 token tiles.
size_t qkv_attention_pair_lds(const Model &M, bool quantised = false) {
  return qkv_attention_lds(M, true) + (quantised ? (size_t)kQpThreads * 32 : 0);
}

bool qkv_attention_pair_supported(const Model &M) {
  return M.d == 128 && M.dh == 16 && M.grouped && M.L <= 16 * (kQpThreads / 64) * kQpTilesPerWave &&
         qkv_attention_pair_lds(M) <= M.lds_max;
}

// The lane-pair form writes the Eq. 2 codes of O itself when a word has at most one row per lane
// pair.

bool qkv_attention_pair_quantises(const Model &M) {
  return qkv_attention_pair_supported(M) && M.L <= kQpThreads / 2 && qkv_attention_pair_lds(M, true) <= M.lds_max;
}

template <int D>
static hipError_t run_qkv_attention_pair(const Model &M, const QkvAttnArgs &a, size_t lds, hipStream_t s) {
  const int64_t per_cu = std::max<int64_t>(1, (int64_t)(M.lds_max / lds));
  const int64_t blocks = std::min<int64_t>(a.words, (int64_t)M.cu_count * per_cu);
  if (a.oq && a.tab1_n > 0) hipLaunchKernelGGL((k_qkv_attention_pair<D, true, true>), dim3((unsigned)blocks), dim3(kQpThreads), lds, s, a);
  else if (a.oq) hipLaunchKernelGGL((k_qkv_attention_pair<D, true>), dim3((unsigned)blocks), dim3(kQpThreads), lds, s, a);
  else hipLaunchKernelGGL((k_qkv_attention_pair<D, false>), dim3((unsigned)blocks), dim3(kQpThreads), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_qkv_attention(const Model &M, int layer, const int8_t *xq, const float *ax, int64_t words,
                                float *o, int8_t *oq, float *ao, bool lane_order, hipStream_t s) {
  if (words <= 0) return hipSuccess;
  if (!qkv_attention_supported(M)) return hipErrorInvalidValue;
  const LayerWeights &W = M.layer[layer];
  if (lane_order && !W.qkv_tb) return hipErrorInvalidValue;
  QkvAttnArgs a{};
  a.xq = xq;
  a.ax = ax;
  a.bpack = lane_order ? W.qkv_tb : W.qkv;
  a.bias = W.b_qkv;
  a.sq[0] = W.sq_qs;
  a.sq[1] = W.sq[1];
  a.sq[2] = W.sq[2];
  a.words = words;
  a.L = M.L;
  a.hf = M.hf;
  a.meta1 = (const int2 *)M.g1_meta; a.meta2 = (const int2 *)M.g2_meta;
  a.tab1 = (const uint2 *)M.g1_tab; a.tab2 = (const uint2 *)M.g2_tab;
  a.o = o;
  a.resident = qkv_attention_resident(M) ? 1 : 0;
  const size_t lds = qkv_attention_lds(M, a.resident != 0);
  hipError_t e = hipErrorInvalidValue;
  if (oq && qkv_attention_pair_quantises(M)) {   // O straight to its codes, no fp32 rows
    a.oq = oq;
    a.ao = ao;
    if (qkv_attention_lists_lds(M) <= M.lds_max) {   // and the lists in LDS
      a.tab1_n = M.g1_groups;
      a.tab2_n = M.g2_groups;
      return run_qkv_attention_pair<128>(M, a, qkv_attention_lists_lds(M), s);
    }
    return run_qkv_attention_pair<128>(M, a, qkv_attention_pair_lds(M, true), s);
  }
  if (qkv_attention_pair_supported(M)) e = run_qkv_attention_pair<128>(M, a, qkv_attention_pair_lds(M), s);
  else if (M.d == 64 && M.dh == 8) e = run_qkv_attention<64, 8>(M, a, lds, s);
  else if (M.d == 128 && M.dh == 16) e = run_qkv_attention<128, 16>(M, a, lds, s);
  else if (M.d == 128 && M.dh == 8) e = run_qkv_attention<128, 8>(M, a, lds, s);
  else if (M.d == 64 && M.dh == 16) e = run_qkv_attention<64, 16>(M, a, lds, s);
  if (e != hipSuccess || !oq) return e;
  const int64_t rows = words * M.L;
  const dim3 grid((unsigned)((rows + 15) / 16));
  if (M.d == 64) hipLaunchKernelGGL(k_quant_rows<64>, grid, dim3(256), 0, s, o, rows, oq, ao);
  else hipLaunchKernelGGL(k_quant_rows<128>, grid, dim3(256), 0, s, o, rows, oq, ao);
  return hipGetLastError();
}

bool qkv_attention_i16_supported(const Model &M) {
  if (!((M.d == 64 || M.d == 128) && (M.dh == 8 || M.dh == 16) && M.grouped)) return false;
  const size_t lds = M.d == 64 ? qkv_attention_i16_lds_bytes<64>(M.L) : qkv_attention_i16_lds_bytes<128>(M.L);
  return lds <= M.lds_max;
}

template <int D, int DH>
static hipError_t run_qkv_attention_i16(const Model &M, const QkvAttnArgs &a, size_t lds, hipStream_t s) {
  const int64_t per_cu = std::max<int64_t>(1, (int64_t)(M.lds_max / lds));
  const int64_t blocks = std::min<int64_t>(a.words, (int64_t)M.cu_count * per_cu);
  hipLaunchKernelGGL((k_qkv_attention_i16<D, DH>), dim3((unsigned)blocks), dim3(kQaThreads), lds, s, a);
  return hipGetLastError();
}

// Keys in fp32, values in int16 (16-dimension heads), when that layout fits LDS.
bool qkv_attention_v16_supported(const Model &M) {
  if (!((M.d == 64 || M.d == 128) && M.dh == 16 && M.grouped)) return false;
  if (M.L > 16 * (kQvThreads / 64) * kQvTilesPerWave) return false;
  const size_t lds = M.d == 64 ? qkv_attention_v16_lds_bytes<64>(M.L) : qkv_attention_v16_lds_bytes<128>(M.L);
  return lds <= M.lds_max;
}

template <int D>
static hipError_t run_qkv_attention_v16(const Model &M, const QkvAttnArgs &a, size_t lds, hipStream_t s) {
  const int64_t per_cu = std::max<int64_t>(1, (int64_t)(M.lds_max / lds));
  const int64_t blocks = std::min<int64_t>(a.words, (int64_t)M.cu_count * per_cu);
  hipLaunchKernelGGL((k_qkv_attention_v16<D>), dim3((unsigned)blocks), dim3(kQvThreads), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_qkv_attention_i16(const Model &M, int layer, const int8_t *xq, const float *ax, int64_t words,
                                    float *o, bool lane_order, hipStream_t s) {
  if (words <= 0) return hipSuccess;
  if (!qkv_attention_i16_supported(M)) return hipErrorInvalidValue;
  const LayerWeights &W = M.layer[layer];
  if (lane_order && !W.qkv_tb) return hipErrorInvalidValue;
  QkvAttnArgs a{};
  a.xq = xq;
  a.ax = ax;
  a.bpack = lane_order ? W.qkv_tb : W.qkv;
  a.bias = W.b_qkv;
  a.sq[0] = W.sq_qs;
  a.sq[1] = W.sq[1];
  a.sq[2] = W.sq[2];
  a.words = words;
  a.L = M.L;
  a.hf = M.hf;
  a.meta1 = (const int2 *)M.g1_meta; a.meta2 = (const int2 *)M.g2_meta;
  a.tab1 = (const uint2 *)M.g1_tab; a.tab2 = (const uint2 *)M.g2_tab;
  a.o = o;
  if (qkv_attention_v16_supported(M)) {
    const size_t lv = M.d == 64 ? qkv_attention_v16_lds_bytes<64>(M.L) : qkv_attention_v16_lds_bytes<128>(M.L);
    return M.d == 64 ? run_qkv_attention_v16<64>(M, a, lv, s) : run_qkv_attention_v16<128>(M, a, lv, s);
  }
  const size_t lds = M.d == 64 ? qkv_attention_i16_lds_bytes<64>(M.L) : qkv_attention_i16_lds_bytes<128>(M.L);
  if (M.d == 128 && M.dh == 16) return run_qkv_attention_i16<128, 16>(M, a, lds, s);
  if (M.d == 64 && M.dh == 16) return run_qkv_attention_i16<64, 16>(M, a, lds, s);
  if (M.d == 64 && M.dh == 8) return run_qkv_attention_i16<64, 8>(M, a, lds, s);
  if (M.d == 128 && M.dh == 8) return run_qkv_attention_i16<128, 8>(M, a, lds, s);
  return hipErrorInvalidValue;
}

// Rows one node type at a time: head partitioning (every list holds one node type), d = 128 with
// 16-dimension heads, the larger node type's keys and values fit LDS.
bool qkv_attention_split_supported(const Model &M) {
  if (!(M.d == 128 && M.dh == 16 && M.grouped && M.g1s_tab && M.g2s_tab)) return false;   // tables: HPSA only
  if (M.L > 16 * (kQsThreads / 64) * kQsTilesPerWave) return false;
  return qkv_attention_split_lds_bytes<128>(std::max(M.n, M.m), M.L) <= M.lds_max;
}

hipError_t launch_qkv_attention_split(const Model &M, int layer, const int8_t *xq, const float *ax, int64_t words,
                                      float *o, bool lane_order, hipStream_t s) {
  if (words <= 0) return hipSuccess;
  if (!qkv_attention_split_supported(M)) return hipErrorInvalidValue;
  const LayerWeights &W = M.layer[layer];
  if (lane_order && !W.qkv_tb) return hipErrorInvalidValue;
  QkvAttnArgs a{};
  a.xq = xq;
  a.ax = ax;
  a.bpack = lane_order ? W.qkv_tb : W.qkv;
  a.bias = W.b_qkv;
  a.sq[0] = W.sq_qs;
  a.sq[1] = W.sq[1];
  a.sq[2] = W.sq[2];
  a.words = words;
  a.L = M.L;
  a.hf = M.hf;
  a.meta1 = (const int2 *)M.g1_meta; a.meta2 = (const int2 *)M.g2_meta;
  a.tab1s = (const uint2 *)M.g1s_tab; a.tab2s = (const uint2 *)M.g2s_tab;
  a.n_var = M.n;
  a.kv_cap = std::max(M.n, M.m);
  a.o = o;
  const size_t lds = qkv_attention_split_lds_bytes<128>(a.kv_cap, M.L);
  const int64_t per_cu = std::max<int64_t>(1, (int64_t)(M.lds_max / lds));
  const int64_t blocks = std::min<int64_t>(words, (int64_t)M.cu_count * per_cu);
  hipLaunchKernelGGL((k_qkv_attention_split<128>), dim3((unsigned)blocks), dim3(kQsThreads), lds, s, a);
  return hipGetLastError();
}

// Words the layered decode's attention kernel processes at once (one word per block, as many
// blocks as stay resident on the device): chunks of words are best sized in multiples of it.
int64_t attention_word_slots(const Model &M, int form) {
  size_t lds = 0;
  switch (form) {
    case 1:   // fp32 keys and values of the whole word
      if (!qkv_attention_pair_supported(M))
        return (int64_t)M.cu_count * qkv_attention_blocks_per_cu(M, qkv_attention_lds(M, qkv_attention_resident(M)));
      lds = qkv_attention_pair_lds(M);
      break;
    case 2:   // int16 accumulators
      lds = qkv_attention_v16_supported(M) ? (M.d == 64 ? qkv_attention_v16_lds_bytes<64>(M.L) : qkv_attention_v16_lds_bytes<128>(M.L))
                                           : (M.d == 64 ? qkv_attention_i16_lds_bytes<64>(M.L) : qkv_attention_i16_lds_bytes<128>(M.L));
      break;
    case 3:   // one node type's rows at a time
      lds = qkv_attention_split_lds_bytes<128>(std::max(M.n, M.m), M.L);
      break;
    default:  // the unfused kernels take rows, not words
      return 1;
  }
  return (int64_t)M.cu_count * std::max<int64_t>(1, (int64_t)(M.lds_max / std::max<size_t>(lds, 1)));
}

bool token_block_supported(const Model &M) {
  return (M.d == 64 || M.d == 128) && M.dff == 4 * M.d && M.layer[0].tb_o != nullptr;
}

template <int D, bool OQ, bool Z, bool E>
static hipError_t run_token_block(const Model &M, const TokenBlockArgs &a, hipStream_t s) {
  constexpr size_t lds = token_block_lds<D>();
  const int64_t strips = (a.rows + 15) / 16;
  const int64_t per_cu = std::max<int64_t>(1, (int64_t)(M.lds_max / lds));
  const int64_t blocks = std::min<int64_t>((strips + kTbWaves - 1) / kTbWaves, (int64_t)M.cu_count * per_cu);
  hipLaunchKernelGGL((k_token_block<D, OQ, Z, E>), dim3((unsigned)std::max<int64_t>(blocks, 1)), dim3(kTbWaves * 64), lds, s, a);
  return hipGetLastError();
}
// the instantiation for the arguments' form: codes or fp32 O, last layer, first layer
template <int D, bool OQ, bool Z>
static hipError_t run_token_block_e(const Model &M, const TokenBlockArgs &a, hipStream_t s) {
  return a.t ? run_token_block<D, OQ, Z, true>(M, a, s) : run_token_block<D, OQ, Z, false>(M, a, s);
}
template <int D, bool OQ>
static hipError_t run_token_block_z(const Model &M, const TokenBlockArgs &a, hipStream_t s) {
  return a.z ? run_token_block_e<D, OQ, true>(M, a, s) : run_token_block_e<D, OQ, false>(M, a, s);
}
template <int D>
static hipError_t run_token_block_oq(const Model &M, const TokenBlockArgs &a, hipStream_t s) {
  return a.oq ? run_token_block_z<D, true>(M, a, s) : run_token_block_z<D, false>(M, a, s);
}
template <int D, int K>
static const void *token_block_kernel() {
  return (const void *)k_token_block<D, (K & 1) != 0, (K & 2) != 0, (K & 4) != 0>;
}

hipError_t launch_token_block(const Model &M, int layer, const float *o, const int8_t *oq, const float *ao,
                              float *x, int64_t rows, int8_t *xq, float *ax, hipStream_t s, float *z, const float *t) {
  if (rows <= 0) return hipSuccess;
  if (!token_block_supported(M)) return hipErrorInvalidValue;
  const LayerWeights &W = M.layer[layer];
  TokenBlockArgs a{};
  a.o = o;
  a.oq = oq;
  a.ao = ao;
  a.x = x;
  a.fo = W.tb_o;
  a.f1 = W.tb_1;
  a.f2 = W.tb_2;
  a.vec = W.tb_vec;
  a.b1 = W.b_ff1;
  a.sq_o = W.sq[3];    // aecct_linear order: q, k, v, o, ff1, ff2
  a.sq_1 = W.sq[4];
  a.sq_2 = W.sq[5];
  a.eps = M.eps;
  a.rows = rows;
  a.xq = xq;
  a.ax = ax;
  a.z = z;
  a.w1 = M.head_w1_lo;
  a.head_b1 = M.head_b1;
  a.t = t;
  a.elo = M.embed_lo;
  a.plo = M.pos_lo;
  a.L = M.L;
  if (!oq == !o || (z && !M.head_w1_lo) || (t && (!M.embed_lo || rows > INT32_MAX))) return hipErrorInvalidValue;
  return M.d == 64 ? run_token_block_oq<64>(M, a, s) : run_token_block_oq<128>(M, a, s);
}

hipError_t launch_head_tiled(const Model &M, const float *x, const float *y, int64_t words, uint8_t *bits,
                             float *logits, bool lane_order, float *zbuf, hipStream_t s, bool z_ready) {
  if (words <= 0) return hipSuccess;
  if (lane_order && M.d != 64 && M.d != 128) return hipErrorInvalidValue;
  HeadArgs a{x, y, M.n, M.L, M.head_w1, M.head_wo, M.head_bo, M.head_b1, bits, logits};
  const int64_t rows = words * M.L;
  const unsigned zgrid = (unsigned)std::min<int64_t>((rows + 15) / 16, (int64_t)M.cu_count * 64);
  if (!z_ready) switch (M.d) {
    case 32: hipLaunchKernelGGL((k_head_z<32, false>), dim3(zgrid), dim3(256), 0, s, a, rows, zbuf); break;
    case 64:
      if (lane_order) hipLaunchKernelGGL((k_head_z<64, true>), dim3(zgrid), dim3(256), 0, s, a, rows, zbuf);
      else hipLaunchKernelGGL((k_head_z<64, false>), dim3(zgrid), dim3(256), 0, s, a, rows, zbuf);
      break;
    case 128:
      if (lane_order) hipLaunchKernelGGL((k_head_z<128, true>), dim3(zgrid), dim3(256), 0, s, a, rows, zbuf);
      else hipLaunchKernelGGL((k_head_z<128, false>), dim3(zgrid), dim3(256), 0, s, a, rows, zbuf);
      break;
    default: return hipErrorInvalidValue;
  }
  const dim3 grid((unsigned)((words + kHeadWords - 1) / kHeadWords), (unsigned)((M.n + kHeadOuts - 1) / kHeadOuts));
  hipLaunchKernelGGL(k_head_gemm, grid, dim3(256), 0, s, a, words, (const float *)zbuf);
  return hipGetLastError();
}

hipError_t launch_head(const Model &M, const float *x, const float *y, int64_t words, uint8_t *bits,
                       float *logits, bool lane_order, hipStream_t s) {
  if (words <= 0) return hipSuccess;
  if (lane_order && M.d != 64 && M.d != 128) return hipErrorInvalidValue;
  HeadArgs a{x, y, M.n, M.L, M.head_w1, M.head_wo, M.head_bo, M.head_b1, bits, logits};
  const size_t shm = sizeof(float) * (size_t)M.L;
  const dim3 grid((unsigned)words);
  switch (M.d) {
    case 32: hipLaunchKernelGGL((k_head<32, false>), grid, dim3(256), shm, s, a); break;
    case 64:
      if (lane_order) hipLaunchKernelGGL((k_head<64, true>), grid, dim3(256), shm, s, a);
      else hipLaunchKernelGGL((k_head<64, false>), grid, dim3(256), shm, s, a);
      break;
    case 128:
      if (lane_order) hipLaunchKernelGGL((k_head<128, true>), grid, dim3(256), shm, s, a);
      else hipLaunchKernelGGL((k_head<128, false>), grid, dim3(256), shm, s, a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// The largest dynamic LDS each kernel that takes it may use on the model's device, set once per
// model at create time (the launches only choose a size within it).
hipError_t set_layered_kernel_attributes(const Model &M) {
  const void *fns[] = {
      (const void *)k_qkv_attention<64, 8>,      (const void *)k_qkv_attention<128, 16>,
      (const void *)k_qkv_attention<128, 8>,     (const void *)k_qkv_attention<64, 16>,
      (const void *)k_qkv_attention<64, 8, true>, (const void *)k_qkv_attention<128, 16, true>,
      (const void *)k_qkv_attention<128, 8, true>,
      (const void *)k_qkv_attention_pair<128, false>, (const void *)k_qkv_attention_pair<128, true>,
      (const void *)k_qkv_attention_pair<128, true, true>,
      (const void *)k_qkv_attention_i16<128, 16>,
      (const void *)k_qkv_attention_i16<64, 16>, (const void *)k_qkv_attention_i16<64, 8>,
      (const void *)k_qkv_attention_i16<128, 8>, (const void *)k_qkv_attention_v16<64>,
      (const void *)k_qkv_attention_v16<128>,    (const void *)k_qkv_attention_split<128>,
      token_block_kernel<64, 0>(),  token_block_kernel<64, 1>(),  token_block_kernel<64, 2>(),
      token_block_kernel<64, 3>(),  token_block_kernel<64, 4>(),  token_block_kernel<64, 5>(),
      token_block_kernel<64, 6>(),  token_block_kernel<64, 7>(),  token_block_kernel<128, 0>(),
      token_block_kernel<128, 1>(), token_block_kernel<128, 2>(), token_block_kernel<128, 3>(),
      token_block_kernel<128, 4>(), token_block_kernel<128, 5>(), token_block_kernel<128, 6>(),
      token_block_kernel<128, 7>(),                   (const void *)k_embed_words<64>,
      (const void *)k_embed_words<128>};
  for (const void *f : fns) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)M.lds_max);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_word_quant(const Model &M, const float *x, int64_t words, int K, bool relu, int8_t *q, float *a,
                             hipStream_t s) {
  if (words <= 0) return hipSuccess;
  if (K % 32) return hipErrorInvalidValue;
  const int64_t per_word = (int64_t)M.L * K;
  const unsigned grid = (unsigned)std::min<int64_t>(words, (int64_t)M.cu_count * 8);
  if (relu) hipLaunchKernelGGL(k_word_quant<true>, dim3(grid), dim3(kWqThreads), 0, s, x, words, per_word, M.L, q, a);
  else hipLaunchKernelGGL(k_word_quant<false>, dim3(grid), dim3(kWqThreads), 0, s, x, words, per_word, M.L, q, a);
  return hipGetLastError();
}

hipError_t launch_ffn1_f32(const Model &M, int layer, const int8_t *x1q, const float *a1, int64_t rows, float *h,
                           hipStream_t s) {
  const LayerWeights &W = M.layer[layer];
  GemmArgs a = gemm_base(x1q, a1, W.ff1, rows);
  a.sq[0] = W.sq[4];
  a.bias = W.b_ff1;
  a.out_f = h;
  switch (M.d) {
    case 32: return run_gemm<32, 128, EPI_F32>(M, a, s);
    case 64: return run_gemm<64, 256, EPI_F32>(M, a, s);
    case 128: return run_gemm<128, 512, EPI_F32>(M, a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace aecct
