// Quantisation-aware training step of AECCT on the GPU: the second training phase of Section 6,
// in which the encoder's in-block linear maps are AAP linear layers (Section 4.1) over latent
// fp32 weights.  Forward with Eq. 1 ternarisation of the current weights and Eq. 2 absmax int8
// activations (both passing gradients straight through their rounding), the cross entropy of the
// multiplicative noise, and the backward pass to every parameter.  fp32 throughout; every
// reduction runs in a fixed order (split partial sums reduced in index order), so a step is
// deterministic.
//
// Layouts: activations row-major [rows][features] with row b * L + r for token r of word b;
// weights [in][out] as in the inference ABI.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "aecct_internal.h"
#include "device_common.h"

namespace aecct {
namespace train {

constexpr int kThreads = 256;

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// ------------------------------------------------------------------------------------------
// Eq. 1 on the current latent weights, one block per matrix: gamma = Percentile(|W|, 0.5) (the
// order statistics at floor(pos) and floor(pos) + 1 for pos = (count - 1) / 2, interpolated in
// double and rounded once to fp32), s = fp32(gamma * delta), T = RoundClip(W / fp32(s + eps),
// -1, 1) with rounding half to even (a zero denominator maps a weight to its sign).  The order
// statistics come from a radix selection over the bit patterns of |W| (non-negative floats order
// like their bits), one 8-bit digit per pass.
// ------------------------------------------------------------------------------------------
using AapJob = TrainAapJob;
constexpr int kAapThreads = 1024, kAapWaves = kAapThreads / 64;

// Bucket b's running total over the wave histograms, and the bucket holding the k-th key (k
// counted from 0 among the keys matching the current prefix) with k's rank inside it: wave 0
// scans the 256 buckets as four per lane.
__device__ void select_bucket(const uint32_t (*hist)[256], uint32_t k, uint32_t *pick) {
  if (threadIdx.x >= 64) return;
  const int lane = threadIdx.x;
  uint32_t c[4], t = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t v = 0;
    for (int w = 0; w < kAapWaves; ++w) v += hist[w][4 * lane + j];
    c[j] = v;
    t += v;
  }
  uint32_t incl = t;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t up = __shfl_up(incl, o, 64);
    if (lane >= o) incl += up;
  }
  const uint32_t excl = incl - t;
  if (excl <= k && k < incl) {
    uint32_t kk = k - excl;
    int j = 0;
    while (j < 3 && kk >= c[j]) kk -= c[j++];
    pick[0] = 4 * lane + j;
    pick[1] = kk;
  }
}

// The k-th smallest |w| (k from 0) as a bit pattern: non-negative floats order like their bits,
// so four passes pick its 8-bit digits from the most significant down, each pass counting the
// keys that match the digits found so far into per-wave histograms.
__device__ uint32_t radix_select(const float *w, int64_t count, uint32_t k, uint32_t (*hist)[256], uint32_t *pick) {
  uint32_t prefix = 0, mask = 0;
  uint32_t *flat = &hist[0][0];
  const int wave = threadIdx.x >> 6;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = threadIdx.x; b < kAapWaves * 256; b += kAapThreads) flat[b] = 0;
    __syncthreads();
    for (int64_t e = threadIdx.x; e < count; e += kAapThreads) {
      const uint32_t key = __float_as_uint(fabsf(w[e]));
      if ((key & mask) == prefix) atomicAdd(&hist[wave][(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    select_bucket(hist, k, pick);
    __syncthreads();
    prefix |= pick[0] << shift;
    mask |= 255u << shift;
    k = pick[1];
    __syncthreads();
  }
  return prefix;
}

__global__ __launch_bounds__(kAapThreads) void k_aap(TrainAapJobs jobs, float eps) {
  __shared__ uint32_t hist[kAapWaves][256];
  __shared__ uint32_t pick[2];
  __shared__ uint32_t wle[kAapWaves], wgt[kAapWaves];
  __shared__ float sden;
  const AapJob J = jobs.j[blockIdx.x];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint32_t lo = (uint32_t)((J.count - 1) / 2);
  const uint32_t a_lo = radix_select(J.w, J.count, lo, hist, pick);
  // the next order statistic: a_lo again if more than lo + 1 keys are <= a_lo, else the least
  // key above it
  uint32_t le = 0, gt = 0xffffffffu;
  for (int64_t e = threadIdx.x; e < J.count; e += kAapThreads) {
    const uint32_t key = __float_as_uint(fabsf(J.w[e]));
    if (key <= a_lo) ++le;
    else gt = min(gt, key);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    le += __shfl_xor(le, o, 64);
    gt = min(gt, (uint32_t)__shfl_xor(gt, o, 64));
  }
  if (lane == 0) {
    wle[wave] = le;
    wgt[wave] = gt;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t n_le = 0, g = 0xffffffffu;
    for (int w = 0; w < kAapWaves; ++w) {
      n_le += wle[w];
      g = min(g, wgt[w]);
    }
    const uint32_t a_hi = ((int64_t)lo + 1 >= J.count || n_le > lo + 1) ? a_lo : g;
    const double pos = 0.5 * (double)(J.count - 1);
    const double frac = pos - (double)lo;
    const double flo = (double)__uint_as_float(a_lo), fhi = (double)__uint_as_float(a_hi);
    const float gamma = (float)(flo + frac * (fhi - flo));
    const float s = gamma * J.delta[0];
    *J.gamma = gamma;
    *J.scale = s;
    sden = s + eps;
  }
  __syncthreads();
  const float den = sden;
  for (int64_t e = threadIdx.x; e < J.count; e += kAapThreads) {
    const float x = J.w[e];
    float r = den == 0.0f ? (x > 0.0f ? 1.0f : (x < 0.0f ? -1.0f : 0.0f)) : rintf(x / den);
    J.t[e] = fminf(1.0f, fmaxf(-1.0f, r));
  }
}

// ------------------------------------------------------------------------------------------
// Pre-processing and embedding (Section 3): t = [|y|, 1 - 2 s(y)], X = t E (+ P); one wavefront
// per token row.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_embed(const float *y, int64_t rows, int n, int L, int d,
                                                    const int32_t *chk_ptr, const int32_t *chk_idx, const float *E,
                                                    const float *P, float *x, float *tv) {
  const int64_t r = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  const int64_t w = r / L;
  const int i = (int)(r - w * L);
  const float *yw = y + w * n;
  float t;
  if (i < n) {
    t = fabsf(yw[i]);
  } else {
    int s = 0;
    for (int e = chk_ptr[i - n]; e < chk_ptr[i - n + 1]; ++e) s ^= yw[chk_idx[e]] < 0.0f ? 1 : 0;
    t = s ? -1.0f : 1.0f;
  }
  for (int c = lane; c < d; c += 64) x[r * d + c] = fmaf(t, E[(int64_t)i * d + c], P ? P[(int64_t)i * d + c] : 0.0f);
  if (lane == 0) tv[r] = t;
}

// Eq. 2 per token row and the value the codes stand for, q alpha / 127 (0 when alpha = 0); of
// max(x, 0) when RELU.  One wavefront per row.
template <bool RELU>
__global__ __launch_bounds__(kThreads) void k_quant_dequant(const float *x, int64_t rows, int K, float *xh) {
  const int64_t r = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  const float *xr = x + r * K;
  float a = 0.0f;
  constexpr int kHeld = 8;   // rows up to 512 wide are read whole before their maximum is formed
  if (K <= 64 * kHeld) {
    float v[kHeld];
#pragma unroll
    for (int u = 0; u < kHeld; ++u) v[u] = lane + 64 * u < K ? xr[lane + 64 * u] : 0.0f;
#pragma unroll
    for (int u = 0; u < kHeld; ++u) {
      if (RELU) v[u] = fmaxf(v[u], 0.0f);
      a = fmaxf(a, fabsf(v[u]));
    }
    a = wave_max(a);
    const float inv = inv127(a);
#pragma unroll
    for (int u = 0; u < kHeld; ++u) {
      const int c = lane + 64 * u;
      if (c < K) xh[r * K + c] = a == 0.0f ? 0.0f : (float)quant_code(v[u], inv) * a / 127.0f;
    }
    return;
  }
  for (int c = lane; c < K; c += 64) {
    const float v = RELU ? fmaxf(xr[c], 0.0f) : xr[c];
    a = fmaxf(a, fabsf(v));
  }
  a = wave_max(a);
  const float inv = inv127(a);
  for (int c = lane; c < K; c += 64) {
    const float v = RELU ? fmaxf(xr[c], 0.0f) : xr[c];
    xh[r * K + c] = a == 0.0f ? 0.0f : (float)quant_code(v, inv) * a / 127.0f;
  }
}

// ------------------------------------------------------------------------------------------
// fp32 GEMM: C[M][N] = beta C + scale (op(A) op(B)) + bias[N], op(A) = A [M][K] (lda) or, with TA,
// the transpose of A stored [K][M]; op(B) = B [K][N] (ldb) or, with TB, the transpose of B stored
// [N][K].  64 x 64 output tiles, 16-deep K steps through LDS, 4 x 4 outputs per thread, FMAs in
// ascending k.  With gridDim.z > 1 each z takes one contiguous k range and writes its raw sum to
// part[z][M][N]; k_gemm_reduce then adds the ranges in index order and applies the epilogue.
// ------------------------------------------------------------------------------------------
struct GemmF32 {
  const float *A, *B;
  float *C;
  int64_t M, N, K;
  int64_t lda, ldb, ldc;
  int64_t kchunk;
  const float *scale;   // device scalar or null (1)
  const float *bias;    // [N] or null
  int beta;             // 1: accumulate into C
  float *part;          // [splits][M][N] when split
};

template <bool TA, bool TB>
__global__ __launch_bounds__(kThreads) void k_gemm(GemmF32 g) {
  __shared__ float As[16][64 + 4];
  __shared__ float Bs[16][64 + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int64_t m0 = (int64_t)blockIdx.y * 64, n0 = (int64_t)blockIdx.x * 64;
  const int64_t kb = (int64_t)blockIdx.z * g.kchunk, ke = std::min<int64_t>(g.K, kb + g.kchunk);
  float acc[4][4] = {};
  for (int64_t k0 = kb; k0 < ke; k0 += 16) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + kThreads * u;
      int mm, kk;
      if (TA) { kk = idx >> 6; mm = idx & 63; } else { mm = idx >> 4; kk = idx & 15; }
      const int64_t gm = m0 + mm, gk = k0 + kk;
      float v = 0.0f;
      if (gm < g.M && gk < ke) v = TA ? g.A[gk * g.lda + gm] : g.A[gm * g.lda + gk];
      As[kk][mm] = v;
      int nn;
      if (TB) { nn = idx >> 4; kk = idx & 15; } else { kk = idx >> 6; nn = idx & 63; }
      const int64_t gn = n0 + nn, gk2 = k0 + kk;
      float w = 0.0f;
      if (gn < g.N && gk2 < ke) w = TB ? g.B[gn * g.ldb + gk2] : g.B[gk2 * g.ldb + gn];
      Bs[kk][nn] = w;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][4 * ty + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][4 * tx + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  const bool split = gridDim.z > 1;
  const float sc = g.scale ? *g.scale : 1.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t r = m0 + 4 * ty + i;
    if (r >= g.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t c = n0 + 4 * tx + j;
      if (c >= g.N) continue;
      if (split) {
        g.part[((int64_t)blockIdx.z * g.M + r) * g.N + c] = acc[i][j];
      } else {
        float v = sc * acc[i][j] + (g.bias ? g.bias[c] : 0.0f);
        if (g.beta) v += g.C[r * g.ldc + c];
        g.C[r * g.ldc + c] = v;
      }
    }
  }
}

// The same product on v_mfma_f32_16x16x4_f32 for operands whose contiguous dimension and leading
// dimensions are multiples of 4 floats (16-byte loads): blocks of BM x 128 outputs (BM = 128, or 64
// for short reductions, which then get twice the blocks), four wavefronts of BM / 2 x 64
// (BM / 32 x 4 MFMA tiles), k-steps of 32 staged through LDS, the next step's operands loaded into
// registers while the current one is multiplied.  LDS rows of BM + 16 and 144 floats put the four k
// rows an MFMA fragment reads 16 banks apart.  MFMA layout (lane l): A row l & 15 at k = l >> 4,
// B column l & 15 at k = l >> 4, D rows 4 (l >> 4) + i, column l & 15.
typedef float v4f __attribute__((ext_vector_type(4)));
constexpr int kMfTile = 128, kMfK = 32;

__device__ __forceinline__ float4 load4_if(const float *p, bool ok) {
  float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  if (ok) v = *(const float4 *)p;
  return v;
}

template <bool TA, bool TB, int BM>
__global__ __launch_bounds__(kThreads) void k_gemm_mfma(GemmF32 g) {
  constexpr int BN = kMfTile, AP = BM / 32, BP = BN / 32, TM = BM / 32;
  __shared__ __attribute__((aligned(16))) float As[kMfK][BM + 16];
  __shared__ __attribute__((aligned(16))) float Bs[kMfK][BN + 16];
  const float *__restrict__ A = g.A;
  const float *__restrict__ B = g.B;
  const int64_t M = g.M, N = g.N, lda = g.lda, ldb = g.ldb;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = (wave >> 1) * (BM / 2), wn = (wave & 1) * 64;
  const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
  const int64_t kb = (int64_t)blockIdx.z * g.kchunk, ke = std::min<int64_t>(g.K, kb + g.kchunk);
  // Thread t stages float4 number t + 256 u of each 32 x W operand tile (W = BM or 128).  Stored
  // k-major ([k][m] or [k][n]): k row t / (W / 4) + u 1024 / W, columns 4 (t mod W / 4) .. +3.
  // Stored with k contiguous: tile row (t >> 3) + 32 u, k offsets 4 (t & 7) .. +3.
  const int kmA_r = tid / (BM / 4), kmA_c = (tid % (BM / 4)) * 4, kmB_r = tid >> 5, kmB_c = (tid & 31) * 4;
  const int kc_r = tid >> 3, kc_k = (tid & 7) * 4;
  float4 ra[AP], rb[BP];
  v4f acc[TM][4];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
  const int fr = lane >> 4, fc = lane & 15;
  for (int64_t k0 = kb, first = 1; k0 < ke; k0 += kMfK, first = 0) {
    if (first) {
      // the first step's operands (later steps' were read during the previous step)
#pragma unroll
      for (int u = 0; u < AP; ++u) {
        if (TA) {
          const int64_t gk = k0 + kmA_r + u * (1024 / BM);
          ra[u] = load4_if(A + gk * lda + m0 + kmA_c, gk < ke && m0 + kmA_c < M);
        } else {
          const int64_t gm = m0 + kc_r + 32 * u;
          ra[u] = load4_if(A + gm * lda + k0 + kc_k, gm < M && k0 + kc_k < ke);
        }
      }
#pragma unroll
      for (int u = 0; u < BP; ++u) {
        if (TB) {
          const int64_t gn = n0 + kc_r + 32 * u;
          rb[u] = load4_if(B + gn * ldb + k0 + kc_k, gn < N && k0 + kc_k < ke);
        } else {
          const int64_t gk = k0 + kmB_r + 8 * u;
          rb[u] = load4_if(B + gk * ldb + n0 + kmB_c, gk < ke && n0 + kmB_c < N);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < AP; ++u) {
      if (TA) {
        *(float4 *)&As[kmA_r + u * (1024 / BM)][kmA_c] = ra[u];
      } else {
        const int mm = kc_r + 32 * u;
        As[kc_k][mm] = ra[u].x; As[kc_k + 1][mm] = ra[u].y; As[kc_k + 2][mm] = ra[u].z; As[kc_k + 3][mm] = ra[u].w;
      }
    }
#pragma unroll
    for (int u = 0; u < BP; ++u) {
      if (TB) {
        const int nn = kc_r + 32 * u;
        Bs[kc_k][nn] = rb[u].x; Bs[kc_k + 1][nn] = rb[u].y; Bs[kc_k + 2][nn] = rb[u].z; Bs[kc_k + 3][nn] = rb[u].w;
      } else {
        *(float4 *)&Bs[kmB_r + 8 * u][kmB_c] = rb[u];
      }
    }
    __syncthreads();
    const int64_t k1 = k0 + kMfK;
    if (k1 < ke) {
#pragma unroll
      for (int u = 0; u < AP; ++u) {
        if (TA) {
          const int64_t gk = k1 + kmA_r + u * (1024 / BM);
          ra[u] = load4_if(A + gk * lda + m0 + kmA_c, gk < ke && m0 + kmA_c < M);
        } else {
          const int64_t gm = m0 + kc_r + 32 * u;
          ra[u] = load4_if(A + gm * lda + k1 + kc_k, gm < M && k1 + kc_k < ke);
        }
      }
#pragma unroll
      for (int u = 0; u < BP; ++u) {
        if (TB) {
          const int64_t gn = n0 + kc_r + 32 * u;
          rb[u] = load4_if(B + gn * ldb + k1 + kc_k, gn < N && k1 + kc_k < ke);
        } else {
          const int64_t gk = k1 + kmB_r + 8 * u;
          rb[u] = load4_if(B + gk * ldb + n0 + kmB_c, gk < ke && n0 + kmB_c < N);
        }
      }
    }
#pragma unroll
    for (int ks = 0; ks < kMfK / 4; ++ks) {
      float av[TM], bv[4];
#pragma unroll
      for (int t = 0; t < TM; ++t) av[t] = As[4 * ks + fr][wm + 16 * t + fc];
#pragma unroll
      for (int t = 0; t < 4; ++t) bv[t] = Bs[4 * ks + fr][wn + 16 * t + fc];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  // split partial sums raw into their slice of part, else scale, bias and the optional C
  const bool split = gridDim.z > 1;
  float *const P = split ? g.part + (int64_t)blockIdx.z * M * N : g.C;
  const int64_t ld = split ? N : g.ldc;
  const float sc = (!split && g.scale) ? *g.scale : 1.0f;
  const bool beta = !split && g.beta;
  const float *bias = split ? nullptr : g.bias;
  const bool full = m0 + BM <= M && n0 + BN <= N;
  float bj[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t c = n0 + wn + 16 * j + fc;
    bj[j] = (bias && c < N) ? bias[c] : 0.0f;
  }
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t r = m0 + wm + 16 * i + 4 * fr + v;
      if (!full && r >= M) continue;
      float *prow = P + r * ld + n0 + wn + fc;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (!full && n0 + wn + 16 * j + fc >= N) continue;
        float o = sc * acc[i][j][v] + bj[j];
        if (beta) o += prow[16 * j];
        prow[16 * j] = o;
      }
    }
}

// ------------------------------------------------------------------------------------------
// Products with a ternary operand: C[M][N] = beta C + scale (A B) + bias[N] where B holds only
// -1, 0, +1 (Eq. 1's T, or its transpose) and A is fp32.  Each fp32 a splits exactly into three
// bf16 parts, a = hi + mid + lo (hi the leading 8 significant bits by truncation, mid the next 8,
// lo the remaining at most 8), each part times a ternary entry is exact, and the three
// v_mfma_f32_16x16x32_bf16 products accumulate in fp32: the result is an fp32-accumulated sum of
// exact products, as in the fp32 kernels, at the bf16 matrix rate.  B comes pre-packed as bf16 MFMA
// B fragments (k_pack_tern).  A wave computes 16 rows x 16 NJ columns, a block four waves.
// ------------------------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Up to three ternary matrices in one product, either side by side in C's columns (segments of
// seg_n columns: the query, key and value maps over one read of their shared input) or one after
// another along k (segments of kseg k-steps of A's row: the input gradient summed over the three
// maps from the packed [rows][3 d] gradient).  Segment s has its own fragments and scale, a column
// segment its own bias; C = D + sum_s scale_s (A_s T_s) + bias, D an optional addend laid out like C
// (C itself to accumulate).
struct GemmTern {
  const float *A;
  const uint4 *B[3];       // fragment (nt, kt) at (nt * kt_s + kt) * 64, kt_s the segment's k-steps:
                           // lane l holds column 16 nt + (l & 15), k = 32 kt + 8 (l >> 4) + e, bf16 e = 0..7
  float *C;
  const float *D;
  int64_t M, N, K, lda, ldc;
  const float *scale[3];   // device scalar or null (1)
  const float *bias[3];    // [seg_n] or null
  int64_t seg_n;           // a multiple of the block's 16 NJ columns
  int kseg;                // k-steps per k segment (K / 32 when there is one)
};

template <typename T>
__device__ __forceinline__ T pick3(const T (&v)[3], int i) {   // a selected kernel argument, no indexing
  return i == 0 ? v[0] : (i == 1 ? v[1] : v[2]);
}

// Ternary matrix T [R][C] (fp32 -1 / 0 / +1, row-major) as bf16 B fragments of B = T (k = row,
// n = column) or, with trans, B = T^T (k = column, n = row); one job per blockIdx.y.
__global__ __launch_bounds__(kThreads) void k_pack_tern(TernPackJobs jobs) {
  const TernPackJob &J = jobs.j[blockIdx.y];
  const float *T = J.T;
  const int R = J.R, Cc = J.C, trans = J.trans;
  uint4 *out = (uint4 *)J.out;
  const int K = trans ? Cc : R, N = trans ? R : Cc, KT = K / 32;
  const int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (u >= (int64_t)(N / 16) * KT * 64) return;
  const int l = (int)(u & 63), f = (int)(u >> 6), nt = f / KT, kt = f - nt * KT;
  const int n = 16 * nt + (l & 15), k0 = 32 * kt + 8 * (l >> 4);
  uint32_t h[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float t = trans ? T[(int64_t)n * Cc + k0 + e] : T[(int64_t)(k0 + e) * Cc + n];
    h[e] = t > 0.0f ? 0x3F80u : (t < 0.0f ? 0xBF80u : 0u);   // bf16 of +1, -1, 0
  }
  out[u] = make_uint4(h[0] | h[1] << 16, h[2] | h[3] << 16, h[4] | h[5] << 16, h[6] | h[7] << 16);
}

// the bf16 bit patterns of eight fp32 values that are exact in bf16 (low 16 bits zero)
__device__ __forceinline__ bf16x8 bf16_hi8(const float (&v)[8]) {
  uint4 w;
  w.x = __builtin_amdgcn_perm(__builtin_bit_cast(uint32_t, v[1]), __builtin_bit_cast(uint32_t, v[0]), 0x07060302u);
  w.y = __builtin_amdgcn_perm(__builtin_bit_cast(uint32_t, v[3]), __builtin_bit_cast(uint32_t, v[2]), 0x07060302u);
  w.z = __builtin_amdgcn_perm(__builtin_bit_cast(uint32_t, v[5]), __builtin_bit_cast(uint32_t, v[4]), 0x07060302u);
  w.w = __builtin_amdgcn_perm(__builtin_bit_cast(uint32_t, v[7]), __builtin_bit_cast(uint32_t, v[6]), 0x07060302u);
  return __builtin_bit_cast(bf16x8, w);
}

// the three bf16 parts of eight fp32 values as MFMA operands
__device__ __forceinline__ void split_bf16x3(const float4 &x0, const float4 &x1, bf16x8 &ph, bf16x8 &pm, bf16x8 &pl) {
  const float a[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
  float hi[8], mid[8], lo[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    hi[e] = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, a[e]) & 0xFFFF0000u);
    const float rm = a[e] - hi[e];
    mid[e] = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, rm) & 0xFFFF0000u);
    lo[e] = rm - mid[e];
  }
  ph = bf16_hi8(hi);
  pm = bf16_hi8(mid);
  pl = bf16_hi8(lo);
}

// The MFMA takes the ternary fragment as its first operand and A's as its second, so it forms the
// transposed tile: lane (col, grp) ends with row 16 t + col, columns 16 j + 4 grp .. + 3 of C, one
// 16-byte store (and, with beta, one 16-byte load) per tile.  Both operands of k-step kt + S - 1 are
// loaded before step kt is computed, from a ring of S register slots: the vector-memory counter
// retires loads in issue order, so a B fragment loaded just before its use would also wait for
// every A prefetch issued ahead of it.  C goes out with ordinary stores: the next kernel reads it,
// partly from the caches (nontemporal stores measured slower over a training step).
template <int NJ, int S>
__global__ __launch_bounds__(kThreads) void k_gemm_tern(GemmTern g) {
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, col = l & 15, grp = l >> 4;
  const int64_t m0 = (int64_t)blockIdx.y * 64 + 16 * wave, n0 = (int64_t)blockIdx.x * (16 * NJ);
  const int sg = (int)(n0 / g.seg_n);
  const int64_t ns = n0 - sg * g.seg_n;   // the block's first column inside its segment
  const int KT = (int)(g.K / 32), ks = g.kseg;
  const int64_t r = m0 + col;
  const float *arow = g.A + (r < g.M ? r : g.M - 1) * g.lda + 8 * grp;   // rows past M: a copy, never stored
  f32x4 acc[NJ];
  float4 o[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    acc[j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    o[j] = float4{0.0f, 0.0f, 0.0f, 0.0f};
  }
  float4 a[S][2];
  uint4 b[S][NJ];
  auto issue = [&](int kt, float4 (&as)[2], uint4 (&bs)[NJ]) {
    const int s = kt / ks;   // the k segment (0 with one)
    const uint4 *bcol = pick3(g.B, sg + s) + (ns / 16) * ks * 64 + l;
#pragma unroll
    for (int j = 0; j < NJ; ++j) bs[j] = bcol[(j * ks + kt - s * ks) * 64];
    as[0] = *(const float4 *)(arow + 32 * kt);
    as[1] = *(const float4 *)(arow + 32 * kt + 4);
  };
  int kend = ks;   // the current k segment ends before step kend
#pragma unroll
  for (int s = 0; s < S - 1; ++s)
    if (s < KT) issue(s, a[s], b[s]);
  for (int k0 = 0; k0 < KT; k0 += S) {
#pragma unroll
    for (int s = 0; s < S; ++s) {   // step k0 + s sits in slot s
      const int kt = k0 + s;
      if (kt >= KT) break;
      if (kt + S - 1 < KT) issue(kt + S - 1, a[(s + S - 1) % S], b[(s + S - 1) % S]);
      bf16x8 ph, pm, pl;
      split_bf16x3(a[s][0], a[s][1], ph, pm, pl);
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const bf16x8 bb = __builtin_bit_cast(bf16x8, b[s][j]);
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bb, pl, acc[j], 0, 0, 0);
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bb, pm, acc[j], 0, 0, 0);
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bb, ph, acc[j], 0, 0, 0);
      }
      if (kt + 1 == kend) {   // a k segment's products, scaled, into o
        const float *sp = pick3(g.scale, sg + kt / ks);
        const float sc = sp ? *sp : 1.0f;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          o[j].x += sc * acc[j][0];
          o[j].y += sc * acc[j][1];
          o[j].z += sc * acc[j][2];
          o[j].w += sc * acc[j][3];
          acc[j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        }
        kend += ks;
      }
    }
  }
  if (r >= g.M) return;
  const float *bias = pick3(g.bias, sg);
  if (bias) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const float4 bj = *(const float4 *)(bias + ns + 16 * j + 4 * grp);
      o[j].x += bj.x;
      o[j].y += bj.y;
      o[j].z += bj.z;
      o[j].w += bj.w;
    }
  }
  float *crow = g.C + r * g.ldc + n0 + 4 * grp;
  const float *drow = g.D ? g.D + r * g.ldc + n0 + 4 * grp : nullptr;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    float4 u = o[j];
    if (drow) {
      const float4 dv = *(const float4 *)(drow + 16 * j);
      u.x += dv.x;
      u.y += dv.y;
      u.z += dv.z;
      u.w += dv.w;
    }
    *(float4 *)(crow + 16 * j) = u;
  }
}

// Split-k partial products summed in a fixed order: a block covers 64 outputs, its four lanes per
// output sum the splits z = lane, lane + 4, ... and are added in lane order.
__global__ __launch_bounds__(kThreads) void k_gemm_reduce(GemmF32 g, int splits) {
  __shared__ float red[4][64];
  const int cl = threadIdx.x & 63, rl = threadIdx.x >> 6;
  const int64_t e = (int64_t)blockIdx.x * 64 + cl, MN = g.M * g.N;
  float s0 = 0.0f, s1 = 0.0f;
  if (e < MN) {
    int z = rl;
    for (; z + 4 < splits; z += 8) {
      s0 += g.part[(int64_t)z * MN + e];
      s1 += g.part[(int64_t)(z + 4) * MN + e];
    }
    if (z < splits) s0 += g.part[(int64_t)z * MN + e];
  }
  red[rl][cl] = s0 + s1;
  __syncthreads();
  if (rl != 0 || e >= MN) return;
  const float s = ((red[0][cl] + red[1][cl]) + red[2][cl]) + red[3][cl];
  const int64_t r = e / g.N, c = e - r * g.N;
  float v = (g.scale ? *g.scale : 1.0f) * s + (g.bias ? g.bias[c] : 0.0f);
  if (g.beta) v += g.C[r * g.ldc + c];
  g.C[r * g.ldc + c] = v;
}

// ------------------------------------------------------------------------------------------
// Head-partitioned attention (Section 4.2) of the training step: one thread per (row, head) over
// the row's neighbour list (first ring for heads below h_f, else the second-ring list, which
// holds the union of both rings under CASA); natural-base softmax of q.k / sqrt(d_h) with the
// maximum subtracted.  Forward stores O and the row's log-sum-exp; the backward recomputes
// p_ij = exp(s_ij - lse_i).  The masks are symmetric, so the key and value gradients are gathered
// per key row over its own list, without atomics.
// ------------------------------------------------------------------------------------------
using AttnT = TrainAttn;

// Thread gid to (row, head): the first-ring heads of every row first (row-major, a row's h_f heads
// on adjacent lanes), then the second-ring heads, so that a wavefront walks one kind of list and
// its lanes run loops of similar length (with both kinds in one wavefront the first-ring lanes idled
// through the longer second-ring lists), while a row's heads of one kind still read adjacent
// stretches of each neighbour's row.
__device__ __forceinline__ void attn_row_head(const AttnT &p, int64_t gid, int64_t &row, int &h) {
  const int64_t n1 = p.rows * p.hf;
  if (gid < n1) {
    row = gid / p.hf;
    h = (int)(gid - row * p.hf);
  } else {
    const int hs = p.heads - p.hf;
    const int64_t g2 = gid - n1;
    row = g2 / hs;
    h = p.hf + (int)(g2 - row * hs);
  }
}

template <int DH>
__device__ __forceinline__ float dot_dh(const float *a, const float *b) {
  float s = a[0] * b[0];
#pragma unroll
  for (int t = 1; t < DH; ++t) s = fmaf(a[t], b[t], s);
  return s;
}

template <int DH>
__global__ __launch_bounds__(kThreads) void k_attn_fwd(AttnT p) {
  const int64_t gid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (gid >= p.rows * p.heads) return;
  int64_t row;
  int h;
  attn_row_head(p, gid, row, h);
  const int64_t base = (row / p.L) * p.L;
  const int i = (int)(row - base);
  const int32_t *ptr = h < p.hf ? p.m1_ptr : p.m2_ptr, *idx = h < p.hf ? p.m1_idx : p.m2_idx;
  const int d = p.d, ld = 3 * d;
  const float kappa = 1.0f / sqrtf((float)DH);
  float q[DH];
#pragma unroll
  for (int t = 0; t < DH; ++t) q[t] = p.qkv[row * ld + h * DH + t];
  // one pass with a running maximum: when a score raises it, the sum and the accumulated values so
  // far are rescaled by exp(old - new) (each key read once instead of once for the maximum and once
  // for the weights)
  float mu = -INFINITY, S = 0.0f, acc[DH] = {};
  for (int e = ptr[i]; e < ptr[i + 1]; ++e) {
    const int64_t j = base + idx[e];
    const float s = dot_dh<DH>(q, p.qkv + j * ld + d + h * DH) * kappa;
    if (s > mu) {
      const float c = expf(mu - s);   // 0 at the first key
      S *= c;
#pragma unroll
      for (int t = 0; t < DH; ++t) acc[t] *= c;
      mu = s;
    }
    const float pe = expf(s - mu);
    S += pe;
#pragma unroll
    for (int t = 0; t < DH; ++t) acc[t] = fmaf(pe, p.qkv[j * ld + 2 * d + h * DH + t], acc[t]);
  }
#pragma unroll
  for (int t = 0; t < DH; ++t) p.o[row * d + h * DH + t] = acc[t] / S;
  p.lse[row * p.heads + h] = mu + logf(S);
}

template <int DH>
__global__ __launch_bounds__(kThreads) void k_attn_bwd_q(AttnT p) {
  const int64_t gid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (gid >= p.rows * p.heads) return;
  int64_t row;
  int h;
  attn_row_head(p, gid, row, h);
  const int64_t base = (row / p.L) * p.L;
  const int i = (int)(row - base);
  const int32_t *ptr = h < p.hf ? p.m1_ptr : p.m2_ptr, *idx = h < p.hf ? p.m1_idx : p.m2_idx;
  const int d = p.d, ld = 3 * d;
  const float kappa = 1.0f / sqrtf((float)DH);
  float q[DH], go[DH], dq[DH] = {};
#pragma unroll
  for (int t = 0; t < DH; ++t) {
    q[t] = p.qkv[row * ld + h * DH + t];
    go[t] = p.dout[row * d + h * DH + t];
  }
  const float D = dot_dh<DH>(go, p.o + row * d + h * DH);
  const float lse = p.lse[row * p.heads + h];
  for (int e = ptr[i]; e < ptr[i + 1]; ++e) {
    const int64_t j = base + idx[e];
    const float *kj = p.qkv + j * ld + d + h * DH;
    const float pij = expf(dot_dh<DH>(q, kj) * kappa - lse);
    const float ds = pij * (dot_dh<DH>(go, p.qkv + j * ld + 2 * d + h * DH) - D) * kappa;
#pragma unroll
    for (int t = 0; t < DH; ++t) dq[t] = fmaf(ds, kj[t], dq[t]);
  }
#pragma unroll
  for (int t = 0; t < DH; ++t) p.dqkv[row * ld + h * DH + t] = dq[t];
  p.Dv[row * p.heads + h] = D;
}

template <int DH>
__global__ __launch_bounds__(kThreads) void k_attn_bwd_kv(AttnT p) {
  const int64_t gid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (gid >= p.rows * p.heads) return;
  int64_t row;   // the key / value row j
  int h;
  attn_row_head(p, gid, row, h);
  const int64_t base = (row / p.L) * p.L;
  const int j = (int)(row - base);
  const int32_t *ptr = h < p.hf ? p.m1_ptr : p.m2_ptr, *idx = h < p.hf ? p.m1_idx : p.m2_idx;
  const int d = p.d, ld = 3 * d;
  const float kappa = 1.0f / sqrtf((float)DH);
  float k[DH], v[DH], dk[DH] = {}, dv[DH] = {};
#pragma unroll
  for (int t = 0; t < DH; ++t) {
    k[t] = p.qkv[row * ld + d + h * DH + t];
    v[t] = p.qkv[row * ld + 2 * d + h * DH + t];
  }
  for (int e = ptr[j]; e < ptr[j + 1]; ++e) {    // rows i whose list holds j (symmetric masks)
    const int64_t i = base + idx[e];
    const float *qi = p.qkv + i * ld + h * DH;
    const float *gi = p.dout + i * d + h * DH;
    const float pij = expf(dot_dh<DH>(qi, k) * kappa - p.lse[i * p.heads + h]);
    const float ds = pij * (dot_dh<DH>(gi, v) - p.Dv[i * p.heads + h]) * kappa;
#pragma unroll
    for (int t = 0; t < DH; ++t) {
      dv[t] = fmaf(pij, gi[t], dv[t]);
      dk[t] = fmaf(ds, qi[t], dk[t]);
    }
  }
#pragma unroll
  for (int t = 0; t < DH; ++t) {
    p.dqkv[row * ld + d + h * DH + t] = dk[t];
    p.dqkv[row * ld + 2 * d + h * DH + t] = dv[t];
  }
}

// ------------------------------------------------------------------------------------------
// LayerNorm of the Post-LN block (Section 6), one wavefront per row: forward of R = a + b, keeping
// the normalised row xn and 1 / sqrt(var + eps); backward dR = rho (dxn - mean dxn - xn mean(dxn
// xn)) with dxn = dy g.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_ln_fwd(const float *a, const float *b, int64_t rows, int d,
                                                     const float *g, const float *beta, float eps, float *out,
                                                     float *xn, float *rho, float *xh) {
  const int64_t r = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  float v[2], s = 0.0f;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int c = lane + 64 * u;
    v[u] = c < d ? a[r * d + c] + b[r * d + c] : 0.0f;
    s += v[u];
  }
  const float mean = wave_sum(s) / (float)d;
  float q = 0.0f;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int c = lane + 64 * u;
    if (c < d) q = fmaf(v[u] - mean, v[u] - mean, q);
  }
  const float rh = 1.0f / sqrtf(wave_sum(q) / (float)d + eps);
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int c = lane + 64 * u;
    if (c >= d) continue;
    const float x = (v[u] - mean) * rh;
    xn[r * d + c] = x;
    v[u] = fmaf(x, g[c], beta[c]);
    out[r * d + c] = v[u];
  }
  if (lane == 0) rho[r] = rh;
  if (!xh) return;
  // the output row's Eq. 2 codes and their values, as k_quant_dequant forms them from out
  float am = 0.0f;
#pragma unroll
  for (int u = 0; u < 2; ++u)
    if (lane + 64 * u < d) am = fmaxf(am, fabsf(v[u]));
  am = wave_max(am);
  const float inv = inv127(am);
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int c = lane + 64 * u;
    if (c < d) xh[r * d + c] = am == 0.0f ? 0.0f : (float)quant_code(v[u], inv) * am / 127.0f;
  }
}

__global__ __launch_bounds__(kThreads) void k_ln_bwd(const float *dy, const float *g, const float *xn,
                                                     const float *rho, int64_t rows, int d, float *dR) {
  const int64_t r = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  float dx[2], x[2], s1 = 0.0f, s2 = 0.0f;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int c = lane + 64 * u;
    dx[u] = c < d ? dy[r * d + c] * g[c] : 0.0f;
    x[u] = c < d ? xn[r * d + c] : 0.0f;
    s1 += dx[u];
    s2 = fmaf(dx[u], x[u], s2);
  }
  const float m1 = wave_sum(s1) / (float)d, m2 = wave_sum(s2) / (float)d;
  const float rh = rho[r];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int c = lane + 64 * u;
    if (c < d) dR[r * d + c] = rh * (dx[u] - m1 - x[u] * m2);
  }
}

// ------------------------------------------------------------------------------------------
// Column sums over rows, deterministic in two passes: v(r, c) = A[r][c] (x B[r][c]) (x w[r]) summed
// over r for each of A's C columns.  With dual (B given) each column also sums A alone, as column
// C + c of the result.  Result column c goes to o[c / seg][c % seg] (several bias vectors from one
// pass over a packed matrix, or the two sums of the dual form to two vectors).  A block covers cw
// columns (a power of two up to 64) with 256 / cw row lanes; lane l of a block sums the rows l,
// l + lanes, ... of its chunk (four interleaved partial sums; the factors present and the dual
// form are template parameters, as a run-time test between one row's loads and the next row's
// held each load until the previous one had landed), the lanes are combined by a fixed tree in LDS.  Pass one writes a
// partial row per chunk, pass two sums the partial rows with the same kernel.
// ------------------------------------------------------------------------------------------
struct ColOut {
  float *o[3];
  int seg;
  int64_t ld;   // distance between the rows of partial sums (pass one); 0 for the final sums
};

template <bool HB, bool HW, bool DUAL>
__global__ __launch_bounds__(kThreads) void k_colsum(const float *A, int64_t lda, const float *Bm, const float *w,
                                                     int64_t rows, int C, int cw_log2, int64_t chunk, ColOut out,
                                                     int accumulate) {
  constexpr int nv = DUAL ? 2 : 1;
  __shared__ float red[nv][kThreads];
  const int cw = 1 << cw_log2, lanes = kThreads >> cw_log2;
  const int cl = threadIdx.x & (cw - 1), rl = threadIdx.x >> cw_log2;
  const int c = blockIdx.x * cw + cl;
  const int64_t r0 = (int64_t)blockIdx.y * chunk, r1 = std::min<int64_t>(rows, r0 + chunk);
  float s[nv][4] = {};
  auto add = [&](int k, int64_t r) {
    const float a = A[r * lda + c];
    float v = a;
    if (HB) v *= Bm[r * C + c];
    if (HW) v *= w[r];
    s[0][k] += v;
    if (DUAL) s[nv - 1][k] += a;
  };
  if (c < C) {
    int64_t r = r0 + rl;
    for (; r + 3 * lanes < r1; r += 4 * lanes) {
      add(0, r);
      add(1, r + lanes);
      add(2, r + 2 * lanes);
      add(3, r + 3 * lanes);
    }
    for (; r < r1; r += lanes) add(0, r);
  }
#pragma unroll
  for (int k = 0; k < nv; ++k) red[k][threadIdx.x] = (s[k][0] + s[k][1]) + (s[k][2] + s[k][3]);
  __syncthreads();
  for (int st = lanes >> 1; st > 0; st >>= 1) {
    if (rl < st)
#pragma unroll
      for (int k = 0; k < nv; ++k) red[k][threadIdx.x] += red[k][threadIdx.x + (st << cw_log2)];
    __syncthreads();
  }
  if (rl == 0 && c < C)
#pragma unroll
    for (int k = 0; k < nv; ++k) {
      const int cc = c + k * C;
      float *o = out.o[cc / out.seg] + (int64_t)blockIdx.y * out.ld + cc % out.seg;
      *o = accumulate ? *o + red[k][threadIdx.x] : red[k][threadIdx.x];
    }
}

// ------------------------------------------------------------------------------------------
// Small elementwise steps.
// ------------------------------------------------------------------------------------------
// ReLU backward (the Eq. 2 code of the hidden row passes the gradient straight through)
__global__ __launch_bounds__(kThreads) void k_relu_bwd(float *dg, const float *f, int64_t count) {
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e < count && !(f[e] > 0.0f)) dg[e] = 0.0f;
}
// the same over 16-byte groups, every group written whole (zeroing only the dropped elements left
// partly written lines behind)
__global__ __launch_bounds__(kThreads) void k_relu_bwd4(float4 *dg, const float4 *f, int64_t count4) {
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e >= count4) return;
  const float4 fv = f[e];
  float4 g = dg[e];
  g.x = fv.x > 0.0f ? g.x : 0.0f;
  g.y = fv.y > 0.0f ? g.y : 0.0f;
  g.z = fv.z > 0.0f ? g.z : 0.0f;
  g.w = fv.w > 0.0f ? g.w : 0.0f;
  dg[e] = g;
}

// z = X w1 + b1 per row (Section 3 head, W_{d->1}); one wavefront per row
__global__ __launch_bounds__(kThreads) void k_rowdot(const float *x, int64_t rows, int d, const float *w1,
                                                     const float *b1, float *z) {
  const int64_t r = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  float s = 0.0f;
  for (int c = lane; c < d; c += 64) s = fmaf(x[r * d + c], w1[c], s);
  s = wave_sum(s);
  if (lane == 0) z[r] = s + b1[0];
}

// dX = dz w1^T (the head's W_{d->1} backward)
__global__ __launch_bounds__(kThreads) void k_outer(const float *dz, int64_t rows, const float *w1, int d, float *dx) {
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e >= rows * d) return;
  dx[e] = dz[e / d] * w1[e % d];
}

// Loss of the multiplicative noise (Section 6): target z = [y x_s < 0] (x_s = +1 if xs is null),
// l = softplus(-f) + z f = BCE-with-logits(-f, z); df = (z - sigmoid(-f)) / count.  Per-block
// sums of l in part[blockIdx].
__global__ __launch_bounds__(kThreads) void k_loss(const float *f, const float *y, const float *xs, int64_t count,
                                                   float inv_count, float *df, float *part) {
  __shared__ float red[kThreads / 64];
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  float l = 0.0f;
  if (e < count) {
    const float fv = f[e];
    const float sg = xs ? xs[e] : 1.0f;
    const float z = y[e] * sg < 0.0f ? 1.0f : 0.0f;
    const float nf = -fv;
    l = fmaxf(nf, 0.0f) + log1pf(expf(-fabsf(nf))) + z * fv;
    const float sig = 1.0f / (1.0f + expf(fv));          // sigmoid(-f)
    df[e] = (z - sig) * inv_count;
  }
  l = wave_sum(l);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = l;
  __syncthreads();
  if (threadIdx.x == 0) {
    float s = 0.0f;
    for (int k = 0; k < kThreads / 64; ++k) s += red[k];
    part[blockIdx.x] = s;
  }
}

__global__ __launch_bounds__(64) void k_loss_final(const float *part, int n, float inv_count, float *loss) {
  if (threadIdx.x != 0) return;
  float s = 0.0f;
  for (int k = 0; k < n; ++k) s += part[k];
  *loss = s * inv_count;
}

// dE[i][c] = sum_b t[b L + i] dX[b L + i][c] (the embedding is t_i E_i)
__global__ __launch_bounds__(kThreads) void k_embed_grad(const float *t, const float *dx, int64_t words, int L, int d,
                                                         float *de) {
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e >= (int64_t)L * d) return;
  const int64_t i = e / d, c = e - i * d;
  float s = 0.0f;
  for (int64_t b = 0; b < words; ++b) s = fmaf(t[b * L + i], dx[(b * L + i) * d + c], s);
  de[e] = s;
}

// The straight-through Eq. 1 gradients of one matrix, one block per matrix: G = Xh^T dY arrives in
// dW; dW = G s / (s + eps) and d delta = gamma sum(G T) - s gamma / (s + eps)^2 sum(G W).
using DeltaJob = TrainDeltaJob;

__global__ __launch_bounds__(kAapThreads) void k_delta_grad(TrainDeltaJobs jobs, float eps) {
  __shared__ float r1[kAapWaves], r2[kAapWaves];
  const DeltaJob J = jobs.j[blockIdx.x];
  const float s = *J.scale, gamma = *J.gamma;
  const float fac = s / (s + eps);
  float a[2] = {0.0f, 0.0f}, b[2] = {0.0f, 0.0f};
  int64_t e = threadIdx.x;
  for (; e + kAapThreads < J.count; e += 2 * kAapThreads) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t x = e + u * kAapThreads;
      const float gv = J.dw[x];
      a[u] = fmaf(gv, J.t[x], a[u]);
      b[u] = fmaf(gv, J.w[x], b[u]);
      J.dw[x] = gv * fac;
    }
  }
  if (e < J.count) {
    const float gv = J.dw[e];
    a[0] = fmaf(gv, J.t[e], a[0]);
    b[0] = fmaf(gv, J.w[e], b[0]);
    J.dw[e] = gv * fac;
  }
  const float sa_ = wave_sum(a[0] + a[1]), sb_ = wave_sum(b[0] + b[1]);
  if ((threadIdx.x & 63) == 0) {
    r1[threadIdx.x >> 6] = sa_;
    r2[threadIdx.x >> 6] = sb_;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float sa = 0.0f, sb = 0.0f;
    for (int k = 0; k < kAapWaves; ++k) {
      sa += r1[k];
      sb += r2[k];
    }
    const float den = s + eps;
    *J.ddelta = gamma * sa - s * gamma / (den * den) * sb;
  }
}

}  // namespace train

// ------------------------------------------------------------------------------------------
// launch helpers (declared in aecct_internal.h)
// ------------------------------------------------------------------------------------------
namespace {
inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }
}

hipError_t train_aap(const TrainAapJobs &jobs, float eps, hipStream_t s) {
  if (jobs.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(train::k_aap, dim3((unsigned)jobs.n), dim3(train::kAapThreads), 0, s, jobs, eps);
  return hipGetLastError();
}

hipError_t train_delta_grad(const TrainDeltaJobs &jobs, float eps, hipStream_t s) {
  if (jobs.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(train::k_delta_grad, dim3((unsigned)jobs.n), dim3(train::kAapThreads), 0, s, jobs, eps);
  return hipGetLastError();
}

hipError_t train_embed(const float *y, int64_t rows, int n, int L, int d, const int32_t *chk_ptr,
                       const int32_t *chk_idx, const float *E, const float *P, float *x, float *t, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(train::k_embed, dim3(blocks_for(rows, 4)), dim3(train::kThreads), 0, s, y, rows, n, L, d, chk_ptr,
                     chk_idx, E, P, x, t);
  return hipGetLastError();
}

hipError_t train_quant(const float *x, int64_t rows, int K, bool relu, float *xh, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (relu) hipLaunchKernelGGL(train::k_quant_dequant<true>, dim3(blocks_for(rows, 4)), dim3(train::kThreads), 0, s, x, rows, K, xh);
  else hipLaunchKernelGGL(train::k_quant_dequant<false>, dim3(blocks_for(rows, 4)), dim3(train::kThreads), 0, s, x, rows, K, xh);
  return hipGetLastError();
}

hipError_t train_gemm(bool ta, bool tb, const float *A, int64_t lda, const float *B, int64_t ldb, float *C, int64_t ldc,
                      int64_t M, int64_t N, int64_t K, const float *scale, const float *bias, bool accumulate,
                      float *part, int64_t part_floats, int cu_count, hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  train::GemmF32 g{A, B, C, M, N, K, lda, ldb, ldc, K, scale, bias, accumulate ? 1 : 0, part};
  // the MFMA kernel reads 16-byte vectors along each operand's contiguous dimension
  auto al16 = [](const float *p) { return ((uintptr_t)p & 15u) == 0; };
  const bool mfma = al16(A) && al16(B) && lda % 4 == 0 && ldb % 4 == 0 && (ta ? M : K) % 4 == 0 &&
                    (tb ? K : N) % 4 == 0;
  // reductions of at most 256, and products of at most 128 x 512 outputs, get 64-row tiles: twice
  // the blocks to cover their short k loops, or the compute units
  const int64_t tm = mfma ? (K <= 256 || M * N <= 128 * 512 ? 64 : train::kMfTile) : 64, tn = mfma ? train::kMfTile : 64;
  const int64_t tiles = ((M + tm - 1) / tm) * ((N + tn - 1) / tn);
  // split long reductions over k so that about two blocks per compute unit are busy (k chunks of at
  // least 128)
  int64_t splits = std::max<int64_t>(1, std::min<int64_t>((2 * (int64_t)cu_count + tiles - 1) / tiles, (K + 127) / 128));
  splits = std::min<int64_t>(splits, part_floats / (M * N));
  if (splits < 1) splits = 1;
  const int64_t kq = mfma ? train::kMfK : 16;
  g.kchunk = (((K + splits - 1) / splits) + kq - 1) / kq * kq;
  if (g.kchunk < kq) g.kchunk = kq;
  splits = (K + g.kchunk - 1) / g.kchunk;
  if (splits < 1) splits = 1;
  const dim3 grid((unsigned)((N + tn - 1) / tn), (unsigned)((M + tm - 1) / tm), (unsigned)splits);
  if (mfma) {
#define AECCT_MF_GO(TA_, TB_)                                                                          \
  do {                                                                                                 \
    if (tm == 64) hipLaunchKernelGGL((train::k_gemm_mfma<TA_, TB_, 64>), grid, dim3(train::kThreads), 0, s, g); \
    else hipLaunchKernelGGL((train::k_gemm_mfma<TA_, TB_, 128>), grid, dim3(train::kThreads), 0, s, g);        \
  } while (0)
    if (ta && tb) AECCT_MF_GO(true, true);
    else if (ta) AECCT_MF_GO(true, false);
    else if (tb) AECCT_MF_GO(false, true);
    else AECCT_MF_GO(false, false);
#undef AECCT_MF_GO
  } else if (ta && tb) {
    hipLaunchKernelGGL((train::k_gemm<true, true>), grid, dim3(train::kThreads), 0, s, g);
  } else if (ta) {
    hipLaunchKernelGGL((train::k_gemm<true, false>), grid, dim3(train::kThreads), 0, s, g);
  } else if (tb) {
    hipLaunchKernelGGL((train::k_gemm<false, true>), grid, dim3(train::kThreads), 0, s, g);
  } else {
    hipLaunchKernelGGL((train::k_gemm<false, false>), grid, dim3(train::kThreads), 0, s, g);
  }
  if (splits > 1)
    hipLaunchKernelGGL(train::k_gemm_reduce, dim3(blocks_for(M * N, 64)), dim3(train::kThreads), 0, s, g,
                       (int)splits);
  return hipGetLastError();
}

bool train_tern_shape_ok(int64_t N, int64_t K) { return K % 32 == 0 && N % 64 == 0; }

bool train_tern_operands_ok(const float *A, int64_t lda, const float *C, int64_t ldc, const float *bias, int64_t N,
                            int64_t K) {
  // 16-byte rows of A and C, 16-byte groups of the bias
  const auto al16 = [](const float *q) { return ((uintptr_t)q & 15u) == 0; };
  return train_tern_shape_ok(N, K) && lda % 4 == 0 && ldc % 4 == 0 && al16(A) && al16(C) && (!bias || al16(bias));
}

hipError_t train_pack_tern(const TernPackJobs &jobs, hipStream_t s) {
  if (jobs.n <= 0) return hipSuccess;
  int64_t lanes = 0;
  for (int i = 0; i < jobs.n; ++i) {
    const TernPackJob &J = jobs.j[i];
    if (!train_tern_shape_ok(J.trans ? J.R : J.C, J.trans ? J.C : J.R)) return hipErrorInvalidValue;
    lanes = std::max<int64_t>(lanes, (int64_t)J.R * J.C / 8);   // one lane per 8 entries
  }
  hipLaunchKernelGGL(train::k_pack_tern, dim3(blocks_for(lanes, train::kThreads), (unsigned)jobs.n), dim3(train::kThreads), 0,
                     s, jobs);
  return hipGetLastError();
}

namespace {
hipError_t gemm_tern_go(const train::GemmTern &g, hipStream_t s) {
  constexpr int S = 3;   // operands two k-steps ahead
  const unsigned gy = (unsigned)((g.M + 63) / 64);
  // a block's 16 NJ columns never straddle two column segments: seg_n is a multiple of 64 (and of
  // 128 for NJ = 8)
  if (g.seg_n % 128 == 0)
    hipLaunchKernelGGL((train::k_gemm_tern<8, S>), dim3((unsigned)(g.N / 128), gy), dim3(train::kThreads), 0, s, g);
  else
    hipLaunchKernelGGL((train::k_gemm_tern<4, S>), dim3((unsigned)(g.N / 64), gy), dim3(train::kThreads), 0, s, g);
  return hipGetLastError();
}
}  // namespace

hipError_t train_gemm_tern_seg(const float *A, int64_t lda, const void *const *frag, float *C, int64_t ldc, int64_t M,
                               int64_t seg_n, int nseg, int64_t K, const float *const *scale, const float *const *bias,
                               bool accumulate, hipStream_t s) {
  if (M <= 0 || seg_n <= 0) return hipSuccess;
  if (nseg < 1 || nseg > 3) return hipErrorInvalidValue;
  for (int k = 0; k < nseg; ++k)
    if (!train_tern_operands_ok(A, lda, C + k * seg_n, ldc, bias[k], seg_n, K)) return hipErrorInvalidValue;
  train::GemmTern g{A, {}, C, accumulate ? C : nullptr, M, seg_n * nseg, K, lda, ldc, {}, {}, seg_n, (int)(K / 32)};
  for (int k = 0; k < nseg; ++k) {
    g.B[k] = (const uint4 *)frag[k];
    g.scale[k] = scale[k];
    g.bias[k] = bias[k];
  }
  return gemm_tern_go(g, s);
}

hipError_t train_gemm_tern_ksum(const float *A, int64_t lda, const void *const *frag, int nseg, int64_t kseg,
                                const float *const *scale, const float *D, float *C, int64_t ldc, int64_t M, int64_t N,
                                hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (nseg < 1 || nseg > 3 || kseg <= 0 || kseg % 32 != 0) return hipErrorInvalidValue;
  if (!train_tern_operands_ok(A, lda, C, ldc, nullptr, N, kseg * nseg) || (D && ((uintptr_t)D & 15u) != 0))
    return hipErrorInvalidValue;
  train::GemmTern g{A, {}, C, D, M, N, kseg * nseg, lda, ldc, {}, {}, N, (int)(kseg / 32)};
  for (int k = 0; k < nseg; ++k) {
    g.B[k] = (const uint4 *)frag[k];
    g.scale[k] = scale[k];
  }
  return gemm_tern_go(g, s);
}

hipError_t train_gemm_tern(const float *A, int64_t lda, const void *frag, float *C, int64_t ldc, int64_t M, int64_t N,
                           int64_t K, const float *scale, const float *bias, bool accumulate, hipStream_t s) {
  return train_gemm_tern_seg(A, lda, &frag, C, ldc, M, N, 1, K, &scale, &bias, accumulate, s);
}

hipError_t train_attention(int which, int dh, const TrainAttn &a, hipStream_t s) {
  const TrainAttn &p = a;
  if (p.rows <= 0) return hipSuccess;
  const dim3 grid(blocks_for(p.rows * p.heads, train::kThreads));
#define AECCT_TRAIN_ATTN(DH)                                                                                 \
  if (which == 0) hipLaunchKernelGGL(train::k_attn_fwd<DH>, grid, dim3(train::kThreads), 0, s, p);          \
  else if (which == 1) hipLaunchKernelGGL(train::k_attn_bwd_q<DH>, grid, dim3(train::kThreads), 0, s, p);   \
  else hipLaunchKernelGGL(train::k_attn_bwd_kv<DH>, grid, dim3(train::kThreads), 0, s, p);
  switch (dh) {
    case 4: AECCT_TRAIN_ATTN(4) break;
    case 8: AECCT_TRAIN_ATTN(8) break;
    case 16: AECCT_TRAIN_ATTN(16) break;
    default: return hipErrorInvalidValue;
  }
#undef AECCT_TRAIN_ATTN
  return hipGetLastError();
}

hipError_t train_ln_fwd(const float *a, const float *b, int64_t rows, int d, const float *g, const float *beta, float eps,
                        float *out, float *xn, float *rho, float *xh, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d > 128) return hipErrorInvalidValue;
  hipLaunchKernelGGL(train::k_ln_fwd, dim3(blocks_for(rows, 4)), dim3(train::kThreads), 0, s, a, b, rows, d, g, beta, eps,
                     out, xn, rho, xh);
  return hipGetLastError();
}

hipError_t train_ln_bwd(const float *dy, const float *g, const float *xn, const float *rho, int64_t rows, int d,
                        float *dR, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d > 128) return hipErrorInvalidValue;
  hipLaunchKernelGGL(train::k_ln_bwd, dim3(blocks_for(rows, 4)), dim3(train::kThreads), 0, s, dy, g, xn, rho, rows, d, dR);
  return hipGetLastError();
}

namespace {
// C columns of A summed into the Ct = C (or 2 C, dual) result columns of fin
hipError_t colsum_run(const float *A, int64_t lda, const float *Bm, const float *w, int64_t rows, int C, bool dual,
                      const train::ColOut &fin, bool accumulate, float *part, int64_t part_floats, hipStream_t s) {
  if (C <= 0) return hipSuccess;
  const int Ct = dual ? 2 * C : C;
  int cwl = 0;
  while ((1 << cwl) < C && cwl < 6) ++cwl;
  const int lanes = train::kThreads >> cwl;
  const unsigned cblocks = blocks_for(C, 1 << cwl);
  // about 1024 blocks in all, each lane summing at least 8 rows
  int64_t chunks = std::min<int64_t>((rows + 8 * lanes - 1) / (8 * lanes), std::max<int64_t>(1, 1024 / cblocks));
  chunks = std::max<int64_t>(1, std::min<int64_t>(chunks, part_floats / Ct));
  const int64_t chunk = std::max<int64_t>(1, (rows + chunks - 1) / chunks);
  chunks = std::max<int64_t>(1, (rows + chunk - 1) / chunk);
  using K = decltype(&train::k_colsum<false, false, false>);
  K pass1 = dual ? (w ? train::k_colsum<true, true, true> : train::k_colsum<true, false, true>)
                 : Bm ? (w ? train::k_colsum<true, true, false> : train::k_colsum<true, false, false>)
                      : (w ? train::k_colsum<false, true, false> : train::k_colsum<false, false, false>);
  if (chunks == 1) {
    hipLaunchKernelGGL(pass1, dim3(cblocks, 1), dim3(train::kThreads), 0, s, A, lda, Bm, w, rows, C, cwl, chunk, fin,
                       accumulate ? 1 : 0);
    return hipGetLastError();
  }
  const train::ColOut pt{{part, nullptr, nullptr}, Ct, (int64_t)Ct};
  hipLaunchKernelGGL(pass1, dim3(cblocks, (unsigned)chunks), dim3(train::kThreads), 0, s, A, lda, Bm, w, rows, C, cwl,
                     chunk, pt, 0);
  // pass two over the partial rows: a block per column, its 256 lanes over the partial rows (a few
  // loads a lane, then the LDS tree), which takes a fraction of the 16-lanes-a-column form's time
  hipLaunchKernelGGL((train::k_colsum<false, false, false>), dim3((unsigned)Ct, 1), dim3(train::kThreads), 0, s, (const float *)part,
                     (int64_t)Ct, (const float *)nullptr, (const float *)nullptr, chunks, Ct, 0, chunks, fin,
                     accumulate ? 1 : 0);
  return hipGetLastError();
}
}  // namespace

hipError_t train_colsum(const float *A, int64_t lda, const float *Bm, const float *w, int64_t rows, int C, float *out,
                        bool accumulate, float *part, int64_t part_floats, hipStream_t s) {
  return colsum_run(A, lda, Bm, w, rows, C, false, train::ColOut{{out, nullptr, nullptr}, std::max(C, 1), 0},
                    accumulate, part, part_floats, s);
}

hipError_t train_colsum_dual(const float *A, int64_t lda, const float *Bm, int64_t rows, int C, float *out_ab,
                             float *out_a, float *part, int64_t part_floats, hipStream_t s) {
  if (!Bm) return hipErrorInvalidValue;
  return colsum_run(A, lda, Bm, nullptr, rows, C, true, train::ColOut{{out_ab, out_a, nullptr}, std::max(C, 1), 0},
                    false, part, part_floats, s);
}

hipError_t train_colsum_split(const float *A, int64_t lda, int64_t rows, int seg, int nseg, float *const *outs,
                              float *part, int64_t part_floats, hipStream_t s) {
  if (nseg < 1 || nseg > 3 || seg <= 0) return hipErrorInvalidValue;
  train::ColOut fin{{outs[0], nseg > 1 ? outs[1] : nullptr, nseg > 2 ? outs[2] : nullptr}, seg, 0};
  return colsum_run(A, lda, nullptr, nullptr, rows, seg * nseg, false, fin, false, part, part_floats, s);
}

hipError_t train_relu_bwd(float *dg, const float *f, int64_t count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  if (count % 4 == 0 && ((uintptr_t)dg & 15u) == 0 && ((uintptr_t)f & 15u) == 0)
    hipLaunchKernelGGL(train::k_relu_bwd4, dim3(blocks_for(count / 4, train::kThreads)), dim3(train::kThreads), 0, s,
                       (float4 *)dg, (const float4 *)f, count / 4);
  else
    hipLaunchKernelGGL(train::k_relu_bwd, dim3(blocks_for(count, train::kThreads)), dim3(train::kThreads), 0, s, dg, f,
                       count);
  return hipGetLastError();
}

hipError_t train_rowdot(const float *x, int64_t rows, int d, const float *w1, const float *b1, float *z, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(train::k_rowdot, dim3(blocks_for(rows, 4)), dim3(train::kThreads), 0, s, x, rows, d, w1, b1, z);
  return hipGetLastError();
}

hipError_t train_outer(const float *dz, int64_t rows, const float *w1, int d, float *dx, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(train::k_outer, dim3(blocks_for(rows * d, train::kThreads)), dim3(train::kThreads), 0, s, dz, rows,
                     w1, d, dx);
  return hipGetLastError();
}

hipError_t train_loss(const float *f, const float *y, const float *xs, int64_t count, float *df, float *part,
                      float *loss, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  const unsigned nb = blocks_for(count, train::kThreads);
  const float inv = 1.0f / (float)count;
  hipLaunchKernelGGL(train::k_loss, dim3(nb), dim3(train::kThreads), 0, s, f, y, xs, count, inv, df, part);
  hipLaunchKernelGGL(train::k_loss_final, dim3(1), dim3(64), 0, s, part, (int)nb, inv, loss);
  return hipGetLastError();
}

hipError_t train_embed_grad(const float *t, const float *dx, int64_t words, int L, int d, float *de, hipStream_t s) {
  hipLaunchKernelGGL(train::k_embed_grad, dim3(blocks_for((int64_t)L * d, train::kThreads)), dim3(train::kThreads), 0, s,
                     t, dx, words, L, d, de);
  return hipGetLastError();
}

}  // namespace aecct
