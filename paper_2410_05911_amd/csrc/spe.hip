// Spectral positional encoding of the Tanner graph (Section 4.3): a create-time step that
// produces the fixed positional table the decode adds to the token embedding.
//
// Host, float64: the Tanner-graph Laplacian D - A, its full eigendecomposition (Householder
// reduction to tridiagonal form with the reflections accumulated, then implicit symmetric QR
// steps with Wilkinson shifts, rotations accumulated into the same rows), and a canonical
// basis of every eigenspace.
//
// GPU: the per-node self-attention.  Every eigen-row of node j is an affine function of the
// two scalars (lambda_i, phi_i[j]): Z_i = lambda_i w_in[0] + phi_i[j] w_in[1] + b_in, so each
// projection is lambda_i a + phi_i[j] b + c with a = w_in[0] W, b = w_in[1] W, c = b_in W + bias.
// A head's score between rows i and i' is then the bilinear form
//     (lambda_i, phi_i, 1) M (lambda_i', phi_i', 1)^T,   M = [a;b;c]_q [a;b;c]_k^T / sqrt(dk)
// (3 x 3 per head), whose third column does not depend on i' and cancels in the softmax; and
// the attention output of row i is A_i a_v + B_i b_v + c_v, where A_i and B_i are the softmax
// means of lambda and phi over i'.  The reduction over rows and the output map are linear, so
// a node needs only R_A = sum_i w_red[i] A_i and R_B = sum_i w_red[i] B_i per head: the kernel
// computes those (L^2 score/exp pairs per node and head, from a 2-float row per eigen-row in
// LDS), and the host finishes SPE_j with d_pe^2 operations.  Same arithmetic as the textbook
// form up to rounding; fp32 on the GPU.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cfloat>
#include <cmath>
#include <cstdint>
#include <new>
#include <numeric>
#include <vector>

#include "../../include/aecct.h"

namespace {

constexpr int kMaxTokens = 4096;
constexpr double kClusterTol = 1e-8;
constexpr double kAcceptTol = 1e-6;
constexpr int kSpeThreads = 256;
constexpr int kSpeRows = 4;   // rows per thread per pass: each LDS read serves four rows

// ---------------------------------------------------------------- eigendecomposition (host)

// A (n x n, symmetric, row-major) -> tridiagonal diag/off, with W = Q^T (rows) such that
// A = Q T Q^T.  A is overwritten.
void householder_tridiagonal(std::vector<double> &A, int n, std::vector<double> &W, std::vector<double> &diag,
                             std::vector<double> &off) {
  std::vector<double> v(n), p(n), w(n), y(n);
  for (int k = 0; k + 2 < n; ++k) {
    const int r = n - k - 1;
    double *x = &A[(size_t)k * n + k + 1];   // row k right of the diagonal (= column k below it)
    double tail = 0.0;
    for (int t = 1; t < r; ++t) tail += x[t] * x[t];
    if (tail == 0.0) continue;               // already tridiagonal in this column
    const double sigma = std::sqrt(x[0] * x[0] + tail);
    const double alpha = x[0] >= 0.0 ? -sigma : sigma;
    v[0] = x[0] - alpha;
    for (int t = 1; t < r; ++t) v[t] = x[t];
    double vn = 0.0;
    for (int t = 0; t < r; ++t) vn += v[t] * v[t];
    vn = std::sqrt(vn);
    for (int t = 0; t < r; ++t) v[t] /= vn;
    // trailing block S <- H S H with H = I - 2 v v^T: S -= v w^T + w v^T, w = 2 (S v - (v.S v) v)
    double K = 0.0;
    for (int i = 0; i < r; ++i) {
      const double *row = &A[(size_t)(k + 1 + i) * n + k + 1];
      double s = 0.0;
      for (int t = 0; t < r; ++t) s += row[t] * v[t];
      p[i] = s;
      K += v[i] * s;
    }
    for (int i = 0; i < r; ++i) w[i] = 2.0 * (p[i] - K * v[i]);
    for (int i = 0; i < r; ++i) {
      double *row = &A[(size_t)(k + 1 + i) * n + k + 1];
      for (int t = 0; t < r; ++t) row[t] -= v[i] * w[t] + w[i] * v[t];
    }
    x[0] = alpha;
    A[(size_t)(k + 1) * n + k] = alpha;
    for (int t = 1; t < r; ++t) {
      x[t] = 0.0;
      A[(size_t)(k + 1 + t) * n + k] = 0.0;
    }
    // W <- H W on rows k+1..n-1
    std::fill(y.begin(), y.end(), 0.0);
    for (int i = 0; i < r; ++i) {
      const double *row = &W[(size_t)(k + 1 + i) * n];
      for (int c = 0; c < n; ++c) y[c] += v[i] * row[c];
    }
    for (int i = 0; i < r; ++i) {
      double *row = &W[(size_t)(k + 1 + i) * n];
      const double f = 2.0 * v[i];
      for (int c = 0; c < n; ++c) row[c] -= f * y[c];
    }
  }
  for (int i = 0; i < n; ++i) diag[i] = A[(size_t)i * n + i];
  for (int i = 0; i + 1 < n; ++i) off[i] = A[(size_t)i * n + i + 1];
}

// Implicit symmetric QR on the tridiagonal (diag, off); each plane rotation R of rows k, k+1
// is also applied to W (W <- R W), so that on return row i of W is the eigenvector of diag[i].
bool tridiagonal_qr(std::vector<double> &diag, std::vector<double> &off, std::vector<double> &W, int n) {
  double tnorm = 0.0;
  for (int i = 0; i < n; ++i)
    tnorm = std::max(tnorm, std::fabs(diag[i]) + (i > 0 ? std::fabs(off[i - 1]) : 0.0) +
                                (i + 1 < n ? std::fabs(off[i]) : 0.0));
  auto negligible = [&](int i) {   // off[i] couples i and i + 1
    const double e = std::fabs(off[i]);
    return e <= DBL_EPSILON * (std::fabs(diag[i]) + std::fabs(diag[i + 1])) || e <= DBL_EPSILON * tnorm;
  };
  long iters = 0;
  const long max_iters = 64L * n + 64;
  int hi = n - 1;
  while (hi > 0) {
    if (negligible(hi - 1)) {
      off[hi - 1] = 0.0;
      --hi;
      continue;
    }
    int lo = hi - 1;
    while (lo > 0 && !negligible(lo - 1)) --lo;
    if (lo > 0) off[lo - 1] = 0.0;
    if (++iters > max_iters) return false;
    // Wilkinson shift: the eigenvalue of the trailing 2 x 2 block nearer its last entry
    const double half = 0.5 * (diag[hi - 1] - diag[hi]);
    const double b = off[hi - 1];
    const double mu = diag[hi] - b * b / (half + (half >= 0.0 ? 1.0 : -1.0) * std::hypot(half, b));
    double x = diag[lo] - mu, z = off[lo];
    for (int k = lo; k < hi; ++k) {
      const double r = std::hypot(x, z);
      const double c = r == 0.0 ? 1.0 : x / r, s = r == 0.0 ? 0.0 : z / r;
      if (k > lo) off[k - 1] = r;                 // the bulge below it is now zero
      const double a = diag[k], e = off[k], f = diag[k + 1];
      diag[k] = c * c * a + 2.0 * c * s * e + s * s * f;
      diag[k + 1] = s * s * a - 2.0 * c * s * e + c * c * f;
      off[k] = c * s * (f - a) + e * (c * c - s * s);
      if (k + 1 < hi) {
        z = s * off[k + 1];                       // new bulge at (k, k + 2)
        off[k + 1] *= c;
        x = off[k];
      }
      double *wk = &W[(size_t)k * n], *wk1 = &W[(size_t)(k + 1) * n];
      for (int t = 0; t < n; ++t) {
        const double u = wk[t], v = wk1[t];
        wk[t] = c * u + s * v;
        wk1[t] = c * v - s * u;
      }
    }
  }
  return true;
}

// Canonical basis of every eigenspace (see aecct.h): rows of `vec` (ascending eigenvalues)
// are replaced, cluster by cluster.
bool canonical_basis(const std::vector<double> &lam, std::vector<double> &vec, int n) {
  double big = 1.0;
  for (double l : lam) big = std::max(big, std::fabs(l));
  const double tol = kClusterTol * big;
  std::vector<double> u(n), basis;
  int s = 0;
  while (s < n) {
    int e = s + 1;
    while (e < n && lam[e] - lam[e - 1] <= tol) ++e;
    const int r = e - s;
    basis.assign((size_t)r * n, 0.0);
    int taken = 0;
    for (int c = 0; c < n && taken < r; ++c) {
      if (taken == 0) {   // nothing to remove yet: the squared norm is the projector's diagonal
        double pcc = 0.0;
        for (int k = s; k < e; ++k) pcc += vec[(size_t)k * n + c] * vec[(size_t)k * n + c];
        if (!(pcc > kAcceptTol)) continue;
      }
      std::fill(u.begin(), u.end(), 0.0);
      for (int k = s; k < e; ++k) {
        const double f = vec[(size_t)k * n + c];
        const double *row = &vec[(size_t)k * n];
        for (int t = 0; t < n; ++t) u[t] += f * row[t];
      }
      for (int pass = 0; pass < 2; ++pass)
        for (int q = 0; q < taken; ++q) {
          const double *b = &basis[(size_t)q * n];
          double dot = 0.0;
          for (int t = 0; t < n; ++t) dot += b[t] * u[t];
          for (int t = 0; t < n; ++t) u[t] -= dot * b[t];
        }
      double nn = 0.0;
      for (int t = 0; t < n; ++t) nn += u[t] * u[t];
      if (!(nn > kAcceptTol)) continue;
      const double inv = 1.0 / std::sqrt(nn);
      double *b = &basis[(size_t)taken * n];
      for (int t = 0; t < n; ++t) b[t] = u[t] * inv;
      ++taken;
    }
    if (taken != r) return false;
    std::copy(basis.begin(), basis.end(), vec.begin() + (size_t)s * n);
    s = e;
  }
  return true;
}

// ---------------------------------------------------------------- per-node attention (GPU)

// Block (j, h): for the L eigen-rows i of node j, the softmax means A_i, B_i of lambda and
// phi under head h's scores, reduced with w_red into out[j][h] = (R_A, R_B).
//   tok_lam [L] fp32 eigenvalues; phi_t [L][L] with phi_t[j][i] = phi_i[j];
//   coef [heads][6] = log2(e) * (M00, M01, M10, M11, M20, M21) of the head's score form.
__global__ __launch_bounds__(kSpeThreads) void k_spe_node_attention(const float *__restrict__ tok_lam,
                                                                    const float *__restrict__ phi_t,
                                                                    const float *__restrict__ w_red,
                                                                    const float *__restrict__ coef, int L,
                                                                    int heads, float *__restrict__ out) {
  __shared__ float2 tok[kMaxTokens];
  __shared__ float part[2][kSpeThreads / 64];
  const int j = blockIdx.x / heads, h = blockIdx.x - j * heads;
  for (int i = threadIdx.x; i < L; i += kSpeThreads) tok[i] = make_float2(tok_lam[i], phi_t[(size_t)j * L + i]);
  __syncthreads();
  const float m00 = coef[h * 6 + 0], m01 = coef[h * 6 + 1], m10 = coef[h * 6 + 2];
  const float m11 = coef[h * 6 + 3], m20 = coef[h * 6 + 4], m21 = coef[h * 6 + 5];
  float ra = 0.0f, rb = 0.0f;
  const int per_pass = kSpeThreads * kSpeRows;
  for (int base = 0; base < L; base += per_pass) {
    float g0[kSpeRows], g1[kSpeRows], wr[kSpeRows], mx[kSpeRows];
#pragma unroll
    for (int k = 0; k < kSpeRows; ++k) {
      const int i = base + k * kSpeThreads + (int)threadIdx.x;
      const bool valid = i < L;
      const float2 t = tok[valid ? i : 0];
      g0[k] = fmaf(t.x, m00, fmaf(t.y, m10, m20));
      g1[k] = fmaf(t.x, m01, fmaf(t.y, m11, m21));
      wr[k] = valid ? w_red[i] : 0.0f;
      mx[k] = -INFINITY;
    }
    for (int q = 0; q < L; ++q) {
      const float2 t = tok[q];
#pragma unroll
      for (int k = 0; k < kSpeRows; ++k) mx[k] = fmaxf(mx[k], fmaf(g0[k], t.x, g1[k] * t.y));
    }
    float S[kSpeRows], SA[kSpeRows], SB[kSpeRows];
#pragma unroll
    for (int k = 0; k < kSpeRows; ++k) S[k] = SA[k] = SB[k] = 0.0f;
    for (int q = 0; q < L; ++q) {
      const float2 t = tok[q];
#pragma unroll
      for (int k = 0; k < kSpeRows; ++k) {
        const float e = __builtin_amdgcn_exp2f(fmaf(g0[k], t.x, fmaf(g1[k], t.y, -mx[k])));
        S[k] += e;
        SA[k] = fmaf(e, t.x, SA[k]);
        SB[k] = fmaf(e, t.y, SB[k]);
      }
    }
#pragma unroll
    for (int k = 0; k < kSpeRows; ++k) {
      ra = fmaf(wr[k], SA[k] / S[k], ra);
      rb = fmaf(wr[k], SB[k] / S[k], rb);
    }
  }
  for (int off = 32; off > 0; off >>= 1) {
    ra += __shfl_xor(ra, off);
    rb += __shfl_xor(rb, off);
  }
  const int wave = threadIdx.x / 64;
  if ((threadIdx.x & 63) == 0) {
    part[0][wave] = ra;
    part[1][wave] = rb;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float sa = 0.0f, sb = 0.0f;
    for (int w = 0; w < kSpeThreads / 64; ++w) {
      sa += part[0][w];
      sb += part[1][w];
    }
    out[(size_t)blockIdx.x * 2 + 0] = sa;
    out[(size_t)blockIdx.x * 2 + 1] = sb;
  }
}

bool all_finite(const float *a, int64_t count) {
  if (!a) return true;
  for (int64_t i = 0; i < count; ++i)
    if (!std::isfinite(a[i])) return false;
  return true;
}

struct DeviceBuffers {
  void *p = nullptr;
  ~DeviceBuffers() {
    if (p) (void)hipFree(p);
  }
};

}  // namespace

extern "C" aecct_status aecct_tanner_spectrum(const uint8_t *H, int32_t m, int32_t n, double *eigvals,
                                              double *eigvecs) {
  if (!H || !eigvals || !eigvecs || m < 1 || n < 1 || (int64_t)m + n > kMaxTokens) return AECCT_ERR_INVALID_ARG;
  for (int64_t i = 0; i < (int64_t)m * n; ++i)
    if (H[i] > 1) return AECCT_ERR_INVALID_ARG;
  const int L = n + m;
  std::vector<double> A, W, diag, off;
  try {
    A.assign((size_t)L * L, 0.0);
    W.assign((size_t)L * L, 0.0);
    diag.assign(L, 0.0);
    off.assign(L, 0.0);
  } catch (const std::bad_alloc &) {
    return AECCT_ERR_OUT_OF_MEMORY;
  }
  for (int j = 0; j < m; ++j)
    for (int i = 0; i < n; ++i)
      if (H[(size_t)j * n + i]) {
        A[(size_t)i * L + n + j] = -1.0;
        A[(size_t)(n + j) * L + i] = -1.0;
        A[(size_t)i * L + i] += 1.0;
        A[(size_t)(n + j) * L + n + j] += 1.0;
      }
  for (int i = 0; i < L; ++i) W[(size_t)i * L + i] = 1.0;
  householder_tridiagonal(A, L, W, diag, off);
  if (!tridiagonal_qr(diag, off, W, L)) return AECCT_ERR_UNSUPPORTED;
  std::vector<int> order(L);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return diag[a] < diag[b]; });
  std::vector<double> lam(L), vec((size_t)L * L);
  for (int i = 0; i < L; ++i) {
    lam[i] = diag[order[i]];
    std::copy(&W[(size_t)order[i] * L], &W[(size_t)order[i] * L] + L, &vec[(size_t)i * L]);
  }
  if (!canonical_basis(lam, vec, L)) return AECCT_ERR_UNSUPPORTED;
  std::copy(lam.begin(), lam.end(), eigvals);
  std::copy(vec.begin(), vec.end(), eigvecs);
  return AECCT_OK;
}

extern "C" aecct_status aecct_spe_table_from_spectrum(const double *eigvals, const double *eigvecs, int32_t L,
                                                      const aecct_spe_params *p, int32_t d, float *pos) {
  if (!eigvals || !eigvecs || !p || !pos || L < 1 || L > kMaxTokens) return AECCT_ERR_INVALID_ARG;
  const int dp = p->d_pe, heads = p->heads;
  if (heads < 1 || dp < heads || dp % heads != 0 || dp > d) return AECCT_ERR_INVALID_ARG;
  if (!p->w_in || !p->w_q || !p->w_k || !p->w_v || !p->w_o || !p->w_red) return AECCT_ERR_INVALID_ARG;
  if (!all_finite(p->w_in, 2 * dp) || !all_finite(p->b_in, dp) || !all_finite(p->w_red, L) ||
      !std::isfinite(p->b_red))
    return AECCT_ERR_INVALID_ARG;
  const float *wm[4] = {p->w_q, p->w_k, p->w_v, p->w_o}, *bm[4] = {p->b_q, p->b_k, p->b_v, p->b_o};
  for (int x = 0; x < 4; ++x)
    if (!all_finite(wm[x], (int64_t)dp * dp) || !all_finite(bm[x], dp)) return AECCT_ERR_INVALID_ARG;
  for (int64_t i = 0; i < (int64_t)L; ++i)
    if (!std::isfinite(eigvals[i])) return AECCT_ERR_INVALID_ARG;
  for (int64_t i = 0; i < (int64_t)L * L; ++i)
    if (!std::isfinite(eigvecs[i])) return AECCT_ERR_INVALID_ARG;

  // the three projections as lambda * a + phi * b + c (float64)
  const int dk = dp / heads;
  std::vector<double> abc(3 * 3 * (size_t)dp, 0.0);   // [x in q,k,v][a,b,c][col]
  auto bin = [&](int t) { return p->b_in ? (double)p->b_in[t] : 0.0; };
  for (int x = 0; x < 3; ++x)
    for (int col = 0; col < dp; ++col) {
      double a = 0.0, b = 0.0, c = bm[x] ? (double)bm[x][col] : 0.0;
      for (int t = 0; t < dp; ++t) {
        const double wt = wm[x][(size_t)t * dp + col];
        a += (double)p->w_in[t] * wt;
        b += (double)p->w_in[dp + t] * wt;
        c += bin(t) * wt;
      }
      abc[((size_t)x * 3 + 0) * dp + col] = a;
      abc[((size_t)x * 3 + 1) * dp + col] = b;
      abc[((size_t)x * 3 + 2) * dp + col] = c;
    }
  std::vector<float> coef((size_t)heads * 6);
  const double scale = 1.4426950408889634 / std::sqrt((double)dk);   // log2(e) / sqrt(dk)
  for (int h = 0; h < heads; ++h)
    for (int r = 0; r < 3; ++r)
      for (int s = 0; s < 2; ++s) {
        double acc = 0.0;
        for (int t = h * dk; t < (h + 1) * dk; ++t)
          acc += abc[((size_t)0 * 3 + r) * dp + t] * abc[((size_t)1 * 3 + s) * dp + t];
        coef[(size_t)h * 6 + r * 2 + s] = (float)(acc * scale);
      }
  std::vector<float> lam_f(L), phi_t, red_out((size_t)L * heads * 2);
  try {
    phi_t.resize((size_t)L * L);
  } catch (const std::bad_alloc &) {
    return AECCT_ERR_OUT_OF_MEMORY;
  }
  for (int i = 0; i < L; ++i) {
    lam_f[i] = (float)eigvals[i];
    for (int j = 0; j < L; ++j) phi_t[(size_t)j * L + i] = (float)eigvecs[(size_t)i * L + j];
  }

  int dev_count = 0;
  if (hipGetDeviceCount(&dev_count) != hipSuccess || dev_count < 1) return AECCT_ERR_DEVICE;
  const size_t n_lam = (size_t)L, n_phi = (size_t)L * L, n_red = (size_t)L, n_coef = coef.size(),
               n_out = red_out.size();
  const size_t total = (n_lam + n_phi + n_red + n_coef + n_out) * sizeof(float);
  DeviceBuffers buf;
  if (hipMalloc(&buf.p, total) != hipSuccess) {
    buf.p = nullptr;
    (void)hipGetLastError();
    return AECCT_ERR_OUT_OF_MEMORY;
  }
  float *d_lam = (float *)buf.p, *d_phi = d_lam + n_lam, *d_red = d_phi + n_phi, *d_coef = d_red + n_red,
        *d_out = d_coef + n_coef;
  if (hipMemcpy(d_lam, lam_f.data(), n_lam * sizeof(float), hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(d_phi, phi_t.data(), n_phi * sizeof(float), hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(d_red, p->w_red, n_red * sizeof(float), hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(d_coef, coef.data(), n_coef * sizeof(float), hipMemcpyHostToDevice) != hipSuccess)
    return AECCT_ERR_DEVICE;
  hipLaunchKernelGGL(k_spe_node_attention, dim3((unsigned)(L * heads)), dim3(kSpeThreads), 0, nullptr, d_lam,
                     d_phi, d_red, d_coef, L, heads, d_out);
  if (hipGetLastError() != hipSuccess) return AECCT_ERR_DEVICE;
  if (hipMemcpy(red_out.data(), d_out, n_out * sizeof(float), hipMemcpyDeviceToHost) != hipSuccess)
    return AECCT_ERR_DEVICE;

  // SPE_j = (concat_h R_A a_v + R_B b_v + W c_v) w_o + W b_o + b_red, W = sum of w_red
  double wsum = 0.0;
  for (int i = 0; i < L; ++i) wsum += (double)p->w_red[i];
  std::vector<double> o(dp);
  for (int j = 0; j < L; ++j) {
    for (int h = 0; h < heads; ++h) {
      const double RA = red_out[((size_t)j * heads + h) * 2 + 0], RB = red_out[((size_t)j * heads + h) * 2 + 1];
      for (int t = h * dk; t < (h + 1) * dk; ++t)
        o[t] = RA * abc[((size_t)2 * 3 + 0) * dp + t] + RB * abc[((size_t)2 * 3 + 1) * dp + t] +
               wsum * abc[((size_t)2 * 3 + 2) * dp + t];
    }
    float *row = pos + (size_t)j * d;
    for (int c = 0; c < d - dp; ++c) row[c] = 0.0f;
    for (int c = 0; c < dp; ++c) {
      double acc = wsum * (p->b_o ? (double)p->b_o[c] : 0.0) + (double)p->b_red;
      for (int t = 0; t < dp; ++t) acc += o[t] * (double)p->w_o[(size_t)t * dp + c];
      row[d - dp + c] = (float)acc;
    }
  }
  return AECCT_OK;
}

extern "C" aecct_status aecct_spe_table(const uint8_t *H, int32_t m, int32_t n, const aecct_spe_params *p,
                                        int32_t d, float *pos) {
  if (!H || !p || !pos || m < 1 || n < 1 || (int64_t)m + n > kMaxTokens) return AECCT_ERR_INVALID_ARG;
  const int L = n + m;
  std::vector<double> lam, vec;
  try {
    lam.resize(L);
    vec.resize((size_t)L * L);
  } catch (const std::bad_alloc &) {
    return AECCT_ERR_OUT_OF_MEMORY;
  }
  const aecct_status st = aecct_tanner_spectrum(H, m, n, lam.data(), vec.data());
  if (st != AECCT_OK) return st;
  return aecct_spe_table_from_spectrum(lam.data(), vec.data(), L, p, d, pos);
}
