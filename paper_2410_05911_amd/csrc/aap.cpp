// AAP weight import (Section 4.1, Eq. 1): trained fp32 weights of one linear map to the
// ternary matrix and the per-matrix scale gamma*delta that the decode kernels run on.
// A create-time host step: the matrices are small (at most d x 4d) and read once.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <new>
#include <vector>

#include "../../include/aecct.h"

extern "C" aecct_status aecct_aap_ternarize(const float *w, int64_t count, float percentile, float delta,
                                            float eps, int8_t *ternary, float *scale) {
  if (!w || !ternary || !scale || count < 1) return AECCT_ERR_INVALID_ARG;
  if (!(percentile >= 0.0f && percentile <= 1.0f)) return AECCT_ERR_INVALID_ARG;
  if (!std::isfinite(delta) || !(delta > 0.0f) || !std::isfinite(eps) || !(eps >= 0.0f))
    return AECCT_ERR_INVALID_ARG;
  std::vector<float> a;
  try {
    a.resize((size_t)count);
  } catch (const std::bad_alloc &) {
    return AECCT_ERR_OUT_OF_MEMORY;
  }
  for (int64_t i = 0; i < count; ++i) {
    if (!std::isfinite(w[i])) return AECCT_ERR_INVALID_ARG;
    a[(size_t)i] = std::fabs(w[i]);
  }
  // gamma: the two order statistics around pos = p (count - 1) by selection (linear time)
  const double pos = (double)percentile * (double)(count - 1);
  const int64_t lo = std::min<int64_t>((int64_t)std::floor(pos), count - 1);
  const double frac = pos - (double)lo;
  std::nth_element(a.begin(), a.begin() + lo, a.end());
  const float a_lo = a[(size_t)lo];
  const float a_hi = lo + 1 < count ? *std::min_element(a.begin() + lo + 1, a.end()) : a_lo;
  const float gamma = (float)((double)a_lo + frac * ((double)a_hi - (double)a_lo));
  const float s = gamma * delta;
  const float den = s + eps;
  for (int64_t i = 0; i < count; ++i) {
    int8_t t;
    if (den == 0.0f) {
      t = w[i] > 0.0f ? 1 : (w[i] < 0.0f ? -1 : 0);
    } else {
      const float r = std::rint(w[i] / den);        // ties to even (default rounding mode)
      t = r > 0.0f ? (int8_t)std::min(r, 1.0f) : (int8_t)std::max(r, -1.0f);
    }
    ternary[i] = t;
  }
  *scale = s;
  return AECCT_OK;
}
