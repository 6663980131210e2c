// Helpers shared by the two quantize-on-append kernels (BF16 and fp32 Keys and
// Values): binary16 scale storage (App. D.1) and the exact rounding of the
// residual quotients of Eq. 1.
#pragma once

#include "qwm_common.h"

#include <type_traits>

namespace qwm {
namespace {

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E) step S.
// Keeps register-array indices static where #pragma unroll gives up on large bodies.
template <int B, int E, int S = 1, typename F>
__device__ inline void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + S, E, S>(f);
  }
}

__device__ inline float f16_round(float s) {
  // FP16 storage of a scale (App. D.1): saturate, then round to nearest even.
  s = fminf(s, 65504.0f);
  return (float)(_Float16)s;
}

__device__ inline uint16_t f16_bits(float exact) {
  return __builtin_bit_cast(uint16_t, (_Float16)exact);
}

// rint(x/s) for N residuals x = xv - mu with the IEEE quotient of Eq. 1, without
// N full divisions. t = x * RN(1/s) lies within 3 * 2^-24 * |x/s| of RN(x/s);
// every residual satisfies |x/s| <= 3.01 here (the range spans 3 steps), so the
// two differ by less than 2^-20 and round to the same integer unless t is
// within 2^-19 of a half-integer (or |t| > 4, out of this bound). If any lane
// of the wave meets such a case the whole chunk takes the exact division.
template <int N>
__device__ inline void round_quotients(const float (&xv)[N], const float (&mu)[N], float s, float inv,
                                       float (&t)[N]) {
  // the largest |q - k| and |q| of the chunk decide it: two compares instead of
  // two per channel, each of which fed a scalar OR chain
  float dmax = 0.0f, qmax = 0.0f;
#pragma unroll
  for (int c = 0; c < N; ++c) {
    const float q = (xv[c] - mu[c]) * inv;
    const float k = rintf(q);
    dmax = fmaxf(dmax, fabsf(q - k));
    qmax = fmaxf(qmax, fabsf(q));
    t[c] = k;
  }
  const bool near = dmax > 0.5f - 0x1p-19f || qmax > 4.0f;
  if (__any(near)) {
    const float sd = s != 0.0f ? s : 1.0f;
#pragma unroll
    for (int c = 0; c < N; ++c) t[c] = rintf((xv[c] - mu[c]) / sd);
  }
}

}  // namespace
}  // namespace qwm
