// fp64 mixed distance r^2 between two encoded configurations (Sec. 3.2, second kernel
// equation, with the per-type distances of Sec. 4.1), used by the Gram matrix, the
// fp64 recomputation of ill-conditioned candidates and the term inspection.
#pragma once
#include "common.h"

namespace bgp {

// `a(q)` and `b(q)` return code word q of the two configurations (unscaled codes).
template <class GA, class GB>
__device__ __forceinline__ double r2_f64(const GA &a, const GB &b, const Weights64 &w) {
  double r2 = 0.0;
  for (int q = 0; q < w.n_num; ++q) {
    const double d = (double)__uint_as_float(a(q)) - (double)__uint_as_float(b(q));
    r2 = fma(w.num_w[q] * d, d, r2);
  }
  for (int q = 0; q < w.n_bits; ++q)
    r2 = fma(w.bits_w[q], (double)__popc(a(w.w_bits0 + q) ^ b(w.w_bits0 + q)), r2);
  for (int q = 0; q < w.n_eq; ++q)
    if (a(w.w_eq0 + q) != b(w.w_eq0 + q)) r2 += w.eq_w[q];
  for (int q = 0; q < w.n_dot; ++q) {
    uint32_t dt = __builtin_amdgcn_udot4(a(w.w_dot0 + 2 * q), b(w.w_dot0 + 2 * q), 0u, false);
    dt = __builtin_amdgcn_udot4(a(w.w_dot0 + 2 * q + 1), b(w.w_dot0 + 2 * q + 1), dt, false);
    r2 = fma(w.dot_w2[q], (double)(w.dot_s2[q] - (int32_t)dt), r2);
  }
  return r2;
}

// Matern-5/2 of the distance r = sqrt(r2): s (1 + sqrt5 r + 5 r^2 / 3) exp(-sqrt5 r).
__device__ __forceinline__ double matern52_f64(double r2, double s) {
  const double r = sqrt(r2);
  const double sqrt5 = 2.23606797749978969640917366873128;
  return s * (1.0 + sqrt5 * r + (5.0 / 3.0) * r2) * exp(-sqrt5 * r);
}

}  // namespace bgp
