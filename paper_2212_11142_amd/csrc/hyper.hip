// GP hyperparameter fit (Sec. 3.2, GP hyperparameter optimisation): batched evaluation of
// the objective (log marginal likelihood of the feasible observations plus gamma
// log-densities of the lengthscales) and its gradient, the choice of the best sampled
// settings, and the L-BFGS iteration of every kept setting.
//
// A setting is theta = (log l_1..log l_d, log s, t) with noise variance floor + e^t. For
// each setting b of a batch (launch plane b):
//   K = s Matern52(r) + noise I,  r^2 = sum_p T_p / l_p^2  (T_p: squared distance of
//       parameter p divided by its maximum, computed once per call),
//   L = chol(K), X = L^-1 (blocked fp64 factorisation and inverse, chol.hip),
//   value = -1/2 |X y|^2 - sum_i log L_ii - nf/2 log 2 pi + sum_p log Gamma(l_p),
//   alpha = X^T (X y),  K^-1 = X^T X,
//   d value / d theta_q = 1/2 sum_ij (alpha_i alpha_j - K^-1_ij) dK_ij/d theta_q + prior',
//       dK/d log l_p = dk/dr^2 (-2 T_p / l_p^2), dK/d log s = K - noise I, dK/dt = e^t I,
//       dk/dr^2 = -(5/6) s (1 + sqrt5 r) e^(-sqrt5 r).
// Every sum runs in a fixed order (wave butterflies, then wavefronts in order, then
// blocks in order), so results do not depend on scheduling.
#include <cmath>

#include "common.h"

namespace bgp {
namespace {

constexpr double kSqrt5 = 2.23606797749978969640917366873128;
constexpr double kLog2Pi = 1.83787706640934548356065947281123;
constexpr int CH = kHypGradChunk;
constexpr double kArmijoC1 = 1e-4;
constexpr int kMaxHalvings = kLbfgsMaxHalvings;
constexpr double kCurvatureEps = 1e-10;

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ double wave_max(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  return v;
}
// Sum over a 256-thread block (every thread gets it); red: 4 doubles of LDS.
__device__ __forceinline__ double block_sum(double v, double *red) {
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const double r = ((red[0] + red[1]) + red[2]) + red[3];
  __syncthreads();
  return r;
}

__device__ __forceinline__ double clamp_exp(double t) { return exp(fmin(t, 709.0)); }

__device__ __forceinline__ void pair_of(int64_t q, int &i, int &j) {  // q -> (i >= j)
  int r = (int)((sqrt(8.0 * (double)q + 1.0) - 1.0) * 0.5);
  while ((int64_t)(r + 1) * (r + 2) / 2 <= q) ++r;
  while ((int64_t)r * (r + 1) / 2 > q) --r;
  i = r;
  j = (int)(q - (int64_t)r * (r + 1) / 2);
}

// ------------------------------------------------------------------------ pair terms
__global__ __launch_bounds__(256) void hyp_terms_k(const uint32_t *codes, int32_t R,
                                                    const TermDesc *td, int32_t d, int32_t nf,
                                                    double *T) {
  const int64_t nn = (int64_t)nf * nf;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= nn) return;
  const int i = (int)(idx / nf), j = (int)(idx - (int64_t)i * nf);
  const uint32_t *a = codes + (int64_t)i * R, *b = codes + (int64_t)j * R;
  for (int p = 0; p < d; ++p) {
    const TermDesc t = td[p];
    const uint32_t a0 = a[t.word], b0 = b[t.word];
    double v;
    if (t.kind == GP_REAL || t.kind == GP_INT || t.kind == GP_ORD) {
      const double df = (double)__uint_as_float(a0) - (double)__uint_as_float(b0);
      v = df * df;
    } else if (t.kind == GP_CAT) {
      if (t.bit >= 0) {
        const uint32_t fm = (t.m >= 32 ? 0xffffffffu : ((1u << t.m) - 1u)) << t.bit;
        v = ((a0 ^ b0) & fm) ? 1.0 : 0.0;
      } else {
        v = a0 != b0 ? 1.0 : 0.0;
      }
    } else if (t.dist == GP_PERM_KENDALL) {
      v = (double)__popc(a0 ^ b0) / (double)(t.m * (t.m - 1) / 2);
    } else if (t.dist == GP_PERM_NAIVE) {
      v = a0 != b0 ? 1.0 : 0.0;
    } else {
      const uint32_t a1 = a[t.word + 1], b1 = b[t.word + 1];
      if (t.dist == GP_PERM_HAMMING) {
        v = (double)((__popc(a0 ^ b0) + __popc(a1 ^ b1)) / 2) / (double)t.m;
      } else {  // Spearman: sum (pi_i - pi'_i)^2 = 2 (S2 - pi . pi')
        const int s2 = (t.m - 1) * t.m * (2 * t.m - 1) / 6;
        uint32_t dt = __builtin_amdgcn_udot4(a0, b0, 0u, false);
        dt = __builtin_amdgcn_udot4(a1, b1, dt, false);
        v = (double)(2 * (s2 - (int32_t)dt)) / (double)((t.m * t.m * t.m - t.m) / 3);
      }
    }
    T[(int64_t)p * nn + idx] = v;
  }
}

// ------------------------------------------------------------------------------ Gram
__device__ __forceinline__ double hyp_r2(const HypArgs &a, const double *w, int64_t idx,
                                         int64_t nn) {
  double r2 = 0.0;
  for (int p = 0; p < a.d; ++p) r2 = fma(a.T[(int64_t)p * nn + idx], w[p], r2);
  return r2;
}

// Setting b's Gram matrix K (rows 0..nf-1 of its plane) and the identity rows below it
// (rows nf..2nf-1, whose factorisation panels give L^-1); the first workgroup of a plane
// also resets its status (1 for an inactive setting, which is skipped).
__global__ __launch_bounds__(256) void hyp_gram_k(const HypArgs a, double *K) {
  __shared__ double w[kMaxD];
  const int b = blockIdx.y;
  const bool inactive = a.active && !a.active[b];
  if (blockIdx.x == 0 && threadIdx.x == 0) a.info[b] = inactive ? 1 : 0;
  if (inactive) return;
  const double *th = a.theta + (int64_t)b * a.theta_ld;
  if (threadIdx.x < a.d) w[threadIdx.x] = exp(-2.0 * th[threadIdx.x]);
  __syncthreads();
  const int64_t nn = (int64_t)a.nf * a.nf;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= nn) return;
  const int i = (int)(idx / a.nf), j = (int)(idx - (int64_t)i * a.nf);
  const double s = clamp_exp(th[a.d]);
  const double r2 = hyp_r2(a, w, idx, nn), r = sqrt(r2);
  double k = s * (1.0 + kSqrt5 * r + (5.0 / 3.0) * r2) * exp(-kSqrt5 * r);
  if (i == j) k += a.noise_floor + clamp_exp(th[a.d + 1]);
  double *Kb = K + (int64_t)b * a.sA;
  Kb[(int64_t)i * a.ld + j] = k;
  Kb[(int64_t)(a.nf + i) * a.ld + j] = i == j ? 1.0 : 0.0;
}

// ----------------------------------------------------------------------------- value
// z = X y (X = L^-1 lower triangular): one wavefront per row, four rows per workgroup.
__global__ __launch_bounds__(256) void hyp_z_k(const HypArgs a, const double *Xb, double *z) {
  const int b = blockIdx.y;
  if ((a.active && !a.active[b]) || a.info[b]) return;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= a.nf) return;
  const double *row = Xb + (int64_t)b * a.sM + (int64_t)i * a.ld;
  double acc0 = 0.0, acc1 = 0.0;
  for (int j = lane; j <= i; j += 128) {
    acc0 = fma(row[j], a.y[j], acc0);
    if (j + 64 <= i) acc1 = fma(row[j + 64], a.y[j + 64], acc1);
  }
  const double v = wave_sum(acc0 + acc1);
  if (lane == 0) z[(int64_t)b * a.nf + i] = v;
}

// value = -1/2 |z|^2 - sum log L_ii - nf/2 log 2 pi + prior (-inf when not a kernel)
__device__ __forceinline__ void hyp_value_wg(const HypArgs &a, int b, const double *Lb,
                                             const double *z, double *value, double *red) {
  const int tid = threadIdx.x;
  if (a.active && !a.active[b]) return;
  if (a.info[b]) {
    if (tid == 0) value[b] = -INFINITY;
    return;
  }
  const int nf = a.nf;
  const double *L = Lb + (int64_t)b * a.sM, *zb = z + (int64_t)b * nf;
  double q = 0.0, hl = 0.0;
  for (int i = tid; i < nf; i += 256) {
    q = fma(zb[i], zb[i], q);
    hl += log(L[(int64_t)i * a.ld + i]);
  }
  q = block_sum(q, red);
  hl = block_sum(hl, red);
  if (tid == 0) {
    double v = -0.5 * q - hl - 0.5 * nf * kLog2Pi;
    if (a.has_prior) {
      const double *th = a.theta + (int64_t)b * a.theta_ld;
      for (int p = 0; p < a.d; ++p)
        v += a.prior_c0 + (a.prior_shape - 1.0) * th[p] - a.prior_rate * exp(th[p]);
    }
    if (!isfinite(v)) {
      v = -INFINITY;
      a.info[b] = 2;  // no gradient
    }
    value[b] = v;
  }
}


// alpha = X^T z: a workgroup per 64 columns, its wavefronts split the rows (i = w mod 4)
// and their partial sums are added in wavefront order. The workgroup after the last
// column block forms the setting's value instead (its "no gradient" status, set when the
// value is not finite, only stops the gradient: alpha of such a setting is not used).
__global__ __launch_bounds__(256) void hyp_alpha_k(const HypArgs a, const double *Xb,
                                                    const double *z, double *alpha,
                                                    const double *Lb, double *value) {
  __shared__ double part[4][64];
  const int b = blockIdx.y;
  if ((int)blockIdx.x == (int)gridDim.x - 1) {
    hyp_value_wg(a, b, Lb, z, value, &part[0][0]);
    return;
  }
  if ((a.active && !a.active[b]) || a.info[b]) return;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nf = a.nf;
  const int j = blockIdx.x * 64 + lane;
  const double *X = Xb + (int64_t)b * a.sM, *zb = z + (int64_t)b * nf;
  double acc = 0.0;
  if (j < nf) {
    // eight rows' loads in flight together (rows above the diagonal are read and left out,
    // the sum keeps its order)
    int i = blockIdx.x * 64 + w;
    for (; i + 28 < nf; i += 32) {
      double x[8], zz[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        x[u] = X[(int64_t)(i + 4 * u) * a.ld + j];
        zz[u] = zb[i + 4 * u];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (i + 4 * u >= j) acc = fma(x[u], zz[u], acc);
    }
    for (; i < nf; i += 4)
      if (i >= j) acc = fma(X[(int64_t)i * a.ld + j], zb[i], acc);
  }
  part[w][lane] = acc;
  __syncthreads();
  if (w == 0 && j < nf)
    alpha[(int64_t)b * nf + j] = (part[0][lane] + part[1][lane]) + (part[2][lane] + part[3][lane]);
}

// -------------------------------------------------------------------------- gradient
// Launch plane (b, chunk): pairs i >= j in a grid-stride loop; every pair's coefficient
// C = w_ij (alpha_i alpha_j - K^-1_ij) dk/dr^2 (w_ij = 2 off the diagonal) multiplies
// T_p for the chunk's CH lengthscales; chunk 0 also sums the output-scale and noise
// terms. Partial sums per block go to `part`, summed in block order by hyp_grad_final_k.
__global__ __launch_bounds__(256) void hyp_grad_k(const HypArgs a, const double *Kinv,
                                                   const double *alpha, double *part) {
  __shared__ double w[kMaxD];
  __shared__ double red[4];
  const int b = blockIdx.y, chunk = blockIdx.z, tid = threadIdx.x;
  if ((a.active && !a.active[b]) || a.info[b]) return;
  const double *th = a.theta + (int64_t)b * a.theta_ld;
  if (tid < a.d) w[tid] = exp(-2.0 * th[tid]);
  __syncthreads();
  const int nf = a.nf;
  const double s = clamp_exp(th[a.d]);
  const int64_t nn = (int64_t)nf * nf, npairs = (int64_t)nf * (nf + 1) / 2;
  const double *Ki = Kinv + (int64_t)b * a.sA, *al = alpha + (int64_t)b * nf;
  const int p0 = chunk * CH;
  double acc[CH];
#pragma unroll
  for (int c = 0; c < CH; ++c) acc[c] = 0.0;
  double acc_s = 0.0, acc_n = 0.0;
  // With all lengthscales in one chunk, a pair's d terms are loaded once, for r^2 and
  // for the sums (same operations in the same order as the two-pass form).
  const bool one_chunk = a.d <= CH;
  for (int64_t q = (int64_t)blockIdx.x * 256 + tid; q < npairs; q += (int64_t)gridDim.x * 256) {
    int i, j;
    pair_of(q, i, j);
    const int64_t idx = (int64_t)i * nf + j;
    double tv[CH];
    double r2 = 0.0;
    if (one_chunk) {
#pragma unroll
      for (int c = 0; c < CH; ++c) tv[c] = c < a.d ? a.T[(int64_t)c * nn + idx] : 0.0;
#pragma unroll
      for (int c = 0; c < CH; ++c)
        if (c < a.d) r2 = fma(tv[c], w[c], r2);
    } else {
      r2 = hyp_r2(a, w, idx, nn);
#pragma unroll
      for (int c = 0; c < CH; ++c)
        tv[c] = p0 + c < a.d ? a.T[(int64_t)(p0 + c) * nn + idx] : 0.0;
    }
    const double r = sqrt(r2);
    const double e = exp(-kSqrt5 * r);
    const double dk = -(5.0 / 6.0) * s * (1.0 + kSqrt5 * r) * e;
    const double wt = (i == j) ? 1.0 : 2.0;
    const double G = al[i] * al[j] - Ki[(int64_t)i * a.ld + j];
    const double C = wt * G * dk;
#pragma unroll
    for (int c = 0; c < CH; ++c)
      if (p0 + c < a.d) acc[c] = fma(C, tv[c], acc[c]);
    if (chunk == 0) {
      const double kf = s * (1.0 + kSqrt5 * r + (5.0 / 3.0) * r2) * e;
      acc_s = fma(wt * G, kf, acc_s);
      if (i == j) acc_n += G;
    }
  }
  double *out = part + (((int64_t)b * gridDim.z + chunk) * gridDim.x + blockIdx.x) * (CH + 2);
#pragma unroll
  for (int c = 0; c < CH + 2; ++c) {
    const double v = block_sum(c < CH ? acc[c] : (c == CH ? acc_s : acc_n), red);
    if (tid == 0) out[c] = v;
  }
}

// Workgroup (b, q): entry q of setting b's gradient; thread k loads block k's partial
// (nblk <= 128) and the two wavefront sums are added in order.
__global__ __launch_bounds__(128) void hyp_grad_final_k(const HypArgs a, const double *part,
                                                         int nblk, int nchunks, double *grad,
                                                         int64_t grad_ld) {
  __shared__ double red[2];
  const int b = blockIdx.x, q = blockIdx.y, tid = threadIdx.x;
  if ((a.active && !a.active[b]) || a.info[b] || q >= a.d + 2) return;
  const double *th = a.theta + (int64_t)b * a.theta_ld;
  const int chunk = q < a.d ? q / CH : 0, c = q < a.d ? q % CH : (q == a.d ? CH : CH + 1);
  const double *pp = part + ((int64_t)b * nchunks + chunk) * nblk * (CH + 2) + c;
  double v = tid < nblk ? pp[(int64_t)tid * (CH + 2)] : 0.0;
  v = wave_sum(v);
  if ((tid & 63) == 0) red[tid >> 6] = v;
  __syncthreads();
  if (tid != 0) return;
  const double sum = red[0] + red[1];
  double g;
  if (q < a.d) {
    g = -exp(-2.0 * th[q]) * sum;
    if (a.has_prior) g += (a.prior_shape - 1.0) - a.prior_rate * exp(th[q]);
  } else if (q == a.d) {
    g = 0.5 * sum;
  } else {
    g = 0.5 * clamp_exp(th[a.d + 1]) * sum;
  }
  grad[(int64_t)b * grad_ld + q] = g;
}

// ------------------------------------------------------------------------- selection
__device__ __forceinline__ bool hyp_before(double v, int i, double w, int j) {
  return v > w || (v == w && i < j);
}

__global__ __launch_bounds__(256) void hyp_select_k(const double *v, int32_t S, int32_t k,
                                                     const double *theta0, int32_t D,
                                                     int32_t *keep, double *x) {
  __shared__ double sv[256];
  __shared__ int si[256];
  __shared__ int picks[kHypBatch];
  const int tid = threadIdx.x;
  double pv = INFINITY;
  int pi = -1;
  for (int r = 0; r < k; ++r) {
    double bv = -INFINITY;
    int bi = INT32_MAX;
    for (int q = tid; q < S; q += 256) {
      const double val = isnan(v[q]) ? -INFINITY : v[q];
      if (hyp_before(pv, pi, val, q) && hyp_before(val, q, bv, bi)) bv = val, bi = q;
    }
    sv[tid] = bv;
    si[tid] = bi;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (tid < st && hyp_before(sv[tid + st], si[tid + st], sv[tid], si[tid])) {
        sv[tid] = sv[tid + st];
        si[tid] = si[tid + st];
      }
      __syncthreads();
    }
    pv = sv[0];
    pi = si[0];
    if (tid == 0) picks[r] = pi;
    __syncthreads();
  }
  for (int e = tid; e < k * D; e += 256) {
    const int r = e / D, c = e - r * D;
    if (picks[r] >= 0 && picks[r] < S) x[e] = theta0[(int64_t)picks[r] * D + c];
  }
  for (int r = tid; r < k; r += 256) keep[r] = picks[r];
}

// ---------------------------------------------------------------------------- L-BFGS
// One wavefront per start; lane l owns entries l and l + 64 of every D-vector (D <= 66).
// The steps follow the oracle's L-BFGS (two-loop recursion, Armijo backtracking by
// halving, curvature test before storing a pair, restart on a non-descent direction).
__global__ __launch_bounds__(64) void lbfgs_init_k(const LbfgsState st, int32_t D) {
  const int k = blockIdx.x, lane = threadIdx.x;
  for (int c = lane; c < D; c += 64) st.xt[(int64_t)k * D + c] = st.x[(int64_t)k * D + c];
  if (lane == 0) {
    st.status[k] = 0;
    st.phase[k] = 0;
    st.it[k] = 0;
    st.halv[k] = 0;
    st.npairs[k] = 0;
    st.head[k] = 0;
    st.active[k] = 1;
    st.F[k] = 0.0;
    st.t[k] = 1.0;
    st.slope[k] = 0.0;
  }
}

struct LVec {  // the two entries of a D-vector held by one lane (0 past D)
  double v[2];
};

__device__ __forceinline__ LVec lv_load(const double *p, int D) {
  LVec r;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int c = threadIdx.x + 64 * h;
    r.v[h] = c < D ? p[c] : 0.0;
  }
  return r;
}
__device__ __forceinline__ void lv_store(double *p, const LVec &a, int D) {
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int c = threadIdx.x + 64 * h;
    if (c < D) p[c] = a.v[h];
  }
}
__device__ __forceinline__ double lv_dot(const LVec &a, const LVec &b) {
  return wave_sum(fma(a.v[1], b.v[1], a.v[0] * b.v[0]));
}

__global__ __launch_bounds__(64) void lbfgs_step_k(const LbfgsState st, const LbfgsParams prm,
                                                    const double *value, const double *grad,
                                                    int64_t grad_ld) {
  const int k = blockIdx.x, lane = threadIdx.x, D = prm.D;
  if (st.status[k] != 0) return;
  const int64_t o = (int64_t)k * D;
  double *x = st.x + o, *xt = st.xt + o, *g = st.g + o, *p = st.p + o;
  // trial point: F = -value and its gradient
  const double Ft = -value[k];
  LVec gt;
  int bad = !isfinite(Ft);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int c = lane + 64 * h;
    gt.v[h] = c < D ? -grad[(int64_t)k * grad_ld + c] : 0.0;
    bad |= !isfinite(gt.v[h]);
  }
  const bool fin = wave_max((double)bad) == 0.0;
  auto finish = [&](int status) {
    if (lane == 0) {
      st.status[k] = status;
      st.active[k] = 0;
    }
  };
  // new direction from the current g (and the stored pairs), then the first trial point
  auto start_line_search = [&](const LVec &gv) {
    LVec d;
    const int np = st.npairs[k];
    bool steepest = np == 0;
    double slope = 0.0;
    if (!steepest) {
      LVec q = gv;
      double al[kLbfgsMem];
      const int head = st.head[k];
      // every stored pair loaded at once (slot of the u-th newest), then both loops run
      // on registers
      LVec Sv[kLbfgsMem], Yv[kLbfgsMem];
      double syv[kLbfgsMem];
#pragma unroll
      for (int u = 0; u < kLbfgsMem; ++u) {
        const int slot = (head - 1 - u + kLbfgsMem) % kLbfgsMem;
        Sv[u] = lv_load(st.S + (o * kLbfgsMem) + (int64_t)slot * D, D);
        Yv[u] = lv_load(st.Y + (o * kLbfgsMem) + (int64_t)slot * D, D);
        syv[u] = st.sy[(int64_t)k * kLbfgsMem + slot];
      }
#pragma unroll
      for (int u = 0; u < kLbfgsMem; ++u) {  // newest to oldest
        al[u] = 0.0;
        if (u < np) {
          al[u] = lv_dot(Sv[u], q) / syv[u];
#pragma unroll
          for (int h = 0; h < 2; ++h) q.v[h] -= al[u] * Yv[u].v[h];
        }
      }
      const double gamma = syv[0] / lv_dot(Yv[0], Yv[0]);  // the newest pair (np >= 1)
      LVec r;
#pragma unroll
      for (int h = 0; h < 2; ++h) r.v[h] = gamma * q.v[h];
#pragma unroll
      for (int u = kLbfgsMem - 1; u >= 0; --u) {  // oldest to newest
        if (u < np) {
          const double be = lv_dot(Yv[u], r) / syv[u];
#pragma unroll
          for (int h = 0; h < 2; ++h) r.v[h] += (al[u] - be) * Sv[u].v[h];
        }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) d.v[h] = -r.v[h];
      slope = lv_dot(gv, d);
      if (!(slope < 0.0)) steepest = true;  // not a descent direction: restart
      if (steepest && lane == 0) {
        st.npairs[k] = 0;
        st.head[k] = 0;
      }
    }
    if (steepest) {
      const double nrm = sqrt(lv_dot(gv, gv));
#pragma unroll
      for (int h = 0; h < 2; ++h) d.v[h] = -gv.v[h] / nrm;
      slope = lv_dot(gv, d);
    }
    lv_store(p, d, D);
    const LVec xv = lv_load(x, D);
    LVec xn;
#pragma unroll
    for (int h = 0; h < 2; ++h) xn.v[h] = xv.v[h] + d.v[h];
    lv_store(xt, xn, D);
    if (lane == 0) {
      st.slope[k] = slope;
      st.t[k] = 1.0;
      st.halv[k] = 0;
      st.phase[k] = 1;
    }
  };

  if (st.phase[k] == 0) {  // first evaluation, at the start itself
    if (lane == 0) st.F[k] = fin ? Ft : INFINITY;
    if (!fin) return finish(5);
    lv_store(g, gt, D);
    const double gmax = wave_max(fmax(fabs(gt.v[0]), fabs(gt.v[1])));
    if (prm.max_iter <= 0) return finish(3);
    if (gmax <= prm.gtol) return finish(1);
    start_line_search(gt);
    return;
  }
  const double F = st.F[k], t = st.t[k];
  const bool accept = fin && Ft <= F + kArmijoC1 * t * st.slope[k];
  if (!accept) {
    const int h2 = st.halv[k] + 1;
    if (h2 > kMaxHalvings) return finish(4);
    const double tn = 0.5 * t;
    const LVec xv = lv_load(x, D), pv = lv_load(p, D);
    LVec xn;
#pragma unroll
    for (int h = 0; h < 2; ++h) xn.v[h] = xv.v[h] + tn * pv.v[h];
    lv_store(xt, xn, D);
    if (lane == 0) {
      st.halv[k] = h2;
      st.t[k] = tn;
    }
    return;
  }
  // accepted: store the pair if it has positive curvature, move
  const LVec xv = lv_load(x, D), xtv = lv_load(xt, D), gv = lv_load(g, D);
  LVec sv, yv;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    sv.v[h] = xtv.v[h] - xv.v[h];
    yv.v[h] = gt.v[h] - gv.v[h];
  }
  const double sy = lv_dot(sv, yv), yy = lv_dot(yv, yv);
  if (sy > kCurvatureEps * yy) {
    const int head = st.head[k];
    lv_store(st.S + (o * kLbfgsMem) + (int64_t)head * D, sv, D);
    lv_store(st.Y + (o * kLbfgsMem) + (int64_t)head * D, yv, D);
    if (lane == 0) {
      st.sy[(int64_t)k * kLbfgsMem + head] = sy;
      st.head[k] = (head + 1) % kLbfgsMem;
      st.npairs[k] = min(st.npairs[k] + 1, kLbfgsMem);
    }
  }
  lv_store(x, xtv, D);
  lv_store(g, gt, D);
  const int it = st.it[k] + 1;
  if (lane == 0) {
    st.F[k] = Ft;
    st.it[k] = it;
  }
  // lane 0's writes of head / npairs must be visible to every lane before the direction
  __syncthreads();
  if (fabs(F - Ft) <= prm.ftol * fmax(fmax(fabs(F), fabs(Ft)), 1.0)) return finish(2);
  if (it >= prm.max_iter) return finish(3);
  const double gmax = wave_max(fmax(fabs(gt.v[0]), fabs(gt.v[1])));
  if (gmax <= prm.gtol) return finish(1);
  start_line_search(gt);
}

__global__ __launch_bounds__(64) void lbfgs_outputs_k(const LbfgsState st, int K, double *value,
                                                      int32_t *iters, int32_t *status) {
  const int k = blockIdx.x * 64 + threadIdx.x;
  if (k >= K) return;
  value[k] = -st.F[k];
  if (iters) iters[k] = st.it[k];
  if (status) status[k] = st.status[k];
}

}  // namespace

hipError_t launch_lbfgs_outputs(const LbfgsState &st, int K, double *value, int32_t *iters,
                                int32_t *status, hipStream_t s) {
  if (K < 1) return hipSuccess;
  hipLaunchKernelGGL(lbfgs_outputs_k, dim3((unsigned)((K + 63) / 64)), dim3(64), 0, s, st, K, value,
                     iters, status);
  return hipGetLastError();
}

hipError_t launch_hyp_terms(const uint32_t *codes, int32_t R, const TermDesc *td, int32_t d,
                            int32_t nf, double *T, hipStream_t s) {
  const int64_t nn = (int64_t)nf * nf;
  if (nn <= 0) return hipSuccess;
  hipLaunchKernelGGL(hyp_terms_k, dim3((unsigned)((nn + 255) / 256)), dim3(256), 0, s, codes, R,
                     td, d, nf, T);
  return hipGetLastError();
}

hipError_t launch_hyp_gram(const HypArgs &a, int B, double *K, hipStream_t s) {
  if (B < 1 || B > kHypBatch || a.d > kMaxD || a.nf < 1) return hipErrorInvalidValue;
  const int64_t nn = (int64_t)a.nf * a.nf;
  hipLaunchKernelGGL(hyp_gram_k, dim3((unsigned)((nn + 255) / 256), (unsigned)B), dim3(256), 0, s,
                     a, K);
  return hipGetLastError();
}

hipError_t launch_hyp_value(const HypArgs &a, int B, const double *L, const double *X,
                            double *value, double *alpha, double *z, hipStream_t s) {
  if (B < 1 || B > kHypBatch || a.nf > kMaxN) return hipErrorInvalidValue;
  hipLaunchKernelGGL(hyp_z_k, dim3((unsigned)((a.nf + 3) / 4), (unsigned)B), dim3(256), 0, s, a, X,
                     z);
  hipLaunchKernelGGL(hyp_alpha_k, dim3((unsigned)((a.nf + 63) / 64 + 1), (unsigned)B), dim3(256), 0,
                     s, a, X, z, alpha, L, value);
  return hipGetLastError();
}

int64_t hyp_grad_part_elems(int B, int d) {
  const int nchunks = (d + CH - 1) / CH;
  return (int64_t)B * std::max(nchunks, 1) * kHypGradBlocks * (CH + 2);
}

hipError_t launch_hyp_grad(const HypArgs &a, int B, const double *Kinv, const double *alpha,
                           double *part, double *grad, int64_t grad_ld, hipStream_t s) {
  if (B < 1 || B > kHypBatch || grad_ld < a.d + 2) return hipErrorInvalidValue;
  const int nchunks = std::max((a.d + CH - 1) / CH, 1);
  const int64_t npairs = (int64_t)a.nf * (a.nf + 1) / 2;
  const int nblk = (int)std::min<int64_t>(kHypGradBlocks, (npairs + 255) / 256);
  hipLaunchKernelGGL(hyp_grad_k, dim3((unsigned)nblk, (unsigned)B, (unsigned)nchunks), dim3(256), 0,
                     s, a, Kinv, alpha, part);
  hipLaunchKernelGGL(hyp_grad_final_k, dim3((unsigned)B, (unsigned)(a.d + 2)), dim3(128), 0, s, a,
                     part, nblk, nchunks, grad, grad_ld);
  return hipGetLastError();
}

hipError_t launch_hyp_select(const double *v, int32_t S, int32_t k, const double *theta0,
                             int32_t D, int32_t *keep, double *x, hipStream_t s) {
  if (k < 1 || k > kHypBatch || k > S) return hipErrorInvalidValue;
  hipLaunchKernelGGL(hyp_select_k, dim3(1), dim3(256), 0, s, v, S, k, theta0, D, keep, x);
  return hipGetLastError();
}

hipError_t launch_lbfgs_init(const LbfgsState &st, int K, int32_t D, hipStream_t s) {
  if (K < 1 || D > 128) return hipErrorInvalidValue;
  hipLaunchKernelGGL(lbfgs_init_k, dim3((unsigned)K), dim3(64), 0, s, st, D);
  return hipGetLastError();
}

hipError_t launch_lbfgs_step(const LbfgsState &st, int K, const LbfgsParams &prm,
                             const double *value, const double *grad, int64_t grad_ld,
                             hipStream_t s) {
  if (K < 1 || prm.D > 128 || grad_ld < prm.D) return hipErrorInvalidValue;
  hipLaunchKernelGGL(lbfgs_step_k, dim3((unsigned)K), dim3(64), 0, s, st, prm, value, grad,
                     grad_ld);
  return hipGetLastError();
}

}  // namespace bgp
