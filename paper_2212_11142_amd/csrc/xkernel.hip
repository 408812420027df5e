// fp32 cross-kernel K*[j][i] = s * Matern52(r(c_j, x_i)) between candidates and the
// model's observations (Sec. 3.2 kernel equations; per-type distances of Sec. 4.1),
// fused with the per-candidate sums the scorer needs on the same pass:
//   mu_j   = sum_i K*[j][i] alpha_i        (posterior mean, fp64 accumulation)
//   sens_j = sum_i K*[j][i] |alpha_i|      (conditioning of mu_j, drives the fp64 pass)
// (the classifier's latent mean is the contraction's job: a linear column of B), so
// the pass needs nothing of the classifier and can run while that is still being fitted.
//
// The numeric part of the squared distance is a dense contraction over the numeric
// parameters, taken on fp64 MFMA (v_mfma_f64_16x16x4f64) with augmented embeddings:
// candidate [a, |a|^2, 1] against observation [-2 b, 1, |b|^2] (a, b the codes scaled by
// 1/l) gives |a - b|^2 = sum_p (u_p - u'_p)^2 / l_p^2 directly, in fp64, so the
// expansion loses nothing to cancellation before its one rounding to fp32. The integer
// semimetrics (popcounts of one-hot / pair-order bit sets, equalities, Spearman dot
// products) and the Matern function stay on the vector ALU.
//
// Mapping: a wavefront takes CB blocks of 16 candidates and walks the observations in
// chunks of 32 (two 16-observation MFMA blocks). In an MFMA result lane l holds
// observations g + 4 v (g = l >> 4, v = 0..3) of a block for candidate l & 15, so each
// lane evaluates 8 pairs per chunk and candidate block. The observation side of a chunk
// is pre-arranged at fit time: the MFMA A operands in lane order, and per lane group g a
// record of its 8 observations' integer words, alpha and |alpha| (one 16-byte load per
// 4 words, the same address for the 16 lanes of a group). A lane's 8 kernel values of
// a chunk are stored contiguously (positions 8 g .. 8 g + 7 of the chunk: observation
// 16 ob + g + 4 v at 8 g + 4 ob + v, the order in which B^T is packed), split into fp16
// high and low parts, as two 16-byte stores.
#include <algorithm>

#include "common.h"

namespace bgp {
namespace {

constexpr float kNegSqrt5Log2e = -3.225964182229561f;  // -sqrt(5) * log2(e)

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx8 __attribute__((ext_vector_type(8)));
typedef double doublex4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// KS: MFMA k-steps of 4 augmented numeric dimensions (n_num + 2 <= 4 KS); NB, NE, ND:
// BITS words, EQ words and Spearman permutations (upper bounds; unused slots are zero on
// both sides); CB: candidate blocks of 16 per wavefront; DBG: the inspection
// instantiation, which also stores every pair's r2 and integer word sums.
template <int KS, int NB, int NE, int ND, int CB, bool DBG>
__global__ __launch_bounds__(64) void xkernel(const XArgs a) {
  constexpr int RW = xrec_words(NB, NE, ND);
  const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
  const int64_t row0 = (int64_t)blockIdx.x * 16 * CB;

  // candidate side: MFMA B operands [k = 4 s + g] of each block, and the integer words
  double bop[CB][KS];
  uint32_t cbw[CB][NB > 0 ? NB : 1], cew[CB][NE > 0 ? NE : 1], cdw[CB][ND > 0 ? 2 * ND : 2];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int64_t j = row0 + 16 * cb + c;
    double nrm = 0.0;
#pragma unroll 4
    for (int q = 0; q < a.n_num; ++q) {
      const double x = (double)__uint_as_float(a.cand[(int64_t)q * a.ldc + j]) * a.num_scale64[q];
      nrm = fma(x, x, nrm);
    }
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int q = 4 * s + g;
      double v = 0.0;
      if (q < a.n_num) v = (double)__uint_as_float(a.cand[(int64_t)q * a.ldc + j]) * a.num_scale64[q];
      else if (q == a.n_num) v = nrm;
      else if (q == a.n_num + 1) v = 1.0;
      bop[cb][s] = v;
    }
#pragma unroll
    for (int q = 0; q < NB; ++q) cbw[cb][q] = q < a.n_bits ? a.cand[(int64_t)(a.w_bits0 + q) * a.ldc + j] : 0u;
#pragma unroll
    for (int q = 0; q < NE; ++q) cew[cb][q] = q < a.n_eq ? a.cand[(int64_t)(a.w_eq0 + q) * a.ldc + j] : 0u;
#pragma unroll
    for (int q = 0; q < 2 * ND; ++q)
      cdw[cb][q] = q < 2 * a.n_dot ? a.cand[(int64_t)(a.w_dot0 + q) * a.ldc + j] : 0u;
  }

  double mu[CB];
  float sens[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) mu[cb] = 0.0, sens[cb] = 0.0f;

  const int nchunk = (a.n + 31) >> 5, per = a.i_chunk >> 5;
  const int kc0 = blockIdx.y * per, kc1 = min(nchunk, kc0 + per);
  const int kwhole = min(kc1, a.n >> 5);  // chunks before it hold 32 observations each

  for (int kc = kc0; kc < kc1; ++kc) {
    // observation side of the chunk
    const double *xa = a.xa64 + ((int64_t)kc * 2 * KS) * 64 + lane;
    double aop[2][KS];
#pragma unroll
    for (int ob = 0; ob < 2; ++ob)
#pragma unroll
      for (int s = 0; s < KS; ++s) aop[ob][s] = xa[(ob * KS + s) * 64];
    u32x4 rec[RW / 4];
    const u32x4 *xr = reinterpret_cast<const u32x4 *>(a.xr + ((int64_t)kc * 4 + g) * RW);
#pragma unroll
    for (int q = 0; q < RW / 4; ++q) rec[q] = xr[q];
    const uint32_t *rw = reinterpret_cast<const uint32_t *>(rec);
    // record: alpha (fp64) [8], |alpha| [8], then per word q its 8 observations
    auto alpha = [&](int t) {
      return __builtin_bit_cast(double, (uint64_t)rw[2 * t] | ((uint64_t)rw[2 * t + 1] << 32));
    };
    auto aabs = [&](int t) { return __uint_as_float(rw[16 + t]); };
    auto word = [&](int q, int t) { return rw[24 + 8 * q + t]; };
    const bool whole = kc < kwhole;  // all 32 observations of the chunk exist

#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      float kv[8];
#pragma unroll
      for (int ob = 0; ob < 2; ++ob) {
        doublex4 d = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int s = 0; s < KS; ++s) d = __builtin_amdgcn_mfma_f64_16x16x4f64(aop[ob][s], bop[cb][s], d, 0, 0, 0);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int t = 4 * ob + v;                 // record slot of observation i
          const int i = 32 * kc + 16 * ob + g + 4 * v;
          const int64_t jd = row0 + 16 * cb + c;
          const bool dbg = DBG && jd < a.dbg_count && i < a.n;
          const int nw = a.n_bits + a.n_eq + a.n_dot;
          int32_t *cnt = DBG ? a.dbg_cnt + (jd * a.n + i) * nw : nullptr;
          float r2 = (float)d[v];
#pragma unroll
          for (int q = 0; q < NB; ++q) {
            const uint32_t pc = __popc(cbw[cb][q] ^ word(q, t));
            if (dbg && q < a.n_bits) cnt[q] = (int32_t)pc;
            r2 = fmaf(a.bits_w[q], (float)pc, r2);
          }
#pragma unroll
          for (int q = 0; q < NE; ++q) {
            const bool ne = cew[cb][q] != word(NB + q, t);
            if (dbg && q < a.n_eq) cnt[a.n_bits + q] = ne ? 1 : 0;
            r2 += ne ? a.eq_w[q] : 0.0f;
          }
#pragma unroll
          for (int q = 0; q < ND; ++q) {
            uint32_t dt = __builtin_amdgcn_udot4(cdw[cb][2 * q], word(NB + NE + 2 * q, t), 0u, false);
            dt = __builtin_amdgcn_udot4(cdw[cb][2 * q + 1], word(NB + NE + 2 * q + 1, t), dt, false);
            const int32_t sd = a.dot_s2[q] - (int32_t)dt;
            if (dbg && q < a.n_dot) cnt[a.n_bits + a.n_eq + q] = sd;
            r2 = fmaf(a.dot_w2[q], (float)sd, r2);
          }
          // the fp64 numeric part of a coincident pair may round to a tiny negative
          // value: the root is taken of |r2| (a free operand modifier)
          if (dbg) a.dbg_r2[jd * a.n + i] = r2;
          const float r = __builtin_amdgcn_sqrtf(fabsf(r2));
          const float e = __builtin_amdgcn_exp2f(r * kNegSqrt5Log2e);
          float k = fmaf(a.A2, r2, fmaf(a.A1, r, a.A0)) * e;
          if (!whole) k = i < a.n ? k : 0.0f;  // padding observations of the last chunk
          mu[cb] = fma((double)k, alpha(t), mu[cb]);
          sens[cb] = fmaf(k, aabs(t), sens[cb]);
          kv[t] = k;
        }
      }
      // positions 8 g + t of the chunk (t = 4 ob + v), already scaled by 2^kexp
      // (through A0..A2), split into fp16 high and low parts (none when only the means
      // are asked for: Kstar null, uniform over the launch)
      if (a.Kstar) {
        const floatx8 k8 = {kv[0], kv[1], kv[2], kv[3], kv[4], kv[5], kv[6], kv[7]};
        const half8 hi = __builtin_convertvector(k8, half8);
        const half8 lo = __builtin_convertvector(k8 - __builtin_convertvector(hi, floatx8), half8);
        half8 *dst = reinterpret_cast<half8 *>(a.Kstar + (row0 + 16 * cb + c) * 2 * a.lda + 64 * kc + 8 * g);
        dst[0] = hi;
        dst[4] = lo;
      }
    }
  }
  // sums over the four lane groups (each holds a quarter of the observations), in a
  // fixed order; the sums were taken over the scaled kernel values: undo the scale
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    double m = mu[cb];
    float sv = sens[cb];
    m += __shfl_xor(m, 16);
    sv += __shfl_xor(sv, 16);
    m += __shfl_xor(m, 32);
    sv += __shfl_xor(sv, 32);
    if (g == 0) {
      const int64_t j = (int64_t)blockIdx.y * a.rows + row0 + 16 * cb + c;
      a.mu[j] = m * (double)a.kinv;
      a.sens[j] = sv * a.kinv;
    }
  }
}

// Sum of the per-split partial results, in split order (deterministic).
__global__ __launch_bounds__(256) void xsplit_reduce(const double *pmu, const float *psens,
                                                     int nsplit, int64_t rows, double *mu,
                                                     float *sens) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= rows) return;
  double m = 0.0;
  float sv = 0.0f;
  for (int q = 0; q < nsplit; ++q) {
    m += pmu[q * rows + j];
    sv += psens[q * rows + j];
  }
  mu[j] = m;
  sens[j] = sv;
}

// Observation side, built once per fit (see the mapping above). XA[kc][ob][s][l] =
// augmented embedding [-2 b, 1, |b|^2] of observation 32 kc + 16 ob + (l & 15), entry
// 4 s + (l >> 4) (zero for observations >= n). XR[kc][g] = the record of observations
// 32 kc + 16 ob + g + 4 v, slot t = 4 ob + v.
__global__ __launch_bounds__(256) void make_xobs_k(const uint32_t *codes, int32_t R, int32_t n,
                                                   XObsLayout lay, const double *num_scale,
                                                   const double *alpha, int32_t n_f,
                                                   double *xa, uint32_t *xr) {
  const int nchunk = (n + 31) >> 5;
  const int64_t na = (int64_t)nchunk * 2 * lay.ks * 64;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx < na) {
    const int l = (int)(idx & 63);
    const int64_t rest = idx >> 6;
    const int s = (int)(rest % lay.ks);
    const int ob = (int)((rest / lay.ks) & 1);
    const int kc = (int)(rest / (2 * lay.ks));
    const int i = 32 * kc + 16 * ob + (l & 15), q = 4 * s + (l >> 4);
    double v = 0.0;
    if (i < n) {
      const uint32_t *cw = codes + (int64_t)i * R;
      if (q < lay.n_num) {
        v = -2.0 * (double)__uint_as_float(cw[q]) * num_scale[q];
      } else if (q == lay.n_num) {
        v = 1.0;
      } else if (q == lay.n_num + 1) {
        double nrm = 0.0;
        for (int p = 0; p < lay.n_num; ++p) {
          const double x = (double)__uint_as_float(cw[p]) * num_scale[p];
          nrm = fma(x, x, nrm);
        }
        v = nrm;
      }
    }
    xa[idx] = v;
    return;
  }
  const int64_t r = idx - na;  // one thread per (chunk, group, slot)
  if (r >= (int64_t)nchunk * 32) return;
  const int t = (int)(r & 7), g = (int)((r >> 3) & 3), kc = (int)(r >> 5);
  const int ob = t >> 2, v = t & 3;
  const int i = 32 * kc + 16 * ob + g + 4 * v;
  uint32_t *o = xr + ((int64_t)kc * 4 + g) * lay.rw;
  const double al = i < n_f ? alpha[i] : 0.0;
  const uint64_t bits = __builtin_bit_cast(uint64_t, al);
  o[2 * t] = (uint32_t)bits;
  o[2 * t + 1] = (uint32_t)(bits >> 32);
  o[16 + t] = __float_as_uint((float)fabs(al));
  const uint32_t *cw = codes + (int64_t)min(i, n - 1) * R;
  const bool in = i < n;
  for (int q = 0; q < lay.nb; ++q) o[24 + 8 * q + t] = (in && q < lay.n_bits) ? cw[lay.w_bits0 + q] : 0u;
  for (int q = 0; q < lay.ne; ++q)
    o[24 + 8 * (lay.nb + q) + t] = (in && q < lay.n_eq) ? cw[lay.w_eq0 + q] : 0u;
  for (int q = 0; q < 2 * lay.nd; ++q)
    o[24 + 8 * (lay.nb + lay.ne + q) + t] = (in && q < 2 * lay.n_dot) ? cw[lay.w_dot0 + q] : 0u;
  if (t == 0)  // record padding
    for (int q = 24 + 8 * (lay.nb + lay.ne + 2 * lay.nd); q < lay.rw; ++q) o[q] = 0u;
}

struct Variant {
  int ks, nb, ne, nd, cb;
};
// Exact fits for common space shapes first, then padded general variants.
constexpr Variant kVariants[] = {
    {2, 1, 0, 0, 4}, {2, 2, 0, 0, 4}, {3, 0, 0, 0, 4}, {3, 1, 0, 0, 4}, {3, 4, 0, 1, 2},
    {3, 4, 2, 2, 2}, {5, 8, 4, 2, 2}, {9, 16, 8, 4, 1}, {17, 64, 64, 16, 1}};
constexpr int kNumVariants = sizeof(kVariants) / sizeof(kVariants[0]);

}  // namespace

int xkernel_variant(int n_num, int n_bits, int n_eq, int n_dot) {
  const int ks = (n_num + 2 + 3) / 4;
  int best = -1, best_cost = 1 << 30;
  for (int v = 0; v < kNumVariants; ++v) {
    const Variant &k = kVariants[v];
    if (ks > k.ks || n_bits > k.nb || n_eq > k.ne || n_dot > k.nd) continue;
    const int cost = 2 * k.ks + 4 * k.nb + 3 * k.ne + 5 * k.nd;  // ~ VALU slots per pair
    if (cost < best_cost) best = v, best_cost = cost;
  }
  return best;
}

XObsLayout xobs_layout(int variant, int n_num, int n_bits, int n_eq, int n_dot, int w_bits0,
                       int w_eq0, int w_dot0) {
  const Variant &k = kVariants[variant];
  XObsLayout l{};
  l.ks = k.ks;
  l.nb = k.nb;
  l.ne = k.ne;
  l.nd = k.nd;
  l.rw = xrec_words(k.nb, k.ne, k.nd);
  l.n_num = n_num;
  l.n_bits = n_bits;
  l.n_eq = n_eq;
  l.n_dot = n_dot;
  l.w_bits0 = w_bits0;
  l.w_eq0 = w_eq0;
  l.w_dot0 = w_dot0;
  return l;
}

size_t xobs_a_doubles(int n, int ks) { return (size_t)((n + 31) / 32) * 2 * ks * 64; }
size_t xobs_r_words(int n, int rw) { return (size_t)((n + 31) / 32) * 4 * rw; }
size_t xobs_a_doubles_max(int n) {
  int ks = 0;
  for (const Variant &k : kVariants) ks = std::max(ks, k.ks);
  return xobs_a_doubles(n, ks);
}
size_t xobs_r_words_max(int n) {
  int rw = 0;
  for (const Variant &k : kVariants) rw = std::max(rw, xrec_words(k.nb, k.ne, k.nd));
  return xobs_r_words(n, rw);
}

hipError_t launch_make_xobs(const uint32_t *codes, int32_t R, int32_t n, const XObsLayout &lay,
                            const double *num_scale, const double *alpha, int32_t n_f,
                            double *xa, uint32_t *xr, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t tot = (int64_t)xobs_a_doubles(n, lay.ks) + (int64_t)((n + 31) / 32) * 32;
  hipLaunchKernelGGL(make_xobs_k, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, codes,
                     R, n, lay, num_scale, alpha, n_f, xa, xr);
  return hipGetLastError();
}

int xkernel_splits(int64_t rows, int n) {
  constexpr int64_t kWaves = 1024;
  const int64_t waves = rows / 64;
  const int chunks = (n + 31) / 32;
  if (waves >= kWaves || chunks <= 1) return 1;
  const int want = (int)std::min<int64_t>(chunks, (kWaves + waves - 1) / std::max<int64_t>(waves, 1));
  const int per = (chunks + want - 1) / want;  // chunks per split
  return (chunks + per - 1) / per;
}

hipError_t launch_xkernel(const XArgs &a0, int variant, const XSplit &sp, hipStream_t s,
                          bool inspect, bool reduce) {
  if (a0.rows <= 0) return hipSuccess;
  if (variant < 0 || variant >= kNumVariants) return hipErrorInvalidValue;
  if (inspect && (!a0.dbg_r2 || !a0.dbg_cnt)) return hipErrorInvalidValue;
  XArgs a = a0;
  const int chunks = (a.n + 31) / 32;
  const int ns = std::max(1, std::min(sp.nsplit, chunks));
  if (ns != xkernel_splits(a.rows, a.n)) return hipErrorInvalidValue;
  a.i_chunk = ((chunks + ns - 1) / ns) * 32;
  if (ns > 1) {
    if (!sp.mu || !sp.sens) return hipErrorInvalidValue;
    a.mu = sp.mu;
    a.sens = sp.sens;
  }
  const int cand_per_wave = 16 * kVariants[variant].cb;
  if (a.rows % cand_per_wave) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(a.rows / cand_per_wave), (unsigned)ns), block(64);
#define BGP_XK(V, KS, NB, NE, ND, CB)                                                        \
  case V:                                                                                    \
    if (inspect) hipLaunchKernelGGL((xkernel<KS, NB, NE, ND, CB, true>), grid, block, 0, s, a); \
    else hipLaunchKernelGGL((xkernel<KS, NB, NE, ND, CB, false>), grid, block, 0, s, a);        \
    break;
  switch (variant) {
    BGP_XK(0, 2, 1, 0, 0, 4)
    BGP_XK(1, 2, 2, 0, 0, 4)
    BGP_XK(2, 3, 0, 0, 0, 4)
    BGP_XK(3, 3, 1, 0, 0, 4)
    BGP_XK(4, 3, 4, 0, 1, 2)
    BGP_XK(5, 3, 4, 2, 2, 2)
    BGP_XK(6, 5, 8, 4, 2, 2)
    BGP_XK(7, 9, 16, 8, 4, 1)
    BGP_XK(8, 17, 64, 64, 16, 1)
    default: return hipErrorInvalidValue;
  }
#undef BGP_XK
  if (ns > 1 && reduce)
    hipLaunchKernelGGL(xsplit_reduce, dim3((unsigned)((a.rows + 255) / 256)), dim3(256), 0, s,
                       sp.mu, sp.sens, ns, a.rows, a0.mu, a0.sens);
  return hipGetLastError();
}

}  // namespace bgp
