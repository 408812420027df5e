// fp32 cross-kernel K*[j][i] = s * Matern52(r(c_j, x_i)) between candidates and the
// model's observations (Sec. 3.2 kernel equations; per-type distances of Sec. 4.1),
// fused with the per-candidate sums the scorer needs on the same pass:
//   mu_j   = sum_i K*[j][i] alpha_i        (posterior mean, fp64 accumulation)
//   sens_j = sum_i K*[j][i] |alpha_i|      (conditioning of mu_j, drives the fp64 pass)
// (the classifier's latent mean is the contraction's job: a linear column of B), so
// the pass needs nothing of the classifier and can run while that is still being fitted.
//
// Mapping (one wavefront per 64 candidates): every lane owns one candidate and keeps
// its code words in registers, pre-scaled by 1/l for numeric parameters. The wave
// walks the observations in chunks of 32; an observation's record is uniform across
// the wave and is read with scalar loads. Small batches (too few candidate waves to
// fill the chip) also split the observations over blockIdx.y and sum the partial
// results in a second, tiny kernel. Each lane buffers its 32 kernel values in
// registers and writes them, split into fp16 high and low parts, as 8 16-byte stores, so
// every 128-byte line of K* is written whole by one lane (the L2 merges the partial-line
// requests).
#include <algorithm>
#include <type_traits>

#include "common.h"

namespace bgp {
namespace {

constexpr float kNegSqrt5Log2e = -3.225964182229561f;  // -sqrt(5) * log2(e)

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef float float2_t __attribute__((ext_vector_type(2)));

typedef __attribute__((address_space(4))) const uint32_t *const_u32p;

// Word offsets of the variant-padded observation x-record.
template <int NN, int NB, int NE, int ND>
struct XLay {
  static constexpr int B0 = NN, E0 = NN + NB, D0 = NN + NB + NE;
  static constexpr int RA = (D0 + 2 * ND + 1) & ~1;
  static constexpr int RX = (RA + 4 + 3) & ~3;
};

// DBG: the inspection instantiation, which also stores every pair's r2 and integer
// semimetric sums (the same values the pair's kernel value is computed from).
template <int NN, int NB, int NE, int ND, bool DBG>
__global__ __launch_bounds__(64) void xkernel(const XArgs a) {
  using L = XLay<NN, NB, NE, ND>;
  constexpr int CPL = 1;  // candidates per lane (rows row0 + 64 h + lane); 2 measured slower
  const int lane = threadIdx.x;
  const int64_t row0 = (int64_t)blockIdx.x * 64 * CPL;

  // Candidate words (natural layout) into registers; padded slots are zero, as are
  // the matching slots of the observation records, so they contribute nothing.
  float cn[CPL][NN > 0 ? NN : 1];
  uint32_t cb[CPL][NB > 0 ? NB : 1];
  uint32_t ce[CPL][NE > 0 ? NE : 1];
  uint32_t cd[CPL][ND > 0 ? 2 * ND : 2];
#pragma unroll
  for (int h = 0; h < CPL; ++h) {
    const int64_t j = row0 + h * 64 + lane;
#pragma unroll
    for (int q = 0; q < NN; ++q)
      cn[h][q] = q < a.n_num ? __uint_as_float(a.cand[(int64_t)q * a.ldc + j]) * a.num_scale[q] : 0.0f;
#pragma unroll
    for (int q = 0; q < NB; ++q)
      cb[h][q] = q < a.n_bits ? a.cand[(int64_t)(a.w_bits0 + q) * a.ldc + j] : 0u;
#pragma unroll
    for (int q = 0; q < NE; ++q)
      ce[h][q] = q < a.n_eq ? a.cand[(int64_t)(a.w_eq0 + q) * a.ldc + j] : 0u;
#pragma unroll
    for (int q = 0; q < 2 * ND; ++q)
      cd[h][q] = q < 2 * a.n_dot ? a.cand[(int64_t)(a.w_dot0 + q) * a.ldc + j] : 0u;
  }

  double mu[CPL];
  float sens[CPL];
#pragma unroll
  for (int h = 0; h < CPL; ++h) mu[h] = 0.0, sens[h] = 0.0f;
  const const_u32p obs = (const_u32p)a.obs;
  const int n = min(a.n, (int)(blockIdx.y + 1) * a.i_chunk);  // end of this split
  // One chunk of 32 observations. Whole chunks carry no per-observation bounds test:
  // with one, every observation's scalar loads sit behind a branch and each pair waits
  // for its own record; without it the loads of later observations issue early.
  auto chunk = [&](const int i0, auto whole_t) {
    constexpr int RW = L::D0 + 2 * ND;  // code words of a record (alpha, |alpha| follow)
    // a whole chunk with records small enough for two to sit in scalar registers runs
    // pipelined and without bounds tests (larger records keep the tested form: untested,
    // their loads are all hoisted and spill)
    constexpr bool pf = decltype(whole_t)::value && RW <= 32;
    typedef __attribute__((address_space(4))) const uint64_t *const_u64p;
    float kv[CPL][32];
    // an observation record: its code words, alpha (fp64) and |alpha| (fp32)
    auto load_rec = [&](int i, uint32_t *w, uint64_t &al, uint32_t &ab) {
      const const_u32p o = obs + i * L::RX;
#pragma unroll
      for (int q = 0; q < RW; ++q) w[q] = o[q];
      al = *(const_u64p)(o + L::RA);
      ab = o[L::RA + 2];
    };
    // the record of the next observation is loaded before the current one is used
    uint32_t nx[RW > 0 ? RW : 1], nx_ab = 0u;
    uint64_t nx_al = 0u;
    if (pf) load_rec(i0, nx, nx_al, nx_ab);
#pragma unroll
    for (int t = 0; t < 32; ++t) {
      const int i = i0 + t;
      float k[CPL];
#pragma unroll
      for (int h = 0; h < CPL; ++h) k[h] = 0.0f;
      if (pf || i < n) {
        uint32_t o[RW > 0 ? RW : 1], o_ab;
        uint64_t o_al;
        if (pf) {
#pragma unroll
          for (int q = 0; q < RW; ++q) o[q] = nx[q];
          o_al = nx_al;
          o_ab = nx_ab;
          // scalar loads return out of order, so any use waits for all of them: wait for
          // this record first, then issue the next one, then compute (the scheduling
          // barriers keep the wait and the next loads between the two computations)
          __builtin_amdgcn_sched_barrier(0);
          __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
          __builtin_amdgcn_sched_barrier(0);
          if (t + 1 < 32) load_rec(i + 1, nx, nx_al, nx_ab);
          __builtin_amdgcn_sched_barrier(0);
        } else {
          load_rec(i, o, o_al, o_ab);
        }
        const double al = __builtin_bit_cast(double, o_al);
        const float aabs = __uint_as_float(o_ab);
#pragma unroll
        for (int h = 0; h < CPL; ++h) {
          const int64_t jd = row0 + h * 64 + lane;  // inspection: pair (jd, i)
          const bool dbg = DBG && jd < a.dbg_count && i < a.n;
          const int nw = a.n_bits + a.n_eq + a.n_dot;
          int32_t *cnt = DBG ? a.dbg_cnt + (jd * a.n + i) * nw : nullptr;
          float r2 = 0.0f;
#pragma unroll
          for (int q = 0; q < NN; ++q) {
            const float d = cn[h][q] - __uint_as_float(o[q]);
            r2 = fmaf(d, d, r2);
          }
#pragma unroll
          for (int q = 0; q < NB; ++q) {
            const uint32_t pc = __popc(cb[h][q] ^ o[L::B0 + q]);
            if (dbg && q < a.n_bits) cnt[q] = (int32_t)pc;
            r2 = fmaf(a.bits_w[q], (float)pc, r2);
          }
#pragma unroll
          for (int q = 0; q < NE; ++q) {
            const bool ne = ce[h][q] != o[L::E0 + q];
            if (dbg && q < a.n_eq) cnt[a.n_bits + q] = ne ? 1 : 0;
            r2 += ne ? a.eq_w[q] : 0.0f;
          }
#pragma unroll
          for (int q = 0; q < ND; ++q) {
            uint32_t dt = __builtin_amdgcn_udot4(cd[h][2 * q], o[L::D0 + 2 * q], 0u, false);
            dt = __builtin_amdgcn_udot4(cd[h][2 * q + 1], o[L::D0 + 2 * q + 1], dt, false);
            const int32_t sd = a.dot_s2[q] - (int32_t)dt;
            if (dbg && q < a.n_dot) cnt[a.n_bits + a.n_eq + q] = sd;
            r2 = fmaf(a.dot_w2[q], (float)sd, r2);
          }
          if (dbg) a.dbg_r2[jd * a.n + i] = r2;
          const float r = __builtin_amdgcn_sqrtf(r2);
          const float e = __builtin_amdgcn_exp2f(r * kNegSqrt5Log2e);
          k[h] = fmaf(a.A2, r2, fmaf(a.A1, r, a.A0)) * e;
          // keep k as one register: folded into the fp16 split at the end of the chunk,
          // its two factors would each stay live until then
          asm("" : "+v"(k[h]));
          mu[h] = fma((double)k[h], al, mu[h]);
          sens[h] = fmaf(k[h], aabs, sens[h]);
        }
      }
#pragma unroll
      for (int h = 0; h < CPL; ++h) kv[h][t] = k[h];
    }
    // columns i0..i0+31 of each candidate's row (zeros past n: lda is a multiple of 32),
    // already scaled by 2^kexp (through A0..A2), split into fp16 high and low parts
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
      half8 hi[4], lo[4];
#pragma unroll
      for (int t = 0; t < 32; t += 2) {
        // pairwise conversions (v_cvt_pk_f16_f32, round to nearest even)
        const float2_t k2 = {kv[h][t], kv[h][t + 1]};
        const half2_t h2 = __builtin_convertvector(k2, half2_t);
        const half2_t l2 = __builtin_convertvector(k2 - __builtin_convertvector(h2, float2_t), half2_t);
        hi[t >> 3][t & 7] = h2[0];
        hi[t >> 3][(t & 7) + 1] = h2[1];
        lo[t >> 3][t & 7] = l2[0];
        lo[t >> 3][(t & 7) + 1] = l2[1];
      }
      half8 *dst = reinterpret_cast<half8 *>(a.Kstar + (row0 + h * 64 + lane) * 2 * a.lda + 2 * i0);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        dst[q] = hi[q];
        dst[4 + q] = lo[q];
      }
    }
  };
  const int i_begin = blockIdx.y * a.i_chunk;
  const int i_whole = i_begin + ((max(n - i_begin, 0)) & ~31);  // end of the whole chunks
  for (int i0 = i_begin; i0 < i_whole; i0 += 32) chunk(i0, std::true_type{});
  if (i_whole < n) chunk(i_whole, std::false_type{});
  // the sums were taken over the scaled kernel values: undo the power-of-two scale
#pragma unroll
  for (int h = 0; h < CPL; ++h) {
    const int64_t j = (int64_t)blockIdx.y * a.rows + row0 + h * 64 + lane;
    a.mu[j] = mu[h] * (double)a.kinv;
    a.sens[j] = sens[h] * a.kinv;
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

struct Variant {
  int nn, nb, ne, nd;
};
// Exact fits for common space shapes first, then padded general variants.
constexpr Variant kVariants[] = {
    {4, 1, 0, 0}, {4, 2, 0, 0}, {8, 1, 0, 0}, {10, 0, 0, 0}, {8, 4, 0, 1},
    {8, 4, 2, 2}, {16, 8, 4, 2}, {32, 16, 8, 4}, {64, 64, 64, 16}};
constexpr int kNumVariants = sizeof(kVariants) / sizeof(kVariants[0]);

}  // namespace

int xkernel_variant(int n_num, int n_bits, int n_eq, int n_dot) {
  int best = -1, best_cost = 1 << 30;
  for (int v = 0; v < kNumVariants; ++v) {
    const Variant &k = kVariants[v];
    if (n_num > k.nn || n_bits > k.nb || n_eq > k.ne || n_dot > k.nd) continue;
    const int cost = 2 * k.nn + 4 * k.nb + 3 * k.ne + 5 * k.nd;  // VALU ops per pair
    if (cost < best_cost) best = v, best_cost = cost;
  }
  return best;
}

void xkernel_layout(int variant, int *B0, int *E0, int *D0, int *RA, int *RX) {
  const Variant &k = kVariants[variant];
  *B0 = k.nn;
  *E0 = k.nn + k.nb;
  *D0 = k.nn + k.nb + k.ne;
  *RA = (*D0 + 2 * k.nd + 1) & ~1;
  *RX = (*RA + 4 + 3) & ~3;
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
                          bool inspect) {
  if (a0.rows <= 0) return hipSuccess;
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
  const dim3 grid((unsigned)(a.rows / 64), (unsigned)ns), block(64);
#define BGP_XK(V, NN, NB, NE, ND)                                                   \
  case V:                                                                          \
    if (inspect) hipLaunchKernelGGL((xkernel<NN, NB, NE, ND, true>), grid, block, 0, s, a); \
    else hipLaunchKernelGGL((xkernel<NN, NB, NE, ND, false>), grid, block, 0, s, a); \
    break;
  switch (variant) {
    BGP_XK(0, 4, 1, 0, 0)
    BGP_XK(1, 4, 2, 0, 0)
    BGP_XK(2, 8, 1, 0, 0)
    BGP_XK(3, 10, 0, 0, 0)
    BGP_XK(4, 8, 4, 0, 1)
    BGP_XK(5, 8, 4, 2, 2)
    BGP_XK(6, 16, 8, 4, 2)
    BGP_XK(7, 32, 16, 8, 4)
    BGP_XK(8, 64, 64, 64, 16)
    default: return hipErrorInvalidValue;
  }
#undef BGP_XK
  if (ns > 1)
    hipLaunchKernelGGL(xsplit_reduce, dim3((unsigned)((a.rows + 255) / 256)), dim3(256), 0, s,
                       sp.mu, sp.sens, ns, a.rows, a0.mu, a0.sens);
  return hipGetLastError();
}

}  // namespace bgp
