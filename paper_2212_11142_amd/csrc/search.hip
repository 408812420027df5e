// Multi-start local search over the acquisition function (Sec. 3.3): the best of the
// scored candidates become starting points, each start moves to its best one-parameter
// neighbour while that improves the acquisition value. The scoring itself is gp_score;
// the kernels here pick the starts, generate the neighbours and take the moves.
//
// Configurations are kept in the raw column formats of the boundary, as 4-byte words:
// a REAL value is 2 words (its float64 bits), INT/ORD/CAT 1 word, a PERM row m words.
//
// Neighbours of a configuration, parameter by parameter in space order (the paper only
// says "all configurations reachable by modifying a single parameter"):
//   REAL  the transformed value (log2 if flagged) minus, then plus, 1/16 of its
//         transformed range (a step leaving the range is not a neighbour);
//   INT   value - 1, value + 1 (within lo..hi);   ORD   index - 1, index + 1;
//   CAT   every other level, ascending;
//   PERM  every exchange of the positions of two items i < j, (i, j) ascending.
// Out-of-range neighbours are scored as copies of the current configuration with a
// zero mask, so their acquisition value is 0 and never wins a strict comparison.
#include "encode_param.h"

namespace bgp {
namespace {

// The descriptor and column tables arrive as kernel arguments (a few KB) and are read
// with data-dependent indices; one parallel copy into LDS replaces chains of dependent
// argument loads.
template <typename T>
__device__ __forceinline__ void ls_stage(T &dst, const T &src) {
  static_assert(sizeof(T) % 4 == 0, "word copy");
  const uint32_t *s = reinterpret_cast<const uint32_t *>(&src);
  uint32_t *d = reinterpret_cast<uint32_t *>(&dst);
  for (int q = threadIdx.x; q < (int)(sizeof(T) / 4); q += blockDim.x) d[q] = s[q];
}

// (value, index) order of the start selection: larger value first, lower index on ties
__device__ __forceinline__ bool ls_before(float v, int64_t i, float w, int64_t j) {
  return v > w || (v == w && i < j);
}

// Block-wide best (in ls_before order) of one (value, index) per thread; all threads
// get the result. A wavefront reduces with lane exchanges, the waves through sv/si (one
// slot per wave).
__device__ __forceinline__ void ls_block_best(float &v, int64_t &i, float *sv, int64_t *si) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float w = __shfl_xor(v, o);
    const int64_t j = __shfl_xor(i, o);
    if (ls_before(w, j, v, i)) {
      v = w;
      i = j;
    }
  }
  const int wid = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sv[wid] = v;
    si[wid] = i;
  }
  __syncthreads();
  v = sv[0];
  i = si[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w)
    if (ls_before(sv[w], si[w], v, i)) {
      v = sv[w];
      i = si[w];
    }
  __syncthreads();  // the slots are free again
}

// k rounds over x[lo, hi): round r takes the best element after the round r-1 pick in
// ls_before order (no exclusion list needed). A NaN value ranks as -inf, so every index
// can be picked and a range of at least k elements yields k picks; missing picks of a
// shorter range are (-inf, INT64_MAX). A thread keeps its first kTopkCache elements in
// registers; elements past those are read again in every round.
constexpr int kTopkCache = 16;
__device__ void ls_topk_range(const float *x, const int64_t *xi, int64_t lo, int64_t hi, int k,
                              float *out_v, int64_t *out_i, float *sv, int64_t *si) {
  auto load = [&](int64_t q, float &v, int64_t &i) {
    v = __builtin_isnan(x[q]) ? -INFINITY : x[q];
    i = xi ? xi[q] : q;
  };
  float cv[kTopkCache];
  int64_t ci[kTopkCache];
#pragma unroll
  for (int c = 0; c < kTopkCache; ++c) {
    const int64_t q = lo + threadIdx.x + (int64_t)c * blockDim.x;
    cv[c] = -INFINITY;
    ci[c] = INT64_MAX;  // an empty slot is never picked
    if (q < hi) load(q, cv[c], ci[c]);
  }
  const int64_t rest = lo + (int64_t)kTopkCache * blockDim.x;
  float pv = INFINITY;
  int64_t pi = -1;
  for (int r = 0; r < k; ++r) {
    float bv = -INFINITY;
    int64_t bi = INT64_MAX;
    auto offer = [&](float v, int64_t i) {
      if (i >= 0 && i != INT64_MAX && ls_before(pv, pi, v, i) && ls_before(v, i, bv, bi)) {
        bv = v;
        bi = i;
      }
    };
#pragma unroll
    for (int c = 0; c < kTopkCache; ++c) offer(cv[c], ci[c]);
    for (int64_t q = rest + threadIdx.x; q < hi; q += blockDim.x) {
      float v;
      int64_t i;
      load(q, v, i);
      offer(v, i);
    }
    ls_block_best(bv, bi, sv, si);
    if (threadIdx.x == 0) {
      out_v[r] = bv;
      out_i[r] = bi;
    }
    pv = bv;
    pi = bi;
  }
}

__global__ __launch_bounds__(256) void ls_topk_partial(const float *acq, const int64_t *map,
                                                        int64_t M, int k, float *pv, int64_t *pi) {
  __shared__ float sv[256];
  __shared__ int64_t si[256];
  const int64_t chunk = (M + gridDim.x - 1) / gridDim.x;
  const int64_t lo = (int64_t)blockIdx.x * chunk, hi = min(M, lo + chunk);
  ls_topk_range(acq, map, lo, max(lo, hi), k, pv + (int64_t)blockIdx.x * k,
                pi + (int64_t)blockIdx.x * k, sv, si);
}

__global__ __launch_bounds__(256) void ls_topk_final(const float *pv, const int64_t *pi, int n,
                                                      int k, float *v, int64_t *idx) {
  __shared__ float sv[256];
  __shared__ int64_t si[256];
  ls_topk_range(pv, pi, 0, n, k, v, idx, sv, si);
}

// cur[s] = configuration start[s] of the candidate columns; cur_acq[s] its value;
// every start active, no moves yet (k <= M, so every start is an index below M)
__global__ __launch_bounds__(256) void ls_gather(const LSDesc dsc0, const LSCols C0, int64_t M,
                                                  const int64_t *start, const float *start_v,
                                                  int k, const LSCols cur0, float *cur_acq,
                                                  int32_t *active, int32_t *steps) {
  __shared__ LSDesc dsc;
  __shared__ LSCols C, cur;
  ls_stage(dsc, dsc0);
  ls_stage(C, C0);
  ls_stage(cur, cur0);
  __syncthreads();
  const int s = blockIdx.x;
  if (s >= k) return;
  const int64_t j = start[s];
  if (j < 0 || j >= M) return;
  for (int p = 0; p < dsc.d; ++p) {
    const int wd = dsc.words[p];
    for (int q = threadIdx.x; q < wd; q += blockDim.x)
      cur.col[p][(int64_t)s * wd + q] = C.col[p][j * wd + q];
  }
  if (threadIdx.x == 0) {
    cur_acq[s] = start_v[s];
    active[s] = 1;
    steps[s] = 0;
  }
}

// The words of parameter p after move mv (in move0 numbering) of the configuration cfg,
// into dst (which may be cfg's own words of p); false when the move leaves the range
// (dst is then unchanged).
__device__ __forceinline__ bool ls_move(const LSDesc &dsc, const uint32_t *cfg, int p, int mv, uint32_t *dst) {
  const uint32_t *src = cfg + dsc.woff[p];
  switch (dsc.kind[p]) {
    case GP_REAL: {
      const double v = __builtin_bit_cast(double, (uint64_t)src[0] | ((uint64_t)src[1] << 32));
      const double tv = dsc.log2[p] ? log2(v) : v;
      const double step = (dsc.t_hi[p] - dsc.t_lo[p]) / 16.0;
      const double t2 = mv == 0 ? tv - step : tv + step;
      if (!(t2 >= dsc.t_lo[p] && t2 <= dsc.t_hi[p])) return false;
      const uint64_t b = __builtin_bit_cast(uint64_t, dsc.log2[p] ? exp2(t2) : t2);
      dst[0] = (uint32_t)b;
      dst[1] = (uint32_t)(b >> 32);
      return true;
    }
    case GP_INT:
    case GP_ORD: {
      const int v = (int)src[0] + (mv == 0 ? -1 : 1);
      if (!(v >= dsc.lo[p] && v <= dsc.hi[p])) return false;
      dst[0] = (uint32_t)v;
      return true;
    }
    case GP_CAT: {
      const int cur_level = (int)src[0];
      dst[0] = (uint32_t)(mv < cur_level ? mv : mv + 1);
      return true;
    }
    default: {  // PERM: pair number mv in (a, b) order, a < b
      const int m = dsc.words[p];
      int a = 0, rem = mv;
      while (rem >= m - 1 - a) {
        rem -= m - 1 - a;
        ++a;
      }
      const int b = a + 1 + rem;
      const uint32_t sa = src[a], sb = src[b];
#pragma unroll
      for (int i = 0; i < 8; ++i)  // static indices: dst may be a register array
        if (i < m) {
          const uint32_t v = src[i];
          dst[i] = i == a ? sb : (i == b ? sa : v);
        }
      return true;
    }
  }
}

// The parameter that neighbour jn moves and its move number
__device__ __forceinline__ int ls_param_of(const LSDesc &dsc, int jn, int &mv) {
  int p = 0;
  while (p + 1 < dsc.d && jn >= dsc.move0[p + 1]) ++p;
  mv = jn - dsc.move0[p];
  return p;
}

// A parameter's raw value as encode_param takes it, from its words w (PERM: into rv)
__device__ __forceinline__ uint64_t ls_raw(const LSDesc &dsc, int p, const uint32_t *w, int (&rv)[8]) {
  if (dsc.kind[p] == GP_REAL) return (uint64_t)w[0] | ((uint64_t)w[1] << 32);
  if (dsc.kind[p] == GP_PERM) {
    const int m = dsc.words[p];
#pragma unroll
    for (int i = 0; i < 8; ++i) rv[i] = i < m ? (int)w[i] : 0;  // rv[i >= m] is not read
  }
  return w[0];
}

// One workgroup per start. Selection: the best neighbour of the previous step (largest
// value, lowest neighbour index on ties) becomes the configuration if it is strictly
// better, else the start is done. Generation: the configuration is encoded once in LDS
// (one thread per parameter); then one thread per neighbour re-encodes only the moved
// parameter and writes the neighbour's code words, validity and mask. A neighbour whose
// move leaves the range is scored as a copy of the configuration with a zero mask, so its
// acquisition value is 0 and never wins a strict comparison; so is every neighbour of an
// inactive start. Block k-1 also writes the padding rows as copies of the last neighbour.
__global__ __launch_bounds__(256) void ls_step(const LSDesc dsc0, const LSCols cur0, int k,
                                               int32_t *active, const float *nb_acq,
                                               float *cur_acq, int32_t *steps, int32_t max_steps,
                                               int gen, const LSEnc e, uint8_t *mask) {
  __shared__ LSDesc dsc;
  __shared__ LSCols cur;
  __shared__ uint32_t cfg[kLsMaxWords];
  __shared__ ParamEnc pes[kMaxD];
  __shared__ uint32_t code[kMaxWords];
  __shared__ uint8_t okp[kMaxD];
  __shared__ float sv[256];
  __shared__ int64_t si[256];
  __shared__ int act_s;
  const int tid = threadIdx.x, s = blockIdx.x;
  if (s >= k) return;  // (uniform over the block)
  // the selection's loads go out with the staging, ahead of its barrier
  const int nnb = dsc0.nnb;
  const float ca = cur_acq[s];  // read before any barrier after which thread 0 may write it
  const int act0 = active[s];
  const float v0 = (nb_acq && tid < nnb) ? nb_acq[(int64_t)s * nnb + tid] : -INFINITY;
  ls_stage(dsc, dsc0);
  ls_stage(cur, cur0);
  for (int q = tid; q < dsc0.d * (int)(sizeof(ParamEnc) / 4); q += blockDim.x)
    reinterpret_cast<uint32_t *>(pes)[q] = reinterpret_cast<const uint32_t *>(e.penc)[q];
  if (tid == 0) act_s = act0;
  __syncthreads();
  for (int w = tid; w < dsc.W; w += blockDim.x) {
    const int p = dsc.wparam[w];
    cfg[w] = cur.col[p][(int64_t)s * dsc.words[p] + (w - dsc.woff[p])];
  }
  __syncthreads();

  if (nb_acq && act0) {  // selection
    float bv = -INFINITY;
    int64_t bi = INT64_MAX;
    if (tid < nnb && ls_before(v0, tid, bv, bi)) bv = v0, bi = tid;
    for (int jn = tid + blockDim.x; jn < nnb; jn += blockDim.x) {
      const float v = nb_acq[(int64_t)s * nnb + jn];
      if (ls_before(v, jn, bv, bi)) bv = v, bi = jn;
    }
    ls_block_best(bv, bi, sv, si);
    const bool move = bi != INT64_MAX && bv > ca;
    if (move && tid == 0) {
      int mv;
      const int p = ls_param_of(dsc, (int)bi, mv);
      ls_move(dsc, cfg, p, mv, cfg + dsc.woff[p]);
      cur_acq[s] = bv;
      steps[s] += 1;
    }
    __syncthreads();
    if (move)
      for (int w = tid; w < dsc.W; w += blockDim.x) {
        const int p = dsc.wparam[w];
        cur.col[p][(int64_t)s * dsc.words[p] + (w - dsc.woff[p])] = cfg[w];
      }
    if (tid == 0) {
      act_s = (move && steps[s] < max_steps) ? 1 : 0;
      active[s] = act_s;
    }
    __syncthreads();
  }
  if (!gen) return;

  // the configuration's codes and per-parameter validity
  for (int w = tid; w < e.R; w += blockDim.x) code[w] = 0u;
  if (s == 0 && tid == 0 && e.clear) *e.clear = 0;
  __syncthreads();
  int bad = 0;
  for (int p = tid; p < dsc.d; p += blockDim.x) {
    const ParamEnc &pe = pes[dsc.penc_of[p]];
    int rv[8];
    const ParamCode c = encode_param(pe, ls_raw(dsc, p, cfg + dsc.woff[p], rv), rv, e.table);
    okp[p] = c.ok ? 1 : 0;
    bad += c.ok ? 0 : 1;
    if (param_field_mask(pe)) {
      atomicOr(&code[pe.word], c.w0);
    } else {
      code[pe.word] = c.w0;
      if (param_code_words(pe) == 2) code[pe.word + 1] = c.w1;
    }
  }
  const int nbad = __syncthreads_count(bad);
  const bool act = act_s != 0;

  const int64_t N = (int64_t)k * dsc.nnb;
  const int nrow = s == k - 1 ? (int)(e.rows - (int64_t)(k - 1) * dsc.nnb) : dsc.nnb;
  for (int r = tid; r < nrow; r += blockDim.x) {
    const int jn = min(r, dsc.nnb - 1);
    const int64_t t = (int64_t)s * dsc.nnb + r;
    int mv;
    const int p = ls_param_of(dsc, jn, mv);
    const ParamEnc &pe = pes[dsc.penc_of[p]];
    uint32_t nw[8];
    const bool ok = ls_move(dsc, cfg, p, mv, nw);
    int w0 = -1, nwd = 0;  // words of the moved parameter's new code
    uint32_t c0 = 0, c1 = 0;
    bool valid = nbad == 0;
    if (ok) {
      int rv[8];
      const ParamCode c = encode_param(pe, ls_raw(dsc, p, nw, rv), rv, e.table);
      w0 = pe.word;
      nwd = param_code_words(pe);
      const uint32_t fm = param_field_mask(pe);
      c0 = fm ? (code[w0] & ~fm) | c.w0 : c.w0;
      c1 = c.w1;
      valid = (nbad - (okp[p] ? 0 : 1)) == 0 && c.ok;
    }
    for (int w = 0; w < e.R; ++w) {
      uint32_t v = code[w];
      if (w == w0) v = c0;
      if (nwd == 2 && w == w0 + 1) v = c1;
      e.cand[(int64_t)w * e.rows + t] = v;
    }
    e.valid[t] = valid ? 1 : 0;
    if (t < N) mask[t] = (ok && act) ? 1 : 0;
  }
}

// Upper bound of each candidate's acquisition value from the cross-kernel's mean alone:
// acq = EI(mu, sigma) p <= EI(mu_lo, smax), since p <= 1, sigma^2 = s - |v|^2 <= s and EI
// falls with mu and rises with sigma; mu_lo takes off a bound of the mean's error in the
// fp32 pipeline and in the fp64 recomputation (1e-5 sens, sens = sum |alpha| K*, against
// about 1e-7 sens), and the result is widened for the fp32 epilogue's rounding and
// rounded up to fp32. Masked and invalid candidates score 0 and get 0. Thread 0 clears
// the compaction counter.
__global__ __launch_bounds__(256) void ls_bound_k(const double *mu64, const float *sens,
                                                   const uint8_t *valid, const uint8_t *mask,
                                                   int64_t M, double fstar, double smax, float *ub,
                                                   int32_t *count) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j == 0) *count = 0;
  if (j >= M) return;
  float u = 0.f;
  if (valid[j] && (!mask || mask[j])) {
    const double mu = mu64[j];
    const double mu_lo = mu - (1e-5 * (double)sens[j] + 1e-12 * (1.0 + fabs(mu)));
    const double imp = fstar - mu_lo, z = imp / smax;
    const double ei = fmax(imp * 0.5 * erfc(-z * 0.70710678118654752440) +
                               smax * 0.39894228040143267794 * exp(-0.5 * z * z),
                           0.0);
    const double b = ei * (1.0 + 1e-3) + 1e-6 * (1.0 + fabs(fstar));
    u = (float)b;
    if ((double)u < b) u = __uint_as_float(__float_as_uint(u) + 1u);  // b > 0: next float up
  }
  ub[j] = u;
}

// The indices j with ub[j] >= *tau, in any order (one atomic per wavefront); *count
// counts all of them, list holds the first cap.
__global__ __launch_bounds__(256) void ls_compact_k(const float *ub, int64_t M, const float *tau,
                                                     int64_t *list, int32_t *count, int64_t cap) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const float t = *tau;
  const bool keep = j < M && ub[j] >= t;
  const uint64_t bal = __ballot(keep);
  if (!bal) return;
  const int lane = threadIdx.x & 63;
  const int leader = __ffsll((unsigned long long)bal) - 1;
  int base = 0;
  if (lane == leader) base = atomicAdd(count, __popcll(bal));
  base = __shfl(base, leader);
  if (keep) {
    const int64_t pos = base + __popcll(bal & ((1ull << lane) - 1ull));
    if (pos < cap) list[pos] = j;
  }
}

// Configurations idx[0..n) of the columns C into rows 0..n of G (one word per thread),
// and (if given) their mask entries into mg.
__global__ __launch_bounds__(256) void ls_gather_rows_k(const LSDesc dsc0, const LSCols C0,
                                                         const int64_t *idx, int64_t n,
                                                         const LSCols G0, const uint8_t *mask,
                                                         uint8_t *mg) {
  __shared__ LSDesc dsc;
  __shared__ LSCols C, G;
  ls_stage(dsc, dsc0);
  ls_stage(C, C0);
  ls_stage(G, G0);
  __syncthreads();
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= n * dsc.W) return;
  const int64_t r = t / dsc.W;
  const int w = (int)(t - r * dsc.W);
  const int p = dsc.wparam[w], wd = dsc.words[p], q = w - dsc.woff[p];
  G.col[p][r * wd + q] = C.col[p][idx[r] * wd + q];
  if (mask && w == 0) mg[r] = mask[idx[r]];
}

}  // namespace

hipError_t launch_ls_bound(const double *mu64, const float *sens, const uint8_t *valid,
                           const uint8_t *mask, int64_t M, double fstar, double smax, float *ub,
                           int32_t *count, hipStream_t s) {
  if (M < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ls_bound_k, dim3((unsigned)((M + 255) / 256)), dim3(256), 0, s, mu64, sens,
                     valid, mask, M, fstar, smax, ub, count);
  return hipGetLastError();
}

hipError_t launch_ls_compact(const float *ub, int64_t M, const float *tau, int64_t *list,
                             int32_t *count, int64_t cap, hipStream_t s) {
  if (M < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ls_compact_k, dim3((unsigned)((M + 255) / 256)), dim3(256), 0, s, ub, M, tau,
                     list, count, cap);
  return hipGetLastError();
}

hipError_t launch_ls_gather_rows(const LSDesc &d, const LSCols &C, const int64_t *idx, int64_t n,
                                 const LSCols &G, const uint8_t *mask, uint8_t *mg, hipStream_t s) {
  const int64_t tot = n * d.W;
  if (n <= 0) return hipSuccess;
  if (d.W < 1 || d.W > kLsMaxWords || (mask && !mg)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ls_gather_rows_k, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, d, C,
                     idx, n, G, mask, mg);
  return hipGetLastError();
}

hipError_t launch_ls_topk(const float *acq, int64_t M, int k, float *pv, int64_t *pi, int parts,
                          float *v, int64_t *idx, hipStream_t s, const int64_t *map) {
  if (k < 1 || k > kLsMaxStarts || parts < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ls_topk_partial, dim3(parts), dim3(256), 0, s, acq, map, M, k, pv, pi);
  hipLaunchKernelGGL(ls_topk_final, dim3(1), dim3(256), 0, s, pv, pi, parts * k, k, v, idx);
  return hipGetLastError();
}

hipError_t launch_ls_gather(const LSDesc &d, const LSCols &C, int64_t M, const int64_t *start,
                            const float *start_v, int k, const LSCols &cur, float *cur_acq,
                            int32_t *active, int32_t *steps, hipStream_t s) {
  if (k < 1 || k > M) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ls_gather, dim3(k), dim3(64), 0, s, d, C, M, start, start_v, k, cur, cur_acq,
                     active, steps);
  return hipGetLastError();
}

hipError_t launch_ls_step(const LSDesc &d, const LSCols &cur, int k, int32_t *active,
                          const float *nb_acq, float *cur_acq, int32_t *steps, int32_t max_steps,
                          bool gen, const LSEnc &e, uint8_t *mask, hipStream_t s) {
  if (k < 1 || k > kLsMaxStarts || d.nnb < 1) return hipErrorInvalidValue;
  if (d.W < 1 || d.W > kLsMaxWords) return hipErrorInvalidValue;
  if (gen) {
    // the padding rows of block k-1 are all its threads' rows past its neighbours
    const int64_t N = (int64_t)k * d.nnb;
    if (e.R < 1 || e.R > kMaxWords || e.rows < N || e.rows - N > kRowTile || !e.cand ||
        !e.valid || !mask || !e.penc || !e.table)
      return hipErrorInvalidValue;
  }
  hipLaunchKernelGGL(ls_step, dim3((unsigned)k), dim3(256), 0, s, d, cur, k, active, nb_acq,
                     cur_acq, steps, max_steps, gen ? 1 : 0, e, mask);
  return hipGetLastError();
}

}  // namespace bgp
