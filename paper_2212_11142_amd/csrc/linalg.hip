// fp64 linear algebra of the model fit: Gram matrix, matrix-vector products,
// K^-1 = L^-T L^-1, and the element-wise steps of the Laplace probit classifier's
// Newton iteration (Rasmussen & Williams 2006, Sec. 3.4, the textbook the paper cites
// for its GP model). The factorisations themselves are in chol.hip.
//
// Matrices are row-major n x n with leading dimension ld.
#include "common.h"
#include "dist64.h"

namespace bgp {
namespace {

__global__ __launch_bounds__(256) void gram_kernel(const uint32_t *codes, int32_t R, int32_t n,
                                                    const Weights64 w, double sv, double noise,
                                                    double *K, int32_t ld) {
  const int b = blockIdx.x * 16 + (threadIdx.x & 15);
  const int a = blockIdx.y * 16 + (threadIdx.x >> 4);
  if (a >= n || b >= n) return;
  const uint32_t *ca = codes + (int64_t)a * R, *cb = codes + (int64_t)b * R;
  auto ga = [&](int q) { return ca[q]; };
  auto gb = [&](int q) { return cb[q]; };
  double k = matern52_f64(r2_f64(ga, gb, w), sv);
  if (a == b) k += noise;
  K[(int64_t)a * ld + b] = k;
}

__device__ __forceinline__ void tri_index(int L, int &bi, int &bj) {
  int i = (int)((sqrt(8.0 * L + 1.0) - 1.0) * 0.5);
  while ((i + 1) * (i + 2) / 2 <= L) ++i;
  while (i * (i + 1) / 2 > L) --i;
  bi = i;
  bj = L - i * (i + 1) / 2;
}

// out = X^T X for lower-triangular X (K^-1 = L^-T L^-1), lower blocks then mirrored.

__global__ __launch_bounds__(64) void gemv_rows(const double *A, int32_t ld, const double *x,
                                                 double *y, int32_t n, int32_t lower) {
  const int r = blockIdx.x;
  const int end = lower ? r + 1 : n;
  double s = 0.0;
  for (int c = threadIdx.x; c < end; c += 64) s = fma(A[(int64_t)r * ld + c], x[c], s);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
  if (threadIdx.x == 0) y[r] = s;
}

// y = A^T x for an n x n upper-triangular A (row stride ld): 64 columns per workgroup,
// the rows r <= c split over its 16 wavefronts (two chains each, so that several loads
// are in flight) in a fixed order, summed in LDS
__global__ __launch_bounds__(1024) void gemv_t_upper(const double *A, int32_t ld, const double *x,
                                                     double *y, int32_t n) {
  __shared__ double part[16][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane;
  double s0 = 0.0, s1 = 0.0;
  if (c < n) {
    int r = w;
    for (; r + 16 <= c; r += 32) {
      s0 = fma(A[(int64_t)r * ld + c], x[r], s0);
      s1 = fma(A[(int64_t)(r + 16) * ld + c], x[r + 16], s1);
    }
    if (r <= c) s0 = fma(A[(int64_t)r * ld + c], x[r], s0);
  }
  part[w][lane] = s0 + s1;
  __syncthreads();
  if (w == 0 && c < n) {
    double t = 0.0;
#pragma unroll
    for (int g = 0; g < 16; ++g) t += part[g][lane];
    y[c] = t;
  }
}

__global__ __launch_bounds__(256) void tril_copy(const double *src, double *dst, int32_t ld,
                                                  int32_t n) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)n * n) return;
  const int r = (int)(idx / n), c = (int)(idx - (int64_t)r * n);
  dst[(int64_t)r * ld + c] = c <= r ? src[(int64_t)r * ld + c] : 0.0;
}

__global__ __launch_bounds__(256) void transpose_k(const double *src, double *dst, int32_t ld,
                                                    int32_t n) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)n * n) return;
  const int r = (int)(idx / n), c = (int)(idx - (int64_t)r * n);
  dst[(int64_t)c * ld + r] = src[(int64_t)r * ld + c];
}

__global__ __launch_bounds__(256) void reduce_min_k(const double *x, int32_t n, double *out) {
  __shared__ double s[256];
  double m = INFINITY;
  for (int i = threadIdx.x; i < n; i += 256) m = fmin(m, x[i]);
  s[threadIdx.x] = m;
  __syncthreads();
  for (int k = 128; k > 0; k >>= 1) {
    if (threadIdx.x < k) s[threadIdx.x] = fmin(s[threadIdx.x], s[threadIdx.x + k]);
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = s[0];
}

// Partial column sums y[s][c] = sum_{r in slice s} A[r][c] x[r] over kGemvSlices row
// slices: workgroup (column group, slice) takes 64 columns, its 16 wavefronts split the
// slice's rows.
__global__ __launch_bounds__(1024) void gemv_cols_k(const double *A, int32_t ld, const double *x,
                                                     double *y, int32_t m, int32_t n,
                                                     const int32_t *halt) {
  __shared__ double part[16][64];
  if (halt && *halt) return;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane, sl = blockIdx.y;
  const int r0 = (int)((int64_t)m * sl / kGemvSlices), r1 = (int)((int64_t)m * (sl + 1) / kGemvSlices);
  double s0 = 0.0, s1 = 0.0;
  if (c < n) {
    int r = r0 + wv;
    for (; r + 48 < r1; r += 64) {  // two steps' loads in flight, the sums in step order
      double av[4], xv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        av[u] = A[(int64_t)(r + 16 * u) * ld + c];
        xv[u] = x[r + 16 * u];
      }
      s0 = fma(av[0], xv[0], s0);
      s1 = fma(av[1], xv[1], s1);
      s0 = fma(av[2], xv[2], s0);
      s1 = fma(av[3], xv[3], s1);
    }
    for (; r + 16 < r1; r += 32) {
      s0 = fma(A[(int64_t)r * ld + c], x[r], s0);
      s1 = fma(A[(int64_t)(r + 16) * ld + c], x[r + 16], s1);
    }
    for (; r < r1; r += 16) s0 = fma(A[(int64_t)r * ld + c], x[r], s0);
  }
  part[wv][lane] = s0 + s1;
  __syncthreads();
  if (wv == 0 && c < n) {
    double t = 0.0;
#pragma unroll
    for (int g = 0; g < 16; ++g) t += part[g][lane];
    y[(int64_t)sl * n + c] = t;
  }
}

// a[r] = b[r] - sw[r] sum_{c >= r} Y[r][c] z[c] for the upper triangular Y (row-major, ld
// n), z the sum of the kGemvSlices partial rows of gemv_cols_k's output: one wavefront
// per row, kNewtonRows rows per workgroup. In place (a == b) is allowed.
constexpr int kNewtonRows = 8;
__global__ __launch_bounds__(64 * kNewtonRows) void newton_a_k(const double *Y, const double *zs,
                                                                const double *b, const double *sw,
                                                                double *a, int32_t n,
                                                                const int32_t *halt) {
  if (*halt) return;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int r = blockIdx.x * kNewtonRows + wv;
  if (r >= n) return;
  double s = 0.0;
  int c = (r & ~63) + lane;
  for (; c + 64 < n; c += 128) {  // two columns' loads in flight, the sum in column order
    double zv[2][kGemvSlices], yv[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int cu = c + 64 * u;
#pragma unroll
      for (int sl = 0; sl < kGemvSlices; ++sl) zv[u][sl] = zs[(int64_t)sl * n + cu];
      yv[u] = Y[(int64_t)r * n + cu];
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      double z = 0.0;
#pragma unroll
      for (int sl = 0; sl < kGemvSlices; ++sl) z += zv[u][sl];
      s = fma(c + 64 * u >= r ? yv[u] : 0.0, z, s);
    }
  }
  for (; c < n; c += 64) {
    double z = 0.0;
#pragma unroll
    for (int sl = 0; sl < kGemvSlices; ++sl) z += zs[(int64_t)sl * n + c];
    const double y = c >= r ? Y[(int64_t)r * n + c] : 0.0;
    s = fma(y, z, s);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
  if (lane == 0) a[r] = b[r] - sw[r] * s;
}

// y[r] = sum_{c < n} K[r][c] b[c], one wavefront per row (four columns' loads in flight,
// the sum in column order) and kNewtonRows rows per workgroup, and the iteration's
// convergence check: each
// workgroup's max |y[r] - f[r]| goes into an atomic max; the workgroup that finishes
// last (its ticket is the last one, so every other max has landed) reads the maximum,
// sets the halt word, publishes the status and clears the counters for the next
// iteration.
__global__ __launch_bounds__(64 * kNewtonRows) void gemv_newton_k(
    const double *K, const double *b, double *y, const double *f, int32_t ld, int32_t n,
    double tol, const int32_t *info, int32_t *halt, NewtonScratch *scr, NewtonStatus *st) {
  __shared__ double dmax[kNewtonRows];
  if (*halt) return;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int r = blockIdx.x * kNewtonRows + wv;
  double s = 0.0;
  if (r < n) {
    const double *Kr = K + (int64_t)r * ld;
    int c = lane;
    for (; c + 192 < n; c += 256) {
      double kv[4], bv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        kv[u] = Kr[c + 64 * u];
        bv[u] = b[c + 64 * u];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) s = fma(kv[u], bv[u], s);
    }
    for (; c < n; c += 64) s = fma(Kr[c], b[c], s);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
  if (lane == 0) {
    double d = 0.0;
    if (r < n) {
      y[r] = s;
      d = fabs(s - f[r]);
    }
    dmax[wv] = d;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double d = dmax[0];
#pragma unroll
    for (int g = 1; g < kNewtonRows; ++g) d = (dmax[g] > d || dmax[g] != dmax[g]) ? dmax[g] : d;
    const unsigned long long old = atomicMax(&scr->dmax, (unsigned long long)__double_as_longlong(d));
    asm volatile("" ::"v"(old));  // the max has been performed before the ticket is taken
    if (atomicAdd(&scr->ticket, 1u) == gridDim.x - 1u) {
      const double dm = __longlong_as_double((long long)atomicOr(&scr->dmax, 0ull));
      const int inf = *info;
      const int h = inf ? 3 : (!isfinite(dm) ? 2 : (dm < tol ? 1 : 0));
      st->delta = dm;
      st->info = inf;
      st->halt = h;
      *halt = h;
      atomicExch(&scr->dmax, 0ull);
      atomicExch(&scr->ticket, 0u);
    }
  }
}

// One workgroup per packed column c: the largest magnitude of the column picks its
// scale 2^e (scaled values in [2^kSplitTop, 2^(kSplitTop+1)) at the top), then every
// value is split into fp16 high and low parts from its fp64 form. The exponent sum is
// kept within the normal fp32 range of cscale.
__global__ __launch_bounds__(256) void pack_bt_k(const double *Linv, int32_t ldl, int32_t nsrc,
                                                  int32_t transposed, const double *rowscale,
                                                  double scale, int32_t kexp, _Float16 *Bt,
                                                  float *cscale, int32_t ldb) {
  __shared__ double red[256];
  const int c = blockIdx.x, tid = threadIdx.x;
  // transposed == 2: column 0 is the dense vector Linv[0..nsrc), the others are zero
  auto val = [&](int k) -> double {
    if (transposed == 2) return (c == 0 && k < nsrc) ? scale * Linv[k] : 0.0;
    if (c >= nsrc || k > c) return 0.0;
    const double x = transposed ? Linv[(int64_t)k * ldl + c] : Linv[(int64_t)c * ldl + k];
    return scale * x * (rowscale ? rowscale[k] : 1.0);
  };
  double mx = 0.0;
  for (int k = tid; k < ldb; k += 256) mx = fmax(mx, fabs(val(k)));
  red[tid] = mx;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (tid < h) red[tid] = fmax(red[tid], red[tid + h]);
    __syncthreads();
  }
  mx = red[0];
  int e = (mx > 0.0 && isfinite(mx)) ? kSplitTop - ilogb(mx) : 0;
  e = min(max(e, -126 - kexp), 126 - kexp);
  _Float16 *row = Bt + (int64_t)c * 2 * ldb;
  for (int k = tid; k < ldb; k += 256) {
    const double v = ldexp(val(k), e);
    const _Float16 h = (_Float16)v;
    const _Float16 l = (_Float16)(v - (double)h);
    const int p = (k >> 5) * 64 + kpos(k & 31);  // the cross-kernel's order within a chunk
    row[p] = h;
    row[p + 32] = l;
  }
  if (tid == 0) cscale[c] = (float)ldexp(1.0, -(kexp + e));
}

__global__ __launch_bounds__(256) void gather_f64_k(const double *src, const int32_t *idx,
                                                     double *dst, int32_t n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) dst[i] = src[idx[i]];
}

__global__ __launch_bounds__(256) void labels_k(const uint8_t *feasible, const int32_t *order,
                                                 double *t, int32_t n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) t[i] = (!feasible || feasible[order[i]]) ? 1.0 : -1.0;
}

inline unsigned blocks_for(int64_t n, int b) { return (unsigned)((n + b - 1) / b); }

}  // namespace

hipError_t launch_gram(const uint32_t *codes, int32_t R, int32_t n, const Weights64 &w, double sv,
                       double noise, double *K, int32_t ld, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  dim3 grid(blocks_for(n, 16), blocks_for(n, 16));
  hipLaunchKernelGGL(gram_kernel, grid, dim3(256), 0, s, codes, R, n, w, sv, noise, K, ld);
  return hipGetLastError();
}

hipError_t launch_tril_copy(const double *src, double *dst, int32_t ld, int32_t n, hipStream_t s) {
  hipLaunchKernelGGL(tril_copy, dim3(blocks_for((int64_t)n * n, 256)), dim3(256), 0, s, src, dst,
                     ld, n);
  return hipGetLastError();
}

hipError_t launch_transpose(const double *src, double *dst, int32_t ld, int32_t n, hipStream_t s) {
  hipLaunchKernelGGL(transpose_k, dim3(blocks_for((int64_t)n * n, 256)), dim3(256), 0, s, src,
                     dst, ld, n);
  return hipGetLastError();
}

hipError_t launch_gemv_rows(const double *A, int32_t ld, const double *x, double *y, int32_t n,
                            int32_t lower, hipStream_t s) {
  hipLaunchKernelGGL(gemv_rows, dim3(n), dim3(64), 0, s, A, ld, x, y, n, lower);
  return hipGetLastError();
}



hipError_t launch_gemv_t_upper(const double *A, int32_t ld, const double *x, double *y, int32_t n,
                               hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(gemv_t_upper, dim3(blocks_for(n, 64)), dim3(1024), 0, s, A, ld, x, y, n);
  return hipGetLastError();
}

hipError_t launch_reduce_min(const double *x, int32_t n, double *out, hipStream_t s) {
  hipLaunchKernelGGL(reduce_min_k, dim3(1), dim3(256), 0, s, x, n, out);
  return hipGetLastError();
}

hipError_t launch_gemv_cols(const double *A, int32_t ld, const double *x, double *y, int32_t m,
                            int32_t n, const int32_t *halt, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(gemv_cols_k, dim3((n + 63) / 64, kGemvSlices), dim3(1024), 0, s, A, ld, x, y,
                     m, n, halt);
  return hipGetLastError();
}

hipError_t launch_newton_a(const double *Y, const double *zs, const double *b, const double *sw,
                           double *a, int32_t n, const int32_t *halt, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(newton_a_k, dim3((n + kNewtonRows - 1) / kNewtonRows), dim3(64 * kNewtonRows),
                     0, s, Y, zs, b, sw, a, n, halt);
  return hipGetLastError();
}

hipError_t launch_gemv_newton(const double *K, const double *b, double *y, const double *f,
                              int32_t ld, int32_t n, double tol, const int32_t *info,
                              int32_t *halt, NewtonScratch *scr, NewtonStatus *st,
                              hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(gemv_newton_k, dim3((n + kNewtonRows - 1) / kNewtonRows), dim3(64 * kNewtonRows),
                     0, s, K, b, y, f, ld, n, tol, info, halt, scr, st);
  return hipGetLastError();
}

hipError_t launch_pack_bt(const double *Linv, int32_t ldl, int32_t nsrc, bool transposed,
                          const double *rowscale, double scale, int32_t kexp, uint16_t *Bt,
                          float *cscale, int32_t ldb, int32_t ncols_pad, hipStream_t s) {
  if (ncols_pad <= 0 || ldb <= 0) return hipSuccess;
  hipLaunchKernelGGL(pack_bt_k, dim3(ncols_pad), dim3(256), 0, s, Linv, ldl, nsrc,
                     transposed ? 1 : 0, rowscale, scale, kexp, reinterpret_cast<_Float16 *>(Bt),
                     cscale, ldb);
  return hipGetLastError();
}

hipError_t launch_pack_vec(const double *v, int32_t n, double scale, int32_t kexp, uint16_t *Bt,
                           float *cscale, int32_t ldb, int32_t ncols_pad, hipStream_t s) {
  if (ncols_pad <= 0 || ldb <= 0 || n > ldb) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pack_bt_k, dim3(ncols_pad), dim3(256), 0, s, v, 0, n, 2, nullptr, scale,
                     kexp, reinterpret_cast<_Float16 *>(Bt), cscale, ldb);
  return hipGetLastError();
}

hipError_t launch_gather_f64(const double *src, const int32_t *idx, double *dst, int32_t n,
                             hipStream_t s) {
  hipLaunchKernelGGL(gather_f64_k, dim3(blocks_for(n, 256)), dim3(256), 0, s, src, idx, dst, n);
  return hipGetLastError();
}

hipError_t launch_labels(const uint8_t *feasible, const int32_t *order, double *t, int32_t n,
                         hipStream_t s) {
  hipLaunchKernelGGL(labels_k, dim3(blocks_for(n, 256)), dim3(256), 0, s, feasible, order, t, n);
  return hipGetLastError();
}

}  // namespace bgp
