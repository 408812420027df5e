// fp64 blocked Cholesky, triangular inverse and triangular solves for the model fit.
//
// Right-looking Cholesky on 64 x 64 blocks with one launch per block column:
//   * chol_panel factors the first diagonal block;
//   * chol_trailing(k) computes the panel L_ik = A_ik D_k^T (D_k = L_kk^-1, so the
//     triangular solve is a GEMM), subtracts L_ik L_jk^T from every trailing block
//     (i >= j), and the workgroup owning block (k+1, k+1) factors it right away, so
//     the next launch already has L_{k+1,k+1} and D_{k+1}.
// Each diagonal factorisation also produces its inverse D_k, which the triangular
// inverse L^-1 and the single-workgroup triangular solves reuse.
// A device int `info` records the first failing pivot (1-based, global row); every
// kernel returns immediately once it is set.
#include "common.h"

namespace bgp {
namespace {

constexpr int NB = kNB;     // 64
constexpr int LP = NB + 1;  // LDS row stride (doubles)
constexpr int HB = 32;      // Tb scratch is HB x (HB + 1) doubles (>= 3 x 64)

__device__ __forceinline__ void tri_index(int L, int &bi, int &bj) {
  int i = (int)((sqrt(8.0 * L + 1.0) - 1.0) * 0.5);
  while ((i + 1) * (i + 2) / 2 <= L) ++i;
  while (i * (i + 1) / 2 > L) --i;
  bi = i;
  bj = L - i * (i + 1) / 2;
}

// acc[u][v] += sum_q Aa[r_u][q] * Bb[c_v][q], r_u = 4 ty + u, c_v = 4 tx + v (LDS, stride LP)
__device__ __forceinline__ void gemm_nt(const double *Aa, const double *Bb, double acc[4][4], int ty,
                                        int tx) {
#pragma unroll 4
  for (int q = 0; q < NB; ++q) {
    double av[4], bv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      av[u] = Aa[(ty * 4 + u) * LP + q];
      bv[u] = Bb[(tx * 4 + u) * LP + q];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[u][v] = fma(av[u], bv[v], acc[u][v]);
  }
}

// 1/x and 1/sqrt(x) from the hardware estimates plus two Newton steps (full fp64
// accuracy to about 1 ulp); used instead of IEEE divide / sqrt, whose latency would sit
// on the serial pivot chain of the block factorisation.
__device__ __forceinline__ double rcp_nr(double x) {
  double r = __builtin_amdgcn_rcp(x);
  r = fma(r, fma(-x, r, 1.0), r);
  return fma(r, fma(-x, r, 1.0), r);
}
__device__ __forceinline__ double rsqrt_nr(double x) {
  double r = __builtin_amdgcn_rsq(x);
  r = r * fma(-0.5 * x * r, r, 1.5);
  return r * fma(-0.5 * x * r, r, 1.5);
}

// Cholesky of the nb x nb (nb <= 64) block in S (LDS, lower part read) and its inverse,
// on all 256 threads: thread (ty, tx) keeps the 4 x 4 sub-block at rows 4 ty..,
// columns 4 tx.. in registers (rows/columns >= nb are padded with the identity).
// Factorisation, right-looking in panels of 4 columns without square roots on the
// serial chain: the owners of a panel publish it (one barrier per panel, double
// buffered); every thread factors the 4 x 4 pivot block itself, brings its own rows'
// and columns' panel entries up to date, and applies the rank-4 update
// a_rc -= sum_p a_rp a_cp / piv_p to its trailing elements. Columns are scaled by
// 1/sqrt(pivot) in one pass at the end.
// Inverse, right-looking in panels of 4 rows: the owners of rows jb..jb+3 of
// X = L^-1 finish them with the 4 x 4 diagonal block of L, publish them, and every
// thread subtracts L[r][jb..jb+3] X[jb..jb+3][c] from its rows below.
// Output: S = L (lower, zero elsewhere), Di = L^-1. *fail = 1-based failing pivot or 0.
__device__ __forceinline__ void factor_invert_block(double *S, double *Di, double *colbuf,
                                                    double *Tb, int *fail, int nb) {
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  double *pb0 = Tb, *pb1 = Tb + 4 * NB;     // panel buffers [64][4]
  double *piv_s = colbuf;                    // pivots, then 1 / L_jj
  double a[4][4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = 4 * ty + u, c = 4 * tx + v;
      a[u][v] = (r < nb && c < nb) ? (c <= r ? S[r * LP + c] : 0.0) : (r == c ? 1.0 : 0.0);
    }
  int bad = 0;
  for (int jb = 0; jb < NB; jb += 4) {
    double *pb = ((jb >> 2) & 1) ? pb1 : pb0;
    const int owner = jb >> 2;
    if (tx == owner) {
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) pb[(4 * ty + u) * 4 + v] = a[u][v];
    }
    __syncthreads();
    // 4 x 4 pivot block, factored locally (unscaled right-looking): w[s][p] is the
    // panel entry of row jb+s when column jb+p becomes the pivot column.
    double w[4][4], ip[4];
#pragma unroll
    for (int s2 = 0; s2 < 4; ++s2)
#pragma unroll
      for (int p = 0; p < 4; ++p) w[s2][p] = pb[(jb + s2) * 4 + p];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      double pv = w[p][p];
      if (!(pv > 0.0) || !isfinite(pv)) {
        if (!bad) bad = jb + p + 1;
        pv = 1.0;
        w[p][p] = 1.0;
      }
      ip[p] = rcp_nr(pv);
#pragma unroll
      for (int s2 = p + 1; s2 < 4; ++s2)
#pragma unroll
        for (int t = p + 1; t <= s2; ++t) w[s2][t] = fma(-w[s2][p] * ip[p], w[t][p], w[s2][t]);
    }
    if (tid == 0) {
#pragma unroll
      for (int p = 0; p < 4; ++p) piv_s[jb + p] = w[p][p];
    }
    // bring the panel entries of the thread's rows and columns up to date
    double cr[4][4], cc[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        cr[u][p] = pb[(4 * ty + u) * 4 + p];
        cc[u][p] = pb[(4 * tx + u) * 4 + p];
      }
#pragma unroll
      for (int p = 1; p < 4; ++p)
#pragma unroll
        for (int q = 0; q < p; ++q) {
          cr[u][p] = fma(-cr[u][q] * ip[q], w[p][q], cr[u][p]);
          cc[u][p] = fma(-cc[u][q] * ip[q], w[p][q], cc[u][p]);
        }
#pragma unroll
      for (int p = 0; p < 4; ++p) cc[u][p] *= ip[p];
    }
    // owners keep the final unscaled panel columns; trailing elements get the rank-4 update
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int r = 4 * ty + u, c = 4 * tx + v;
        if (tx == owner) {
          if (r >= c) a[u][v] = (ty == owner) ? w[u][v] : cr[u][v];
        } else if (c > jb + 3 && r >= c) {
          double t = a[u][v];
#pragma unroll
          for (int p = 0; p < 4; ++p) t = fma(-cr[u][p], cc[v][p], t);
          a[u][v] = t;
        }
      }
  }
  __syncthreads();
  if (tid == 0) *fail = (bad && bad <= nb) ? bad : 0;
  __syncthreads();
  if (*fail) return;
  // scale the columns: L_rc = a_rc / sqrt(piv_c) (c <= r); keep 1 / L_cc for the inverse
  double rs[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) rs[v] = rsqrt_nr(piv_s[4 * tx + v]);
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = 4 * ty + u, c = 4 * tx + v;
      a[u][v] = (c <= r) ? a[u][v] * rs[v] : 0.0;
      S[r * LP + c] = a[u][v];
    }
  __syncthreads();
  if (ty == tx) {
#pragma unroll
    for (int v = 0; v < 4; ++v) piv_s[4 * tx + v] = rcp_nr(a[v][v]);
  }
  double x[4][4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) x[u][v] = (4 * ty + u == 4 * tx + v) ? 1.0 : 0.0;
  __syncthreads();
  for (int jb = 0; jb < NB; jb += 4) {
    double *rb = ((jb >> 2) & 1) ? pb1 : pb0;   // [4][64]
    const int owner = jb >> 2;
    if (ty == owner) {
      // rows jb..jb+3 of X for this thread's columns: forward solve with L's diagonal block
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const double il = piv_s[jb + p];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          double t = x[p][v];
#pragma unroll
          for (int q = 0; q < p; ++q) t = fma(-S[(jb + p) * LP + jb + q], x[q][v], t);
          x[p][v] = t * il;
          rb[p * NB + 4 * tx + v] = x[p][v];
        }
      }
    }
    __syncthreads();
    if (ty > owner) {
      double lr[4][4], xj[4][4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          lr[u][p] = S[(4 * ty + u) * LP + jb + p];
          xj[p][u] = rb[p * NB + 4 * tx + u];
        }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          double t = x[u][v];
#pragma unroll
          for (int p = 0; p < 4; ++p) t = fma(-lr[u][p], xj[p][v], t);
          x[u][v] = t;
        }
    }
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = 4 * ty + u, c = 4 * tx + v;
      const bool in = r < nb && c < nb;
      Di[r * LP + c] = in ? x[u][v] : 0.0;
      if (!in) S[r * LP + c] = 0.0;
    }
  __syncthreads();
}

__device__ __forceinline__ void store_factor(const double *S, const double *Di, double *L, int ldl, double *Dk,
                             int g0, int nb) {
  for (int e = threadIdx.x; e < NB * NB; e += 256) {
    const int r = e / NB, c = e % NB;
    if (r < nb && c < nb) L[(int64_t)(g0 + r) * ldl + g0 + c] = S[r * LP + c];
    Dk[e] = Di[r * LP + c];
  }
}

__global__ __launch_bounds__(256) void chol_panel(const double *A, int32_t lda, double *L,
                                                   int32_t ldl, double *D, int32_t n,
                                                   int32_t *info) {
  __shared__ double S[NB * LP], Di[NB * LP], colbuf[NB], Tb[HB * (HB + 1)];
  __shared__ int fail;
  if (*info) return;
  const int nb = min(NB, n);
  for (int e = threadIdx.x; e < NB * NB; e += 256) {
    const int r = e / NB, c = e % NB;
    S[r * LP + c] = (r < nb && c <= r) ? A[(int64_t)r * lda + c] : 0.0;
  }
  __syncthreads();
  factor_invert_block(S, Di, colbuf, Tb, &fail, nb);
  if (fail) {
    if (threadIdx.x == 0) *info = fail;
    return;
  }
  store_factor(S, Di, L, ldl, D, 0, nb);
}

__global__ __launch_bounds__(256) void chol_trailing(double *A, int32_t lda, double *L,
                                                      int32_t ldl, double *D, int32_t k,
                                                      int32_t n, int32_t *info) {
  __shared__ double Ds[NB * LP], Pi[NB * LP], Pj[NB * LP], Ts[NB * LP];
  __shared__ double colbuf[NB], Tb[HB * (HB + 1)];
  __shared__ int fail;
  if (*info) return;
  int bi, bj;
  tri_index(blockIdx.x, bi, bj);
  const int k0 = k * NB;
  const int i0 = k0 + NB + bi * NB, j0 = k0 + NB + bj * NB;
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const double *Dk = D + (int64_t)k * NB * NB;
  for (int e = tid; e < NB * NB; e += 256) {
    const int r = e / NB, c = e % NB;
    Ds[r * LP + c] = Dk[e];
    Ts[r * LP + c] = (i0 + r < n) ? A[(int64_t)(i0 + r) * lda + k0 + c] : 0.0;
  }
  __syncthreads();
  double acc[4][4] = {};
  gemm_nt(Ts, Ds, acc, ty, tx);  // P_i = A_ik D_k^T = L_ik
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) Pi[(ty * 4 + u) * LP + tx * 4 + v] = acc[u][v];
  __syncthreads();
  if (bi != bj) {
    for (int e = tid; e < NB * NB; e += 256) {
      const int r = e / NB, c = e % NB;
      Ts[r * LP + c] = (j0 + r < n) ? A[(int64_t)(j0 + r) * lda + k0 + c] : 0.0;
    }
    __syncthreads();
    double acc2[4][4] = {};
    gemm_nt(Ts, Ds, acc2, ty, tx);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < 4; ++v) Pj[(ty * 4 + u) * LP + tx * 4 + v] = acc2[u][v];
    __syncthreads();
  }
  const double *Pjj = (bi == bj) ? Pi : Pj;
  double up[4][4] = {};
  gemm_nt(Pi, Pjj, up, ty, tx);
  if (bi == bj) {
    for (int e = tid; e < NB * NB; e += 256) {
      const int r = e / NB, c = e % NB;
      if (i0 + r < n) L[(int64_t)(i0 + r) * ldl + k0 + c] = Pi[r * LP + c];
    }
  }
  if (bi == 0 && bj == 0) {
    // block (k+1, k+1) has received all of its updates: factor it now
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int r = ty * 4 + u, c = tx * 4 + v;
        Ts[r * LP + c] = (i0 + r < n && i0 + c < n) ? A[(int64_t)(i0 + r) * lda + i0 + c] - up[u][v] : 0.0;
      }
    __syncthreads();
    const int nb = min(NB, n - i0);
    factor_invert_block(Ts, Pj, colbuf, Tb, &fail, nb);
    if (fail) {
      if (tid == 0) *info = i0 + fail;
      return;
    }
    store_factor(Ts, Pj, L, ldl, D + (int64_t)(k + 1) * NB * NB, i0, nb);
  } else {
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int r = i0 + ty * 4 + u, c = j0 + tx * 4 + v;
        if (r < n && c < n) A[(int64_t)r * lda + c] -= up[u][v];
      }
  }
}

// X = L^-1: diagonal blocks are the D_k; block row I: X_IJ = -D_I sum_{K=J}^{I-1} L_IK X_KJ.
__global__ __launch_bounds__(256) void place_diag(const double *D, double *X, int32_t ldx,
                                                   int32_t n) {
  const int k = blockIdx.x, g0 = k * NB, nb = min(NB, n - g0);
  for (int e = threadIdx.x; e < NB * NB; e += 256) {
    const int r = e / NB, c = e % NB;
    if (r < nb && c < nb) X[(int64_t)(g0 + r) * ldx + g0 + c] = D[(int64_t)k * NB * NB + e];
  }
}

__global__ __launch_bounds__(256) void trtri_row(const double *L, int32_t ldl, const double *D,
                                                  double *X, int32_t ldx, int32_t n, int32_t I) {
  __shared__ double Ta[NB * LP], Tb[NB * LP];
  const int J = blockIdx.x;
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const int i0 = I * NB, j0 = J * NB;
  double acc[4][4] = {};
  for (int K = J; K < I; ++K) {
    const int k0 = K * NB;
    for (int e = tid; e < NB * NB; e += 256) {
      const int r = e / NB, q = e % NB;
      Ta[r * LP + q] = (i0 + r < n) ? L[(int64_t)(i0 + r) * ldl + k0 + q] : 0.0;
      Tb[q * LP + r] = X[(int64_t)(k0 + r) * ldx + j0 + q];   // transposed: Tb[col][k]
    }
    __syncthreads();
    gemm_nt(Ta, Tb, acc, ty, tx);
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) Tb[(tx * 4 + v) * LP + ty * 4 + u] = acc[u][v];  // T^T
  for (int e = tid; e < NB * NB; e += 256) Ta[(e / NB) * LP + e % NB] = D[(int64_t)I * NB * NB + e];
  __syncthreads();
  double out[4][4] = {};
  gemm_nt(Ta, Tb, out, ty, tx);  // D_I T
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = i0 + ty * 4 + u, c = j0 + tx * 4 + v;
      if (r < n) X[(int64_t)r * ldx + c] = -out[u][v];
    }
}

// Single-workgroup triangular solves with the factor L and its diagonal-block
// inverses: y = L^-1 (w o rhs), out = L^-T y (w = sqrt(W) when given).
__global__ __launch_bounds__(1024) void trsv_both(const double *L, int32_t ldl, const double *D,
                                                   const double *rhs, const double *w,
                                                   double *out, int32_t n) {
  __shared__ double y[kMaxN];
  __shared__ double part[16][NB];
  __shared__ double tmp[NB];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int nbk = (n + NB - 1) / NB;
  for (int i = tid; i < n; i += 1024) y[i] = w ? w[i] * rhs[i] : rhs[i];
  __syncthreads();
  // forward
  for (int k = 0; k < nbk; ++k) {
    const int k0 = k * NB, kb = min(NB, n - k0);
    for (int rr = 0; rr < 4; ++rr) {
      const int r = wv * 4 + rr;
      double s = 0.0;
      if (r < kb)
        for (int c = lane; c < k0; c += 64) s = fma(L[(int64_t)(k0 + r) * ldl + c], y[c], s);
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
      if (lane == 0) tmp[r] = (r < kb) ? y[k0 + r] - s : 0.0;
    }
    __syncthreads();
    for (int rr = 0; rr < 4; ++rr) {
      const int r = wv * 4 + rr;
      double s = D[(int64_t)k * NB * NB + r * NB + lane] * tmp[lane];
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
      if (lane == 0 && r < kb) y[k0 + r] = s;
    }
    __syncthreads();
  }
  // backward: z_k = D_k^T (y_k - sum_{r beyond block k} L[r][k cols] z_r), z stored in y
  for (int k = nbk - 1; k >= 0; --k) {
    const int k0 = k * NB, kb = min(NB, n - k0);
    double s = 0.0;
    if (lane < kb)
      for (int r = k0 + NB + wv; r < n; r += 16) s = fma(L[(int64_t)r * ldl + k0 + lane], y[r], s);
    part[wv][lane] = s;
    __syncthreads();
    if (tid < NB) {
      double t = 0.0;
#pragma unroll
      for (int g = 0; g < 16; ++g) t += part[g][tid];
      tmp[tid] = (tid < kb) ? y[k0 + tid] - t : 0.0;
    }
    __syncthreads();
    if (tid < NB) {
      double z = 0.0;
      for (int q = 0; q < NB; ++q) z = fma(D[(int64_t)k * NB * NB + q * NB + tid], tmp[q], z);
      if (tid < kb) y[k0 + tid] = z;
    }
    __syncthreads();
  }
  for (int i = tid; i < n; i += 1024) out[i] = y[i];
}

// f_new = K a with a = b - w o z2 formed on the fly (block 0 also stores a).
__global__ __launch_bounds__(64) void gemv_newton(const double *K, int32_t ld, const double *b,
                                                   const double *w, const double *z2, double *a,
                                                   double *fnew, int32_t n) {
  const int r = blockIdx.x;
  double s = 0.0;
  for (int c = threadIdx.x; c < n; c += 64) {
    const double ac = b[c] - w[c] * z2[c];
    if (r == 0) a[c] = ac;
    s = fma(K[(int64_t)r * ld + c], ac, s);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
  if (threadIdx.x == 0) fnew[r] = s;
}

__global__ __launch_bounds__(256) void copy_lower_k(const double *src, int32_t lds, double *dst,
                                                     int32_t ldd, int32_t n) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)n * n) return;
  const int r = (int)(idx / n), c = (int)(idx - (int64_t)r * n);
  dst[(int64_t)r * ldd + c] = src[(int64_t)r * lds + c];
}

}  // namespace

hipError_t chol_factor(double *A, int32_t lda, double *L, int32_t ldl, double *D, int32_t n,
                       int32_t *info, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int nbk = (n + NB - 1) / NB;
  hipError_t e = hipMemsetAsync(L, 0, sizeof(double) * (size_t)ldl * n, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(chol_panel, dim3(1), dim3(256), 0, s, A, lda, L, ldl, D, n, info);
  for (int k = 0; k + 1 < nbk; ++k) {
    const int T = nbk - 1 - k;
    hipLaunchKernelGGL(chol_trailing, dim3(T * (T + 1) / 2), dim3(256), 0, s, A, lda, L, ldl, D,
                       k, n, info);
  }
  return hipGetLastError();
}

hipError_t chol_inverse(const double *L, int32_t ldl, const double *D, double *X, int32_t ldx,
                        int32_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int nbk = (n + NB - 1) / NB;
  hipError_t e = hipMemsetAsync(X, 0, sizeof(double) * (size_t)ldx * n, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(place_diag, dim3(nbk), dim3(256), 0, s, D, X, ldx, n);
  for (int I = 1; I < nbk; ++I)
    hipLaunchKernelGGL(trtri_row, dim3(I), dim3(256), 0, s, L, ldl, D, X, ldx, n, I);
  return hipGetLastError();
}

hipError_t chol_solve_both(const double *L, int32_t ldl, const double *D, const double *rhs,
                           const double *w, double *out, int32_t n, hipStream_t s) {
  hipLaunchKernelGGL(trsv_both, dim3(1), dim3(1024), 0, s, L, ldl, D, rhs, w, out, n);
  return hipGetLastError();
}

hipError_t launch_gemv_newton(const double *K, int32_t ld, const double *b, const double *w,
                              const double *z2, double *a, double *fnew, int32_t n, hipStream_t s) {
  hipLaunchKernelGGL(gemv_newton, dim3(n), dim3(64), 0, s, K, ld, b, w, z2, a, fnew, n);
  return hipGetLastError();
}

hipError_t launch_copy_matrix(const double *src, int32_t lds, double *dst, int32_t ldd, int32_t n,
                              hipStream_t s) {
  const int64_t tot = (int64_t)n * n;
  if (tot <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy_lower_k, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, src, lds,
                     dst, ldd, n);
  return hipGetLastError();
}

}  // namespace bgp
