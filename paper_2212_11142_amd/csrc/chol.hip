// fp64 blocked Cholesky for the model fit, with triangular solves and L^-T carried as
// extra rows of the factorisation.
//
// Right-looking Cholesky on NB x NB blocks (NB = 32) with one launch per block column:
//   * chol_panel factors the first diagonal block;
//   * chol_trailing(k) computes the panel L_ik = A_ik D_k^T (D_k = L_kk^-1, so the
//     triangular solve is a GEMM), subtracts L_ik L_jk^T from every trailing block
//     (i >= j), and the workgroup owning block (k+1, k+1) factors it right away, so
//     the next launch already has L_{k+1,k+1} and D_{k+1}.
// Each diagonal factorisation also produces its inverse D_k, with which the panels are
// GEMMs. Optional extra rows E stored below A (rows n.., columns 0..n-1)
// are carried through the same right-looking updates; their final panels form
// L_E = E L^-T, i.e. L_E^T = L^-1 E^T, the forward solve of L against every column of
// E^T, at the cost of parallel workgroups beside the critical one. The last n_ident
// extra rows may be an identity block (L_E = L^-T there): its block row e stays zero
// until step e, so its workgroups start at that step.
// A device int `info` records the first failing pivot (1-based, global row); every
// kernel returns immediately once it is set.
#include <algorithm>

#include "common.h"

namespace bgp {
namespace {

constexpr int NB = kNB;      // factorisation block
constexpr int TT = NB / 16;  // each of the 16 x 16 threads of a workgroup holds a TT x TT tile
constexpr int LP = NB + 1;   // LDS row stride (doubles)
constexpr int kPer = NB * NB / 256;  // elements of a block per thread
static_assert(NB * NB % 256 == 0, "block elements per thread");
static_assert(NB % 16 == 0 && NB <= 64, "block size");

__device__ __forceinline__ void tri_index(int L, int &bi, int &bj) {
  int i = (int)((sqrt(8.0 * L + 1.0) - 1.0) * 0.5);
  while ((i + 1) * (i + 2) / 2 <= L) ++i;
  while (i * (i + 1) / 2 > L) --i;
  bi = i;
  bj = L - i * (i + 1) / 2;
}

// Block products on fp64 MFMA: each of the 4 wavefronts owns one 16 x 16 quadrant of a
// 32 x 32 result. v_mfma_f64_16x16x4f64 takes A[row l & 15][k l >> 4] and
// B[k l >> 4][col l & 15] from lane l and leaves element v of the quadrant's result at
// row (l >> 4) + 4 v, column l & 15 (the layout every "quad" array below follows).
typedef double doublex4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ int quad_row(int v) {
  return 16 * ((int)threadIdx.x >> 7) + (((int)threadIdx.x & 63) >> 4) + 4 * v;
}
__device__ __forceinline__ int quad_col() {
  return 16 * (((int)threadIdx.x >> 6) & 1) + ((int)threadIdx.x & 15);
}

// acc (quadrant layout) += sum_q Aa[r][q] * Bb[c][q] over q < NB (LDS, stride LP); two
// accumulators split the k-chain
__device__ __forceinline__ void gemm_nt(const double *Aa, const double *Bb, doublex4 &acc) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const double *ar = Aa + (16 * (w >> 1) + (lane & 15)) * LP + (lane >> 4);
  const double *br = Bb + (16 * (w & 1) + (lane & 15)) * LP + (lane >> 4);
  doublex4 acc2 = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int q = 0; q < NB; q += 8) {
    acc = __builtin_amdgcn_mfma_f64_16x16x4f64(ar[q], br[q], acc, 0, 0, 0);
    acc2 = __builtin_amdgcn_mfma_f64_16x16x4f64(ar[q + 4], br[q + 4], acc2, 0, 0, 0);
  }
  acc += acc2;
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

constexpr int PW = 4;  // factorisation panel width (columns), a multiple of TT
static_assert(PW % TT == 0 && NB % PW == 0, "panel width");

// Cholesky of the nb x nb (nb <= NB) block in S (LDS, lower part read) and its inverse,
// on all 256 threads: thread (ty, tx) keeps the TT x TT sub-block at rows TT ty..,
// columns TT tx.. in registers (rows/columns >= nb are padded with the identity).
// Factorisation, right-looking in panels of PW columns without square roots on the
// serial chain (A = U D U^T, U unit lower): the owners of a panel publish it (one barrier
// per panel, double buffered, stored column-major); every thread factors the PW x PW
// pivot block itself, brings its own rows' and columns' panel entries up to date (a
// pivot row brought up to date is the eliminated pivot block row, so the owners take
// their final values from the same arrays) and applies the rank-PW update
// a_rc -= sum_p a_rp a_cp / piv_p to its trailing elements, with selects instead of
// branches. The inverse rides along: Y = U^-1 is the same elimination applied to the
// identity (row r of Y loses U[r][p] times the final row p of Y at pivot p), so the
// owners of the panel's rows of Y publish them with the panel, every thread finishes
// those rows for its columns with the pivot block and subtracts them from its rows
// below. At the end L = U D^1/2 and L^-1 = D^-1/2 Y are one scaling pass each.
// Output: S = L (lower, zero elsewhere), Di = L^-1. *fail = 1-based failing pivot or 0.
// Tb: 4 PW NB doubles of panel buffers; colbuf: NB doubles.
__device__ __forceinline__ void factor_invert_block(double *S, double *Di, double *colbuf,
                                                    double *Tb, int *fail, int nb) {
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  double *pb0 = Tb, *pb1 = Tb + PW * NB;  // panel [PW][NB]: column p, row r at p * NB + r
  double *yb0 = Tb + 2 * PW * NB, *yb1 = Tb + 3 * PW * NB;  // rows of Y [PW][NB]
  double a[TT][TT], y[TT][TT];
#pragma unroll
  for (int u = 0; u < TT; ++u)
#pragma unroll
    for (int v = 0; v < TT; ++v) {
      const int r = TT * ty + u, c = TT * tx + v;
      a[u][v] = (r < nb && c < nb) ? (c <= r ? S[r * LP + c] : 0.0) : (r == c ? 1.0 : 0.0);
      y[u][v] = (r == c) ? 1.0 : 0.0;
    }
  int bad = 0;
  for (int jb = 0; jb < NB; jb += PW) {
    const bool odd = (jb / PW) & 1;
    double *pb = odd ? pb1 : pb0, *yb = odd ? yb1 : yb0;
    const int vc0 = TT * tx - jb;  // this thread's first column within the panel
    const bool own_c = vc0 >= 0 && vc0 < PW;
    const int vr0 = TT * ty - jb;  // this thread's first row within the panel
    const bool own_r = vr0 >= 0 && vr0 < PW;
    if (own_c) {
#pragma unroll
      for (int u = 0; u < TT; ++u)
#pragma unroll
        for (int v = 0; v < TT; ++v) pb[(vc0 + v) * NB + TT * ty + u] = a[u][v];
    }
    if (own_r) {
#pragma unroll
      for (int u = 0; u < TT; ++u)
#pragma unroll
        for (int v = 0; v < TT; ++v) yb[(vr0 + u) * NB + TT * tx + v] = y[u][v];
    }
    __syncthreads();
    // PW x PW pivot block, factored locally (unscaled right-looking): w[s][p] is the
    // panel entry of row jb+s when column jb+p becomes the pivot column.
    double w[PW][PW], cr[TT][PW], cc[TT][PW], ip[PW], yr[PW][TT];
#pragma unroll
    for (int p = 0; p < PW; ++p) {
#pragma unroll
      for (int u = 0; u < PW; ++u) w[u][p] = pb[p * NB + jb + u];
#pragma unroll
      for (int u = 0; u < TT; ++u) {
        cr[u][p] = pb[p * NB + TT * ty + u];
        cc[u][p] = pb[p * NB + TT * tx + u];
      }
#pragma unroll
      for (int v = 0; v < TT; ++v) yr[p][v] = yb[p * NB + TT * tx + v];
    }
#pragma unroll
    for (int p = 0; p < PW; ++p) {
      double pv = w[p][p];
      const bool ok = pv > 0.0 && isfinite(pv);
      bad = (!ok && !bad) ? jb + p + 1 : bad;
      pv = ok ? pv : 1.0;
      w[p][p] = pv;
      ip[p] = rcp_nr(pv);
#pragma unroll
      for (int s2 = p + 1; s2 < PW; ++s2)
#pragma unroll
        for (int t = p + 1; t <= s2; ++t) w[s2][t] = fma(-w[s2][p] * ip[p], w[t][p], w[s2][t]);
    }
    if (tid == 0) {
#pragma unroll
      for (int p = 0; p < PW; ++p) colbuf[jb + p] = w[p][p];
    }
    // bring the panel entries of the thread's rows and columns up to date
#pragma unroll
    for (int u = 0; u < TT; ++u) {
#pragma unroll
      for (int p = 1; p < PW; ++p)
#pragma unroll
        for (int q = 0; q < p; ++q) {
          cr[u][p] = fma(-cr[u][q] * ip[q], w[p][q], cr[u][p]);
          cc[u][p] = fma(-cc[u][q] * ip[q], w[p][q], cc[u][p]);
        }
#pragma unroll
      for (int p = 0; p < PW; ++p) cc[u][p] *= ip[p];
    }
    // the panel's rows of Y, finished with the pivot block's unit lower part
#pragma unroll
    for (int s2 = 1; s2 < PW; ++s2)
#pragma unroll
      for (int q = 0; q < s2; ++q)
#pragma unroll
        for (int v = 0; v < TT; ++v) yr[s2][v] = fma(-w[s2][q] * ip[q], yr[q][v], yr[s2][v]);
    // owners keep the final unscaled panel columns; trailing elements get the update
#pragma unroll
    for (int u = 0; u < TT; ++u)
#pragma unroll
      for (int v = 0; v < TT; ++v) {
        const int r = TT * ty + u, c = TT * tx + v;
        double t = a[u][v];
#pragma unroll
        for (int p = 0; p < PW; ++p) t = fma(-cr[u][p], cc[v][p], t);
        double fin = cr[u][v];
#pragma unroll
        for (int o = TT; o < PW; o += TT) fin = (vc0 == o) ? cr[u][o + v] : fin;
        const bool upd = own_c ? (r >= c) : (c >= jb + PW && r >= c);
        a[u][v] = upd ? (own_c ? fin : t) : a[u][v];
        // Y: the panel's rows take their finished values, rows below lose
        // U[r][jb+p] = cr[u][p] / piv_p times them
        double ty_ = y[u][v];
#pragma unroll
        for (int p = 0; p < PW; ++p) ty_ = fma(-cr[u][p] * ip[p], yr[p][v], ty_);
        double yfin = yr[u][v];
#pragma unroll
        for (int o = TT; o < PW; o += TT) yfin = (vr0 == o) ? yr[o + u][v] : yfin;
        y[u][v] = own_r ? yfin : (r >= jb + PW ? ty_ : y[u][v]);
      }
  }
  __syncthreads();
  if (tid == 0) *fail = (bad && bad <= nb) ? bad : 0;
  __syncthreads();
  if (*fail) return;
  // L = U D^1/2 (columns times sqrt(piv_c)), L^-1 = D^-1/2 Y (rows over sqrt(piv_r))
  double rs[TT], rr[TT];
#pragma unroll
  for (int v = 0; v < TT; ++v) {
    rs[v] = rsqrt_nr(colbuf[TT * tx + v]);
    rr[v] = rsqrt_nr(colbuf[TT * ty + v]);
  }
#pragma unroll
  for (int u = 0; u < TT; ++u)
#pragma unroll
    for (int v = 0; v < TT; ++v) {
      const int r = TT * ty + u, c = TT * tx + v;
      const bool in = r < nb && c < nb;
      S[r * LP + c] = (in && c <= r) ? a[u][v] * rs[v] : 0.0;
      Di[r * LP + c] = in ? y[u][v] * rr[u] : 0.0;
    }
  __syncthreads();
}

__device__ __forceinline__ void store_factor(const double *S, const double *Di, double *L, int ldl,
                                             double *Dk, int g0, int nb) {
  for (int e = threadIdx.x; e < NB * NB; e += 256) {
    const int r = e / NB, c = e % NB;
    if (r < nb && c < nb) L[(int64_t)(g0 + r) * ldl + g0 + c] = S[r * LP + c];
    Dk[e] = Di[r * LP + c];
  }
}

__global__ __launch_bounds__(256) void chol_panel(const double *A, int32_t lda, double *L,
                                                   int32_t ldl, double *D, int32_t n,
                                                   int32_t *info, const int32_t *halt,
                                                   const CholBatch bt) {
  __shared__ double S[NB * LP], Di[NB * LP], colbuf[NB], Tb[4 * PW * NB];
  __shared__ int fail;
  {
    const int64_t b = blockIdx.z;
    A += b * bt.sA;
    L += b * bt.sL;
    D += b * bt.sD;
    info += b;
  }
  if (*info || (halt && *halt)) return;
  const int nb = min(NB, n);
  double v[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {  // all loads in flight, then the LDS stores
    const int e = threadIdx.x + 256 * u, r = e / NB, c = e % NB;
    v[u] = (r < nb && c <= r) ? A[(int64_t)r * lda + c] : 0.0;
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int e = threadIdx.x + 256 * u;
    S[(e / NB) * LP + e % NB] = v[u];
  }
  __syncthreads();
  factor_invert_block(S, Di, colbuf, Tb, &fail, nb);
  if (fail) {
    if (threadIdx.x == 0) *info = fail;
    return;
  }
  store_factor(S, Di, L, ldl, D, 0, nb);
}

// Newton setup (see launch_newton_setup): workgroup 0 builds B's first diagonal block
// itself and factors it (dispatched first, it overlaps the rest); the next workgroups
// each write a tile of kSetupRows rows x 256 columns of the stacked matrix [B ; I]; the
// last ones form v = W^1/2 K b for kSetupVRows rows each. Probit terms are computed once
// per row and column of a tile (not per element: they are the costly part), the row
// terms into LDS; the tiles of row 0 also store the vectors.
constexpr int kSetupRows = 32;
constexpr int kSetupVRows = 8;
__global__ __launch_bounds__(256) void newton_setup_k(const double *K, const double *f,
                                                       const double *t, double *grad, double *W,
                                                       double *sw, double *b, double *v,
                                                       double *A, int32_t n, int64_t nfill,
                                                       double *L, double *D, int32_t *info,
                                                       const int32_t *halt) {
  __shared__ double S[NB * LP], Di[NB * LP], colbuf[NB], Tb[4 * PW * NB];
  __shared__ double swr[kSetupRows > NB ? kSetupRows : NB];
  __shared__ int fail;
  if (*info || *halt) return;
  const int tid = threadIdx.x;
  if (blockIdx.x == 0) {
    const int nb = min(NB, n);
    if (tid < nb) {
      double g, w;
      probit_terms(f[tid], t[tid], g, w);
      swr[tid] = sqrt(w);
    }
    __syncthreads();
    double kv[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {  // all loads in flight, then the LDS stores
      const int e = tid + 256 * u, r = e / NB, c = e % NB;
      kv[u] = (r < nb && c <= r) ? K[(int64_t)r * n + c] : 0.0;
    }
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = tid + 256 * u, r = e / NB, c = e % NB;
      S[r * LP + c] = (r < nb && c <= r) ? swr[r] * kv[u] * swr[c] + (r == c ? 1.0 : 0.0) : 0.0;
    }
    __syncthreads();
    factor_invert_block(S, Di, colbuf, Tb, &fail, nb);
    if (fail) {
      if (tid == 0) *info = fail;
      return;
    }
    store_factor(S, Di, L, n, D, 0, nb);
    return;
  }
  if ((int64_t)blockIdx.x > nfill) {
    // v[r] = W_r^1/2 sum_c K[r][c] b[c] for kSetupVRows rows; each thread takes the
    // columns tid, tid + 256, ... (b from the probit terms at f) and every row's partial
    // sums are reduced over the workgroup in a fixed order
    const int r0 = (int)((int64_t)blockIdx.x - nfill - 1) * kSetupVRows;
    double acc[kSetupVRows];
#pragma unroll
    for (int q = 0; q < kSetupVRows; ++q) acc[q] = 0.0;
    for (int c = tid; c < n; c += 256) {
      double gc, wc;
      probit_terms(f[c], t[c], gc, wc);
      const double bc = fma(wc, f[c], gc);
#pragma unroll
      for (int q = 0; q < kSetupVRows; ++q)
        if (r0 + q < n) acc[q] = fma(K[(int64_t)(r0 + q) * n + c], bc, acc[q]);
    }
    const int lane = tid & 63, wv = tid >> 6;
#pragma unroll
    for (int q = 0; q < kSetupVRows; ++q) {
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) acc[q] += __shfl_xor(acc[q], off);
      if (lane == 0) S[wv * kSetupVRows + q] = acc[q];
    }
    __syncthreads();
    if (tid < kSetupVRows && r0 + tid < n) {
      const int r = r0 + tid;
      double g, w;
      probit_terms(f[r], t[r], g, w);
      const double u = (S[tid] + S[kSetupVRows + tid]) + (S[2 * kSetupVRows + tid] + S[3 * kSetupVRows + tid]);
      v[r] = sqrt(w) * u;
    }
    return;
  }
  const int nct = (n + 255) / 256;
  const int tr = (int)(blockIdx.x - 1) / nct, tcol = (int)(blockIdx.x - 1) - tr * nct;
  const int r0 = tr * kSetupRows, rows = 2 * n;
  const int c = tcol * 256 + tid;
  if (r0 < n) {  // workgroup-uniform: the tile has rows of B
    if (tid < kSetupRows && r0 + tid < n) {
      double g, w;
      probit_terms(f[r0 + tid], t[r0 + tid], g, w);
      swr[tid] = sqrt(w);
    }
    __syncthreads();
  }
  if (c >= n) return;
  double gc, wc;
  probit_terms(f[c], t[c], gc, wc);
  const double swc = sqrt(wc);
  if (r0 == 0) {
    grad[c] = gc;
    W[c] = wc;
    sw[c] = swc;
    b[c] = fma(wc, f[c], gc);
  }
  const int rend = min(r0 + kSetupRows, rows);
  for (int r = r0; r < rend; ++r) {
    const double x = r < n ? swr[r - r0] * K[(int64_t)r * n + c] * swc + (r == c ? 1.0 : 0.0)
                           : (r - n == c ? 1.0 : 0.0);
    A[(int64_t)r * n + c] = x;
  }
}

// Global loads of the block steps are unconditional: a row or column index past the
// matrix is clamped to its last one (finite data), and whatever it feeds is either
// multiplied by the zero padding of D_k or never stored. All of a workgroup's loads are
// issued before its first barrier.

// Workgroup (e, bj) of the extra rows at block step k: rows n + e NB.. of A, trailing
// block column j0 = k0 + NB + bj NB. P_e = A_Ek D_k^T (final: L_E panel, stored by bj = 0,
// the only workgroup of block row e when there is no trailing column), P_j = A_jk D_k^T,
// A_Ej -= P_e P_j^T.
__device__ __forceinline__ void extra_rows_step(double *A, int32_t lda, const double *Dk,
                                                double *LE, int32_t ldle, int k, int e, int bj,
                                                int T, int n, int n_extra, bool le_t, double *Ds,
                                                double *Pi, double *Pj, double *Ts, double *Tj) {
  const int k0 = k * NB, ie = e * NB, j0 = k0 + NB + bj * NB;
  const int tid = threadIdx.x, qc = quad_col();
  const int rmax = n - 1, emax = n_extra - 1;
  doublex4 tile;
  double dv[kPer], tv[kPer], jv[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {  // all loads in flight, then the LDS stores
    const int q = tid + 256 * u, r = q / NB, c = q % NB;
    dv[u] = Dk[q];
    tv[u] = A[(int64_t)(n + min(ie + r, emax)) * lda + min(k0 + c, rmax)];
    jv[u] = T > 0 ? A[(int64_t)min(j0 + r, rmax) * lda + k0 + c] : 0.0;
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int q = tid + 256 * u, r = q / NB, c = q % NB;
    Ds[r * LP + c] = dv[u];
    Ts[r * LP + c] = tv[u];
    if (T > 0) Tj[r * LP + c] = jv[u];
  }
  if (T > 0) {
#pragma unroll
    for (int v = 0; v < 4; ++v)
      tile[v] = A[(int64_t)(n + min(ie + quad_row(v), emax)) * lda + min(j0 + qc, rmax)];
  }
  __syncthreads();
  doublex4 acc = {0.0, 0.0, 0.0, 0.0}, acc2 = {0.0, 0.0, 0.0, 0.0};
  gemm_nt(Ts, Ds, acc);               // P_e = A_Ek D_k^T
  if (T > 0) gemm_nt(Tj, Ds, acc2);   // P_j = A_jk D_k^T
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    Pi[quad_row(v) * LP + qc] = acc[v];
    Pj[quad_row(v) * LP + qc] = acc2[v];
  }
  __syncthreads();
  if (bj == 0) {
    for (int q = tid; q < NB * NB; q += 256) {
      const int r = q / NB, c = q % NB;
      if (ie + r < n_extra && k0 + c < n) {
        if (le_t) LE[(int64_t)(k0 + c) * ldle + ie + r] = Pi[r * LP + c];  // L_E^T
        else LE[(int64_t)(ie + r) * ldle + k0 + c] = Pi[r * LP + c];
      }
    }
  }
  if (T == 0) return;
  doublex4 up = {0.0, 0.0, 0.0, 0.0};
  gemm_nt(Pi, Pj, up);
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int r = ie + quad_row(v), c = j0 + qc;
    if (r < n_extra && c < n) A[(int64_t)(n + r) * lda + c] = tile[v] - up[v];
  }
}

__global__ __launch_bounds__(256) void chol_trailing(double *A, int32_t lda, double *L,
                                                      int32_t ldl, double *D, int32_t k,
                                                      int32_t n, int32_t n_extra, double *LE,
                                                      int32_t ldle, int32_t *info,
                                                      const int32_t *halt, const CholBatch bt,
                                                      int32_t le_t) {
  __shared__ double Ds[NB * LP], Pi[NB * LP], Pj[NB * LP], Ts[NB * LP], Tj[NB * LP];
  __shared__ double colbuf[NB], Tb[4 * PW * NB];
  __shared__ int fail;
  {
    const int64_t b = blockIdx.z;  // (a batched launch's extra rows are identity rows)
    A += b * bt.sA;
    L += b * bt.sL;
    D += b * bt.sD;
    if (LE) LE += b * bt.sX;
    info += b;
  }
  if (*info || (halt && *halt)) return;
  const int nbk = (n + NB - 1) / NB, T = nbk - 1 - k, nsq = T * (T + 1) / 2;
  if ((int)blockIdx.x >= nsq) {  // extra rows (identity blocks past step k are not launched)
    const int q = blockIdx.x - nsq, Tc = T > 0 ? T : 1;
    extra_rows_step(A, lda, D + (int64_t)k * NB * NB, LE, ldle, k, q / Tc, q % Tc, T, n, n_extra,
                    le_t != 0,
                    Ds, Pi, Pj, Ts, Tj);
    return;
  }
  int bi, bj;
  tri_index(blockIdx.x, bi, bj);
  const int k0 = k * NB;  // k < nbk - 1 here, so block column k is full
  const int i0 = k0 + NB + bi * NB, j0 = k0 + NB + bj * NB;
  const int tid = threadIdx.x, qc = quad_col();
  const int rmax = n - 1;
  const double *Dk = D + (int64_t)k * NB * NB;
  // A_ij (for bi = bj = 0 the next diagonal block), prefetched for the end
  doublex4 tile;
#pragma unroll
  for (int v = 0; v < 4; ++v)
    tile[v] = A[(int64_t)min(i0 + quad_row(v), rmax) * lda + min(j0 + qc, rmax)];
  double dv[kPer], tv[kPer], jv[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {  // all loads in flight, then the LDS stores
    const int e = tid + 256 * u, r = e / NB, c = e % NB;
    dv[u] = Dk[e];
    tv[u] = A[(int64_t)min(i0 + r, rmax) * lda + k0 + c];
    jv[u] = A[(int64_t)min(j0 + r, rmax) * lda + k0 + c];
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int e = tid + 256 * u, r = e / NB, c = e % NB;
    Ds[r * LP + c] = dv[u];
    Ts[r * LP + c] = tv[u];
    if (bi != bj) Tj[r * LP + c] = jv[u];
  }
  __syncthreads();
  {
    doublex4 acc = {0.0, 0.0, 0.0, 0.0};
    gemm_nt(Ts, Ds, acc);  // P_i = A_ik D_k^T = L_ik
#pragma unroll
    for (int v = 0; v < 4; ++v) Pi[quad_row(v) * LP + qc] = acc[v];
    if (bi != bj) {
      doublex4 acc2 = {0.0, 0.0, 0.0, 0.0};
      gemm_nt(Tj, Ds, acc2);  // P_j
#pragma unroll
      for (int v = 0; v < 4; ++v) Pj[quad_row(v) * LP + qc] = acc2[v];
    }
  }
  __syncthreads();
  const double *Pjj = (bi == bj) ? Pi : Pj;
  doublex4 up = {0.0, 0.0, 0.0, 0.0};
  gemm_nt(Pi, Pjj, up);
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
    for (int v = 0; v < 4; ++v) {
      const int r = quad_row(v);
      Ts[r * LP + qc] = (i0 + r < n && i0 + qc < n) ? tile[v] - up[v] : 0.0;
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
    for (int v = 0; v < 4; ++v) {
      const int r = i0 + quad_row(v), c = j0 + qc;
      if (r < n && c < n) A[(int64_t)r * lda + c] = tile[v] - up[v];
    }
  }
}

// out = X^T X (both triangles) for lower-triangular X: the workgroup of output block
// (bi, bj), bi >= bj, sums X_{R,bi}^T X_{R,bj} over the block rows R >= bi (X is zero
// above them) on fp64 MFMA; the two column blocks go to LDS transposed so that the
// block product of gemm_nt contracts over the rows.
__global__ __launch_bounds__(256) void ata_mfma_k(const double *X, int32_t ld, double *out,
                                                   int32_t n, const int32_t *info,
                                                   const CholBatch bt) {
  __shared__ double Ta[NB * LP], Tb[NB * LP];
  {
    const int64_t b = blockIdx.z;
    if (info && info[b]) return;
    X += b * bt.sX;
    out += b * bt.sA;
  }
  int bi, bj;
  tri_index(blockIdx.x, bi, bj);
  const int nbk = (n + NB - 1) / NB, tid = threadIdx.x, qc = quad_col();
  const int ci = bi * NB, cj = bj * NB;
  doublex4 acc = {0.0, 0.0, 0.0, 0.0};
  // the next block row's values are loaded into registers while this one is multiplied
  double va[kPer], vb[kPer];
  auto load = [&](int Rb) {
    const int r0 = Rb * NB;
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = tid + 256 * u, r = e / NB, c = e % NB;
      const bool rin = r0 + r < n;
      const double *xr = X + (int64_t)(r0 + r) * ld;
      va[u] = (rin && ci + c < n) ? xr[ci + c] : 0.0;
      vb[u] = (rin && cj + c < n) ? xr[cj + c] : 0.0;
    }
  };
  load(bi);
  for (int Rb = bi; Rb < nbk; ++Rb) {
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = tid + 256 * u, r = e / NB, c = e % NB;
      Ta[c * LP + r] = va[u];
      Tb[c * LP + r] = vb[u];
    }
    __syncthreads();
    if (Rb + 1 < nbk) load(Rb + 1);
    gemm_nt(Ta, Tb, acc);  // acc[r][c] += sum_q X[q][ci + r] X[q][cj + c]
    __syncthreads();
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int r = ci + quad_row(v), c = cj + qc;
    if (r < n && c < n) {
      out[(int64_t)r * ld + c] = acc[v];
      out[(int64_t)c * ld + r] = acc[v];
    }
  }
}

__global__ __launch_bounds__(256) void copy_lower_k(const double *src, int32_t lds, double *dst,
                                                     int32_t ldd, int32_t n) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)n * n) return;
  const int r = (int)(idx / n), c = (int)(idx - (int64_t)r * n);
  dst[(int64_t)r * ldd + c] = src[(int64_t)r * lds + c];
}

// dst (2n rows, stride n) = [src; I]: the matrix, then identity rows whose factorisation
// panels give L^-T
__global__ __launch_bounds__(256) void copy_ident_k(const double *src, int32_t lds, double *dst,
                                                     int32_t n) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= 2 * (int64_t)n * n) return;
  const int r = (int)(idx / n), c = (int)(idx - (int64_t)r * n);
  dst[idx] = r < n ? src[(int64_t)r * lds + c] : (r - n == c ? 1.0 : 0.0);
}


}  // namespace

hipError_t launch_copy_ident(const double *src, int32_t lds, double *dst, int32_t n,
                             hipStream_t s) {
  const int64_t tot = 2 * (int64_t)n * n;
  if (tot <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy_ident_k, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, src, lds,
                     dst, n);
  return hipGetLastError();
}

hipError_t chol_factor(double *A, int32_t lda, double *L, int32_t ldl, double *D, int32_t n,
                       int32_t *info, hipStream_t s, int32_t n_extra, double *LE, int32_t ldle,
                       const int32_t *halt, bool clear_upper, int32_t n_ident,
                       bool first_block_done) {
  if (n <= 0) return hipSuccess;
  if (n_extra < 0 || (n_extra > 0 && !LE)) return hipErrorInvalidValue;
  // identity rows: the last n extra rows, starting on a block boundary
  if (n_ident != 0 && (n_ident != n || n_extra < n_ident || (n_extra - n_ident) % NB))
    return hipErrorInvalidValue;
  const int nbk = (n + NB - 1) / NB, ne_dense = (n_extra - n_ident + NB - 1) / NB;
  const int ne_ident = (n_ident + NB - 1) / NB;
  if (clear_upper) {
    hipError_t e = hipMemsetAsync(L, 0, sizeof(double) * (size_t)ldl * n, s);
    if (e != hipSuccess) return e;
  }
  if (!first_block_done)
    hipLaunchKernelGGL(chol_panel, dim3(1), dim3(256), 0, s, A, lda, L, ldl, D, n, info, halt,
                       CholBatch{});
  for (int k = 0; k < nbk; ++k) {
    const int T = nbk - 1 - k;
    const int ne = ne_dense + std::min(k + 1, ne_ident);  // identity block e joins at step e
    const int grid = T * (T + 1) / 2 + ne * (T > 0 ? T : 1);
    if (grid == 0) break;  // last block column without extra rows
    hipLaunchKernelGGL(chol_trailing, dim3(grid), dim3(256), 0, s, A, lda, L, ldl, D, k, n,
                       n_extra, LE, ldle, info, halt, CholBatch{}, 0);
  }
  return hipGetLastError();
}

hipError_t chol_factor_batched(double *A, int32_t lda, double *L, int32_t ldl, double *D,
                               int32_t n, int32_t *info, const CholBatch &bt, hipStream_t s,
                               bool clear_upper, double *X, int32_t ldx) {
  if (n <= 0 || bt.count <= 0) return hipSuccess;
  if (bt.count > 65535 || bt.sL < (int64_t)ldl * n) return hipErrorInvalidValue;
  if (X && (bt.sA < 2 * (int64_t)lda * n || bt.sX < (int64_t)ldx * n)) return hipErrorInvalidValue;
  const int nbk = (n + NB - 1) / NB;
  if (clear_upper) {
    hipError_t e = hipMemsetAsync(L, 0, sizeof(double) * (size_t)bt.sL * bt.count, s);
    if (e != hipSuccess) return e;
  }
  if (X) {  // L^-1's blocks above the diagonal are never written
    hipError_t e = hipMemsetAsync(X, 0, sizeof(double) * (size_t)bt.sX * bt.count, s);
    if (e != hipSuccess) return e;
  }
  const unsigned z = (unsigned)bt.count;
  hipLaunchKernelGGL(chol_panel, dim3(1, 1, z), dim3(256), 0, s, A, lda, L, ldl, D, n, info,
                     nullptr, bt);
  for (int k = 0; k < nbk; ++k) {
    const int T = nbk - 1 - k;
    // with X: the identity rows' block e joins at step e; their panels, stored transposed,
    // are L^-1
    const int ne = X ? std::min(k + 1, nbk) : 0;
    const int grid = T * (T + 1) / 2 + ne * (T > 0 ? T : 1);
    if (grid == 0) break;
    hipLaunchKernelGGL(chol_trailing, dim3(grid, 1, z), dim3(256), 0, s, A, lda, L, ldl, D, k, n,
                       X ? n : 0, X, ldx, info, nullptr, bt, X ? 1 : 0);
  }
  return hipGetLastError();
}


hipError_t launch_newton_setup(const double *K, const double *f, const double *t, double *grad,
                               double *W, double *sw, double *b, double *v, double *A, int32_t n,
                               double *L, double *D, int32_t *info, const int32_t *halt,
                               hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t nfill = (int64_t)((2 * n + kSetupRows - 1) / kSetupRows) * ((n + 255) / 256);
  const int64_t nv = (n + kSetupVRows - 1) / kSetupVRows;
  hipLaunchKernelGGL(newton_setup_k, dim3((unsigned)(1 + nfill + nv)), dim3(256), 0, s, K, f, t,
                     grad, W, sw, b, v, A, n, nfill, L, D, info, halt);
  return hipGetLastError();
}


hipError_t launch_ata_batched(const double *X, int32_t ld, double *out, int32_t n,
                              const int32_t *info, const CholBatch &bt, hipStream_t s) {
  if (n <= 0 || bt.count <= 0) return hipSuccess;
  if (bt.count > 65535) return hipErrorInvalidValue;
  const int nbk = (n + NB - 1) / NB;
  hipLaunchKernelGGL(ata_mfma_k, dim3(nbk * (nbk + 1) / 2, 1, (unsigned)bt.count), dim3(256), 0, s,
                     X, ld, out, n, info, bt);
  return hipGetLastError();
}

hipError_t launch_ata_lower(const double *X, int32_t ld, double *out, int32_t n, hipStream_t s) {
  return launch_ata_batched(X, ld, out, n, nullptr, CholBatch{}, s);
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
