// Posterior-variance contraction, EI / feasibility epilogue, fp64 recomputation of
// ill-conditioned candidates, arg-max and term inspection.
//
// Variance (textbook GP regression; the paper uses the GP of Sec. 3.2 without printing
// these formulas): sigma^2 = s - |L_f^-1 k*|^2. With B = L_f^-T (upper triangular) the
// squared norms are row sums of (K* B)^2. The classifier's predictive variance
// V = s_c - |L_B^-1 W^1/2 k_c*|^2 has the same shape with B = rho W^1/2 L_B^-T. Both are
// one fp32 MFMA GEMM over K* against the packed B^T, whose column tiles stop the
// k-loop at the triangle (tile [c0, c0+128) only needs k < c0+128), and whose epilogue
// reduces each 128-column tile to one partial per row; V = K* B itself is never stored.
#include "common.h"
#include "dist64.h"

namespace bgp {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

// Blocks are dispatched round-robin over the 8 XCDs (block b runs on XCD b % 8). Give
// each XCD a contiguous range of logical tiles so that the column tiles of one row
// block (which share the same K* rows) run on the same XCD and hit its L2.
__device__ __forceinline__ int xcd_remap(int b, int G) {
  const int q = G >> 3, r = G & 7;
  const int x = b & 7, k = b >> 3;
  return x * q + (x < r ? x : r) + k;
}

constexpr int kLdsStride = 36;  // 32 k-values + 4 floats padding per row

__global__ __launch_bounds__(256, 2) void contract_f32(const CArgs a) {
  __shared__ __attribute__((aligned(16))) float As[2][kRowTile * kLdsStride];
  __shared__ __attribute__((aligned(16))) float Bs[2][kColTile * kLdsStride];
  __shared__ float red[2][kRowTile];

  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int rt = L / a.ntiles, t = L - rt * a.ntiles;
  const CTile tl = a.tiles[t];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t row0 = (int64_t)rt * kRowTile;
  const float *Ag = a.A + row0 * a.lda;
  const float *Bg = a.Bt + (int64_t)tl.bcol * a.lda;
  const int nk = tl.kend / kKChunk;

  // global -> register staging: thread covers rows lr + 32 q, columns lc..lc+3
  const int lr = tid >> 3, lc = (tid & 7) * 4;
  floatx4 ra[4], rb[4];
  auto gload = [&](int kc) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      ra[q] = *(const floatx4 *)(Ag + (int64_t)(lr + 32 * q) * a.lda + kc * kKChunk + lc);
      rb[q] = *(const floatx4 *)(Bg + (int64_t)(lr + 32 * q) * a.lda + kc * kKChunk + lc);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      *(floatx4 *)&As[buf][(lr + 32 * q) * kLdsStride + lc] = ra[q];
      *(floatx4 *)&Bs[buf][(lr + 32 * q) * kLdsStride + lc] = rb[q];
    }
  };

  floatx4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[i][k] = floatx4{0.f, 0.f, 0.f, 0.f};

  // wave tile 64 x 64 at (wr, wc); MFMA 16x16x4: lane supplies A[row fr][k] and
  // B[k][col fr] with k = 4 (lane >> 4) + s for step s, so each lane's 4 steps read one
  // contiguous float4 (any k order works as long as A and B agree).
  const int wr = (w >> 1) * 64, wc = (w & 1) * 64;
  const int fr = lane & 15, fk = (lane >> 4) * 4;

  gload(0);
  sstore(0);
  __syncthreads();
  for (int kc = 0; kc < nk; ++kc) {
    const int buf = kc & 1;
    if (kc + 1 < nk) gload(kc + 1);
#pragma unroll
    for (int kk = 0; kk < kKChunk; kk += 16) {
      floatx4 av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        av[i] = *(const floatx4 *)&As[buf][(wr + i * 16 + fr) * kLdsStride + kk + fk];
        bv[i] = *(const floatx4 *)&Bs[buf][(wc + i * 16 + fr) * kLdsStride + kk + fk];
      }
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int k = 0; k < 4; ++k)
            acc[i][k] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i][s], bv[k][s], acc[i][k], 0, 0, 0);
    }
    if (kc + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // Output layout of the 16x16 MFMA: lane holds rows 4 (lane >> 4) + v, column lane & 15.
  float sq[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      float s = 0.f;
#pragma unroll
      for (int k = 0; k < 4; ++k) s = fmaf(acc[i][k][v], acc[i][k][v], s);
      sq[i][v] = s;
    }
#pragma unroll
  for (int off = 1; off < 16; off <<= 1)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) sq[i][v] += __shfl_xor(sq[i][v], off);
  if (fr == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) red[w & 1][wr + i * 16 + (lane >> 4) * 4 + v] = sq[i][v];
  }
  __syncthreads();
  if (tid < kRowTile) a.part[(int64_t)t * a.rows + row0 + tid] = red[0][tid] + red[1][tid];
}

__device__ __forceinline__ float norm_cdf_f(float z) { return 0.5f * erfcf(-z * 0.70710678118654752f); }

__device__ __forceinline__ float ei_f32(float mu, float sigma, float fstar) {
  const float imp = fstar - mu;
  if (!(sigma > 0.f)) return fmaxf(imp, 0.f);
  const float z = imp / sigma;
  const float phi = 0.39894228040143268f * expf(-0.5f * z * z);
  return fmaxf(fmaf(imp, norm_cdf_f(z), sigma * phi), 0.f);
}

__device__ __forceinline__ double ei_f64(double mu, double sigma, double fstar) {
  const double imp = fstar - mu;
  if (!(sigma > 0.0)) return fmax(imp, 0.0);
  const double z = imp / sigma;
  const double Phi = 0.5 * erfc(-z * 0.70710678118654752440);
  const double phi = 0.39894228040143267794 * exp(-0.5 * z * z);
  return fmax(fma(imp, Phi, sigma * phi), 0.0);
}

__global__ __launch_bounds__(256) void epilogue_kernel(const EArgs a, float *pwork) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool in = j < a.M;
  bool flag = false;
  if (in) {
    float s_reg = 0.f, s_cls = 0.f;
    for (int t = 0; t < a.n_reg_tiles; ++t) s_reg += a.part[(int64_t)t * a.rows + j];
    for (int t = a.n_reg_tiles; t < a.ntiles; ++t) s_cls += a.part[(int64_t)t * a.rows + j];
    const bool ok = a.valid[j] != 0;
    float p = 1.f;
    if (a.has_cls) {
      const float V = fmaxf(a.cls_sv - s_cls, 0.f);
      p = norm_cdf_f(a.fbar[j] / sqrtf(1.f + V));
    }
    if (!ok) {
      const float nan = __builtin_nanf("");
      a.mu[j] = nan;
      a.sigma[j] = nan;
      a.ei[j] = nan;
      pwork[j] = 0.f;
      a.acq[j] = 0.f;
    } else {
      pwork[j] = p;
      const float mu = (float)a.mu64[j];
      const float var = a.sv - s_reg;
      flag = var < a.refine_var * a.sv || a.sens[j] > a.refine_sens * fmaxf(fabsf(mu), 1.f);
      if (!flag) {
        const float sigma = sqrtf(fmaxf(var, 0.f));
        const float ei = ei_f32(mu, sigma, a.fstar);
        const bool allowed = a.mask ? a.mask[j] != 0 : true;
        a.mu[j] = mu;
        a.sigma[j] = sigma;
        a.ei[j] = ei;
        a.acq[j] = (allowed && p >= a.eps_f) ? ei * p : 0.f;
      }
    }
  }
  // compact flagged candidates: one atomic per wavefront
  const uint64_t bal = __ballot(flag);
  if (bal) {
    const int lane = threadIdx.x & 63;
    const int leader = __ffsll((unsigned long long)bal) - 1;
    int base = 0;
    if (lane == leader) base = atomicAdd(a.refine_count, __popcll(bal));
    base = __shfl(base, leader);
    if (flag) a.refine_list[base + __popcll(bal & ((1ull << lane) - 1ull))] = (int32_t)j;
  }
}

// fp64 recomputation of flagged candidates: K* row, mu, |L_f^-1 k*|^2, EI, acq.
constexpr int kRefineMaxCB = 8;

__global__ __launch_bounds__(256) void refine_kernel(const RArgs a, const Weights64 w,
                                                      const float *pwork) {
  extern __shared__ double kf[];  // [cb][n_f]
  __shared__ double red[4][2 * kRefineMaxCB];
  __shared__ double fin[2 * kRefineMaxCB];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int count = *a.count;
  const int nf = a.n_f;
  for (int base = blockIdx.x * a.cb; base < count; base += gridDim.x * a.cb) {
    const int nc = min(a.cb, count - base);
    for (int idx = tid; idx < nc * nf; idx += 256) {
      const int c = idx / nf, i = idx - c * nf;
      const int64_t j = a.list[base + c];
      const uint32_t *cj = a.cand + j;
      const uint32_t *oi = a.obs + (int64_t)i * a.R;
      auto ga = [&](int q) { return cj[(int64_t)q * a.ldc]; };
      auto gb = [&](int q) { return oi[q]; };
      kf[c * nf + i] = matern52_f64(r2_f64(ga, gb, w), a.sv);
    }
    __syncthreads();
    double accs[kRefineMaxCB], accm[kRefineMaxCB];
#pragma unroll
    for (int c = 0; c < kRefineMaxCB; ++c) accs[c] = accm[c] = 0.0;
    for (int col = tid; col < nf; col += 256) {
      double v[kRefineMaxCB];
#pragma unroll
      for (int c = 0; c < kRefineMaxCB; ++c) v[c] = 0.0;
      for (int i = 0; i <= col; ++i) {
        const double b = a.B64[(int64_t)i * a.ldb + col];
#pragma unroll
        for (int c = 0; c < kRefineMaxCB; ++c)
          if (c < nc) v[c] = fma(b, kf[c * nf + i], v[c]);
      }
#pragma unroll
      for (int c = 0; c < kRefineMaxCB; ++c) accs[c] = fma(v[c], v[c], accs[c]);
    }
    for (int i = tid; i < nf; i += 256) {
      const double al = a.alpha[i];
#pragma unroll
      for (int c = 0; c < kRefineMaxCB; ++c)
        if (c < nc) accm[c] = fma(kf[c * nf + i], al, accm[c]);
    }
#pragma unroll
    for (int c = 0; c < kRefineMaxCB; ++c) {
      double s = accs[c], m = accm[c];
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        s += __shfl_xor(s, off);
        m += __shfl_xor(m, off);
      }
      if (lane == 0) {
        red[wv][c] = s;
        red[wv][kRefineMaxCB + c] = m;
      }
    }
    __syncthreads();
    if (tid < 2 * kRefineMaxCB) fin[tid] = ((red[0][tid] + red[1][tid]) + red[2][tid]) + red[3][tid];
    __syncthreads();
    if (tid < nc) {
      const int64_t j = a.list[base + tid];
      const double mu = fin[kRefineMaxCB + tid];
      const double sigma = sqrt(fmax(a.sv - fin[tid], 0.0));
      const double ei = ei_f64(mu, sigma, a.fstar);
      const float p = pwork[j];
      const bool allowed = a.mask ? a.mask[j] != 0 : true;
      a.mu[j] = (float)mu;
      a.sigma[j] = (float)sigma;
      a.ei[j] = (float)ei;
      a.acq[j] = (allowed && p >= a.eps_f) ? (float)(ei * (double)p) : 0.f;
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void argmax_partial(const float *acq, int64_t M, float *pval,
                                                       int64_t *pidx) {
  __shared__ float sv[256];
  __shared__ int64_t si[256];
  const int tid = threadIdx.x;
  float best = -1.f;
  int64_t bi = -1;
  for (int64_t j = (int64_t)blockIdx.x * 256 + tid; j < M; j += (int64_t)gridDim.x * 256) {
    const float v = acq[j];
    if (v > best) best = v, bi = j;  // strided ascending j: first max kept
  }
  sv[tid] = best;
  si[tid] = bi;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s) {
      const float v2 = sv[tid + s];
      const int64_t i2 = si[tid + s];
      if (v2 > sv[tid] || (v2 == sv[tid] && i2 >= 0 && (si[tid] < 0 || i2 < si[tid]))) {
        sv[tid] = v2;
        si[tid] = i2;
      }
    }
    __syncthreads();
  }
  if (tid == 0) {
    pval[blockIdx.x] = sv[0];
    pidx[blockIdx.x] = si[0];
  }
}

__global__ __launch_bounds__(256) void argmax_final(const float *pval, const int64_t *pidx, int nb,
                                                     int64_t *out) {
  __shared__ float sv[256];
  __shared__ int64_t si[256];
  const int tid = threadIdx.x;
  float best = -1.f;
  int64_t bi = -1;
  for (int b = tid; b < nb; b += 256) {
    const float v = pval[b];
    const int64_t i = pidx[b];
    if (v > best || (v == best && i >= 0 && (bi < 0 || i < bi))) best = v, bi = i;
  }
  sv[tid] = best;
  si[tid] = bi;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s) {
      const float v2 = sv[tid + s];
      const int64_t i2 = si[tid + s];
      if (v2 > sv[tid] || (v2 == sv[tid] && i2 >= 0 && (si[tid] < 0 || i2 < si[tid]))) {
        sv[tid] = v2;
        si[tid] = i2;
      }
    }
    __syncthreads();
  }
  if (tid == 0) out[0] = si[0] < 0 ? 0 : si[0];
}

// Per-parameter terms (Sec. 4.1) from the same code words the scorer uses.
__global__ __launch_bounds__(256) void terms_kernel(const uint32_t *cand, int64_t ldc,
                                                     const uint32_t *obs, int32_t R, int32_t n,
                                                     int64_t count, const TermDesc *td,
                                                     int32_t d, float *terms) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= count * n) return;
  const int64_t c = idx / n;
  const int i = (int)(idx - c * n);
  const uint32_t *oi = obs + (int64_t)i * R;
  for (int p = 0; p < d; ++p) {
    const TermDesc t = td[p];
    const uint32_t a0 = cand[(int64_t)t.word * ldc + c], b0 = oi[t.word];
    float v;
    if (t.kind == GP_REAL || t.kind == GP_INT || t.kind == GP_ORD) {
      v = __uint_as_float(a0) - __uint_as_float(b0);
    } else if (t.kind == GP_CAT) {
      if (t.bit >= 0) {
        const uint32_t fm = (t.m >= 32 ? 0xffffffffu : ((1u << t.m) - 1u)) << t.bit;
        v = ((a0 ^ b0) & fm) ? 1.f : 0.f;
      } else {
        v = a0 != b0 ? 1.f : 0.f;
      }
    } else if (t.dist == GP_PERM_KENDALL) {
      v = (float)__popc(a0 ^ b0);
    } else if (t.dist == GP_PERM_NAIVE) {
      v = a0 != b0 ? 1.f : 0.f;
    } else {
      const uint32_t a1 = cand[(int64_t)(t.word + 1) * ldc + c], b1 = oi[t.word + 1];
      if (t.dist == GP_PERM_HAMMING) {
        v = (float)((__popc(a0 ^ b0) + __popc(a1 ^ b1)) / 2);
      } else {
        const int s2 = (t.m - 1) * t.m * (2 * t.m - 1) / 6;
        uint32_t dt = __builtin_amdgcn_udot4(a0, b0, 0u, false);
        dt = __builtin_amdgcn_udot4(a1, b1, dt, false);
        v = (float)(2 * (s2 - (int32_t)dt));
      }
    }
    terms[((int64_t)c * n + i) * d + p] = v;
  }
}

__global__ __launch_bounds__(256) void gather_rows_f32(const float *src, int64_t ld_src, float *dst,
                                                        int64_t ld_dst, int64_t rows, int32_t cols) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * cols) return;
  const int64_t r = idx / cols;
  const int c = (int)(idx - r * cols);
  dst[r * ld_dst + c] = src[r * ld_src + c];
}

}  // namespace

hipError_t launch_contract(const CArgs &a, hipStream_t s) {
  const int64_t grid = (int64_t)a.nrowtiles * a.ntiles;
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(contract_f32, dim3((unsigned)grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_epilogue(const EArgs &a, float *pwork, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  hipLaunchKernelGGL(epilogue_kernel, dim3((unsigned)((a.M + 255) / 256)), dim3(256), 0, s, a,
                     pwork);
  return hipGetLastError();
}

int refine_candidates_per_block(int n_f) {
  int cb = (120 * 1024) / (8 * (n_f > 0 ? n_f : 1));
  return cb < 1 ? 1 : (cb > kRefineMaxCB ? kRefineMaxCB : cb);
}

hipError_t launch_refine(const RArgs &a, const Weights64 &w, const float *pwork, int grid,
                         hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  const size_t lds = (size_t)a.cb * a.n_f * sizeof(double);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&refine_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 128 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL(refine_kernel, dim3(grid), dim3(256), lds, s, a, w, pwork);
  return hipGetLastError();
}

hipError_t launch_argmax(const float *acq, int64_t M, float *pval, int64_t *pidx, int nblocks,
                         int64_t *out, hipStream_t s) {
  hipLaunchKernelGGL(argmax_partial, dim3(nblocks), dim3(256), 0, s, acq, M, pval, pidx);
  hipLaunchKernelGGL(argmax_final, dim3(1), dim3(256), 0, s, pval, pidx, nblocks, out);
  return hipGetLastError();
}

hipError_t launch_terms(const uint32_t *cand, int64_t ldc, const uint32_t *obs, int32_t R,
                        int32_t n, int64_t count, const TermDesc *td, int32_t d, float *terms,
                        hipStream_t s) {
  const int64_t tot = count * n;
  if (tot <= 0) return hipSuccess;
  hipLaunchKernelGGL(terms_kernel, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, cand,
                     ldc, obs, R, n, count, td, d, terms);
  return hipGetLastError();
}

hipError_t launch_gather_rows_f32(const float *src, int64_t ld_src, float *dst, int64_t ld_dst,
                                  int64_t rows, int32_t cols, hipStream_t s) {
  const int64_t tot = rows * cols;
  if (tot <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_rows_f32, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, src,
                     ld_src, dst, ld_dst, rows, cols);
  return hipGetLastError();
}

}  // namespace bgp
