// Posterior-variance contraction, EI / feasibility epilogue, fp64 recomputation of
// ill-conditioned candidates, arg-max and term inspection.
//
// Variance (textbook GP regression; the paper uses the GP of Sec. 3.2 without printing
// these formulas): sigma^2 = s - |L_f^-1 k*|^2. With B = L_f^-T (upper triangular) the
// squared norms are row sums of (K* B)^2. The classifier's predictive variance
// V = s_c - |L_B^-1 W^1/2 k_c*|^2 has the same shape with B = rho W^1/2 L_B^-T. Both are
// one GEMM over K* against the packed B^T, whose column tiles stop the k-loop at the
// triangle (tile [c0, c0+128) only needs k < c0+128), and whose epilogue reduces each
// 128-column tile to one partial per row; V = K* B itself is never stored. One spare
// column of a tile may instead hold a dense vector (the classifier's rho g, whose product
// with K* is its latent mean), which runs the full contraction length and is written
// out unsquared. The GEMM
// runs on fp16 MFMA with fp32 accumulation over operands split into high and low fp16
// parts (three products per multiply-add), which keeps the accuracy of an fp32 product
// at 16 times the fp32 MFMA rate.
#include "common.h"
#include "dist64.h"

namespace bgp {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef double doublex4 __attribute__((ext_vector_type(4)));

// Blocks are dispatched round-robin over the 8 XCDs (block b runs on XCD b % 8). Give
// each XCD a contiguous range of logical tiles so that the column tiles of one row
// block (which share the same K* rows) run on the same XCD and hit its L2.
__device__ __forceinline__ int xcd_remap(int b, int G) {
  const int q = G >> 3, r = G & 7;
  const int x = b & 7, k = b >> 3;
  return x * q + (x < r ? x : r) + k;
}

// LDS tile layout: row r of a 32-wide k-chunk holds 8 16-byte chunks (high parts of
// k-values 8q..8q+7 in chunk q < 4, their low parts in chunk 4 + q); chunk q is stored at
// slot q ^ ((r >> 1) & 7). Fragment reads (16 consecutive rows, one
// chunk each) then spread over all banks (no bank conflicts counted, against many for
// the plain layout) without padding rows, which keeps two workgroups per CU in the LDS.
constexpr int kLdsStride = kKChunk;
__device__ __forceinline__ int lds_off(int r, int q) {
  return r * kLdsStride + 4 * (q ^ ((r >> 1) & 7));
}

// Workgroup: a kRowTile x kColTile (128 x 128) output tile on kWR x kWC wavefronts, two
// workgroups per CU (the LDS double buffers take 64 KB each; larger tiles that leave one
// workgroup per CU measured slower, as its barriers then idle the MFMA pipes).
// Wave (wr, hc) owns 64 rows and the 16-column sub-tiles hc, hc + kWC, hc + 2 kWC, ...
// (interleaving the column waves balances the triangular work among them).
constexpr int kWR = kRowTile / 64;           // row waves (64 rows each)
constexpr int kWC = 2;                       // column waves
constexpr int kWaves = kWR * kWC;
constexpr int kCS = kColTile / 16 / kWC;     // 16-column sub-tiles per wave
constexpr int kBlk = kRowTile / 8 / kWaves;  // 8-row DMA blocks per wave and tile
static_assert(kRowTile == kColTile && kBlk * kWaves * 8 == kRowTile, "tile shape");

__global__ __launch_bounds__(64 * kWaves, 2) void contract_split(const CArgs a) {
  // two buffers of each tile as separate LDS objects, so that the compiler can tell the
  // buffer being loaded from the one being read
  __shared__ __attribute__((aligned(16))) float As0[kRowTile * kLdsStride];
  __shared__ __attribute__((aligned(16))) float As1[kRowTile * kLdsStride];
  __shared__ __attribute__((aligned(16))) float Bs0[kColTile * kLdsStride];
  __shared__ __attribute__((aligned(16))) float Bs1[kColTile * kLdsStride];
  __shared__ float red[kWC][kRowTile];

  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int rt = L / a.ntiles, t = L - rt * a.ntiles;
  const CTile tl = a.tiles[t];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t row0 = (int64_t)rt * kRowTile;
  // rows of the split operands take lda 4-byte words, chunk kc the words 32 kc..32 kc+31
  const float *Ag = reinterpret_cast<const float *>(a.A) + row0 * a.lda;
  const float *Bg = reinterpret_cast<const float *>(a.Bt) + (int64_t)tl.bcol * a.lda;
  const int nk = tl.kend / kKChunk;

  // Global -> LDS without register staging (global_load_lds_dwordx4): one instruction
  // moves 64 lanes x 16 B into 1 KB of LDS in lane order, i.e. rows 8 blk .. 8 blk + 7 of
  // the swizzled tile. Lane l fills physical slot l & 7 of row 8 blk + (l >> 3), so it
  // loads the logical 16-byte chunk (l & 7) ^ ((row >> 1) & 7) of that row. Wave w
  // fills blocks w, w + kWaves, ... of A and of B.
  uint32_t goff[kBlk];
#pragma unroll
  for (int q = 0; q < kBlk; ++q) {
    const int r = 8 * (kWaves * q + w) + (lane >> 3);
    goff[q] = (uint32_t)(r * a.lda + 4 * ((lane & 7) ^ ((r >> 1) & 7)));
  }
  auto dma = [&](float *As, float *Bs, int kc) {
    const float *pa = Ag + kc * kKChunk, *pb = Bg + kc * kKChunk;
#pragma unroll
    for (int q = 0; q < kBlk; ++q) {
      const int blk = kWaves * q + w;
      __builtin_amdgcn_global_load_lds(pa + goff[q], As + blk * 256, 16, 0, 0);
      __builtin_amdgcn_global_load_lds(pb + goff[q], Bs + blk * 256, 16, 0, 0);
    }
  };
  // all of this wave's loads have landed in LDS (vmcnt = 0; other counters untouched)
  auto dma_wait = [&]() { __builtin_amdgcn_s_waitcnt(0x0F70); };

  floatx4 acc[4][kCS];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int k = 0; k < kCS; ++k) acc[i][k] = floatx4{0.f, 0.f, 0.f, 0.f};

  // MFMA 16x16x32 (fp16): lane supplies A[row fr][k] and B[k][col fr] for
  // k = 8 (lane >> 4) .. 8 (lane >> 4) + 7, one 16-byte chunk of each row (high parts
  // in chunk lane >> 4, low parts in chunk 4 + (lane >> 4)).
  const int wr = (w / kWC) * 64, hc = __builtin_amdgcn_readfirstlane(w % kWC);
  const int fr = lane & 15, fg = lane >> 4;
  int cc[kCS], kneed[kCS];
  // Column j of a triangular factor block only has rows k <= j: sub-tile k needs
  // k < tri0 + cc[k] + 16; sub-tiles at or past ncol are padding, except the one holding
  // the linear column, which needs the whole length.
  const int lin_sub = tl.lin >= 0 ? (tl.lin & ~15) : -1;
#pragma unroll
  for (int k = 0; k < kCS; ++k) {
    cc[k] = 16 * (kWC * k + hc);
    kneed[k] = cc[k] == lin_sub ? tl.kend : (cc[k] < tl.ncol) ? tl.tri0 + cc[k] + 16 : 0;
  }

  // Per sub-tile the three partial products go round the four row blocks, so an
  // accumulator is updated again only after three other MFMAs.
  auto compute = [&](const float *As, const float *Bs, int kc) {
    __builtin_amdgcn_s_setprio(1);  // MFMA blocks before the other wave's loads
    half8 ah[4], al[4], bh[kCS], bl[kCS];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ah[i] = *(const half8 *)&As[lds_off(wr + i * 16 + fr, fg)];
      al[i] = *(const half8 *)&As[lds_off(wr + i * 16 + fr, 4 + fg)];
    }
#pragma unroll
    for (int k = 0; k < kCS; ++k) {
      bh[k] = *(const half8 *)&Bs[lds_off(cc[k] + fr, fg)];
      bl[k] = *(const half8 *)&Bs[lds_off(cc[k] + fr, 4 + fg)];
    }
    const int kabs = kc * kKChunk;
#pragma unroll
    for (int k = 0; k < kCS; ++k) {
      if (kabs < kneed[k]) {  // wave-uniform
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[i][k] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[i], bh[k], acc[i][k], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[i][k] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[i], bl[k], acc[i][k], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[i][k] = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[i], bh[k], acc[i][k], 0, 0, 0);
      }
    }
    __builtin_amdgcn_s_setprio(0);
  };

  // Chunk kc + 1 streams into the other LDS buffer while chunk kc is computed; the
  // barrier after each chunk both publishes the next buffer and frees the current one.
  // The load is unconditional (past the end it reloads the last chunk into the idle
  // buffer): loads behind branches make the compiler wait for every load in flight.
  const int klast = nk - 1;
  dma(As0, Bs0, 0);
  dma_wait();
  __syncthreads();
  for (int kc = 0; kc < nk; kc += 2) {
    dma(As1, Bs1, min(kc + 1, klast));
    compute(As0, Bs0, kc);
    dma_wait();
    __syncthreads();
    if (kc + 1 >= nk) break;
    dma(As0, Bs0, min(kc + 2, klast));
    compute(As1, Bs1, kc + 1);
    dma_wait();
    __syncthreads();
  }

  // Output layout of the 16x16 MFMA: lane holds rows 4 (lane >> 4) + v, column lane & 15,
  // which is unscaled by its cscale before squaring. The linear column is stored and
  // left out of the squares.
  float cs[kCS], keep[kCS];
#pragma unroll
  for (int k = 0; k < kCS; ++k) {
    cs[k] = a.cscale[tl.bcol + cc[k] + fr];
    keep[k] = (cc[k] + fr == tl.lin) ? 0.f : 1.f;
    if (cc[k] + fr == tl.lin) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          a.lin[row0 + wr + i * 16 + fg * 4 + v] = acc[i][k][v] * cs[k];
    }
  }
  float sq[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      float s = 0.f;
#pragma unroll
      for (int k = 0; k < kCS; ++k) {
        const float x = acc[i][k][v] * cs[k];
        s = fmaf(x * keep[k], x, s);
      }
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
      for (int v = 0; v < 4; ++v) red[hc][wr + i * 16 + (lane >> 4) * 4 + v] = sq[i][v];
  }
  __syncthreads();
  if (tid < kRowTile) {
    float v = 0.f;
#pragma unroll
    for (int c = 0; c < kWC; ++c) v += red[c][tid];
    a.part[(int64_t)t * a.rows + row0 + tid] = v;
  }
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

// The epilogue in two halves. The value model's half (mu, sigma, EI of the candidates
// that keep their fp32 values, and the list of those to recompute in fp64) needs the
// value model only, so a scoring fused with a fit runs it, and the fp64 recomputation's
// block path, beside the classifier's fit. The classifier's half (p, acq) follows the
// classifier's contraction. Both take the recomputation decision from the same inputs.
// Sum of the tile partials t0..t1-1 of row j in tile order, four tiles' loads in flight
// at a time (an absent tile adds 0, which leaves a sum of non-negative partials as is)
__device__ __forceinline__ float tile_sum(const float *part, int64_t rows, int t0, int t1,
                                          int64_t j) {
  float s = 0.f;
  for (int t = t0; t < t1; t += 4) {
    float v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = t + u < t1 ? part[(int64_t)(t + u) * rows + j] : 0.f;
#pragma unroll
    for (int u = 0; u < 4; ++u) s += v[u];
  }
  return s;
}

struct ValueRow {
  bool ok, flag;
  float mu, var;
};
__device__ __forceinline__ ValueRow value_row(const EArgs &a, int64_t j) {
  const float s_reg = tile_sum(a.part, a.rows, 0, a.n_reg_tiles, j);
  ValueRow r;
  r.ok = a.valid[j] != 0;
  double mu = 0.0;
  float sens = 0.0f;
  if (a.nsplit > 1) {  // the split partials in split order, four splits' loads in flight
    for (int q = 0; q < a.nsplit; q += 4) {
      double m4[4];
      float s4[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bool in = q + u < a.nsplit;
        m4[u] = in ? a.pmu[(int64_t)(q + u) * a.rows + j] : 0.0;
        s4[u] = in ? a.psens[(int64_t)(q + u) * a.rows + j] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (q + u < a.nsplit) {
          mu += m4[u];
          sens += s4[u];
        }
    }
  } else {
    mu = a.mu64[j];
    sens = a.sens[j];
  }
  r.mu = (float)mu;
  r.var = a.sv - s_reg;
  r.flag = r.ok && (r.var < a.refine_var * a.sv ||
                    sens > a.refine_sens * fmaxf(fabsf(r.mu), 1.f));
  return r;
}

// The value model's outputs of candidate j (NaN when invalid; left to the fp64
// recomputation when flagged), then the flagged candidates compacted, one atomic per
// wavefront. Every thread of the block calls it (the compaction uses a ballot).
__device__ __forceinline__ void epilogue_value_row(const EArgs &a, int64_t j, const ValueRow &r) {
  bool flag = false;
  if (j < a.M) {
    flag = r.flag;
    if (!r.ok) {
      const float nan = __builtin_nanf("");
      a.mu[j] = nan;
      a.sigma[j] = nan;
      a.ei[j] = nan;
    } else if (!r.flag) {
      const float fstar = a.fstar_dev ? (float)*a.fstar_dev : a.fstar;
      const float sigma = sqrtf(fmaxf(r.var, 0.f));
      a.mu[j] = r.mu;
      a.sigma[j] = sigma;
      a.ei[j] = ei_f32(r.mu, sigma, fstar);
    }
  }
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

// The feasibility probability p of candidate j < M and its acquisition value (left to the
// fp64 recomputation when flagged); reads the EI that epilogue_value_row wrote.
__device__ __forceinline__ void epilogue_cls_row(const EArgs &a, int64_t j, const ValueRow &r,
                                                 float *pwork) {
  float p = 1.f;
  if (a.has_cls) {
    const float s_cls = tile_sum(a.part, a.rows, a.n_reg_tiles, a.ntiles, j);
    const float V = fmaxf(a.cls_sv - s_cls, 0.f);
    p = norm_cdf_f(a.fbar[j] / sqrtf(1.f + V));
  }
  if (!r.ok) {
    pwork[j] = 0.f;
    a.acq[j] = 0.f;
  } else {
    pwork[j] = p;
    if (!r.flag) {
      const bool allowed = a.mask ? a.mask[j] != 0 : true;
      a.acq[j] = (allowed && p > a.eps_f) ? a.ei[j] * p : 0.f;
    }
  }
}

__global__ __launch_bounds__(256) void epilogue_value_kernel(const EArgs a) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  ValueRow r{};
  if (j < a.M) r = value_row(a, j);
  epilogue_value_row(a, j, r);
}

__global__ __launch_bounds__(256) void epilogue_cls_kernel(const EArgs a, float *pwork) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= a.M) return;
  epilogue_cls_row(a, j, value_row(a, j), pwork);
}

// Both halves in one pass, when they run on one stream.
__global__ __launch_bounds__(256) void epilogue_kernel(const EArgs a, float *pwork) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  ValueRow r{};
  if (j < a.M) r = value_row(a, j);
  epilogue_value_row(a, j, r);
  if (j < a.M) epilogue_cls_row(a, j, r, pwork);
}

// fp64 recomputation of flagged candidates: K* row, mu, |L_f^-1 k*|^2, EI, acq. A block
// takes CB flagged candidates at a time (unused slots hold zero rows), stages their fp64
// kernel rows in LDS as kf[i][CB], and gives each thread whole columns of the triangular
// product, whose k-loop is unrolled so that the B loads of 8 rows are in flight together.
constexpr int kRefineMaxCB = 8;
constexpr int kRefineLds = 120 * 1024;

// fp64 kernel row of candidate j against observation i
__device__ __forceinline__ double refine_k(const RArgs &a, const Weights64 &w, int64_t j, int i) {
  const uint32_t *cj = a.cand + j;
  const uint32_t *oi = a.obs + (int64_t)i * a.R;
  auto ga = [&](int q) { return cj[(int64_t)q * a.ldc]; };
  auto gb = [&](int q) { return oi[q]; };
  return matern52_f64(r2_f64(ga, gb, w), a.sv);
}

// outputs of one recomputed candidate from mu and |L_f^-1 k*|^2
__device__ __forceinline__ void refine_store(const RArgs &a, const float *pwork, int64_t j,
                                             double mu, double ssq) {
  const double sigma = sqrt(fmax(a.sv - ssq, 0.0));
  const double ei = ei_f64(mu, sigma, a.fstar);
  const float p = pwork[j];
  const bool allowed = a.mask ? a.mask[j] != 0 : true;
  a.mu[j] = (float)mu;
  a.sigma[j] = (float)sigma;
  a.ei[j] = (float)ei;
  a.acq[j] = (allowed && p > a.eps_f) ? (float)(ei * (double)p) : 0.f;
}

// kf[i][c] (i < n_f, c < CB) = the fp64 kernel row of flagged candidate base + c, zero
// for c >= nc; the nc n_f real values are spread over all threads (a group with few
// candidates still keeps every thread busy)
template <int CB>
__device__ __forceinline__ void refine_rows(const RArgs &a, const Weights64 &w, int base, int nc,
                                            double *kf) {
  const int nf = a.n_f;
  for (int idx = threadIdx.x; idx < nc * nf; idx += blockDim.x) {
    const int i = idx / nc, c = idx - i * nc;
    kf[i * CB + c] = refine_k(a, w, a.list[base + c], i);
  }
  if (nc < CB)
    for (int idx = threadIdx.x; idx < CB * nf; idx += blockDim.x)
      if (idx % CB >= nc) kf[idx] = 0.0;
}

template <int CB>
__global__ __launch_bounds__(256) void refine_kernel(const RArgs a, const Weights64 w,
                                                      const float *pwork) {
  extern __shared__ double kf[];  // [n_f][CB]
  __shared__ double red[4][2 * CB];
  __shared__ double fin[2 * CB];
  __shared__ double vr[4][kRefineColRange][CB];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int count = *a.count;
  const int nf = a.n_f;
  if (count > kRefineBlockMin) return;  // block path
  if (count <= kRefineSplitGroups * CB) {
    // Split path: item (group g, column range rho); v for the range's columns with the
    // rows split over the 4 wavefronts, its squared norm and (rho = 0) mu go to part and
    // mup; refine_finish sums the ranges.
    const int ngroups = (count + CB - 1) / CB, nr = (nf + kRefineColRange - 1) / kRefineColRange;
    for (int item = blockIdx.x; item < ngroups * nr; item += gridDim.x) {
      const int g = item / nr, rho = item - g * nr;
      const int base = g * CB, nc = min(CB, count - base);
      refine_rows<CB>(a, w, base, nc, kf);
      __syncthreads();
      const int col = rho * kRefineColRange + lane;
      double v[CB];
#pragma unroll
      for (int c = 0; c < CB; ++c) v[c] = 0.0;
      if (col < nf) {
        const double *bc = a.B64 + col;  // column col of the upper-triangular B: rows 0..col
        int i = wv;
        for (; i + 28 <= col; i += 32) {
          double b[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) b[u] = bc[(int64_t)(i + 4 * u) * a.ldb];
#pragma unroll
          for (int u = 0; u < 8; ++u)
#pragma unroll
            for (int c = 0; c < CB; ++c) v[c] = fma(b[u], kf[(i + 4 * u) * CB + c], v[c]);
        }
        for (; i <= col; i += 4) {
          const double b = bc[(int64_t)i * a.ldb];
#pragma unroll
          for (int c = 0; c < CB; ++c) v[c] = fma(b, kf[i * CB + c], v[c]);
        }
      }
#pragma unroll
      for (int c = 0; c < CB; ++c) vr[wv][lane][c] = v[c];
      double accm[CB];
#pragma unroll
      for (int c = 0; c < CB; ++c) accm[c] = 0.0;
      if (rho == 0) {
        for (int i = tid; i < nf; i += 256) {
          const double al = a.alpha[i];
#pragma unroll
          for (int c = 0; c < CB; ++c) accm[c] = fma(kf[i * CB + c], al, accm[c]);
        }
      }
      __syncthreads();
#pragma unroll
      for (int c = 0; c < CB; ++c) {
        double sq = 0.0;
        if (wv == 0) {
          const double t = ((vr[0][lane][c] + vr[1][lane][c]) + vr[2][lane][c]) + vr[3][lane][c];
          sq = t * t;
        }
        double m = accm[c];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
          sq += __shfl_xor(sq, off);
          m += __shfl_xor(m, off);
        }
        if (lane == 0) {
          red[wv][c] = sq;
          red[wv][CB + c] = m;
        }
      }
      __syncthreads();
      if (tid < CB) {
        a.part[((int64_t)g * nr + rho) * CB + tid] = red[0][tid];
        if (rho == 0)
          a.mup[g * CB + tid] = ((red[0][CB + tid] + red[1][CB + tid]) + red[2][CB + tid]) + red[3][CB + tid];
      }
      __syncthreads();
    }
    return;
  }
  for (int base = blockIdx.x * CB; base < count; base += gridDim.x * CB) {
    const int nc = min(CB, count - base);
    refine_rows<CB>(a, w, base, nc, kf);
    __syncthreads();
    double accs[CB], accm[CB];
#pragma unroll
    for (int c = 0; c < CB; ++c) accs[c] = accm[c] = 0.0;
    for (int col = tid; col < nf; col += 256) {
      double v[CB];
#pragma unroll
      for (int c = 0; c < CB; ++c) v[c] = 0.0;
      const double *bc = a.B64 + col;  // column col of the upper-triangular B: rows 0..col
      int i = 0;
      for (; i + 8 <= col + 1; i += 8) {
        double b[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) b[u] = bc[(int64_t)(i + u) * a.ldb];
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
          for (int c = 0; c < CB; ++c) v[c] = fma(b[u], kf[(i + u) * CB + c], v[c]);
      }
      for (; i <= col; ++i) {
        const double b = bc[(int64_t)i * a.ldb];
#pragma unroll
        for (int c = 0; c < CB; ++c) v[c] = fma(b, kf[i * CB + c], v[c]);
      }
#pragma unroll
      for (int c = 0; c < CB; ++c) accs[c] = fma(v[c], v[c], accs[c]);
    }
    for (int i = tid; i < nf; i += 256) {
      const double al = a.alpha[i];
#pragma unroll
      for (int c = 0; c < CB; ++c) accm[c] = fma(kf[i * CB + c], al, accm[c]);
    }
#pragma unroll
    for (int c = 0; c < CB; ++c) {
      double s = accs[c], m = accm[c];
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        s += __shfl_xor(s, off);
        m += __shfl_xor(m, off);
      }
      if (lane == 0) {
        red[wv][c] = s;
        red[wv][CB + c] = m;
      }
    }
    __syncthreads();
    if (tid < 2 * CB) fin[tid] = ((red[0][tid] + red[1][tid]) + red[2][tid]) + red[3][tid];
    __syncthreads();
    if (tid < nc) refine_store(a, pwork, a.list[base + tid], fin[CB + tid], fin[tid]);
    __syncthreads();
  }
}

// Split path of the refinement: sums each candidate's column-range partials in order.
__global__ __launch_bounds__(256) void refine_finish(const RArgs a, const float *pwork) {
  const int count = *a.count;
  if (count > kRefineSplitGroups * a.cb) return;
  const int nr = (a.n_f + kRefineColRange - 1) / kRefineColRange;
  const int q = threadIdx.x;
  if (q >= count) return;
  const int g = q / a.cb, c = q - g * a.cb;
  double ssq = 0.0;
  for (int rho = 0; rho < nr; ++rho) ssq += a.part[((int64_t)g * nr + rho) * a.cb + c];
  refine_store(a, pwork, a.list[q], a.mup[g * a.cb + c], ssq);
}

// Block path of the refinement, for many flagged candidates (dense batches near the
// data flag most of them): a work item is a group of 64 flagged candidates and a tile of
// 256 columns of B = L_f^-T, run by a persistent workgroup of 16 wavefronts. Per
// 16-observation chunk, eight staging wavefronts compute the 64 x 16 fp64 kernel values
// and load the 16 x 256 block of B into one LDS buffer while eight compute wavefronts
// accumulate V += K B on fp64 MFMA from the other buffer (each 16 candidates x 128
// columns; column blocks wholly left of the chunk, or wholly past n_f, are skipped, as B
// is upper triangular); one barrier per chunk swaps the buffers. Two wavefronts of each
// role share a SIMD, so that one's latency is covered by the other's work. The
// candidates' codes are staged in LDS per item, alpha and the weights once; a staging
// wavefront reads its observations' codes through the scalar cache (they are the same
// for all its lanes). The tile's squared row norms go to part64; the last tile (whose
// k-range covers all n_f observations) also forms mu = K alpha. refine_block_finish sums
// the tiles in order.
constexpr int kRbK = 16;                     // observations per chunk
constexpr int kRbBS = kRefineBlockCols + 8;  // LDS row stride of the B block (doubles)
constexpr int kRbKS = kRbK + 1;              // LDS row stride of the kernel block
constexpr int kRbRoleWaves = 8;              // compute wavefronts = staging wavefronts
constexpr int kRbWaves = 2 * kRbRoleWaves;
constexpr int kRbObs = kRbK / kRbRoleWaves;  // observations per staging lane and chunk
constexpr int kRbCols = kRefineBlockCols / 2;  // columns per compute wavefront
constexpr int kRbKsD = kRefineBlockRows * kRbKS, kRbBsD = kRbK * kRbBS;  // doubles per buffer
constexpr size_t kRbFixedBytes =
    sizeof(double) * (2 * kRbKsD + 2 * kRbBsD + 4 * kRefineBlockRows + kRefineBlockRows);
constexpr size_t kRbMaxLds = 160 * 1024 - 2048;  // dynamic LDS (the weights take the rest)
static_assert(sizeof(Weights64) <= 2048, "weights in LDS");
static_assert(kRbK % kRbRoleWaves == 0 && kRbRoleWaves == 8, "roles");

// r2_f64 of one configuration (words a(q)) against U observations (words b(u, q)), with
// the same operations in the same order for each of them; the U chains give the ALU
// independent work and share the reads of a(q) and of the weights.
template <int U, class GA, class GB>
__device__ __forceinline__ void r2xu_f64(const GA &a, const GB &b, const Weights64 &w,
                                         double (&r2)[U]) {
#pragma unroll
  for (int u = 0; u < U; ++u) r2[u] = 0.0;
  // (unrolled so that the reads of several words are in flight together)
#pragma unroll 4
  for (int q = 0; q < w.n_num; ++q) {
    const double av = (double)__uint_as_float(a(q)), wq = w.num_w[q];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const double d = av - (double)__uint_as_float(b(u, q));
      r2[u] = fma(wq * d, d, r2[u]);
    }
  }
#pragma unroll 4
  for (int q = 0; q < w.n_bits; ++q) {
    const uint32_t av = a(w.w_bits0 + q);
    const double wq = w.bits_w[q];
#pragma unroll
    for (int u = 0; u < U; ++u) r2[u] = fma(wq, (double)__popc(av ^ b(u, w.w_bits0 + q)), r2[u]);
  }
#pragma unroll 4
  for (int q = 0; q < w.n_eq; ++q) {
    const uint32_t av = a(w.w_eq0 + q);
    const double wq = w.eq_w[q];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (av != b(u, w.w_eq0 + q)) r2[u] += wq;
  }
  for (int q = 0; q < w.n_dot; ++q) {
    const uint32_t a0 = a(w.w_dot0 + 2 * q), a1 = a(w.w_dot0 + 2 * q + 1);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      uint32_t dt = __builtin_amdgcn_udot4(a0, b(u, w.w_dot0 + 2 * q), 0u, false);
      dt = __builtin_amdgcn_udot4(a1, b(u, w.w_dot0 + 2 * q + 1), dt, false);
      r2[u] = fma(w.dot_w2[q], (double)(w.dot_s2[q] - (int32_t)dt), r2[u]);
    }
  }
}

__device__ __forceinline__ void barrier_rb() {
  __asm__ volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  __asm__ volatile("" ::: "memory");
}
__device__ __forceinline__ void wait_lds_rb() { __builtin_amdgcn_s_waitcnt(0xC07F); }  // lgkmcnt(0)

__global__ __launch_bounds__(64 * kRbWaves, 1) void refine_block(const RArgs a, const Weights64 w) {
  extern __shared__ double rb_lds[];
  __shared__ Weights64 wl;  // the weights, read in the kernel values' loops, from LDS
  double *Ks = rb_lds;                          // [2][64][kRbKS]
  double *Bs = Ks + 2 * kRbKsD;                 // [2][16][kRbBS]
  double *mred = Bs + 2 * kRbBsD;               // [4][64]
  double *sqx = mred + 4 * kRefineBlockRows;    // [64] second column halves' row sums
  double *al = sqx + kRefineBlockRows;          // [n_f] alpha
  uint32_t *cw = reinterpret_cast<uint32_t *>(al + a.n_f);  // [R][64]
  const int count = *a.count;
  if (count <= kRefineBlockMin) return;
  const int nf = a.n_f, R = a.R;
  const int nct = (nf + kRefineBlockCols - 1) / kRefineBlockCols;
  const int ngroups = (count + kRefineBlockRows - 1) / kRefineBlockRows;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool stager = wv >= kRbRoleWaves;
  for (int e = tid; e < nf; e += 64 * kRbWaves) al[e] = a.alpha[e];
  for (int e = tid; e < (int)(sizeof(Weights64) / 4); e += 64 * kRbWaves)
    reinterpret_cast<uint32_t *>(&wl)[e] = reinterpret_cast<const uint32_t *>(&w)[e];

  for (int item = blockIdx.x; item < ngroups * nct; item += gridDim.x) {
    const int g = item / nct, ct = item - g * nct;
    const int base = g * kRefineBlockRows, nc = min(kRefineBlockRows, count - base);
    const int c0 = ct * kRefineBlockCols;
    const int kend = min(c0 + kRefineBlockCols, nf);  // columns < kend need rows k < kend
    const bool with_mu = ct == nct - 1;                // kend == nf
    const int nchunks = (kend + kRbK - 1) / kRbK;
    __syncthreads();  // the previous item's buffers and codes are no longer read
    for (int e = tid; e < R * kRefineBlockRows; e += 64 * kRbWaves) {
      const int q = e / kRefineBlockRows, c = e - q * kRefineBlockRows;
      cw[e] = c < nc ? a.cand[(int64_t)q * a.ldc + a.list[base + c]] : 0u;
    }
    __syncthreads();

    // The two roles run loops of their own with the same barriers, so that the compute
    // wavefronts' accumulators are not live in the staging code. The barriers carry no
    // memory fence (a fence would wait for the B loads in flight); each side waits for
    // its own LDS accesses before them.
    if (stager) {
      // Staging wavefront sw: kernel values of candidate `lane` against observations
      // k0 + kRbObs sw .. (the same for all lanes), and 8 rows of one column of the
      // chunk's B (thread t: column t & 255, rows 8 (t >> 8) ..), whose loads for the next
      // chunk are issued while this chunk is staged (rows past kend and columns past n_f
      // read a clamped address; zeros are stored for them).
      const int sw = wv - kRbRoleWaves, t = tid - 64 * kRbRoleWaves;
      const int bc = t & (kRefineBlockCols - 1), br = 8 * (t >> 8);
      auto load_b = [&](double(&bv)[8], int k) {
        const int jc = min(c0 + bc, nf - 1);
#pragma unroll
        for (int i = 0; i < 8; ++i)
          bv[i] = a.B64[(int64_t)min(k * kRbK + br + i, kend - 1) * a.ldb + jc];
      };
      auto stage = [&](const double(&bv)[8], int k, int buf) {
        const int k0 = k * kRbK, i0 = k0 + kRbObs * sw;
        double *kb = Ks + buf * kRbKsD, *bb = Bs + buf * kRbBsD;
        // observation rows, read as constant memory (never written by this kernel)
        typedef __attribute__((address_space(4))) const uint32_t cu32;
        const cu32 *orow[kRbObs];
#pragma unroll
        for (int u = 0; u < kRbObs; ++u)
          orow[u] = (const cu32 *)(a.obs + (int64_t)min(i0 + u, kend - 1) * R);
        double r2[kRbObs];
        r2xu_f64<kRbObs>([&](int q) { return cw[q * kRefineBlockRows + lane]; },
                         [&](int u, int q) { return orow[u][q]; }, wl, r2);
#pragma unroll
        for (int u = 0; u < kRbObs; ++u)
          kb[lane * kRbKS + kRbObs * sw + u] =
              (lane < nc && i0 + u < kend) ? matern52_f64(r2[u], a.sv) : 0.0;
#pragma unroll
        for (int i = 0; i < 8; ++i)
          bb[(br + i) * kRbBS + bc] = (k0 + br + i < kend && c0 + bc < nf) ? bv[i] : 0.0;
      };
      double bv[8];
      load_b(bv, 0);
      stage(bv, 0, 0);
      load_b(bv, 1);
      wait_lds_rb();
      barrier_rb();
      for (int k = 0; k < nchunks; ++k) {
        if (k + 1 < nchunks) {
          stage(bv, k + 1, (k & 1) ^ 1);
          load_b(bv, k + 2);
        }
        wait_lds_rb();
        barrier_rb();
      }
      barrier_rb();  // the compute wavefronts' column halves
    } else {
      // compute wavefront: candidates 16 (wv & 3) .., columns c0 + kRbCols (wv >> 2) ..
      const int rb = wv & 3, ch = wv >> 2;
      const int cb0 = c0 + kRbCols * ch;
      doublex4 acc[kRbCols / 16];
#pragma unroll
      for (int b = 0; b < kRbCols / 16; ++b) acc[b] = doublex4{0.0, 0.0, 0.0, 0.0};
      double mu = 0.0;
      barrier_rb();
      for (int k = 0; k < nchunks; ++k) {
        const int k0 = k * kRbK;
        const double *kb = Ks + (k & 1) * kRbKsD, *bb = Bs + (k & 1) * kRbBsD;
        if (with_mu && ch == 0) {  // thread: candidate lane, observations k0 + 4 rb ..
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int kk = 4 * rb + u;
            if (k0 + kk < nf) mu = fma(kb[lane * kRbKS + kk], al[k0 + kk], mu);
          }
        }
        // V[16 rb + r][c] += sum_kk K[16 rb + r][kk] B[kk][c]: lane supplies K[row l & 15]
        // [kk l >> 4] and B[kk l >> 4][col l & 15] per 4-deep step
#pragma unroll
        for (int b = 0; b < kRbCols / 16; ++b) {
          // wave-uniform: the block has columns >= k0 and columns < kend
          if (cb0 + 16 * b + 15 >= k0 && cb0 + 16 * b < kend) {
#pragma unroll
            for (int ks = 0; ks < kRbK; ks += 4) {
              const double av = kb[(16 * rb + (lane & 15)) * kRbKS + ks + (lane >> 4)];
              const double bv = bb[(ks + (lane >> 4)) * kRbBS + kRbCols * ch + 16 * b + (lane & 15)];
              acc[b] = __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv, acc[b], 0, 0, 0);
            }
          }
        }
        wait_lds_rb();
        barrier_rb();
      }
      // squared row norms of the half tile: lane holds rows (l >> 4) + 4 v of its 16,
      // column l & 15; the second half's go through LDS to the first
      double sq[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        double t = 0.0;
#pragma unroll
        for (int b = 0; b < kRbCols / 16; ++b) t = fma(acc[b][v], acc[b][v], t);
        sq[v] = t;
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1)
#pragma unroll
        for (int v = 0; v < 4; ++v) sq[v] += __shfl_xor(sq[v], off);
      if (ch == 1 && (lane & 15) == 0)
#pragma unroll
        for (int v = 0; v < 4; ++v) sqx[16 * rb + (lane >> 4) + 4 * v] = sq[v];
      if (with_mu && ch == 0) mred[rb * kRefineBlockRows + lane] = mu;
      wait_lds_rb();
      barrier_rb();
      if (ch == 0 && (lane & 15) == 0) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int r = 16 * rb + (lane >> 4) + 4 * v;
          if (r < nc) a.part64[(int64_t)ct * a.cap + base + r] = sq[v] + sqx[r];
        }
      }
    }
    if (with_mu) {
      __syncthreads();
      if (tid < nc)
        a.mu64[base + tid] = ((mred[tid] + mred[kRefineBlockRows + tid]) +
                              mred[2 * kRefineBlockRows + tid]) + mred[3 * kRefineBlockRows + tid];
    }
  }
}

__global__ __launch_bounds__(256) void refine_block_finish(const RArgs a, const float *pwork) {
  const int count = *a.count;
  if (count <= kRefineBlockMin) return;
  const int nct = (a.n_f + kRefineBlockCols - 1) / kRefineBlockCols;
  for (int q = blockIdx.x * 256 + threadIdx.x; q < count; q += gridDim.x * 256) {
    double ssq = 0.0;
    for (int ct = 0; ct < nct; ++ct) ssq += a.part64[(int64_t)ct * a.cap + q];
    refine_store(a, pwork, a.list[q], a.mu64[q], ssq);
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

__global__ __launch_bounds__(256) void gather_rows_split(const _Float16 *src, int32_t lda,
                                                          float inv_scale, float *dst,
                                                          int64_t ld_dst, int64_t rows,
                                                          int32_t cols) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * cols) return;
  const int64_t r = idx / cols;
  const int c = (int)(idx - r * cols);
  const _Float16 *row = src + r * 2 * lda + (c >> 5) * 64 + kpos(c & 31);
  dst[r * ld_dst + c] = ((float)row[0] + (float)row[32]) * inv_scale;  // h + l is exact in fp32
}

}  // namespace

hipError_t launch_contract(const CArgs &a, hipStream_t s) {
  const int64_t grid = (int64_t)a.nrowtiles * a.ntiles;
  if (grid <= 0) return hipSuccess;
  for (int t = 0; t < a.ntiles; ++t) {
    const CTile &tl = a.tiles[t];
    if (tl.kend <= 0 || tl.kend % kKChunk || tl.kend > a.lda) return hipErrorInvalidValue;
    // a linear column lies in a sub-tile of its own, past the triangular columns
    if (tl.lin >= 0 && (!a.lin || tl.lin >= kColTile || (tl.lin & ~15) < tl.ncol))
      return hipErrorInvalidValue;
  }
  hipLaunchKernelGGL(contract_split, dim3((unsigned)grid), dim3(64 * kWaves), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_epilogue_value(const EArgs &a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  hipLaunchKernelGGL(epilogue_value_kernel, dim3((unsigned)((a.M + 255) / 256)), dim3(256), 0, s,
                     a);
  return hipGetLastError();
}

hipError_t launch_epilogue(const EArgs &a, float *pwork, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  hipLaunchKernelGGL(epilogue_kernel, dim3((unsigned)((a.M + 255) / 256)), dim3(256), 0, s, a,
                     pwork);
  return hipGetLastError();
}

hipError_t launch_epilogue_cls(const EArgs &a, float *pwork, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  hipLaunchKernelGGL(epilogue_cls_kernel, dim3((unsigned)((a.M + 255) / 256)), dim3(256), 0, s, a,
                     pwork);
  return hipGetLastError();
}

int refine_candidates_per_block(int n_f) {
  const int nf = n_f > 0 ? n_f : 1;
  for (int cb = kRefineMaxCB; cb > 1; cb >>= 1)
    if ((size_t)cb * nf * sizeof(double) <= (size_t)kRefineLds) return cb;
  return 1;
}

template <int CB>
hipError_t launch_refine_cb(const RArgs &a, const Weights64 &w, const float *pwork, int grid,
                            hipStream_t s) {
  static bool attr_set = false;  // per instantiation
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&refine_kernel<CB>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kRefineLds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const size_t lds = (size_t)CB * a.n_f * sizeof(double);
  hipLaunchKernelGGL(refine_kernel<CB>, dim3(grid), dim3(256), lds, s, a, w, pwork);
  return hipGetLastError();
}

hipError_t launch_refine_block(const RArgs &a, const Weights64 &w, int cus, hipStream_t s) {
  // (its kernel returns at once unless more than kRefineBlockMin are flagged)
  if (a.cap <= kRefineBlockMin) return hipSuccess;
  if (!a.part64 || !a.mu64 || cus < 1) return hipErrorInvalidValue;
  const int nct = (a.n_f + kRefineBlockCols - 1) / kRefineBlockCols;
  const int64_t items = (a.cap + kRefineBlockRows - 1) / kRefineBlockRows * nct;
  const size_t lds = kRbFixedBytes + sizeof(uint32_t) * (size_t)a.R * kRefineBlockRows +
                     sizeof(double) * a.n_f;
  if (lds > kRbMaxLds) return hipErrorInvalidValue;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&refine_block),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)kRbMaxLds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  // persistent: one workgroup per compute unit the stream can use
  hipLaunchKernelGGL(refine_block, dim3((unsigned)std::min<int64_t>(items, cus)),
                     dim3(64 * kRbWaves), lds, s, a, w);
  return hipGetLastError();
}

hipError_t launch_refine_rest(const RArgs &a, const Weights64 &w, const float *pwork, int grid,
                              hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  if ((size_t)a.cb * a.n_f * sizeof(double) > (size_t)kRefineLds) return hipErrorInvalidValue;
  static_assert(kRefineSplitGroups * kRefineMaxCB <= 256, "one finishing workgroup");
  hipError_t e;
  switch (a.cb) {
    case 8: e = launch_refine_cb<8>(a, w, pwork, grid, s); break;
    case 4: e = launch_refine_cb<4>(a, w, pwork, grid, s); break;
    case 2: e = launch_refine_cb<2>(a, w, pwork, grid, s); break;
    case 1: e = launch_refine_cb<1>(a, w, pwork, grid, s); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(refine_finish, dim3(1), dim3(256), 0, s, a, pwork);
  if (a.cap > kRefineBlockMin) {
    if (!a.part64 || !a.mu64) return hipErrorInvalidValue;
    hipLaunchKernelGGL(refine_block_finish, dim3((unsigned)std::min<int64_t>((a.cap + 255) / 256, 1024)),
                       dim3(256), 0, s, a, pwork);
  }
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

hipError_t launch_gather_rows_split(const uint16_t *src, int32_t lda, float inv_scale, float *dst,
                                    int64_t ld_dst, int64_t rows, int32_t cols, hipStream_t s) {
  const int64_t tot = rows * cols;
  if (tot <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_rows_split, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s,
                     reinterpret_cast<const _Float16 *>(src), lda, inv_scale, dst, ld_dst, rows,
                     cols);
  return hipGetLastError();
}

}  // namespace bgp
