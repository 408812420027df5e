// Random-forest feasibility model (Sec. 4.2, hidden constraints): a classification
// forest fitted to the feasible / infeasible labels of the observations predicts the
// probability of feasibility that multiplies the expected improvement.
//
// Trees are CART trees with Gini impurity grown on bootstrap samples with a random
// feature subset per node; all random choices come from Philox4x64-10 streams (key
// (seed, 0), counter (tree, stream, block, 3); stream 0 the bootstrap, stream k + 1
// the feature subset of node k), so the trees are a deterministic function of the
// inputs. Split qualities Q = pos_L neg_L / c_L + pos_R neg_R / c_R (the Gini impurity
// of the children weighted by their sizes, halved) are compared exactly as fractions
// of 64-bit integers: the smallest Q wins, then the smallest feature, then the
// smallest threshold; a split is taken only if Q is below the node's own
// pos neg / c. A threshold is the largest value sent left.
//
// Training: one workgroup per tree, nodes in breadth-first order; per node and tried
// feature the node's (value, label) pairs are sorted in LDS (bitonic), labels
// prefix-summed, every boundary between distinct values scored in parallel and the
// best one reduced; the node's sample range is then partitioned in place (stable).
// Prediction: one wavefront per 64 configurations, their features column-major in
// LDS, the trees walked in order with one 16-byte node load per level.
#include "common.h"

namespace bgp {
namespace {

constexpr int kSortCap = kMaxN;  // node samples sorted at once (n <= kMaxN)

__device__ __forceinline__ void philox4x64(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                           uint64_t k0, uint64_t k1, uint64_t out[4]) {
  constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += W0;
      k1 += W1;
    }
    const uint64_t hi0 = __umul64hi(M0, c0), lo0 = M0 * c0;
    const uint64_t hi1 = __umul64hi(M1, c2), lo1 = M1 * c2;
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
}

// word q of stream (t, s)
__device__ __forceinline__ uint64_t stream_word(uint64_t seed, int t, int s, int q) {
  uint64_t w[4];
  philox4x64((uint64_t)t, (uint64_t)s, (uint64_t)(q >> 2), 3, seed, 0, w);
  const int r = q & 3;
  return r == 0 ? w[0] : (r == 1 ? w[1] : (r == 2 ? w[2] : w[3]));
}

template <typename T>
__device__ __forceinline__ void stage(T &dst, const T &src) {
  static_assert(sizeof(T) % 4 == 0, "word copy");
  const uint32_t *s = reinterpret_cast<const uint32_t *>(&src);
  uint32_t *d = reinterpret_cast<uint32_t *>(&dst);
  for (int q = threadIdx.x; q < (int)(sizeof(T) / 4); q += blockDim.x) d[q] = s[q];
}

// a/b < c/d for nonnegative fractions with a, c < 2^40 and b, d < 2^24
__device__ __forceinline__ bool frac_less(uint64_t a, uint64_t b, uint64_t c, uint64_t d) {
  return a * d < c * b;
}

__device__ __forceinline__ double feature_of(const ForestDesc &D, const CotCols &cols, int p, int q,
                                             int64_t j) {
  const int kind = D.kind[p];
  if (kind == GP_REAL) return static_cast<const double *>(cols.col[p])[j];
  if (kind == GP_PERM) return (double)static_cast<const int32_t *>(cols.col[p])[j * D.m[p] + q];
  return (double)static_cast<const int32_t *>(cols.col[p])[j];
}

__global__ __launch_bounds__(256) void forest_features_k(const ForestDesc *dd, const CotCols cols0,
                                                          int64_t count, int64_t ld, double *X) {
  __shared__ ForestDesc D;
  __shared__ CotCols cols;
  stage(D, *dd);
  stage(cols, cols0);
  __syncthreads();
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= count) return;
  for (int p = 0; p < D.d; ++p)
    for (int q = 0; q < D.m[p]; ++q) X[(int64_t)(D.fofs[p] + q) * ld + j] = feature_of(D, cols, p, q, j);
}

__device__ __forceinline__ int block_sum_int(int v, int *red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const int r = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return r;
}

// Inclusive scan of a[0..P) in place (P <= kSortCap; thread t owns a contiguous chunk).
__device__ void block_scan_int(int *a, int P, int *tsum) {
  const int tid = threadIdx.x, per = (P + 255) / 256, b0 = tid * per, b1 = min(P, b0 + per);
  int run = 0;
  for (int i = b0; i < b1; ++i) {
    run += a[i];
    a[i] = run;
  }
  tsum[tid] = run;
  __syncthreads();
  for (int o = 1; o < 256; o <<= 1) {  // Hillis-Steele over the 256 chunk totals
    const int v = tid >= o ? tsum[tid - o] : 0;
    __syncthreads();
    tsum[tid] += v;
    __syncthreads();
  }
  const int off = tid > 0 ? tsum[tid - 1] : 0;
  for (int i = b0; i < b1; ++i) a[i] += off;
  __syncthreads();
}

__global__ __launch_bounds__(256) void forest_train_k(const ForestDesc *dd, const double *X,
                                                       const uint8_t *y, int32_t *idx_all,
                                                       int32_t *tmp_all, ForestNode *nodes_all,
                                                       int32_t *aux_all, int32_t *n_nodes_out) {
  __shared__ ForestDesc D;
  __shared__ double skey[kSortCap];
  __shared__ int slab[kSortCap];
  __shared__ int sscan[kSortCap];
  __shared__ int tsum[256];
  __shared__ uint64_t bnum[256], bden[256];
  __shared__ int bidx[256];
  __shared__ int perm[kForestMaxF];
  __shared__ int subset[kForestMaxMtry];
  __shared__ int red[4];
  __shared__ int s_nn, s_start, s_end, s_depth;
  __shared__ int s_have, s_f, s_split;
  __shared__ uint64_t s_num, s_den;
  __shared__ double s_thr;
  stage(D, *dd);
  __syncthreads();
  const int t = blockIdx.x, tid = threadIdx.x, n = D.n, F = D.F;
  int32_t *idx = idx_all + (int64_t)t * n, *tmp = tmp_all + (int64_t)t * n;
  ForestNode *nodes = nodes_all + (int64_t)t * D.cap;
  int32_t *aux = aux_all + (int64_t)t * D.cap * 3;
  // bootstrap sample: index i from word i of stream (t, 0)
  for (int i = tid; i < n; i += 256)
    idx[i] = (int32_t)__umul64hi(stream_word(D.seed, t, 0, i), (uint64_t)n);
  if (tid == 0) {
    aux[0] = 0;
    aux[1] = n;
    aux[2] = 0;
    s_nn = 1;
  }
  __syncthreads();
  for (int k = 0; k < s_nn; ++k) {
    if (tid == 0) {
      s_start = aux[3 * k];
      s_end = aux[3 * k + 1];
      s_depth = aux[3 * k + 2];
    }
    __syncthreads();
    const int start = s_start, c = s_end - s_start, depth = s_depth;
    int lp = 0;
    for (int i = tid; i < c; i += 256) lp += y[idx[start + i]] != 0;
    const int pos = block_sum_int(lp, red);
    if (tid == 0) {
      nodes[k].feature = -1;
      nodes[k].left = -1;
      nodes[k].val = (double)pos / (double)c;
    }
    const bool leaf = pos == 0 || pos == c || c < D.min_split || depth >= D.max_depth;
    if (leaf) {
      __syncthreads();
      continue;
    }
    // features tried at this node: partial Fisher-Yates over 0..F-1, then ascending
    for (int f = tid; f < F; f += 256) perm[f] = f;
    __syncthreads();
    if (tid == 0) {
      for (int q = 0; q < D.mtry; ++q) {
        const int r = q + (int)__umul64hi(stream_word(D.seed, t, k + 1, q), (uint64_t)(F - q));
        const int a = perm[q];
        perm[q] = perm[r];
        perm[r] = a;
      }
      for (int q = 0; q < D.mtry; ++q) subset[q] = perm[q];
      for (int q = 1; q < D.mtry; ++q)
        for (int z = q; z > 0 && subset[z - 1] > subset[z]; --z) {
          const int a = subset[z];
          subset[z] = subset[z - 1];
          subset[z - 1] = a;
        }
      s_have = 0;
    }
    __syncthreads();
    int P = 1;
    while (P < c) P <<= 1;
    for (int sq = 0; sq < D.mtry; ++sq) {
      const int f = subset[sq];
      const double *xf = X + (int64_t)f * n;
      for (int i = tid; i < P; i += 256) {
        if (i < c) {
          const int o = idx[start + i];
          skey[i] = xf[o];
          slab[i] = y[o] != 0;
        } else {
          skey[i] = INFINITY;
          slab[i] = 0;
        }
      }
      __syncthreads();
      for (int size = 2; size <= P; size <<= 1)  // bitonic sort by value, ascending
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
          for (int i = tid; i < P / 2; i += 256) {
            const int lo = 2 * i - (i & (stride - 1)), hi = lo + stride;
            const bool asc = (lo & size) == 0;
            const double a = skey[lo], b = skey[hi];
            if ((a > b) == asc && a != b) {
              skey[lo] = b;
              skey[hi] = a;
              const int la = slab[lo];
              slab[lo] = slab[hi];
              slab[hi] = la;
            }
          }
          __syncthreads();
        }
      for (int i = tid; i < P; i += 256) sscan[i] = slab[i];
      __syncthreads();
      block_scan_int(sscan, P, tsum);
      // best boundary of this feature: thread-local, then reduced (ties: lower index)
      uint64_t bn = 0, bd = 0;
      int bi = -1;
      for (int i = tid; i < c - 1; i += 256) {
        if (!(skey[i] < skey[i + 1])) continue;
        const uint64_t cl = i + 1, cr = c - cl, pl = sscan[i], pr = pos - pl;
        const uint64_t num = pl * (cl - pl) * cr + pr * (cr - pr) * cl, den = cl * cr;
        if (bi < 0 || frac_less(num, den, bn, bd)) bn = num, bd = den, bi = i;
      }
      bnum[tid] = bn;
      bden[tid] = bd;
      bidx[tid] = bi;
      __syncthreads();
      for (int st = 128; st > 0; st >>= 1) {
        if (tid < st) {
          const int j2 = tid + st;
          const bool take = bidx[j2] >= 0 &&
                            (bidx[tid] < 0 || frac_less(bnum[j2], bden[j2], bnum[tid], bden[tid]) ||
                             (!frac_less(bnum[tid], bden[tid], bnum[j2], bden[j2]) &&
                              bidx[j2] < bidx[tid]));
          if (take) {
            bnum[tid] = bnum[j2];
            bden[tid] = bden[j2];
            bidx[tid] = bidx[j2];
          }
        }
        __syncthreads();
      }
      if (tid == 0 && bidx[0] >= 0 &&
          (!s_have || frac_less(bnum[0], bden[0], s_num, s_den))) {  // ties: earlier feature
        s_have = 1;
        s_num = bnum[0];
        s_den = bden[0];
        s_f = f;
        s_thr = skey[bidx[0]];
      }
      __syncthreads();
    }
    if (tid == 0)
      s_split = s_have && frac_less(s_num, s_den, (uint64_t)pos * (uint64_t)(c - pos), (uint64_t)c);
    __syncthreads();
    if (!s_split) continue;
    // stable partition of the node's samples: x_f <= thr first
    const int f = s_f;
    const double thr = s_thr, *xf = X + (int64_t)f * n;
    for (int i = tid; i < P; i += 256) sscan[i] = (i < c && xf[idx[start + i]] <= thr) ? 1 : 0;
    __syncthreads();
    block_scan_int(sscan, P, tsum);
    const int nl = sscan[c - 1];
    for (int i = tid; i < c; i += 256) {
      const int incl = sscan[i], isl = (i == 0 ? incl : incl - sscan[i - 1]);
      const int dst = isl ? incl - 1 : nl + (i - incl);
      tmp[start + dst] = idx[start + i];
    }
    __syncthreads();
    for (int i = tid; i < c; i += 256) idx[start + i] = tmp[start + i];
    if (tid == 0) {
      const int l = s_nn;
      nodes[k].feature = f;
      nodes[k].left = l;
      nodes[k].val = thr;
      aux[3 * l] = start;
      aux[3 * l + 1] = start + nl;
      aux[3 * l + 2] = depth + 1;
      aux[3 * (l + 1)] = start + nl;
      aux[3 * (l + 1) + 1] = start + c;
      aux[3 * (l + 1) + 2] = depth + 1;
      s_nn = l + 2;
    }
    __syncthreads();
  }
  if (tid == 0) n_nodes_out[t] = s_nn;
}

__global__ __launch_bounds__(64) void forest_predict_k(const ForestDesc *dd, const ForestNode *nodes,
                                                        const CotCols cols0, int64_t M,
                                                        const float *ei, const uint8_t *mask,
                                                        float eps_f, float *p_out, float *acq) {
  extern __shared__ double feat[];  // [F][64]
  __shared__ ForestDesc D;
  __shared__ CotCols cols;
  stage(D, *dd);
  stage(cols, cols0);
  __syncthreads();
  const int lane = threadIdx.x;
  const int64_t j = (int64_t)blockIdx.x * 64 + lane;
  if (j >= M) return;
  for (int p = 0; p < D.d; ++p)
    for (int q = 0; q < D.m[p]; ++q) feat[(D.fofs[p] + q) * 64 + lane] = feature_of(D, cols, p, q, j);
  double acc = 0.0;
  for (int t = 0; t < D.n_trees; ++t) {
    const ForestNode *nt = nodes + (int64_t)t * D.cap;
    int k = 0;
    ForestNode nd = nt[0];
    while (nd.feature >= 0) {
      k = nd.left + (feat[nd.feature * 64 + lane] <= nd.val ? 0 : 1);
      nd = nt[k];
    }
    acc += nd.val;
  }
  const float pf = (float)(acc / (double)D.n_trees);
  p_out[j] = pf;
  if (acq) {
    const bool allowed = !mask || mask[j];
    acq[j] = (allowed && pf > eps_f) ? ei[j] * pf : 0.0f;
  }
}

}  // namespace

hipError_t launch_forest_features(const ForestDesc *dd, const CotCols &cols, int64_t count,
                                  int64_t ld, double *X, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(forest_features_k, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, dd,
                     cols, count, ld, X);
  return hipGetLastError();
}

hipError_t launch_forest_train(const ForestDesc *dd, int n_trees, const double *X,
                               const uint8_t *y, int32_t *idx, int32_t *tmp, ForestNode *nodes,
                               int32_t *aux, int32_t *n_nodes, hipStream_t s) {
  if (n_trees <= 0) return hipSuccess;
  hipLaunchKernelGGL(forest_train_k, dim3((unsigned)n_trees), dim3(256), 0, s, dd, X, y, idx, tmp,
                     nodes, aux, n_nodes);
  return hipGetLastError();
}

hipError_t launch_forest_predict(const ForestDesc *dd, const ForestDesc &hd, const ForestNode *nodes,
                                 const CotCols &cols, int64_t M, const float *ei,
                                 const uint8_t *mask, float eps_f, float *p, float *acq,
                                 hipStream_t s) {
  if (M <= 0) return hipSuccess;
  const size_t lds = sizeof(double) * 64 * (size_t)hd.F;
  hipLaunchKernelGGL(forest_predict_k, dim3((unsigned)((M + 63) / 64)), dim3(64), lds, s, dd, nodes,
                     cols, M, ei, mask, eps_f, p, acq);
  return hipGetLastError();
}

}  // namespace bgp
