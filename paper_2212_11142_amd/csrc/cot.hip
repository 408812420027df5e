// Chain-of-Trees (Sec. 4.2, known constraints): the feasible partial configurations of
// every group of co-dependent parameters are the leaves of its tree; a configuration is
// drawn uniformly over each tree's leaves (free parameters uniformly over their
// domains), and membership in the chain replaces the evaluation of the constraints.
//
// A tree's leaves are kept as sorted 64-bit keys packing their value indices into bit
// fields (first level most significant), so a draw is one multiply-high, one key load
// and shifts, and a membership test is a binary search. Random words come from Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011),
// key (seed, 0), counter (offset + j, b, 0, 0) for the b-th block of four words of
// configuration j; words are used in order: one per tree, then per free parameter in
// space order one word (REAL, INT, ORD, CAT) or m - 1 words (PERM).
#include "common.h"

namespace bgp {
namespace {

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

// Sequential reader of configuration j's random words.
struct WordStream {
  uint64_t ctr, seed, blk = 0;
  uint64_t buf[4];
  int pos = 4;
  __device__ uint64_t next() {
    if (pos == 4) {
      philox4x64(ctr, blk, 0, 0, seed, 0, buf);
      ++blk;
      pos = 0;
    }
    const int q = pos++;  // registers only: select instead of indexing
    return q == 0 ? buf[0] : (q == 1 ? buf[1] : (q == 2 ? buf[2] : buf[3]));
  }
};

__device__ __forceinline__ uint64_t uniform_index(uint64_t u, uint64_t c) {
  return __umul64hi(u, c);
}

template <typename T>
__device__ __forceinline__ void stage(T &dst, const T &src) {
  static_assert(sizeof(T) % 4 == 0, "word copy");
  const uint32_t *s = reinterpret_cast<const uint32_t *>(&src);
  uint32_t *d = reinterpret_cast<uint32_t *>(&dst);
  for (int q = threadIdx.x; q < (int)(sizeof(T) / 4); q += blockDim.x) d[q] = s[q];
}

__global__ __launch_bounds__(256) void cot_keys_k(const CotDesc *dd, int tree,
                                                   const int32_t *leaves, int64_t n,
                                                   uint64_t *keys, unsigned long long *bad) {
  __shared__ CotDesc D;
  stage(D, *dd);
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int k = D.tcount[tree], t0 = D.tstart[tree];
  bool ok = true;
  uint64_t key = 0, prev = 0;
  for (int l = 0; l < k; ++l) {
    const int p = D.tparam[t0 + l];
    const int32_t v = leaves[i * k + l];
    ok = ok && v >= 0 && v < D.dim[p];
    key |= (uint64_t)((uint32_t)v & D.fmask[p]) << D.shift[p];
    if (i > 0) prev |= (uint64_t)((uint32_t)leaves[(i - 1) * k + l] & D.fmask[p]) << D.shift[p];
  }
  ok = ok && (i == 0 || key > prev);
  keys[i] = key;
  if (!ok) atomicMin(bad, (unsigned long long)i);
}

__global__ __launch_bounds__(256) void cot_sample_k(const CotDesc *dd, const uint64_t *keys,
                                                     int64_t M, uint64_t seed, uint64_t offset,
                                                     const CotCols out0) {
  __shared__ CotDesc D;
  __shared__ CotCols out;
  stage(D, *dd);
  stage(out, out0);
  __syncthreads();
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= M) return;
  WordStream ws;
  ws.ctr = offset + (uint64_t)j;
  ws.seed = seed;
  for (int t = 0; t < D.n_trees; ++t) {
    const uint64_t leaf = uniform_index(ws.next(), (uint64_t)D.nleaves[t]);
    const uint64_t key = keys[D.koff[t] + (int64_t)leaf];
    for (int l = 0; l < D.tcount[t]; ++l) {
      const int p = D.tparam[D.tstart[t] + l];
      const int32_t idx = (int32_t)((key >> D.shift[p]) & D.fmask[p]);
      static_cast<int32_t *>(out.col[p])[j] = D.lo[p] + idx;
    }
  }
  for (int p = 0; p < D.d; ++p) {
    if (D.tree[p] >= 0) continue;
    const int kind = D.kind[p];
    if (kind == GP_REAL) {
#pragma clang fp contract(off)  // lo + (hi - lo) x: a rounded product, then a rounded sum
      const double x = (double)(ws.next() >> 11) * 0x1p-53;
      const double span = D.rhi[p] - D.rlo[p];
      const double t = span * x;
      static_cast<double *>(out.col[p])[j] = D.rlo[p] + t;
    } else if (kind == GP_PERM) {
      const int m = D.dim[p];
      int32_t pi[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) pi[q] = q;
      for (int i = m - 1; i >= 1; --i) {
        const int r = (int)uniform_index(ws.next(), (uint64_t)(i + 1));
        int32_t a = 0, b = 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) {  // registers only: select instead of indexing
          a = q == i ? pi[q] : a;
          b = q == r ? pi[q] : b;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) pi[q] = q == i ? b : (q == r ? a : pi[q]);
      }
      int32_t *dst = static_cast<int32_t *>(out.col[p]) + j * m;
      for (int q = 0; q < m; ++q) {
        int32_t v = 0;
#pragma unroll
        for (int z = 0; z < 8; ++z) v = z == q ? pi[z] : v;
        dst[q] = v;
      }
    } else {
      const int32_t idx = (int32_t)uniform_index(ws.next(), (uint64_t)D.dim[p]);
      static_cast<int32_t *>(out.col[p])[j] = D.lo[p] + idx;
    }
  }
}

__global__ __launch_bounds__(256) void cot_member_k(const CotDesc *dd, const uint64_t *keys,
                                                     const CotCols cols0, int64_t M,
                                                     uint8_t *mask) {
  __shared__ CotDesc D;
  __shared__ CotCols cols;
  stage(D, *dd);
  stage(cols, cols0);
  __syncthreads();
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= M) return;
  bool ok = true;
  for (int t = 0; t < D.n_trees && ok; ++t) {
    uint64_t key = 0;
    for (int l = 0; l < D.tcount[t]; ++l) {
      const int p = D.tparam[D.tstart[t] + l];
      const int32_t v = static_cast<const int32_t *>(cols.col[p])[j] - D.lo[p];
      ok = ok && v >= 0 && v < D.dim[p];
      key |= (uint64_t)((uint32_t)v & D.fmask[p]) << D.shift[p];
    }
    if (!ok) break;
    // lower bound of key in the tree's sorted keys
    const uint64_t *kt = keys + D.koff[t];
    int64_t lo = 0, n = D.nleaves[t];
    while (n > 0) {
      const int64_t h = n >> 1;
      if (kt[lo + h] < key) {
        lo += h + 1;
        n -= h + 1;
      } else {
        n = h;
      }
    }
    ok = lo < D.nleaves[t] && kt[lo] == key;
  }
  mask[j] = ok ? 1 : 0;
}

}  // namespace

hipError_t launch_cot_keys(const CotDesc *dd, int tree, const int32_t *leaves, int64_t n,
                           uint64_t *keys, unsigned long long *bad, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(cot_keys_k, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, dd, tree,
                     leaves, n, keys, bad);
  return hipGetLastError();
}

hipError_t launch_cot_sample(const CotDesc *dd, const uint64_t *keys, int64_t M, uint64_t seed,
                             uint64_t offset, const CotCols &out, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(cot_sample_k, dim3((unsigned)((M + 255) / 256)), dim3(256), 0, s, dd, keys, M,
                     seed, offset, out);
  return hipGetLastError();
}

hipError_t launch_cot_member(const CotDesc *dd, const uint64_t *keys, const CotCols &cols,
                             int64_t M, uint8_t *mask, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(cot_member_k, dim3((unsigned)((M + 255) / 256)), dim3(256), 0, s, dd, keys,
                     cols, M, mask);
  return hipGetLastError();
}

}  // namespace bgp
