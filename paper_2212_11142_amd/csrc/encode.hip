// Encoding of raw parameter columns into code words (Sec. 3.2 input normalisation,
// Sec. 4.1 parameter types, Sec. 4.2 log transform of exponential parameters).
//
// One thread per configuration. Numeric codes are u = fl32((t(v) - t_lo) / den) with
// each step one IEEE fp64 operation, t = identity or log2. Categorical levels become
// one-hot bit fields (or an equality word above 32 levels); permutations (position
// vectors, pi[i] = position of item i) become Kendall pair bits, Hamming one-hot
// positions, Spearman position bytes or a packed equality word.
#include "common.h"

namespace bgp {
namespace {

struct EncodeArgs {
  const void *col[kMaxD];
  const ParamEnc *penc;
  const double *table;
  const int32_t *rowmap;   // source row of output row j, or null (identity)
  uint32_t *out;
  uint8_t *valid;
  float *num_out;          // [count][n_num] or null
  int32_t *clear;          // set to 0 by thread 0 (scorer's counter), or null
  int64_t count, rows_out, s_word, s_row;
  int32_t d, n_num;
};

__device__ __forceinline__ void put(const EncodeArgs &a, int64_t j, int w, uint32_t v) {
  a.out[(int64_t)w * a.s_word + j * a.s_row] = v;
}

__global__ __launch_bounds__(256) void encode_kernel(EncodeArgs a) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j == 0 && a.clear) *a.clear = 0;
  if (j >= a.rows_out) return;
  int64_t src = j < a.count ? j : a.count - 1;   // padding rows repeat the last one
  if (a.rowmap) src = a.rowmap[src];
  bool ok = true;
  uint32_t acc = 0;
  int accw = -1;
  for (int q = 0; q < a.d; ++q) {
    const ParamEnc pe = a.penc[q];
    const int kind = pe.kind;
    if (kind == GP_REAL || kind == GP_INT || kind == GP_ORD) {
      double t;
      if (kind == GP_REAL) {
        const double v = static_cast<const double *>(a.col[pe.col])[src];
        ok = ok && isfinite(v) && (!(pe.flags & 1) || v > 0.0);
        t = (pe.flags & 1) ? log2(v) : v;
      } else if (kind == GP_INT) {
        const int32_t v = static_cast<const int32_t *>(a.col[pe.col])[src];
        ok = ok && (double)v >= pe.lo && (double)v <= pe.hi;
        t = (pe.flags & 1) ? log2((double)v) : (double)v;
      } else {
        int32_t l = static_cast<const int32_t *>(a.col[pe.col])[src];
        ok = ok && l >= 0 && l < pe.levels;
        l = l < 0 ? 0 : (l >= pe.levels ? pe.levels - 1 : l);
        t = a.table[pe.table + l];
      }
      float u = 0.0f;
      if (pe.den != 0.0) u = (float)((t - pe.t_lo) / pe.den);
      put(a, j, pe.word, __float_as_uint(u));
      if (a.num_out && j < a.count) a.num_out[j * a.n_num + pe.num_index] = u;
    } else if (kind == GP_CAT) {
      int32_t l = static_cast<const int32_t *>(a.col[pe.col])[src];
      ok = ok && l >= 0 && l < pe.levels;
      l = l < 0 ? 0 : (l >= pe.levels ? pe.levels - 1 : l);
      if (pe.bit >= 0) {
        if (pe.word != accw) {
          if (accw >= 0) put(a, j, accw, acc);
          accw = pe.word;
          acc = 0;
        }
        acc |= 1u << (pe.bit + l);
      } else {
        put(a, j, pe.word, (uint32_t)l);
      }
    } else {  // GP_PERM
      const int m = pe.levels;
      const int dist = (pe.flags >> 8) & 0xff;
      const int32_t *row = static_cast<const int32_t *>(a.col[pe.col]) + src * m;
      int p[8];
      uint32_t seen = 0;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        int v = i < m ? row[i] : i;
        ok = ok && (i >= m || (v >= 0 && v < m));
        v &= 7;
        p[i] = v;
        if (i < m) seen |= 1u << v;
      }
      ok = ok && seen == ((1u << m) - 1u);
      if (dist == GP_PERM_KENDALL) {
        uint32_t bits = 0;
        int idx = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int k = i + 1; k < 8; ++k)
            if (k < m) {
              bits |= (uint32_t)(p[i] > p[k]) << idx;
              ++idx;
            }
        put(a, j, pe.word, bits);
      } else if (dist == GP_PERM_HAMMING) {
        uint32_t w0 = 0, w1 = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (i < m) {
            const uint32_t b = 1u << (8 * (i & 3) + p[i]);
            if (i < 4) w0 |= b; else w1 |= b;
          }
        put(a, j, pe.word, w0);
        put(a, j, pe.word + 1, w1);
      } else if (dist == GP_PERM_SPEARMAN) {
        uint32_t w0 = 0, w1 = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (i < m) {
            const uint32_t b = (uint32_t)p[i] << (8 * (i & 3));
            if (i < 4) w0 |= b; else w1 |= b;
          }
        put(a, j, pe.word, w0);
        put(a, j, pe.word + 1, w1);
      } else {  // naive: the whole permutation as one value
        uint32_t w0 = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (i < m) w0 |= (uint32_t)p[i] << (4 * i);
        put(a, j, pe.word, w0);
      }
    }
  }
  if (accw >= 0) put(a, j, accw, acc);
  if (a.valid) a.valid[j] = ok ? 1 : 0;
}

}  // namespace

hipError_t launch_encode(const void *const *cols, int32_t d, const ParamEnc *penc,
                         const double *table, int64_t count, int64_t rows_out,
                         const int32_t *rowmap, uint32_t *out, int64_t s_word,
                         int64_t s_row, uint8_t *valid, float *num_out, int32_t n_num,
                         int32_t *clear, hipStream_t s) {
  if (rows_out <= 0) return hipSuccess;
  EncodeArgs a{};
  for (int i = 0; i < d; ++i) a.col[i] = cols[i];
  a.penc = penc;
  a.table = table;
  a.rowmap = rowmap;
  a.out = out;
  a.valid = valid;
  a.num_out = num_out;
  a.count = count;
  a.rows_out = rows_out;
  a.s_word = s_word;
  a.s_row = s_row;
  a.d = d;
  a.n_num = n_num;
  a.clear = clear;
  const int64_t blocks = (rows_out + 255) / 256;
  hipLaunchKernelGGL(encode_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace bgp
