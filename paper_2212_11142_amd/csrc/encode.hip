// Encoding of raw parameter columns into code words (Sec. 3.2 input normalisation,
// Sec. 4.1 parameter types, Sec. 4.2 log transform of exponential parameters).
//
// One thread per configuration; the code of each parameter value is encode_param's.
#include "encode_param.h"

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

// Each thread loads the raw values of kEncGroup parameters before it encodes them and
// stores their codes, so the loads of a group are in flight together instead of each
// waiting behind the previous code's store (what rules small batches).
constexpr int kEncGroup = 8;
__global__ __launch_bounds__(256) void encode_kernel(EncodeArgs a) {
  __shared__ uint64_t raw_s[kEncGroup][256];
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j == 0 && a.clear) *a.clear = 0;
  if (j >= a.rows_out) return;
  int64_t src = j < a.count ? j : a.count - 1;   // padding rows repeat the last one
  if (a.rowmap) src = a.rowmap[src];
  // parameter descriptions, read as constant memory (never written by this kernel)
  auto penc = [&](int q) {
    typedef __attribute__((address_space(4))) const uint32_t cu32;
    const cu32 *w = (const cu32 *)(a.penc + q);
    ParamEnc e;
    uint32_t *dst = reinterpret_cast<uint32_t *>(&e);
#pragma unroll
    for (int i = 0; i < (int)(sizeof(ParamEnc) / 4); ++i) dst[i] = w[i];
    return e;
  };
  bool ok = true;
  uint32_t acc = 0;
  int accw = -1;
  for (int q0 = 0; q0 < a.d; q0 += kEncGroup) {
    // Branch-free loads: the first word of the row (of a parameter past d: of the last
    // parameter's row) and, for REAL, the second; PERM rows are read below.
    const uint32_t *lo_p[kEncGroup], *hi_p[kEncGroup];
#pragma unroll
    for (int g = 0; g < kEncGroup; ++g) {
      const ParamEnc pe = penc(min(q0 + g, a.d - 1));
      const int kind = pe.kind;
      const int w = kind == GP_REAL ? 2 : (kind == GP_PERM ? pe.levels : 1);
      lo_p[g] = static_cast<const uint32_t *>(a.col[pe.col]) + src * w;
      hi_p[g] = lo_p[g] + (kind == GP_REAL ? 1 : 0);
    }
    // REAL: the float64 bits; INT, ORD, CAT: the int32 value. Kept in this thread's LDS
    // slots so that the encoding below is one loop body, not kEncGroup copies of it.
    uint32_t lo[kEncGroup], hi[kEncGroup];
#pragma unroll
    for (int g = 0; g < kEncGroup; ++g) {
      lo[g] = *lo_p[g];
      hi[g] = *hi_p[g];
    }
#pragma unroll
    for (int g = 0; g < kEncGroup; ++g) raw_s[g][threadIdx.x] = (uint64_t)lo[g] | ((uint64_t)hi[g] << 32);
#pragma unroll 1
    for (int g = 0; g < kEncGroup; ++g) {
      const int q = q0 + g;
      if (q >= a.d) break;
      const ParamEnc pe = penc(q);
      int rv[8];
      if (pe.kind == GP_PERM) {  // the row's words, all loads in flight together
        const int m = pe.levels;
        const int32_t *row = static_cast<const int32_t *>(a.col[pe.col]) + src * m;
#pragma unroll
        for (int i = 0; i < 8; ++i) rv[i] = row[i < m ? i : m - 1];
      }
      const ParamCode c = encode_param(pe, raw_s[g][threadIdx.x], rv, a.table);
      ok = ok && c.ok;
      if (pe.kind == GP_CAT && pe.bit >= 0) {  // one-hot fields of a shared word
        if (pe.word != accw) {
          if (accw >= 0) put(a, j, accw, acc);
          accw = pe.word;
          acc = 0;
        }
        acc |= c.w0;
      } else {
        put(a, j, pe.word, c.w0);
        if (param_code_words(pe) == 2) put(a, j, pe.word + 1, c.w1);
        if (a.num_out && j < a.count && pe.kind != GP_CAT && pe.kind != GP_PERM)
          a.num_out[j * a.n_num + pe.num_index] = c.u;
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
