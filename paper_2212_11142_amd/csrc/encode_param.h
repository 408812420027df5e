// Code words of one parameter value (Sec. 3.2 input normalisation, Sec. 4.1 parameter
// types, Sec. 4.2 log transform), shared by the batch encoder and the local search so that
// both produce the same bits for the same value.
//
// Numeric codes are u = fl32((t(v) - t_lo) / den) with each step one IEEE fp64 operation,
// t = identity or log2. A categorical level is one bit of a one-hot field (several fields
// share a word) or, above 32 levels, the level itself in a word of its own. A permutation
// (position vector, pi[i] = position of item i) becomes Kendall pair bits, Hamming one-hot
// positions, Spearman position bytes or one packed equality word.
#pragma once
#include "common.h"

namespace bgp {

struct ParamCode {
  uint32_t w0, w1;  // the words at pe.word and (two-word codes) pe.word + 1; a one-hot
                    // categorical gives its field's bit, to be merged into the word
  float u;          // the numeric code (REAL, INT, ORD)
  bool ok;          // the value lies in the parameter's domain
};

// Words of the code that start at pe.word (a one-hot field counts its shared word).
__device__ __forceinline__ int param_code_words(const ParamEnc &pe) {
  if (pe.kind != GP_PERM) return 1;
  const int dist = (pe.flags >> 8) & 0xff;
  return (dist == GP_PERM_HAMMING || dist == GP_PERM_SPEARMAN) ? 2 : 1;
}

// Bits of the word at pe.word that a one-hot categorical owns (0: the word is its own).
__device__ __forceinline__ uint32_t param_field_mask(const ParamEnc &pe) {
  if (pe.kind != GP_CAT || pe.bit < 0) return 0u;
  const uint32_t f = pe.levels >= 32 ? 0xffffffffu : ((1u << pe.levels) - 1u);
  return f << pe.bit;
}

// raw: a REAL value's float64 bits, an INT value or ORD/CAT index in the low word;
// rv: a PERM row's m values (unused otherwise). Out-of-range levels are clamped for the
// code and reported through ok.
__device__ __forceinline__ ParamCode encode_param(const ParamEnc &pe, uint64_t raw,
                                                  const int (&rv)[8], const double *table) {
  ParamCode c{0u, 0u, 0.f, true};
  const int kind = pe.kind;
  if (kind == GP_REAL || kind == GP_INT || kind == GP_ORD) {
    double t;
    if (kind == GP_REAL) {
      const double v = __builtin_bit_cast(double, raw);
      c.ok = isfinite(v) && (!(pe.flags & 1) || v > 0.0);
      t = (pe.flags & 1) ? log2(v) : v;
    } else if (kind == GP_INT) {
      const int32_t v = (int32_t)(uint32_t)raw;
      c.ok = (double)v >= pe.lo && (double)v <= pe.hi;
      t = (pe.flags & 1) ? log2((double)v) : (double)v;
    } else {
      int32_t l = (int32_t)(uint32_t)raw;
      c.ok = l >= 0 && l < pe.levels;
      l = l < 0 ? 0 : (l >= pe.levels ? pe.levels - 1 : l);
      t = table[pe.table + l];
    }
    float u = 0.0f;
    if (pe.den != 0.0) u = (float)((t - pe.t_lo) / pe.den);
    c.u = u;
    c.w0 = __float_as_uint(u);
  } else if (kind == GP_CAT) {
    int32_t l = (int32_t)(uint32_t)raw;
    c.ok = l >= 0 && l < pe.levels;
    l = l < 0 ? 0 : (l >= pe.levels ? pe.levels - 1 : l);
    c.w0 = pe.bit >= 0 ? 1u << (pe.bit + l) : (uint32_t)l;
  } else {  // GP_PERM
    const int m = pe.levels;
    const int dist = (pe.flags >> 8) & 0xff;
    int p[8];
    uint32_t seen = 0;
    bool ok = true;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      int v = i < m ? rv[i] : i;
      ok = ok && (i >= m || (v >= 0 && v < m));
      v &= 7;
      p[i] = v;
      if (i < m) seen |= 1u << v;
    }
    c.ok = ok && seen == ((1u << m) - 1u);
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
      c.w0 = bits;
    } else if (dist == GP_PERM_HAMMING || dist == GP_PERM_SPEARMAN) {
      uint32_t w0 = 0, w1 = 0;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (i < m) {
          const uint32_t b = dist == GP_PERM_HAMMING ? 1u << (8 * (i & 3) + p[i])
                                                     : (uint32_t)p[i] << (8 * (i & 3));
          if (i < 4) w0 |= b; else w1 |= b;
        }
      c.w0 = w0;
      c.w1 = w1;
    } else {  // naive: the whole permutation as one value
      uint32_t w0 = 0;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (i < m) w0 |= (uint32_t)p[i] << (4 * i);
      c.w0 = w0;
    }
  }
  return c;
}

}  // namespace bgp
