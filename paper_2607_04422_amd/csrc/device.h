// Device helpers for the NVFP4 Newton-Schulz kernels (gfx950).
//
// Number formats follow Section 2 ("NVFP4 format"): E2M1 element codes, one
// E4M3FN scale per 16-element block, one FP32 tensor scale; RTN rounding
// (Section 2 "Others", Section 3.4).  Everything here is written with bit
// operations and comparisons; the library is compiled with FP contraction off
// and IEEE division so that each helper computes one fixed sequence of
// correctly rounded binary32/binary64 operations.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define FP4R_DEV __device__ __forceinline__

namespace fp4r {

// s_g = amax / (6 * 448): the largest block scale maps to the largest E4M3.
constexpr float kSgDivisor = 2688.0f;

// Random 16x16 Hadamard: flip the signs selected by `mask` (bit i set means
// d_i = -1), then the Sylvester butterfly with strides 1, 2, 4, 8, then * 1/4.
// A row block x becomes x diag(d) H / 4; a column block y becomes
// H diag(d) y / 4, the transpose of the same map.  (Sections 2, 3.4.)
FP4R_DEV void rotate16(float (&u)[16], uint32_t mask) {
#pragma unroll
  for (int i = 0; i < 16; ++i)
    if ((mask >> i) & 1u) u[i] = -u[i];
#pragma unroll
  for (int h = 1; h < 16; h <<= 1) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if ((i & h) == 0) {
        const float p = u[i], q = u[i + h];
        u[i] = p + q;
        u[i + h] = p - q;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) u[i] *= 0.25f;
}

// E4M3FN code of v in [0, 448], round to nearest, ties to the even code.
FP4R_DEV uint32_t e4m3_rne(float v) {
  if (v < 0.015625f) {                           // below 2^-6: grid m * 2^-9, m = 0..8
    return (uint32_t)__builtin_rintf(v * 512.0f);  // exact scaling, RNE to an integer
  }
  const uint32_t b = __float_as_uint(v);
  const uint32_t e = (b >> 23) - 120u;           // E4M3 biased exponent (bias 7)
  const uint32_t mant = b & 0x7FFFFFu;
  const uint32_t m3 = mant >> 20, rem = mant & 0xFFFFFu;
  uint32_t code = (e << 3) | m3;
  if (rem > 0x80000u || (rem == 0x80000u && (m3 & 1u))) code += 1u;  // carries into the exponent
  return code;
}

// Value of a non-negative E4M3FN code (0..126).
FP4R_DEV float e4m3_value(uint32_t c) {
  const uint32_t e = (c >> 3) & 15u, m = c & 7u;
  if (e == 0) return (float)m * 0.001953125f;   // m * 2^-9
  return __uint_as_float(((e + 120u) << 23) | (m << 20));
}

// E2M1 magnitude index of y in [0, 6]: the number of grid midpoints below y,
// a tie at a midpoint resolved towards the even index.
FP4R_DEV uint32_t e2m1_index(float y) {
  return (uint32_t)(y > 0.25f) + (uint32_t)(y >= 0.75f) + (uint32_t)(y > 1.25f) +
         (uint32_t)(y >= 1.75f) + (uint32_t)(y > 2.5f) + (uint32_t)(y >= 3.5f) +
         (uint32_t)(y > 5.0f);
}

FP4R_DEV double e2m1_value64(uint32_t idx) {
  // 0, 0.5, 1, 1.5 = idx/2 for idx < 4; 2, 3, 4, 6 above.
  return idx < 4 ? 0.5 * (double)idx : (idx == 7 ? 6.0 : (double)(idx - 2));
}

// One candidate block scaling (block maximum mapped to M * s * s_g).
struct BlockCand {
  uint32_t scale;   // E4M3 code
  uint64_t codes;   // 16 nibbles, element i in bits 4i..4i+3
  double err;       // sum of squared decode errors, element order, binary64
};

FP4R_DEV BlockCand quant_candidate(const float (&u)[16], float bmax, float sg, float M) {
  BlockCand r;
  const float den = M * sg;
  const float v = fminf(bmax / den, 448.0f);
  r.scale = e4m3_rne(v);
  const float s = e4m3_value(r.scale);
  const float rs = s * sg;
  const double s64 = (double)s, sg64 = (double)sg;
  r.codes = 0;
  r.err = 0.0;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const uint32_t neg = __float_as_uint(u[i]) >> 31;
    uint32_t idx = 0;
    if (rs > 0.0f) idx = e2m1_index(fminf(fabsf(u[i]) / rs, 6.0f));
    r.codes |= (uint64_t)((neg << 3) | idx) << (4 * i);
    double dec = (e2m1_value64(idx) * s64) * sg64;   // exact: <= 30 significant bits
    if (neg) dec = -dec;
    const double d = (double)u[i] - dec;
    r.err = r.err + d * d;
  }
  return r;
}

// Quantise one (already rotated) block given the tensor scale.
FP4R_DEV void quant_block(const float (&u)[16], float sg, bool adaptive, uint32_t& scale,
                          uint64_t& codes) {
  if (sg == 0.0f) {   // all-zero tensor: zero scales, zero magnitudes, signs kept
    codes = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) codes |= (uint64_t)((__float_as_uint(u[i]) >> 31) << 3) << (4 * i);
    scale = 0;
    return;
  }
  float bmax = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) bmax = fmaxf(bmax, fabsf(u[i]));
  BlockCand c6 = quant_candidate(u, bmax, sg, 6.0f);
  if (adaptive) {
    BlockCand c4 = quant_candidate(u, bmax, sg, 4.0f);
    if (c4.err < c6.err) c6 = c4;
  }
  scale = c6.scale;
  codes = c6.codes;
}

// Global scale from the bit pattern of the (non-negative) amax.
FP4R_DEV float tensor_scale_from_amax(uint32_t amax_bits) {
  return __uint_as_float(amax_bits) / kSgDivisor;
}

FP4R_DEV float warp_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

}  // namespace fp4r
