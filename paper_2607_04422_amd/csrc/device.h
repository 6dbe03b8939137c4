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

// -1.0f where bit i of mask is set, else 1.0f (integer operations only, so a
// uniform mask gives a scalar value).
FP4R_DEV float sign_factor(uint32_t mask, int i) {
  return __uint_as_float(0x3F800000u | (((mask >> i) & 1u) << 31));
}

// Random 16x16 Hadamard: flip the signs selected by `mask` (bit i set means
// d_i = -1), then the Sylvester butterfly with strides 1, 2, 4, 8, then * 1/4.
// A row block x becomes x diag(d) H / 4; a column block y becomes
// H diag(d) y / 4, the transpose of the same map.  (Sections 2, 3.4.)
// hadamard16 stops before the factor 1/4 (its outputs are 4 times the rotated
// values, exactly, wherever those are normal numbers).
FP4R_DEV void hadamard16(float (&u)[16], uint32_t mask) {
  // signs and the stride-1 stage together: fl(s_i u_i +- s_j u_j) as one fma of
  // exact products (the signs are built from bits of the uniform mask, so they
  // stay scalar operands and s_i costs no vector work)
#pragma unroll
  for (int i = 0; i < 16; i += 2) {
    const float si = sign_factor(mask, i), sj = sign_factor(mask, i + 1);
    const float t = sj * u[i + 1];
    const float p = fmaf(si, u[i], t), q = fmaf(si, u[i], -t);
    u[i] = p;
    u[i + 1] = q;
  }
#pragma unroll
  for (int h = 2; h < 16; h <<= 1) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if ((i & h) == 0) {
        const float p = u[i], q = u[i + h];
        u[i] = p + q;
        u[i + h] = p - q;
      }
    }
  }
}

FP4R_DEV void quarter16(float (&u)[16]) {
#pragma unroll
  for (int i = 0; i < 16; ++i) u[i] *= 0.25f;
}

FP4R_DEV void rotate16(float (&u)[16], uint32_t mask) {
  hadamard16(u, mask);
  quarter16(u);
}

// Inverse of rotate16: (diag(d) H / 4)^-1 = (H / 4) diag(d) since H H = 16 I, i.e.
// the unsigned butterfly (strides 1, 2, 4, 8, binary32), then * 1/4, then the signs.
FP4R_DEV void unrotate16(float (&u)[16], uint32_t mask) {
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
  for (int i = 0; i < 16; ++i) u[i] = (u[i] * 0.25f) * sign_factor(mask, i);
}

// SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): output `index` (1-based) of the
// generator started at `state`; splitmix64_mix is its output function applied to
// the advanced state state + gamma * index.
FP4R_DEV uint64_t splitmix64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
FP4R_DEV uint64_t splitmix64_at(uint64_t state, uint64_t index) {
  return splitmix64_mix(state + 0x9E3779B97F4A7C15ull * index);
}

// Binary32 -> BF16 bit pattern, round to nearest, ties to even (finite inputs).
FP4R_DEV uint16_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// Binary32 value of an E4M3FN code (bit 7 ignored): (8 + m) 2^(e - 10), or m 2^-9
// for the subnormal codes.
FP4R_DEV float e4m3_value(uint32_t code) {
  const uint32_t e = (code >> 3) & 15u, m = code & 7u;
  return e ? __uint_as_float(((e + 120u) << 23) | (m << 20)) : (float)m * 0.001953125f;
}

// The largest magnitude over a block after rotate16, times 4: the same butterfly
// up to the last stage, whose pair (fl(p + q), fl(p - q)) has the larger magnitude
// fl(|p| + |q|).  Multiplying the result by 1/4 gives max |rotate16(u)| exactly
// (rounding is monotone, so the factor commutes with the maximum).
FP4R_DEV float rot16_absmax4(float (&u)[16], uint32_t mask) {
#pragma unroll
  for (int i = 0; i < 16; i += 2) {
    const float si = sign_factor(mask, i), sj = sign_factor(mask, i + 1);
    const float t = sj * u[i + 1];
    const float p = fmaf(si, u[i], t), q = fmaf(si, u[i], -t);
    u[i] = p;
    u[i + 1] = q;
  }
#pragma unroll
  for (int h = 2; h < 8; h <<= 1) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if ((i & h) == 0) {
        const float p = u[i], q = u[i + h];
        u[i] = p + q;
        u[i + h] = p - q;
      }
    }
  }
  float m = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) m = fmaxf(m, fabsf(u[i]) + fabsf(u[i + 8]));
  return m;
}

// Binary32 rounding of a positive binary64 value downwards / upwards.
FP4R_DEV float rd32(double x) {
  float f = (float)x;
  if ((double)f > x) f = __uint_as_float(__float_as_uint(f) - 1u);
  return f;
}
FP4R_DEV float ru32(double x) {
  float f = (float)x;
  if ((double)f < x) f = __uint_as_float(__float_as_uint(f) + 1u);
  return f;
}

// E2M1 magnitude index of fl32(a / r) for a >= 0, r > 0, without dividing.
// The index counts the grid midpoints t crossed by y = fl32(a / r): y > t for
// t in {0.25, 1.25, 2.5, 5} and y >= t for t in {0.75, 1.75, 3.5} (ties to the
// even index).  Every t has an even binary32 significand, so y > t exactly when
// the quotient exceeds the binary32 midpoint t + ulp(t)/2, and y >= t exactly
// when it reaches the midpoint t - ulp(t^-)/2 below t.  Those midpoints have 25
// significant bits, so midpoint * r is exact in binary64, and for a binary32 a:
// a > X  <=>  a > RD32(X),  a >= X  <=>  a >= RU32(X).
struct E2m1Thresholds {
  float t[7];
};

FP4R_DEV E2m1Thresholds e2m1_thresholds(float r) {
  const double rd = (double)r;
  E2m1Thresholds th;
  th.t[0] = rd32((0.25 + 0x1p-26) * rd);
  th.t[1] = ru32((0.75 - 0x1p-25) * rd);
  th.t[2] = rd32((1.25 + 0x1p-24) * rd);
  th.t[3] = ru32((1.75 - 0x1p-24) * rd);
  th.t[4] = rd32((2.5 + 0x1p-23) * rd);
  th.t[5] = ru32((3.5 - 0x1p-23) * rd);
  th.t[6] = rd32((5.0 + 0x1p-22) * rd);
  return th;
}

// The thresholds increase, so the count is found by bisection: bit 2 of the
// index is a >= t3, bit 1 compares with t5 or t1, bit 0 with t6, t4, t2 or t0
// (the comparison kinds, >= at odd and > at even positions, match each level).
FP4R_DEV uint32_t e2m1_index_thr(float a, const E2m1Thresholds& th) {
  const bool b2 = a >= th.t[3];
  const bool b1 = a >= (b2 ? th.t[5] : th.t[1]);
  const float lo = b1 ? th.t[2] : th.t[0], hi = b1 ? th.t[6] : th.t[4];
  const bool b0 = a > (b2 ? hi : lo);
  return (b2 ? 4u : 0u) | (b1 ? 2u : 0u) | (b0 ? 1u : 0u);
}

// Twice the E2M1 magnitude of an index: {0, 1, 2, 3, 4, 6, 8, 12} (one nibble each).
FP4R_DEV uint32_t e2m1_twice(uint32_t idx) { return (0xC8643210u >> (idx << 2)) & 15u; }

// One candidate block scaling (block maximum mapped to M * s * s_g).
struct BlockCand {
  uint64_t codes;   // 16 nibbles, element i in bits 4i..4i+3
  float err;        // sum of squared decode errors in binary32 (fma, element order)
  float s2;         // (s s_g)^2 in binary32, for the error bound
  float s;          // the E4M3 scale value
};

// Codes and error sums of a candidate whose scale rs = s s_g is positive, with the
// E2M1 rounding done by the hardware conversion (round to nearest even, saturating,
// sign kept) on u * r, r ~ 1/rs.  fl32(u / rs) lies strictly between the products
// with r (1 - 2^-19) and with r (1 + 2^-19) (r is within 2^-23 of 1/rs, each
// product within 2^-24), and the rounding is monotone, so when both bracket values
// give the same codes, fl32(u / rs) gives them too: those are the codes.  Returns
// false when the codes differ (an element lies next to a grid midpoint) or r is not
// finite.
FP4R_DEV bool quant_candidate_hw(const float (&u)[16], float rs, BlockCand& r) {
  const float rinv = __builtin_amdgcn_rcpf(rs);
  if (!(rinv < 1e38f)) return false;
  const float rup = rinv * (1.0f + 0x1p-19f), rdn = rinv * (1.0f - 0x1p-19f);
  uint32_t c[2] = {0u, 0u}, cd[2] = {0u, 0u};
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int w = k >> 2;
    const float a = u[2 * k], b = u[2 * k + 1];
    switch (k & 3) {
#define FP4R_CVT(SEL)                                                                  \
  case SEL:                                                                            \
    c[w] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c[w], a * rup, b * rup, 1.0f, SEL);  \
    cd[w] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(cd[w], a * rdn, b * rdn, 1.0f, SEL); \
    break;
      FP4R_CVT(0)
      FP4R_CVT(1)
      FP4R_CVT(2)
      FP4R_CVT(3)
#undef FP4R_CVT
    }
  }
  if (c[0] != cd[0] || c[1] != cd[1]) return false;
  r.codes = (uint64_t)c[0] | ((uint64_t)c[1] << 32);
  // decoded values q (= tw / 2, signed) back from the codes; u - q rs has the
  // magnitude of |u| - tw (rs / 2), so the sum equals the element-order fma sum
  float err = 0.0f;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int w = k >> 2;
    float2 q;
    switch (k & 3) {
      case 0: q = __builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c[w], 1.0f, 0)); break;
      case 1: q = __builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c[w], 1.0f, 1)); break;
      case 2: q = __builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c[w], 1.0f, 2)); break;
      default: q = __builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c[w], 1.0f, 3)); break;
    }
    const float d0 = fmaf(-q.x, rs, u[2 * k]);
    err = fmaf(d0, d0, err);
    const float d1 = fmaf(-q.y, rs, u[2 * k + 1]);
    err = fmaf(d1, d1, err);
  }
  r.err = err;
  return true;
}

// The E4M3 value nearest to v in [0, 448] (ties to the even code), in binary32.
// From 2^-6 up the grid keeps 3 significand bits: round the binary32 significand
// at bit 20 (ties to even) and clear the bits below (a carry moves into the
// exponent by itself); below 2^-6 the grid is m 2^-9.
FP4R_DEV float e4m3_round(float v) {
  const uint32_t b = __float_as_uint(v);
  const float sn = __uint_as_float((b + 0x7FFFFu + ((b >> 20) & 1u)) & 0xFFF00000u);
  const float ss = __builtin_rintf(v * 512.0f) * 0.001953125f;
  return v < 0.015625f ? ss : sn;
}

// E4M3FN code of a value s of the grid (0 <= s <= 448) given in binary32.
FP4R_DEV uint32_t e4m3_code(float s) {
  return s < 0.015625f ? (uint32_t)(s * 512.0f) : (__float_as_uint(s) >> 20) - 960u;
}

// E4M3 value of min(fl32(bmax / den), 448) for den > 0.  The quotient is taken as
// bmax * rcp(den), within 4 ulp of fl32(bmax / den) (rcp within 1 ulp of 1/den,
// one rounding each); the E4M3 rounding only changes at its midpoints, where the
// 20 bits below the 3-bit mantissa read 0x80000, so a value at least 16 ulp away
// from one (and in the normal E4M3 range, where the rounding reads those bits)
// rounds like the quotient itself.  Other values take the correctly rounded
// division.
FP4R_DEV float scale_value(float bmax, float den) {
  const float rd = __builtin_amdgcn_rcpf(den);
  float v = fminf(bmax * rd, 448.0f);
  const uint32_t rem = __float_as_uint(v) & 0xFFFFFu;
  const bool fast = (rd < 1e38f) & (rd > 1e-37f) & (v >= 0.015625f) & (rem - 0x7FFF0u >= 32u);
  if (!fast) v = fminf(bmax / den, 448.0f);
  return e4m3_round(v);
}

// u holds kf times the block (kf = 1, or 4 for hadamard16 outputs); every scale
// below is kf times its reference value, which is exact (a power-of-two factor on
// normal numbers), so codes and scale codes are those of the block itself and the
// error sums are kf^2 times its own.
// Codes and binary32 error sum of a candidate with effective scale rs = s s_g kf
// (r.s is left to the caller).
FP4R_DEV void cand_codes(const float (&u)[16], float rs, BlockCand& r) {
  r.s2 = rs * rs;
  r.codes = 0;
  r.err = 0.0f;
  if (rs > 0.0f && quant_candidate_hw(u, rs, r)) return;
  if (rs > 0.0f) {
    // elements next to a grid midpoint: the exact threshold comparisons
    r.codes = 0;
    r.err = 0.0f;
    const E2m1Thresholds th = e2m1_thresholds(rs);
    const float h = 0.5f * rs;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t neg = __float_as_uint(u[i]) >> 31;
      const float a = fabsf(u[i]);
      const uint32_t idx = e2m1_index_thr(a, th);
      r.codes |= (uint64_t)((neg << 3) | idx) << (4 * i);
      const uint32_t tw = e2m1_twice(idx);
      const float d = fmaf(-(float)tw, h, a);
      r.err = fmaf(d, d, r.err);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t neg = __float_as_uint(u[i]) >> 31;
      r.codes |= (uint64_t)(neg << 3) << (4 * i);
      r.err = fmaf(u[i], u[i], r.err);
    }
  }
}

FP4R_DEV BlockCand quant_candidate(const float (&u)[16], float bmax, float sg, float M, float kf) {
  BlockCand r;
  const float s = scale_value(bmax, (M * sg) * kf);
  r.s = s;
  cand_codes(u, (s * sg) * kf, r);
  return r;
}

// The candidate's squared error in binary64, summed in element order: the
// reference definition of the 4/6 choice (on the block itself: u / kf, rounded
// to binary32 as the rotation's factor 1/4 rounds).
FP4R_DEV double cand_err64(const float (&u)[16], const BlockCand& c, float sg, float kf) {
  const double half_ss = 0.5 * ((double)c.s * (double)sg);   // exact: 4 + 24 significant bits
  double e = 0.0;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const double dec = (double)e2m1_twice((uint32_t)(c.codes >> (4 * i)) & 7u) * half_ss;
    const float ui = kf == 1.0f ? u[i] : u[i] * 0.25f;
    const double d = (double)fabsf(ui) - dec;   // exact; d^2 as for the signed difference
    e = e + d * d;
  }
  return e;
}

// Quantise one (already rotated) block given the tensor scale; u holds kf times
// the block (kf = 1 or 4, and 4 only where the tensor scale is at least 2^-40:
// then an element whose quarter is subnormal lies far below every grid step, and
// differences below the normal range change the binary32 error sums by far less
// than their bound, so the choice and the codes are those of the block).  With want_n2,
// `n2` receives sum_i (2 q_i)^2 M^2 with M the scale's integer significand (8..15,
// or the mantissa of a subnormal scale): the block's sum of squared decoded values
// is n2 2^(2 e - 22), e = max(exponent field, 1); otherwise n2 is 0.
//
// Adaptive 4/6 keeps M = 4 iff its binary64 squared error is strictly smaller.
// The binary32 sums decide when they are far apart: with S = s s_g, decoded
// values |dec_i| <= 6 S and D_i the exact errors, each fma-computed difference
// is within 2^-24 (|dec_i| + |D_i|) of D_i and the sum adds 16 roundings, so
// |err32 - E| <= 2^-24 (E + 576 S^2) + 2^-19.8 E < 2^-14 S^2 + 2^-19 E =: B.
// If err4 + 2 (B4 + B6) < err6 the exact E4 < E6 by more than any binary64
// rounding, and symmetrically; otherwise both are recomputed in binary64.
FP4R_DEV void quant_block(const float (&u)[16], float sg, bool adaptive, uint32_t& scale,
                          uint64_t& codes, uint32_t& n2, bool want_n2 = true, float kf = 1.0f) {
  n2 = 0;
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
  BlockCand c6 = quant_candidate(u, bmax, sg, 6.0f, kf);
  if (adaptive) {
    const BlockCand c4 = quant_candidate(u, bmax, sg, 4.0f, kf);
    const float b = 2.0f * (0x1p-14f * (c4.s2 + c6.s2) + 0x1p-18f * (c4.err + c6.err));
    bool use4;
    if (c4.err + b < c6.err) use4 = true;
    else if (c6.err + b < c4.err) use4 = false;
    else use4 = cand_err64(u, c4, sg, kf) < cand_err64(u, c6, sg, kf);
    if (use4) c6 = c4;
  }
  scale = e4m3_code(c6.s);
  codes = c6.codes;
  if (!want_n2) return;
  // sum of q^2 from the codes decoded to f16 pairs (q and q^2 exact; the sums are
  // multiples of 1/4 below 2^10, exact in the binary32 accumulator)
  const uint32_t w[2] = {(uint32_t)codes, (uint32_t)(codes >> 32)};
  float k2 = 0.0f;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    __attribute__((ext_vector_type(2))) _Float16 q;
    switch (k & 3) {
      case 0: q = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w[k >> 2], 1.0f, 0); break;
      case 1: q = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w[k >> 2], 1.0f, 1); break;
      case 2: q = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w[k >> 2], 1.0f, 2); break;
      default: q = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w[k >> 2], 1.0f, 3); break;
    }
    k2 = __builtin_amdgcn_fdot2(q, q, k2, false);
  }
  // n2 = 4 k2 M^2 < 2^24: exact in binary32
  const float mant = (float)((scale >> 3) ? 8u + (scale & 7u) : (scale & 7u));
  n2 = (uint32_t)((4.0f * k2) * (mant * mant));
}

// BF16 value of a bit pattern (exact).
FP4R_DEV float bf16_value(uint32_t h) { return __uint_as_float((h & 0xFFFFu) << 16); }

// Block quantisation with a BF16 block scale and no tensor scale (the AdamW second
// moment, Section 3.3): s = bf16(fl32(bmax / M)) for M = 6, and M = 4 with adaptive
// 4/6; element codes and the 4/6 choice exactly as quant_block (the error bound
// there holds for any effective scale).  `scale` receives the BF16 bits.
FP4R_DEV void quant_block_bf16(const float (&u)[16], bool adaptive, uint32_t& scale, uint64_t& codes) {
  float bmax = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) bmax = fmaxf(bmax, fabsf(u[i]));
  BlockCand c6;
  c6.s = bf16_value(bf16_rne(bmax / 6.0f));
  cand_codes(u, c6.s, c6);
  if (adaptive) {
    BlockCand c4;
    c4.s = bf16_value(bf16_rne(bmax / 4.0f));
    cand_codes(u, c4.s, c4);
    const float b = 2.0f * (0x1p-14f * (c4.s2 + c6.s2) + 0x1p-18f * (c4.err + c6.err));
    bool use4;
    if (c4.err + b < c6.err) use4 = true;
    else if (c6.err + b < c4.err) use4 = false;
    else use4 = cand_err64(u, c4, 1.0f, 1.0f) < cand_err64(u, c6, 1.0f, 1.0f);
    if (use4) c6 = c4;
  }
  scale = bf16_rne(c6.s);
  codes = c6.codes;
}

// The first-moment update of one 16-element block at flat offset e0: decode of the
// previous state (q s exact, times its tensor scale with one rounding, then the
// inverse rotation) when has_prev, then m = fl32(b1 m_hat + b2 g) with exact
// products and one binary64 rounding.
FP4R_DEV void mom_block(const float (&x)[16], const uint8_t* codes, const uint8_t* scales, int64_t e0,
                        float sgp, bool has_prev, uint32_t prev_mask, bool rotate, float b1, float b2,
                        float (&mv)[16]) {
  float mh[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) mh[i] = 0.0f;
  if (has_prev) {
    const uint2 cw = *reinterpret_cast<const uint2*>(codes + e0 / 2);
    const float s = e4m3_value(scales[e0 / 16]);
    const uint32_t w[2] = {cw.x, cw.y};
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      float2 q;
      switch (k & 3) {
        case 0: q = __builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[k >> 2], 1.0f, 0)); break;
        case 1: q = __builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[k >> 2], 1.0f, 1)); break;
        case 2: q = __builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[k >> 2], 1.0f, 2)); break;
        default: q = __builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[k >> 2], 1.0f, 3)); break;
      }
      mh[2 * k] = (q.x * s) * sgp;       // q s exact, one rounding
      mh[2 * k + 1] = (q.y * s) * sgp;
    }
    if (rotate) unrotate16(mh, prev_mask);
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) mv[i] = (float)__builtin_fma((double)b1, (double)mh[i], (double)b2 * (double)x[i]);
}

// Chain bound of one 4-block stage of a row (the NVFP4 products accumulate a
// stage in binary32 when rho sigma < 2^48, see gemm_fp4.hip):
//   rho = sum_b n2_b 4^(e_b - e_min),  e = max(exponent field, 1) over blocks with
// a non-zero scale (a zero block adds nothing and does not lower e_min).
FP4R_DEV uint32_t block_exp(uint32_t scale) {
  return (scale & 0x7Fu) ? max((scale >> 3) & 15u, 1u) : 15u;
}
FP4R_DEV float stage_rho(const uint32_t (&n2)[4], const uint32_t (&e)[4]) {
  const uint32_t emin = min(min(e[0], e[1]), min(e[2], e[3]));
  double r = 0.0;
#pragma unroll
  for (int b = 0; b < 4; ++b) r += ldexp((double)n2[b], 2 * (int)(e[b] - emin));
  return ru32(r);   // the sum is exact in binary64 (terms n2 < 2^19 times 4^k, k <= 14)
}

// Lane moves within a row of 16 lanes (DPP; every source lane of the patterns used
// exists, and all lanes of the wave must be active): quad_perm broadcasts of lane k
// of each quad (0x00, 0x55, 0xAA, 0xFF), xor 1 (0xB1), xor 2 (0x4E), mirror within
// 8 lanes (0x141) and within 16 lanes (0x140).
template <int CTRL>
FP4R_DEV uint32_t dpp_u(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
}

// The stage bound of the row whose four blocks sit in lanes 4i .. 4i + 3.  All
// lanes of the wave must be active.
FP4R_DEV float quad_stage_rho(uint32_t n2, uint32_t e) {
  const uint32_t qn[4] = {dpp_u<0x00>(n2), dpp_u<0x55>(n2), dpp_u<0xAA>(n2), dpp_u<0xFF>(n2)};
  const uint32_t qe[4] = {dpp_u<0x00>(e), dpp_u<0x55>(e), dpp_u<0xAA>(e), dpp_u<0xFF>(e)};
  return stage_rho(qn, qe);
}

// Maximum of non-negative values over each 16 lanes / over the wave (compared as
// bit patterns, which order non-negative floats); all lanes of the wave must be
// active, and every lane gets the result.
FP4R_DEV uint32_t row16_max_bits(uint32_t b) {
  b = max(b, dpp_u<0xB1>(b));
  b = max(b, dpp_u<0x4E>(b));
  b = max(b, dpp_u<0x141>(b));
  return max(b, dpp_u<0x140>(b));
}
FP4R_DEV float row16_max_pos(float v) { return __uint_as_float(row16_max_bits(__float_as_uint(v))); }
FP4R_DEV float wave_max_pos(float v) {
  const uint32_t b = row16_max_bits(__float_as_uint(v));
  const uint32_t r0 = __builtin_amdgcn_readlane(b, 0), r1 = __builtin_amdgcn_readlane(b, 16);
  const uint32_t r2 = __builtin_amdgcn_readlane(b, 32), r3 = __builtin_amdgcn_readlane(b, 48);
  return __uint_as_float(max(max(r0, r1), max(r2, r3)));
}

// Global scale fl32(amax / 2688) from the bit pattern of the (non-negative) amax.
// From 2^-100 up as q = amax y (y the binary32 nearest to 1/2688) corrected once by
// the exact remainder, q + (amax - 2688 q) y: equal to the correctly rounded
// quotient for every binary32 amax >= 2^-119 (checked exhaustively against IEEE
// division), and every intermediate is a normal number from 2^-100 up.
FP4R_DEV float tensor_scale_from_amax(uint32_t amax_bits) {
  const float a = __uint_as_float(amax_bits);
  if (!(a >= 0x1p-100f)) return a / kSgDivisor;
  const float y = 0x1.861862p-12f;
  const float q = a * y;
  return fmaf(fmaf(-q, kSgDivisor, a), y, q);
}

FP4R_DEV float warp_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

}  // namespace fp4r
