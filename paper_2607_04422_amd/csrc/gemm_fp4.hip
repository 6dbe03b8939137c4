// Matrix products of the Newton-Schulz step on gfx950 MFMA.
//
// All three products of a step (Section 3.4 display equation) have both
// operands contiguous along the contraction index:
//   A = qX qX^T        (K = n, symmetric: upper tiles only, mirrored)
//   B = b A + c qA qA^T (K = m, symmetric; epilogue reads A, may overwrite it)
//   X <- a X + qB qXt^T (K = m; epilogue reads X_k and writes X_{k+1} in place)
//
// NVFP4 operands (exact bridge): codes and E4M3 scales are decoded to f16
// while staging into LDS (q * s needs at most 6 significant bits and lies in
// [2^-10, 2688], so it is exact in f16).  One MFMA 32x32x16 covers exactly one
// 16-element block: all its products are integer multiples of s_a s_b / 4 with
// |sum| < 2^19 of those units, so the MFMA result (accumulator input 0) is the
// exact block sum.  Block sums are accumulated in binary64 and the epilogue
// forms the output in binary64 and rounds once to binary32, so every product
// equals the binary32 rounding of its exact value.
//
// Chained blocks.  Element values are q s with q = k/2 (|k| <= 12) and
// s = M 2^(e-10) (E4M3: M <= 15, e >= 1; subnormal scales as M = m, e = 1), so
// every product of a row i of the first operand and a row j of the second over
// a group G of blocks is a multiple of u = 2^(ea_min(i) + eb_min(j) - 22), the
// minima over G.  Any partial sum of those products, in any order, is at most
// their sum of magnitudes, and by Cauchy-Schwarz at most sqrt(T_a(i) T_b(j)),
// T being the sum of squared values over G.  With rho_i = T_a(i) 2^(22 - 2 ea_min(i))
// = sum_b n2_b 4^(e_b - ea_min(i)) (n2 = sum (2q)^2 M^2 per block; sigma_j alike)
// the bound is below 2^24 u whenever rho_i sigma_j < 2^48; then every partial
// sum is exactly representable in binary32, and the MFMAs of the group may
// accumulate into one binary32 register, folded into binary64 once.  The encoder
// stores rho per stage (four blocks) and 16 rows, rounded up to binary32, and
// each compute wave tests the maxima over its own rows (diagonal tiles of
// symmetric products test tile-wide maxima, so that (i, j) and (j, i) add the
// same binary32 values in the same order and the product stays exactly
// symmetric).
#include "device.h"
#include "internal.h"

#include <type_traits>

namespace fp4r {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Tile configuration of the exact NVFP4 product: WAVES_M x WAVES_N waves, each
// owning TM x TN MFMA 32x32 tiles; K is staged through LDS 64 elements (four
// NVFP4 blocks) at a time, double-buffered.
#ifndef FP4R_FP4_WAVES_M
#define FP4R_FP4_WAVES_M 4
#endif
#ifndef FP4R_FP4_WAVES_N
#define FP4R_FP4_WAVES_N 2
#endif
#ifndef FP4R_FP4_TM
#define FP4R_FP4_TM 1
#endif
#ifndef FP4R_FP4_TN
#define FP4R_FP4_TN 2
#endif
constexpr int KS = 64;   // K per LDS stage (4 NVFP4 blocks)
// Chained accumulation of block groups whose exactness bound holds (1) or one
// binary64 fold per block (0).
#ifndef FP4R_FP4_CHAIN
#define FP4R_FP4_CHAIN 1
#endif

// LDS layout of one decoded ROWS x 64 operand stage: block kb (16 f16, two 16-byte
// halves h) of row r at byte
//   kb_base(kb) + 32 r + 16 (h ^ bit 2 of r),   kb_base(kb) = 32 ROWS kb + {0, 64, 144, 208}[kb].
// A 16-byte access is served per 8 lanes.  MFMA operand reads (8 consecutive rows,
// one block and half) then cover all 32 banks, and so do the loader's writes
// (rows r, r + 1 times the four blocks: the block bases differ by 0, 64, 16 and 80
// modulo 128 bytes).  The block and buffer offsets are constants, so one address
// register per operand tile serves every block of both buffers.
FP4R_DEV int lds_row_off(int row, int h) { return row * 32 + ((h ^ ((row >> 2) & 1)) << 4); }
template <int ROWS>
constexpr int lds_kb_base(int kb) {
  return 32 * ROWS * kb + (kb == 0 ? 0 : kb == 1 ? 64 : kb == 2 ? 144 : 208);
}
template <int ROWS>
constexpr int lds_stage_bytes() { return lds_kb_base<ROWS>(3) + 32 * ROWS; }
static_assert(lds_kb_base<128>(2) == 32 * 128 * 2 + 64 * 2 + 16 && lds_kb_base<128>(3) == 32 * 128 * 3 + 64 * 3 + 16,
              "block bases");

// Output tile coordinates.  Symmetric products enumerate the upper triangle
// row by row; others are row-major over (tiles_m x tiles_n).
FP4R_DEV void tile_coords(int64_t t, int tiles_m, int tiles_n, bool sym, int& tm, int& tn) {
  if (!sym) {
    tm = (int)(t / tiles_n);
    tn = (int)(t % tiles_n);
    return;
  }
  int r = 0;
  int64_t left = t;
  while (left >= tiles_n - r) {
    left -= tiles_n - r;
    ++r;
  }
  tm = r;
  tn = r + (int)left;
}

// ---------------------------------------------------------------------------
// NVFP4 operand staging: each thread loads whole 16-element blocks (8 code
// bytes + 1 scale byte), decodes them to f16 and writes them to LDS.

template <int ROWS, int NT>
struct Fp4Stage {
  static constexpr int kPer = ROWS * 4 / NT;   // blocks per thread per stage
  static_assert(kPer == 1, "each thread stages one block of each operand per stage");
  uint2 codes[kPer];
  uint32_t scales[kPer];
};

// Where a thread's blocks come from: raw buffer resources over the tile's rows
// of codes and scales (the hardware range check returns 0 for rows past the
// matrix, so the tail tile needs no branch).  Thread t stages row t / 4, block
// t % 4 of every 64-element stage: scale byte (t / 4) nkb + t % 4 + 4 s and the
// codes at eight times that offset, the same offsets for both operands.
constexpr int kBufWord3 = 0x00020000;          // raw 32-bit data format, no swizzle
constexpr uint32_t kBufOutOfRange = 0x7FFFFFF0u;

struct Fp4Src {
  __amdgpu_buffer_rsrc_t codes, scales;
};

template <int ROWS>
FP4R_DEV Fp4Src fp4_src(const Fp4Operand& op, int64_t mat, int64_t rows, int64_t K, int64_t row0) {
  const int64_t nkb = K / 16;
  const int64_t live = rows - row0 < ROWS ? rows - row0 : ROWS;
  Fp4Src s;
  s.codes = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(op.codes + mat * op.codes_bstride + row0 * (K / 2)), (short)0, (int)(live * (K / 2)), kBufWord3);
  s.scales = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(op.scales + mat * op.scales_bstride + row0 * nkb), (short)0, (int)(live * nkb), kBufWord3);
  return s;
}

template <int ROWS, int NT>
FP4R_DEV void fp4_load(const Fp4Src& src, int nkb, int stage, Fp4Stage<ROWS, NT>& s) {
  // blocks past the end of K read as 0 (nkb < 2^17; the block index is recomputed
  // from the thread index, which is cheaper than keeping it live)
  const int kq = (int)(threadIdx.x & 3);
  const bool valid = stage * 4 + kq < nkb;
  const uint32_t o = (threadIdx.x >> 2) * (uint32_t)nkb + (uint32_t)(kq + 4 * stage);
  const uint32_t oc = valid ? 8u * o : kBufOutOfRange;
  const uint32_t os = valid ? o : kBufOutOfRange;
  const auto c = __builtin_amdgcn_raw_buffer_load_b64(src.codes, (int)oc, 0, 0);
  s.codes[0] = make_uint2(c[0], c[1]);
  s.scales[0] = __builtin_amdgcn_raw_buffer_load_b8(src.scales, (int)os, 0, 0);
}

template <int SEL>
FP4R_DEV f16x2 fp4_pair(uint32_t w, f16x2 s2) {
  // two E2M1 codes (low nibble first) -> two f16, then the exact product with the block scale
  const f16x2 q = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, SEL);
  return q * s2;
}

// Chain records of one operand: the encoder stores, per 64-element stage and 16
// rows, the largest rho (see the header), [K/64][rows/16].  Two ways to bring
// them to a compute wave (chosen per product by measurement):
// * table: before the stage loop each wave evaluates rho sigma over its own row
//   groups for every stage (one stage per lane) into its column of an LDS table,
//   so the loop reads one value per stage (K up to 64 kRecStages);
// * scalar: per stage the wave reads its groups' records through the constant
//   address space (written by an earlier kernel, never by this one), so the
//   wave-uniform loads become scalar loads, one stage ahead.
constexpr int kRecStages = 256;   // table: longer K (over 16384) folds every block
typedef const float __attribute__((address_space(4))) cfloat;

// Largest record of groups [g0, g0 + n) of stage s, clamped to the operand's
// groups (a tail tile's missing rows are zero and need no record).
FP4R_DEV float rho_records_max(const float* rec, int64_t ngroups, int s, int g0, int n) {
  cfloat* p = (cfloat*)(rec + (int64_t)s * ngroups);
  float m = 0.0f;
  for (int g = 0; g < n; ++g) m = fmaxf(m, p[min((int64_t)(g0 + g), ngroups - 1)]);
  return m;
}

// Decodes the staged blocks into the LDS stage at `lds`.
template <int ROWS, int NT>
FP4R_DEV void fp4_store(char* lds, const Fp4Stage<ROWS, NT>& s) {
#pragma unroll
  for (int j = 0; j < Fp4Stage<ROWS, NT>::kPer; ++j) {
    const int idx = threadIdx.x + NT * j;
    const int r = idx >> 2, kb = idx & 3;
    // the E4M3 scale in both halves, converted exactly (every E4M3 value is an f16)
    const f16x2 s2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8((s.scales[j] & 0xFFu) * 0x0101u, 1.0f, false);
    const uint32_t w[2] = {s.codes[j].x, s.codes[j].y};
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const f16x2 p0 = fp4_pair<0>(w[half], s2), p1 = fp4_pair<1>(w[half], s2);
      const f16x2 p2 = fp4_pair<2>(w[half], s2), p3 = fp4_pair<3>(w[half], s2);
      f16x8 v;
      v[0] = p0[0]; v[1] = p0[1]; v[2] = p1[0]; v[3] = p1[1];
      v[4] = p2[0]; v[5] = p2[1]; v[6] = p3[0]; v[7] = p3[1];
      const int kbo = 32 * ROWS * kb + 64 * kb + 16 * (kb >> 1);   // lds_kb_base<ROWS>(kb)
      *reinterpret_cast<f16x8*>(lds + kbo + lds_row_off(r, half)) = v;
    }
  }
}

// ---------------------------------------------------------------------------
// Rotated amaxes of an output, for the tensor scale of the operand encoded from
// it next (Section 3.2: the scale follows the largest magnitude after the 16-point
// rotation).  The rotation is the encoder's binary32 butterfly (signs, strides 1,
// 2, 4, 8, factor 1/4); only the largest magnitude is wanted, which permits three
// exact shortcuts:
// * the signs enter the stride-1 stage: fl(s_i u_i +- s_j u_j) is one fma of exact
//   products;
// * a stage across lanes may produce the difference with its sign flipped in the
//   lane holding the higher position: the later stages pair positions that agree
//   in that bit, so the flip reaches the final value unchanged (a sign only);
// * of the last stage's pair fl(p + q), fl(p - q) the larger magnitude is
//   fl(|p| + |q|), and the factor 1/4 commutes with the maximum (rounding is
//   monotone), so it is applied once to the final maximum.

template <int CTRL>
FP4R_DEV float dpp_f(float v) {
  // every source lane of the patterns used here exists (bound_ctrl only spares the old value)
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

// Row direction, four consecutive elements per lane: lane p = lane % 4 of a quad
// holds positions 4p .. 4p + 3 of a 16-element block; sg = their signs (+-1),
// s4 = +1 for even p, -1 for odd p.  Returns the unscaled maximum magnitude of
// the quad's block (every lane of the quad gets the same value).  All lanes of
// the wave must be active.
FP4R_DEV float rot_rows_max4(float4 u, const float (&sg)[4], float s4) {
  const float t1 = sg[1] * u.y, t3 = sg[3] * u.w;
  const float a0 = __builtin_fmaf(sg[0], u.x, t1), a1 = __builtin_fmaf(sg[0], u.x, -t1);
  const float a2 = __builtin_fmaf(sg[2], u.z, t3), a3 = __builtin_fmaf(sg[2], u.z, -t3);
  const float b0 = a0 + a2, b2 = a0 - a2, b1 = a1 + a3, b3 = a1 - a3;
  // stride 4: partner p ^ 1
  const float c0 = __builtin_fmaf(dpp_f<kDppXor1>(b0), s4, b0);
  const float c1 = __builtin_fmaf(dpp_f<kDppXor1>(b1), s4, b1);
  const float c2 = __builtin_fmaf(dpp_f<kDppXor1>(b2), s4, b2);
  const float c3 = __builtin_fmaf(dpp_f<kDppXor1>(b3), s4, b3);
  // stride 8: partner p ^ 2
  const float m0 = fabsf(c0) + fabsf(dpp_f<kDppXor2>(c0));
  const float m1 = fabsf(c1) + fabsf(dpp_f<kDppXor2>(c1));
  const float m2 = fabsf(c2) + fabsf(dpp_f<kDppXor2>(c2));
  const float m3 = fabsf(c3) + fabsf(dpp_f<kDppXor2>(c3));
  return fmaxf(fmaxf(m0, m1), fmaxf(m2, m3));
}

// Column direction, on the MFMA 32x32 output layout: v[B .. B + 7] of a lane are
// rows (e & 3) + 4 hb + 8 (e >> 2), e = 0 .. 7, of a 16-row block of its column
// (hb = lane / 32); sg = the signs of those rows, s4 = +1 (hb = 0) or -1.
// Returns the unscaled maximum magnitude over the lane's 8 outputs.  All lanes of
// the wave must be active.
template <int B>
FP4R_DEV float rot_cols_max8(const float (&v)[16], const float (&sg)[8], float s4) {
  float a[8], b[8], c[8];
#pragma unroll
  for (int e = 0; e < 8; e += 2) {
    const float t = sg[e + 1] * v[B + e + 1];
    a[e] = __builtin_fmaf(sg[e], v[B + e], t);
    a[e + 1] = __builtin_fmaf(sg[e], v[B + e], -t);
  }
#pragma unroll
  for (int e = 0; e < 8; e += 4) {
    b[e] = a[e] + a[e + 2];
    b[e + 2] = a[e] - a[e + 2];
    b[e + 1] = a[e + 1] + a[e + 3];
    b[e + 3] = a[e + 1] - a[e + 3];
  }
  // stride 4: both halves' values of the pair in every lane
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const auto lh = __builtin_amdgcn_permlane32_swap(__float_as_uint(b[e]), __float_as_uint(b[e]), false, false);
    c[e] = __builtin_fmaf(__uint_as_float(lh[1]), s4, __uint_as_float(lh[0]));
  }
  float m = 0.0f;
#pragma unroll
  for (int e = 0; e < 4; ++e) m = fmaxf(m, fabsf(c[e]) + fabsf(c[e + 4]));
  return m;
}

// Maximum of a non-negative value over the wave (bit pattern, uniform).
FP4R_DEV uint32_t wave_max_bits(float v) {
  v = fmaxf(v, dpp_f<kDppXor1>(v));
  v = fmaxf(v, dpp_f<kDppXor2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f<kDppMirror>(v));
  const uint32_t b = __float_as_uint(v);
  const uint32_t r0 = __builtin_amdgcn_readlane(b, 0), r1 = __builtin_amdgcn_readlane(b, 16);
  const uint32_t r2 = __builtin_amdgcn_readlane(b, 32), r3 = __builtin_amdgcn_readlane(b, 48);
  const uint32_t m01 = r0 > r1 ? r0 : r1, m23 = r2 > r3 ? r2 : r3;
  return m01 > m23 ? m01 : m23;
}

// ---------------------------------------------------------------------------
// Exact NVFP4 product.

#ifndef FP4R_FP4_WAVES_PER_EU
#define FP4R_FP4_WAVES_PER_EU 4
#endif

template <int MODE, int WM_, int WN_, int TM, int TN>
__global__ __launch_bounds__(WM_* WN_ * 64) __attribute__((amdgpu_waves_per_eu(FP4R_FP4_WAVES_PER_EU)))
void k_gemm_fp4(GemmFp4Args g, int tiles_m, int tiles_n, int64_t tiles_per_mat) {
  constexpr int BM = WM_ * TM * 32, BN = WN_ * TN * 32, NT = WM_ * WN_ * 64;
  // padded row of the FP32 output tile staged in LDS: rows stay 16-byte aligned, and
  // the two half-waves of an MFMA-layout write (rows 4 apart) fall 32 banks apart
  constexpr int kLdT = BN + 8;
  constexpr int kStA = lds_stage_bytes<BM>(), kStB = lds_stage_bytes<BN>();
  constexpr size_t kMainBytes = (size_t)2 * (kStA + kStB);
  constexpr size_t kEpiBytes = (size_t)BM * kLdT * sizeof(float);
  constexpr int kGa = BM / 16, kGb = BN / 16;   // 16-row groups per operand tile
  __shared__ __attribute__((aligned(16))) char smem[kMainBytes > kEpiBytes ? kMainBytes : kEpiBytes];
  constexpr bool kTable = MODE != kModeUpdateX;   // record delivery (see above)
  __shared__ uint8_t wflags[FP4R_FP4_CHAIN && kTable ? kRecStages : 1][NT / 64];
  __shared__ uint32_t red[2][NT / 64];   // per-wave amaxes (rows, columns)
  char(*lds_a)[kStA] = reinterpret_cast<char(*)[kStA]>(smem);
  char(*lds_b)[kStB] = reinterpret_cast<char(*)[kStB]>(smem + 2 * kStA);
  constexpr bool kSym = MODE != kModeUpdateX;
  const int64_t mat = blockIdx.x / tiles_per_mat;
  int tm, tn;
  tile_coords(blockIdx.x % tiles_per_mat, tiles_m, tiles_n, kSym, tm, tn);
  const int64_t row0 = (int64_t)tm * BM, col0 = (int64_t)tn * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN_, wn = wave % WN_;
  const int nkb = (int)(g.K / 16);   // K <= 2^21
  const int nstages = (int)((nkb + 3) / 4);

  double acc[TM][TN][16];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0;

  const Fp4Src src_a = fp4_src<BM>(g.a, mat, g.M, g.K, row0);
  const Fp4Src src_b = fp4_src<BN>(g.b, mat, g.N, g.K, col0);
  // a group chains if rho sigma < 2^48; the limit leaves room for the rounding of
  // the binary32 product rho * sigma
  constexpr float kLimStage = 281474976710656.0f * (1.0f - 1.0f / 65536.0f);   // 2^48 (1 - 2^-16)
#if FP4R_FP4_CHAIN
  static_assert(kGa == kGb, "square tiles");
  // the rows a compute wave covers: TM * 2 loader groups of A, TN * 2 of B;
  // diagonal tiles of symmetric products use all groups (see the header)
  const int uwave = __builtin_amdgcn_readfirstlane(wave);
  const bool diag = kSym && tm == tn;
  const bool chain_on = g.a.rhog != nullptr && g.b.rhog != nullptr && (!kTable || nstages <= kRecStages);
  const int ga0 = diag ? 0 : (uwave / WN_) * TM * 2, nga = diag ? kGa : TM * 2;
  const int gb0 = diag ? 0 : (uwave % WN_) * TN * 2, ngb = diag ? kGb : TN * 2;
  const float* rec_a = chain_on ? g.a.rhog + mat * g.a.rhog_bstride : nullptr;
  const float* rec_b = chain_on ? g.b.rhog + mat * g.b.rhog_bstride : nullptr;
  const float* rec8_a = chain_on && g.a.rho8 ? g.a.rho8 + mat * g.a.rho8_bstride : nullptr;
  const float* rec8_b = chain_on && g.b.rho8 ? g.b.rho8 + mat * g.b.rho8_bstride : nullptr;
  // the largest record over groups g0 .. g0 + ng - 1 of record row `idx`
  // (missing groups of a tail tile read 0: their rows are zero)
  auto group_max = [&](const float* rec, int64_t groups_all, int64_t idx, int64_t g0, int ng) {
    float mx = 0.0f;
    for (int k = 0; k < ng; ++k)
      if (g0 + k < groups_all) mx = fmaxf(mx, rec[idx * groups_all + g0 + k]);
    return mx;
  };
  // chain flags of stages s0 .. s0 + kRecStages - 1 for this wave's rows into
  // wflags[.][wave] (one stage per lane): bit 0 = the stage chains, bit 1 (even
  // stages) = the stage and the next chain as one group.  Only this wave touches
  // its column, so no barrier is needed.
  auto fill_flags = [&](int s0) {
    if (!kTable) return;
    const int64_t nga_all = g.M / 16, ngb_all = g.N / 16;
    const int64_t a0 = row0 / 16 + ga0, b0 = col0 / 16 + gb0;
#pragma unroll
    for (int h = 0; h < kRecStages / 64; ++h) {
      const int ss = lane + 64 * h;
      const int64_t sg = (int64_t)s0 + ss;
      uint32_t f = 0;
      if (chain_on && sg < nstages) {
        if (group_max(rec_a, nga_all, sg, a0, nga) * group_max(rec_b, ngb_all, sg, b0, ngb) < kLimStage) f |= 1u;
        if (rec8_a && rec8_b && (sg & 1) == 0 && sg + 1 < nstages &&
            group_max(rec8_a, nga_all, sg / 2, a0, nga) * group_max(rec8_b, ngb_all, sg / 2, b0, ngb) < kLimStage)
          f |= 2u;
      }
      wflags[ss][wave] = (uint8_t)f;
    }
  };
  auto stage_flags = [&](int s) { return (uint32_t)wflags[s % kRecStages][wave]; };
  auto stage_bound = [&](int s) {
    if (!chain_on || s >= nstages) return __builtin_inff();
    return rho_records_max(rec_a, g.M / 16, s, (int)(row0 / 16) + ga0, nga) *
           rho_records_max(rec_b, g.N / 16, s, (int)(col0 / 16) + gb0, ngb);
  };
#endif

  // stage -> LDS buffer `buf` (decoded operands)
  // The decode into LDS runs at raised wave priority: a wave that has finished its
  // MFMAs then gets the issue slots ahead of waves still in their MFMA or fold phase,
  // and reaches the barrier sooner (measured: update product -1 to -2 %, Gram of qX
  // -0.3 to -1.4 %; the Gram of qA, with its short K, lost 2 % and keeps the default).
  auto put = [&](int buf, const Fp4Stage<BM, NT>& xa, const Fp4Stage<BN, NT>& xb) {
    if constexpr (MODE != kModeGramB) __builtin_amdgcn_s_setprio(1);
    fp4_store<BM, NT>(lds_a[buf], xa);
    fp4_store<BN, NT>(lds_b[buf], xb);
    if constexpr (MODE != kModeGramB) __builtin_amdgcn_s_setprio(0);
  };

  const f32x16 zero = {};
  f32x16 p[TM][TN];   // the binary32 chain registers
  // MFMAs and binary64 folds of the stage in LDS buffer `buf` (kbs blocks).  fl:
  // bit k - 1 set = block k accumulates onto block k - 1 (blocks past the end of K
  // are zero in LDS and join any group).  Odd stages (odd_tag true) start on the
  // chain registers as left by the previous stage; fold_end folds the registers
  // at the end, and even stages then clear them for the odd stage after them.
  auto compute = [&](auto odd_tag, int buf, int kbs, uint32_t fl, bool fold_end) {
    constexpr bool ODD = decltype(odd_tag)::value;
    if (kbs <= 0) return;
    const char* la = lds_a[buf];
    const char* lb = lds_b[buf];
#if FP4R_FP4_CHAIN
    // the TM x TN tiles' chains run interleaved, block by block
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      f16x8 av[TM], bv[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        av[i] = *reinterpret_cast<const f16x8*>(
            la + lds_kb_base<BM>(kb) + lds_row_off((wm * TM + i) * 32 + (lane & 31), lane >> 5));
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bv[j] = *reinterpret_cast<const f16x8*>(
            lb + lds_kb_base<BN>(kb) + lds_row_off((wn * TN + j) * 32 + (lane & 31), lane >> 5));
      const bool chained = kb > 0 ? ((fl >> (kb - 1)) & 1u) != 0 : ODD;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          if (kb > 0 && !chained) {
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = acc[i][j][e] + (double)p[i][j][e];
          }
          p[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[i], bv[j], chained ? p[i][j] : zero, 0, 0, 0);
        }
      __builtin_amdgcn_sched_barrier(0);   // keep operand loads next to their use
    }
    if (fold_end) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[i][j][e] = acc[i][j][e] + (double)p[i][j][e];
          if (!ODD) p[i][j] = zero;
        }
    }
#else
    (void)fl; (void)fold_end;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      if (kb >= kbs) break;
      f16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const f16x8*>(
            la + lds_kb_base<BM>(kb) + lds_row_off((wm * TM + i) * 32 + (lane & 31), lane >> 5));
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const f16x8*>(
            lb + lds_kb_base<BN>(kb) + lds_row_off((wn * TN + j) * 32 + (lane & 31), lane >> 5));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const f32x16 p = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[i], bfr[j], zero, 0, 0, 0);
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[i][j][e] = acc[i][j][e] + (double)p[e];
        }
    }
#endif
  };
  auto blocks_in = [&](int s) { return nkb - s * 4 < 4 ? nkb - s * 4 : 4; };

  Fp4Stage<BM, NT> sa;
  Fp4Stage<BN, NT> sb;
  fp4_load<BM, NT>(src_a, nkb, 0, sa);
  fp4_load<BN, NT>(src_b, nkb, 0, sb);
  put(0, sa, sb);
  if (FP4R_FP4_CHAIN) fill_flags(0);
  __syncthreads();
  // Stage s is computed from LDS buffer s % 2 while stage s + 1 loads into
  // registers; it is decoded into the other buffer after the MFMAs.
  if (kTable) {
    // two stages per iteration, buffers as constants; a stage pair may chain as
    // one group of eight blocks (one fold per 128 elements); the last stage loads
    // and decodes nothing
    for (int s = 0; s < nstages; s += 2) {
      const uint32_t f0 = FP4R_FP4_CHAIN ? stage_flags(s) : 0u;
      const bool pair = (f0 & 2u) != 0, has_odd = s + 1 < nstages;
      if (has_odd) {
        fp4_load<BM, NT>(src_a, nkb, s + 1, sa);
        fp4_load<BN, NT>(src_b, nkb, s + 1, sb);
      }
      compute(std::false_type(), 0, blocks_in(s), (pair || (f0 & 1u)) ? 7u : 0u, !pair);
      if (has_odd) put(1, sa, sb);
      __syncthreads();
      if (!has_odd) break;
      const uint32_t f1 = FP4R_FP4_CHAIN ? stage_flags(s + 1) : 0u;
      const bool more = s + 2 < nstages;
      if (more) {
        fp4_load<BM, NT>(src_a, nkb, s + 2, sa);
        fp4_load<BN, NT>(src_b, nkb, s + 2, sb);
      }
      compute(std::true_type(), 1, blocks_in(s + 1), (pair || (f1 & 1u)) ? 7u : 0u, true);
      if (more) put(0, sa, sb);
      __syncthreads();
    }
  } else {
    float st = FP4R_FP4_CHAIN ? stage_bound(0) : 0.0f;
    // (unconditional loads and stores past the last stage: measured faster here)
    for (int s = 0; s < nstages; ++s) {
      fp4_load<BM, NT>(src_a, nkb, s + 1, sa);   // reads 0 past the last stage
      fp4_load<BN, NT>(src_b, nkb, s + 1, sb);
      compute(std::false_type(), s & 1, blocks_in(s), st < kLimStage ? 7u : 0u, true);
      put((s & 1) ^ 1, sa, sb);
      if (FP4R_FP4_CHAIN) st = stage_bound(s + 1);
      __syncthreads();
    }
  }

  // epilogue: binary64 formula, one rounding to binary32, staged through LDS
  // (the main loop's buffers are free after the last barrier)
  const double sga = (double)g.sc[mat].sg[g.slot_a], sgb = (double)g.sc[mat].sg[g.slot_b];
  const double alpha = sga * sgb;   // exact: product of two binary32 values
  const double ca = (double)g.ca, cb = (double)g.cb, cc = (double)g.cc;
  float* out = g.out + mat * g.out_bstride;
  const float* aux = g.aux ? g.aux + mat * g.out_bstride : nullptr;
  float* tile = reinterpret_cast<float*>(smem);
  // the epilogue operand (A for B, X_k for X_{k+1}) of all of this lane's
  // outputs, loaded up front (in-range index for lanes past the edge)
  float xin[TM][TN][16];
  if (MODE != kModeGramA) {
    const int64_t live = g.M - row0 < BM ? g.M - row0 : BM;
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc((void*)(aux + row0 * g.N), (short)0, (int)(live * g.N * 4), kBufWord3);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int rl = (wm * TM + i) * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
          const int64_t c = col0 + (wn * TN + j) * 32 + (lane & 31);
          const uint32_t off = c < g.N ? (uint32_t)((rl * g.N + c) * 4) : kBufOutOfRange;
          xin[i][j][e] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, (int)off, 0, 0));
        }
  }
  // this lane's outputs in binary32 (zero outside the matrix), also staged in LDS
  float val[TM][TN][16];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int rl = (wm * TM + i) * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        const int cl = (wn * TN + j) * 32 + (lane & 31);
        double v = alpha * acc[i][j][e];
        if (MODE == kModeGramB) v = cb * (double)xin[i][j][e] + cc * v;
        if (MODE == kModeUpdateX) v = ca * (double)xin[i][j][e] + v;
        const bool in = row0 + rl < g.M && col0 + cl < g.N;
        val[i][j][e] = in ? (float)v : 0.0f;
        tile[rl * kLdT + cl] = val[i][j][e];
      }
  // off-diagonal tiles of symmetric products (and a transposed final output): the
  // transposed tile straight from registers (four consecutive rows of a column
  // form a row segment of it)
  const bool mirror = kSym && tm != tn;
  const bool fin = !kSym && g.fin_count > 0;
  float* const fin_out = fin ? g.fin_out[mat] : nullptr;
  const int64_t fin_ld = fin ? g.fin_ld[mat] : 0;
  const bool fin_tall = fin && g.fin_tall[mat] != 0;
  if (fin_tall) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const int rb = (wm * TM + i) * 32 + 8 * e4 + 4 * (lane >> 5);
          const int cl = (wn * TN + j) * 32 + (lane & 31);
          const int64_t ur = col0 + cl, uc = row0 + rb;
          if (ur < g.N && uc < g.M)
            *reinterpret_cast<float4*>(fin_out + ur * fin_ld + uc) =
                make_float4(val[i][j][4 * e4], val[i][j][4 * e4 + 1], val[i][j][4 * e4 + 2], val[i][j][4 * e4 + 3]);
        }
  }
  if (mirror) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const int rb = (wm * TM + i) * 32 + 8 * e4 + 4 * (lane >> 5);
          const int cl = (wn * TN + j) * 32 + (lane & 31);
          const int64_t mr = col0 + cl, mc = row0 + rb;
          if (mr < g.N && mc < g.M)
            *reinterpret_cast<float4*>(out + mr * g.N + mc) =
                make_float4(val[i][j][4 * e4], val[i][j][4 * e4 + 1], val[i][j][4 * e4 + 2], val[i][j][4 * e4 + 3]);
        }
  }
  // rotated amaxes: 16-row blocks of every column (the mirrored tile's rows, or
  // X_{k+1} along m) from registers, 16-column blocks of every row from LDS
  const bool do_rows = g.amax_row_slot >= 0;
  const bool do_cols = g.amax_col_slot >= 0 && (!kSym || mirror);
  float cmax = 0.0f, rmax = 0.0f;
  if (do_cols) {
    if (g.amax_rotate) {
      const int hb = lane >> 5;
      float sg[8];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        sg[e] = ((g.amax_mask >> ((e & 3) + 4 * hb + 8 * (e >> 2))) & 1u) ? -1.0f : 1.0f;
      const float s4 = hb ? -1.0f : 1.0f;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          cmax = fmaxf(cmax, rot_cols_max8<0>(val[i][j], sg, s4));
          cmax = fmaxf(cmax, rot_cols_max8<8>(val[i][j], sg, s4));
        }
    } else {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e) cmax = fmaxf(cmax, fabsf(val[i][j][e]));
    }
  }
  __syncthreads();
  // rows of the tile: 32 lanes per row, one 16-byte slot each (coalesced stores;
  // a quad of lanes holds one 16-column block)
  {
    constexpr int kSlots = BN / 4;
    static_assert(NT % kSlots == 0 && (BM * kSlots) % NT == 0, "the row pass covers the tile");
    const int p = lane & 3;
    float sg[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) sg[w] = ((g.amax_mask >> (4 * p + w)) & 1u) ? -1.0f : 1.0f;
    const float s4 = (p & 1) ? -1.0f : 1.0f;
    constexpr int kIt = BM * kSlots / NT;
    float4 u[kIt];
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int idx = threadIdx.x + NT * it;
      u[it] = *reinterpret_cast<const float4*>(tile + (idx / kSlots) * kLdT + 4 * (idx % kSlots));
    }
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int idx = threadIdx.x + NT * it;
      const int64_t r = row0 + idx / kSlots, c = col0 + 4 * (idx % kSlots);
      if (r < g.M && c < g.N && !fin_tall)
        *reinterpret_cast<float4*>(fin ? fin_out + r * fin_ld + c : out + r * g.N + c) = u[it];
    }
    if (do_rows && g.amax_rotate) {
#pragma unroll
      for (int it = 0; it < kIt; ++it) rmax = fmaxf(rmax, rot_rows_max4(u[it], sg, s4));
    } else if (do_rows) {
#pragma unroll
      for (int it = 0; it < kIt; ++it)
        rmax = fmaxf(rmax, fmaxf(fmaxf(fabsf(u[it].x), fabsf(u[it].y)), fmaxf(fabsf(u[it].z), fabsf(u[it].w))));
    }
  }
  // one maximum per direction and workgroup, recorded on the workgroup's amax line
  if (do_rows || do_cols) {
    const uint32_t wr = wave_max_bits(rmax), wc = wave_max_bits(cmax);
    if (lane == 0) {
      red[0][wave] = wr;
      red[1][wave] = wc;
    }
    __syncthreads();
    if (threadIdx.x < 2 && (threadIdx.x == 0 ? do_rows : do_cols)) {
      uint32_t m = 0;
#pragma unroll
      for (int w = 0; w < NT / 64; ++w) m = m > red[threadIdx.x][w] ? m : red[threadIdx.x][w];
      const float mf = g.amax_rotate ? 0.25f * __uint_as_float(m) : __uint_as_float(m);
      amax_record(&g.sc[mat], threadIdx.x == 0 ? g.amax_row_slot : g.amax_col_slot, blockIdx.x, mf);
    }
  }
}

hipError_t launch_gemm_fp4(GemmMode mode, const GemmFp4Args& g, hipStream_t st) {
  constexpr int WM_ = FP4R_FP4_WAVES_M, WN_ = FP4R_FP4_WAVES_N, TM = FP4R_FP4_TM, TN = FP4R_FP4_TN;
  constexpr int BM = WM_ * TM * 32, BN = WN_ * TN * 32, NT = WM_ * WN_ * 64;
  static_assert(BM == BN, "symmetric products need square tiles");
  static_assert((BM * 4) % NT == 0, "each thread stages whole blocks");
  const int tiles_m = (int)((g.M + BM - 1) / BM), tiles_n = (int)((g.N + BN - 1) / BN);
  const bool sym = mode != kModeUpdateX;
  const int64_t per = sym ? (int64_t)tiles_m * (tiles_m + 1) / 2 : (int64_t)tiles_m * tiles_n;
  const dim3 grid((uint32_t)(per * g.batch));
  switch (mode) {
    case kModeGramA:
      hipLaunchKernelGGL((k_gemm_fp4<kModeGramA, WM_, WN_, TM, TN>), grid, dim3(NT), 0, st, g, tiles_m, tiles_n, per);
      break;
    case kModeGramB:
      hipLaunchKernelGGL((k_gemm_fp4<kModeGramB, WM_, WN_, TM, TN>), grid, dim3(NT), 0, st, g, tiles_m, tiles_n, per);
      break;
    default:
      hipLaunchKernelGGL((k_gemm_fp4<kModeUpdateX, WM_, WN_, TM, TN>), grid, dim3(NT), 0, st, g, tiles_m, tiles_n, per);
  }
  return hipGetLastError();
}

}  // namespace fp4r
