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
// equals the binary32 rounding of its exact value whenever the binary64 running
// sums are exact (every partial sum within 53 bits of the smallest product unit,
// which holds unless the block exponents of a row span more than about 20 binades).
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
// accumulate into one binary32 register, folded into binary64 once.  The encoders
// store rho per 16 rows for every 64-element stage (four blocks), rounded up to
// binary32.  Each compute wave tests the maxima over its own rows (diagonal tiles
// of symmetric products test tile-wide maxima, so that (i, j) and (j, i) add the
// same binary32 values in the same order and the product stays exactly symmetric)
// and runs every stage either as one group or as one group per block.
//
// Work per wave (Gram of qX and update product): a 64 x 64 output tile (2 x 2
// MFMA tiles), 64 binary64 accumulators and 64 binary32 chain registers per lane;
// four waves share a 128 x 128 workgroup tile and two workgroups a CU (two waves
// per SIMD, 236-248 of their 256 VGPRs).  The Gram of qA runs 32 x 64 per wave,
// eight waves per workgroup, four per SIMD.  Per MFMA the exact path issues 8 fold
// instructions (one conversion and one binary64 add per output and stage) and 4-5
// decode instructions; per stage a wave waits for its LDS operand reads, for the
// staged loads of the next stage and at the barrier, which the other waves of its
// SIMD cover only in part.  Groups longer than one stage would keep the chain
// registers live beside the binary64 accumulators, which does not fit: every
// arrangement tried spilled 36-200 binary32 registers per lane, at 32 x 64 per
// wave (128 registers) and at 64 x 64 (256).
//
// Binary32 accumulation (GemmFp4Args::acc32, the library's FP4ROOT_F_FP32_ACCUM):
// the same loop with one chain over the whole contraction (zeroed once, never
// folded, no chain records), as tensor-core NVFP4 products accumulate in FP32.
// Each product is then within the binary32 accumulation bound of its exact value
// rather than equal to its rounding.  Its spare registers carry operand loads two
// stages ahead.
#include "device.h"
#include "internal.h"

#include <atomic>
#include <type_traits>
#include <utility>

namespace fp4r {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Tile configurations of the exact NVFP4 product: WAVES_M x WAVES_N waves, each
// owning TM x TN MFMA 32x32 tiles, WPE waves per SIMD; K is staged through LDS 64
// elements (four NVFP4 blocks) at a time, double-buffered.  Every workgroup tile is
// 128 x 128 and two workgroups share a CU.  Wide: 64 x 64 outputs per wave (four
// waves per workgroup, two per SIMD), half the LDS operand reads per MFMA of
// Narrow's 32 x 64 per wave (eight waves per workgroup, four per SIMD).  A wide
// workgroup alone on a CU (the last, partly filled round of a launch) has one wave
// per SIMD, which cannot overlap MFMA and VALU work, so launches of the Gram of qX
// and the update product take Wide only when they fill whole rounds of resident
// workgroups or at least kWideMinRounds of them; the Gram of qA (short
// contraction) always takes Narrow.
#ifndef FP4R_FP4_CFG_WIDE
#define FP4R_FP4_CFG_WIDE 2, 2, 2, 2, 2
#endif
#ifndef FP4R_FP4_CFG_NARROW
#define FP4R_FP4_CFG_NARROW 4, 2, 1, 2, 4
#endif
#ifndef FP4R_FP4_WIDE_MIN_ROUNDS
#define FP4R_FP4_WIDE_MIN_ROUNDS 4
#endif
// products (bit = mode) whose operand decode runs at raised wave priority
#ifndef FP4R_FP4_DECODE_PRIO
#define FP4R_FP4_DECODE_PRIO 7
#endif
template <int WM_, int WN_, int TM_, int TN_, int WPE_>
struct Fp4Tiling {
  static constexpr int WM = WM_, WN = WN_, TM = TM_, TN = TN_, WPE = WPE_;
};
using Fp4Wide = Fp4Tiling<FP4R_FP4_CFG_WIDE>;
using Fp4Narrow = Fp4Tiling<FP4R_FP4_CFG_NARROW>;
constexpr int kWideMinRounds = FP4R_FP4_WIDE_MIN_ROUNDS;
constexpr int KS = 64;   // K per LDS stage (4 NVFP4 blocks)

// LDS layout of one decoded ROWS x 64 operand stage: block kb (16 f16, two
// 16-byte halves h) of row r at byte
//   base(kb) + 32 r + 16 (h ^ sw(r)),   base(kb) = 32 ROWS kb + {0, 16, 64, 80}[kb],
// sw(r) = bit 2 of r xor bit 3 of r.  gfx950 serves a 16-byte LDS read 16 lanes
// per cycle over 64 banks (256 bytes) and a 16-byte write 8 lanes per cycle over
// 32 banks (128 bytes); lanes that share banks in one cycle conflict (measured
// with the SQ_LDS_BANK_CONFLICT counter on known patterns).  The MFMA operand
// reads (16 consecutive rows of one block and half per 16 lanes) fall in distinct
// banks through the swizzle.  The loader's writes (2 rows x the 4 blocks per 8
// lanes) fall in distinct banks through the block offsets, which are 0, 1, 4 and
// 5 sixteen-byte units modulo 128 bytes against the rows' 2 units apart.  The
// offsets are constants, so one address register per operand tile serves every
// block of both buffers.
FP4R_DEV int lds_row_off(int row, int h) { return row * 32 + ((h ^ ((row >> 2) & 1) ^ ((row >> 3) & 1)) << 4); }
template <int ROWS>
__host__ __device__ constexpr int lds_kb_base(int kb) { return 32 * ROWS * kb + 16 * ((kb & 1) + 4 * (kb >> 1)); }
template <int ROWS>
constexpr int lds_stage_bytes() { return lds_kb_base<ROWS>(3) + 32 * ROWS; }
static_assert(lds_kb_base<128>(0) % 128 == 0 && lds_kb_base<128>(1) % 128 == 16 && lds_kb_base<128>(2) % 128 == 64 &&
                  lds_kb_base<128>(3) % 128 == 80,
              "block offsets");

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
// bytes + 1 scale byte), decodes them to f16 and writes them to LDS.  Block
// slot idx = thread + NT j (j < kPer) stages row idx / 4, block idx % 4 of the
// stage.  The operands are stage-major (the encoders write them so): the 32 code
// bytes and 4 scale bytes of one row and stage follow those of the previous row,
// so a stage of the tile's rows is one contiguous run and lane idx reads bytes
// 8 idx .. 8 idx + 7 of it (whole 128-byte lines per wave).

template <int ROWS, int NT>
struct Fp4Stage {
  static constexpr int kPer = ROWS * 4 / NT;   // blocks per thread per stage
  static_assert(kPer >= 1 && ROWS * 4 == kPer * NT, "whole blocks per thread");
  uint2 codes[kPer];
  uint32_t scales[kPer];
};

FP4R_DEV int stage_row(int idx) { return idx >> 2; }
FP4R_DEV int stage_kb(int idx) { return idx & 3; }

constexpr int kBufWord3 = 0x00020000;          // raw 32-bit data format, no swizzle
constexpr uint32_t kBufOutOfRange = 0x7FFFFFF0u;

// The tile's rows of one operand: stage 0 of its codes and scales, the bytes from
// one stage to the next, and how many of its ROWS rows exist (a tail tile has fewer).
struct Fp4Src {
  const uint8_t* codes;
  const uint8_t* scales;
  int64_t code_stage, scale_stage;
  int live, nstages;
};

template <int ROWS>
FP4R_DEV Fp4Src fp4_src(const Fp4Operand& op, int64_t mat, int64_t rows, int64_t K, int64_t row0) {
  Fp4Src s;
  s.codes = op.codes + mat * op.codes_bstride + row0 * 32;
  s.scales = op.scales + mat * op.scales_bstride + row0 * 4;
  s.code_stage = rows * 32;
  s.scale_stage = rows * 4;
  s.live = (int)(rows - row0 < ROWS ? rows - row0 : ROWS);
  s.nstages = (int)((K + 63) / 64);
  return s;
}

template <int ROWS, int NT>
FP4R_DEV void fp4_load(const Fp4Src& src, int nkb, int stage, Fp4Stage<ROWS, NT>& s) {
  // one buffer resource per stage over the tile's rows of that stage: rows past the
  // matrix, blocks past the end of K and stages past the last read as 0
  const bool in_k = stage < src.nstages;
  const int64_t st = in_k ? stage : 0;
  const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(src.codes + st * src.code_stage), (short)0, in_k ? src.live * 32 : 0, kBufWord3);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(src.scales + st * src.scale_stage), (short)0, in_k ? src.live * 4 : 0, kBufWord3);
#pragma unroll
  for (int j = 0; j < Fp4Stage<ROWS, NT>::kPer; ++j) {
    const int idx = (int)threadIdx.x + NT * j;
    const bool valid = stage * 4 + stage_kb(idx) < nkb;
    const uint32_t oc = valid ? 8u * (uint32_t)idx : kBufOutOfRange;
    const uint32_t os = valid ? (uint32_t)idx : kBufOutOfRange;
    const auto c = __builtin_amdgcn_raw_buffer_load_b64(rc, (int)oc, 0, 0);
    s.codes[j] = make_uint2(c[0], c[1]);
    s.scales[j] = __builtin_amdgcn_raw_buffer_load_b8(rs, (int)os, 0, 0);
  }
}

template <int SEL>
FP4R_DEV f16x2 fp4_pair(uint32_t w, f16x2 s2) {
  // two E2M1 codes (low nibble first) -> two f16, then the exact product with the block scale
  const f16x2 q = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, SEL);
  return q * s2;
}

// Decodes the staged blocks into the LDS stage at `lds`.
template <int ROWS, int NT>
FP4R_DEV void fp4_store(char* lds, const Fp4Stage<ROWS, NT>& s) {
#pragma unroll
  for (int j = 0; j < Fp4Stage<ROWS, NT>::kPer; ++j) {
    const int idx = (int)threadIdx.x + NT * j;
    const int r = stage_row(idx), kb = stage_kb(idx);
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
      *reinterpret_cast<f16x8*>(lds + lds_kb_base<ROWS>(kb) + lds_row_off(r, half)) = v;
    }
    // one block at a time: few temporaries live beside the accumulators
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Chain records of one operand (see the header): per 64-element stage and 16 rows,
// [rows/16][K/64] (group-major).  Before the stage loop
// each wave evaluates rho sigma over its own row groups for every stage (up to
// kRecStages, K = 32768) into its column of an LDS byte table; the loop reads one
// byte per stage.
constexpr int kRecStages = 512;

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

// Accumulation form of one stage (uniform over a wave): one group per block, or
// the stage as one group.
enum StageForm { kFormBlock = 0, kFormStage = 1, kFormRun = 2 };
template <int F>
using form_t = std::integral_constant<int, F>;

// One output tile of one product: workgroup wg of the product's tiles_per_mat *
// batch tiles; fin (may be null) routes a last update's output to the callers'
// matrices.  Every kernel entry below runs this body.
template <int MODE, int WM_, int WN_, int TM, int TN, bool ACC32>
FP4R_DEV void gemm_fp4_tile(const GemmFp4Args& g, int64_t wg, int tiles_m, int tiles_n, int64_t tiles_per_mat,
                            const GemmFin* finp) {
  constexpr int BM = WM_ * TM * 32, BN = WN_ * TN * 32, NT = WM_ * WN_ * 64, NW = WM_ * WN_;
  // padded row of the FP32 output tile staged in LDS: rows stay 16-byte aligned, and
  // the two half-waves of an MFMA-layout write (rows 4 apart) fall 32 banks apart
  constexpr int kLdT = BN + 8;
  constexpr int kStA = lds_stage_bytes<BM>(), kStB = lds_stage_bytes<BN>();
  constexpr size_t kMainBytes = (size_t)2 * (kStA + kStB);
  constexpr size_t kEpiBytes = (size_t)BM * kLdT * sizeof(float);
  constexpr int kGa = BM / 16, kGb = BN / 16;   // 16-row groups per operand tile
  __shared__ __attribute__((aligned(16))) char smem[kMainBytes > kEpiBytes ? kMainBytes : kEpiBytes];
  __shared__ uint8_t wflags[kRecStages][NW];
  __shared__ uint32_t red[2][NW];   // per-wave amaxes (rows, columns)
  char* const la0 = smem;
  char* const la1 = smem + kStA;
  char* const lb0 = smem + 2 * kStA;
  char* const lb1 = smem + 2 * kStA + kStB;
  constexpr bool kSym = MODE != kModeUpdateX;
  const int64_t mat = wg / tiles_per_mat;
  int tm, tn;
  tile_coords(wg % tiles_per_mat, tiles_m, tiles_n, kSym, tm, tn);
  const int64_t row0 = (int64_t)tm * BM, col0 = (int64_t)tn * BN;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
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
  constexpr float kLim = 281474976710656.0f * (1.0f - 1.0f / 65536.0f);   // 2^48 (1 - 2^-16)
  // the rows a compute wave covers: TM * 2 groups of A, TN * 2 of B; diagonal
  // tiles of symmetric products use all groups of the tile (see the header)
  const bool diag = kSym && tm == tn;
  const bool chain_on = g.a.rhog != nullptr && g.b.rhog != nullptr;
  const int ga0 = diag ? 0 : wm * TM * 2, nga = diag ? kGa : TM * 2;
  const int gb0 = diag ? 0 : wn * TN * 2, ngb = diag ? kGb : TN * 2;
  const float* rec_a = chain_on ? g.a.rhog + mat * g.a.rhog_bstride : nullptr;
  const float* rec_b = chain_on ? g.b.rhog + mat * g.b.rhog_bstride : nullptr;
  // the largest record of stage `ss` over groups g0 .. g0 + ng - 1 (records are
  // group-major, [rows/16][K/64], so the lanes of a wave read consecutive stages;
  // missing groups of a tail tile read 0: their rows are zero)
  const int64_t nst_all = g.K / 64;
  auto group_max = [&](const float* rec, int64_t groups_all, int64_t ss, int64_t g0, int ng) {
    float mx = 0.0f;
    for (int k = 0; k < ng; ++k)
      if (g0 + k < groups_all) mx = fmaxf(mx, rec[(g0 + k) * nst_all + ss]);
    return mx;
  };
  // chain flags of every stage for this wave's rows into wflags[.][wave] (one
  // stage per lane and pass): bit 0 = the stage chains.  Only this wave touches its column, so no
  // barrier is needed.  Stages past kRecStages (K over 64 kRecStages) fold every block.
  auto fill_flags = [&]() {
    const int64_t nga_all = g.M / 16, ngb_all = g.N / 16;
    const int64_t a0 = row0 / 16 + ga0, b0 = col0 / 16 + gb0;
    const int nfill = nstages < kRecStages ? nstages : kRecStages;
    for (int s0 = 0; s0 < nfill; s0 += 64) {
      const int ss = s0 + lane;
      uint32_t f = 0;
      if (chain_on && ss < nfill) {
        if (group_max(rec_a, nga_all, ss, a0, nga) * group_max(rec_b, ngb_all, ss, b0, ngb) < kLim) f |= 1u;
      }
      if (ss < kRecStages) wflags[ss][wave] = (uint8_t)f;
    }
  };
  auto stage_flags = [&](int s) { return !ACC32 && s < kRecStages ? (uint32_t)wflags[s][wave] : 0u; };

  // stage -> LDS buffers (decoded operands)
  // The decode runs at raised wave priority: a wave that has finished its MFMAs
  // then gets the issue slots ahead of waves still in their MFMA or fold phase, and
  // reaches the barrier sooner (the Gram of qA, with its short K, keeps the default).
  auto put = [&](char* la, char* lb, const Fp4Stage<BM, NT>& xa, const Fp4Stage<BN, NT>& xb) __attribute__((always_inline)) {
    constexpr bool kPrio = (FP4R_FP4_DECODE_PRIO >> MODE) & 1;
    if constexpr (kPrio) __builtin_amdgcn_s_setprio(1);
    fp4_store<BM, NT>(la, xa);
    fp4_store<BN, NT>(lb, xb);
    if constexpr (kPrio) __builtin_amdgcn_s_setprio(0);
  };

  const f32x16 zero = {};
  f32x16 p[TM][TN];   // the binary32 chain registers
  auto fold = [&](int i, int j) __attribute__((always_inline)) {
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[i][j][e] = acc[i][j][e] + (double)p[i][j][e];
  };
  // MFMAs of the stage in (la, lb).  A group starts with accumulator input 0 and
  // is folded into binary64 as soon as it ends (after its last block, or at the end
  // of the stage), so the chain registers are dead while the next stage decodes.
  // Form Run (binary32 accumulation) adds every block to the chain registers, which
  // start at zero before the first stage and are never folded.  Blocks past the end
  // of K are zero in LDS and join any group.
  auto compute = [&](auto form_tag, const char* la, const char* lb) __attribute__((always_inline)) {
    constexpr int F = decltype(form_tag)::value;
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
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const bool fresh = F == kFormBlock || (F == kFormStage && kb == 0);
          p[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[i], bv[j], fresh ? zero : p[i][j], 0, 0, 0);
        }
      __builtin_amdgcn_sched_barrier(0);   // keep operand loads next to their use
      if (F == kFormBlock && kb < 3) {
        // every block a group of its own (rare: the stage bound failed)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) fold(i, j);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    if constexpr (F != kFormRun) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) fold(i, j);
    }
  };
  // one stage that is a group of its own (form Stage) or folds every block (Block);
  // with binary32 accumulation every stage continues the one chain (form Run)
  auto run_single = [&](uint32_t f, const char* la, const char* lb) __attribute__((always_inline)) {
    if constexpr (ACC32) {
      compute(form_t<kFormRun>(), la, lb);
    } else {
      if (f & 1u) compute(form_t<kFormStage>(), la, lb);
      else compute(form_t<kFormBlock>(), la, lb);
    }
  };
  if constexpr (ACC32) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) p[i][j] = zero;
  }

  // With binary32 accumulation the registers allow operand loads two stages ahead, in
  // two register sets (even and odd stages).  The exact products load one stage ahead:
  // their 32 x 64 form would spill, and their 64 x 64 form, which fits at 256 VGPRs,
  // ran its update product 1-2 % slower that way.
  constexpr bool kAhead2 = ACC32;
  if constexpr (kAhead2) {
    Fp4Stage<BM, NT> sa[2];
    Fp4Stage<BN, NT> sb[2];
    fp4_load<BM, NT>(src_a, nkb, 0, sa[0]);
    fp4_load<BN, NT>(src_b, nkb, 0, sb[0]);
    fp4_load<BM, NT>(src_a, nkb, 1, sa[1]);
    fp4_load<BN, NT>(src_b, nkb, 1, sb[1]);
    put(la0, lb0, sa[0], sb[0]);
    fp4_load<BM, NT>(src_a, nkb, 2, sa[0]);
    fp4_load<BN, NT>(src_b, nkb, 2, sb[0]);
    if constexpr (!ACC32) fill_flags();
    __syncthreads();
    // pairs of stages, then an odd last stage after the loop (one exit, so the
    // loop-carried chain registers keep their registers)
    int s = 0;
    for (; s + 1 < nstages; s += 2) {
      run_single(stage_flags(s), la0, lb0);
      put(la1, lb1, sa[1], sb[1]);
      fp4_load<BM, NT>(src_a, nkb, s + 3, sa[1]);
      fp4_load<BN, NT>(src_b, nkb, s + 3, sb[1]);
      __syncthreads();
      run_single(stage_flags(s + 1), la1, lb1);
      if (s + 2 < nstages) {
        put(la0, lb0, sa[0], sb[0]);
        fp4_load<BM, NT>(src_a, nkb, s + 4, sa[0]);
        fp4_load<BN, NT>(src_b, nkb, s + 4, sb[0]);
      }
      __syncthreads();
    }
    if (s < nstages) run_single(stage_flags(s), la0, lb0);
  } else {
  Fp4Stage<BM, NT> sa;
  Fp4Stage<BN, NT> sb;
  fp4_load<BM, NT>(src_a, nkb, 0, sa);
  fp4_load<BN, NT>(src_b, nkb, 0, sb);
  put(la0, lb0, sa, sb);
  // stage 1 loads while the flags are computed (reads 0 past the last stage)
  fp4_load<BM, NT>(src_a, nkb, 1, sa);
  fp4_load<BN, NT>(src_b, nkb, 1, sb);
  if constexpr (!ACC32) fill_flags();
  __syncthreads();
  // Two stages per iteration with the LDS buffers as constants: stage s computes
  // from one buffer while stage s + 1, loaded during the previous stage, decodes
  // into the other; the loads of stage s + 2 are issued into the same registers
  // right after that decode, so they have the barrier and a whole stage of MFMAs
  // to arrive.  Loads past the last stage read 0 and are never decoded.
  for (int s = 0; s < nstages; s += 2) {
    const bool has_odd = s + 1 < nstages, more = s + 2 < nstages;
    run_single(stage_flags(s), la0, lb0);
    if (has_odd) {
      put(la1, lb1, sa, sb);
      fp4_load<BM, NT>(src_a, nkb, s + 2, sa);
      fp4_load<BN, NT>(src_b, nkb, s + 2, sb);
    }
    __syncthreads();
    if (!has_odd) break;
    run_single(stage_flags(s + 1), la1, lb1);
    if (more) {
      put(la0, lb0, sa, sb);
      fp4_load<BM, NT>(src_a, nkb, s + 3, sa);
      fp4_load<BN, NT>(src_b, nkb, s + 3, sb);
    }
    __syncthreads();
  }
  }
  if constexpr (ACC32) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = (double)p[i][j][e];
  }

  // epilogue: binary64 formula, one rounding to binary32, staged through LDS
  // (the main loop's buffers are free after its last barrier), one MFMA tile at
  // a time
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
  // off-diagonal tiles of symmetric products (and a transposed final output): the
  // transposed tile straight from registers (four consecutive rows of a column
  // form a row segment of it)
  const bool mirror = kSym && tm != tn;
  const bool fin = !kSym && finp != nullptr && finp->count > 0;
  float* const fin_out = fin ? finp->out[mat] : nullptr;
  const int64_t fin_ld = fin ? finp->ld[mat] : 0;
  const bool fin_tall = fin && finp->tall[mat] != 0;
  const bool do_rows = g.amax_row_slot >= 0;
  const bool do_cols = g.amax_col_slot >= 0 && (!kSym || mirror);
  float cmax = 0.0f, rmax = 0.0f;
  const int hb = lane >> 5;
  float csg[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) csg[e] = ((g.amax_mask >> ((e & 3) + 4 * hb + 8 * (e >> 2))) & 1u) ? -1.0f : 1.0f;
  const float cs4 = hb ? -1.0f : 1.0f;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      // this lane's outputs of MFMA tile (i, j) in binary32 (zero outside the matrix)
      float val[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int rl = (wm * TM + i) * 32 + 8 * (e >> 2) + 4 * hb + (e & 3);
        const int cl = (wn * TN + j) * 32 + (lane & 31);
        double v = alpha * acc[i][j][e];
        if (MODE == kModeGramB) v = cb * (double)xin[i][j][e] + cc * v;
        if (MODE == kModeUpdateX) v = ca * (double)xin[i][j][e] + v;
        const bool in = row0 + rl < g.M && col0 + cl < g.N;
        val[e] = in ? (float)v : 0.0f;
        tile[rl * kLdT + cl] = val[e];
      }
      const int cl = (wn * TN + j) * 32 + (lane & 31);
      if (fin_tall || mirror) {
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const int rb = (wm * TM + i) * 32 + 8 * e4 + 4 * hb;
          const int64_t tr = col0 + cl, tc = row0 + rb;
          if (tr < g.N && tc < g.M) {
            float* dst = fin_tall ? fin_out + tr * fin_ld + tc : out + tr * g.N + tc;
            *reinterpret_cast<float4*>(dst) = make_float4(val[4 * e4], val[4 * e4 + 1], val[4 * e4 + 2], val[4 * e4 + 3]);
          }
        }
      }
      // rotated amaxes of 16-row blocks of every column (the mirrored tile's rows,
      // or X_{k+1} along m) from registers
      if (do_cols) {
        if (g.amax_rotate) {
          cmax = fmaxf(cmax, rot_cols_max8<0>(val, csg, cs4));
          cmax = fmaxf(cmax, rot_cols_max8<8>(val, csg, cs4));
        } else {
#pragma unroll
          for (int e = 0; e < 16; ++e) cmax = fmaxf(cmax, fabsf(val[e]));
        }
      }
    }
  __syncthreads();
  // rows of the tile: 32 lanes per row, one 16-byte slot each (coalesced stores;
  // a quad of lanes holds one 16-column block), and the rotated amaxes of
  // 16-column blocks of every row
  {
    constexpr int kSlots = BN / 4;
    static_assert(NT % kSlots == 0 && (BM * kSlots) % NT == 0, "the row pass covers the tile");
    const int pq = lane & 3;
    float sg[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) sg[w] = ((g.amax_mask >> (4 * pq + w)) & 1u) ? -1.0f : 1.0f;
    const float s4 = (pq & 1) ? -1.0f : 1.0f;
    constexpr int kIt = BM * kSlots / NT;
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int idx = threadIdx.x + NT * it;
      const float4 u = *reinterpret_cast<const float4*>(tile + (idx / kSlots) * kLdT + 4 * (idx % kSlots));
      const int64_t r = row0 + idx / kSlots, c = col0 + 4 * (idx % kSlots);
      if (r < g.M && c < g.N && !fin_tall)
        *reinterpret_cast<float4*>(fin ? fin_out + r * fin_ld + c : out + r * g.N + c) = u;
      if (do_rows) {
        if (g.amax_rotate) rmax = fmaxf(rmax, rot_rows_max4(u, sg, s4));
        else rmax = fmaxf(rmax, fmaxf(fmaxf(fabsf(u.x), fabsf(u.y)), fmaxf(fabsf(u.z), fabsf(u.w))));
      }
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
      for (int w = 0; w < NW; ++w) m = m > red[threadIdx.x][w] ? m : red[threadIdx.x][w];
      const float mf = g.amax_rotate ? 0.25f * __uint_as_float(m) : __uint_as_float(m);
      amax_record(&g.sc[mat], threadIdx.x == 0 ? g.amax_row_slot : g.amax_col_slot, blockIdx.x, mf);
    }
  }
}

// One product per launch (its arguments at fixed offsets).
template <int MODE, int WM_, int WN_, int TM, int TN, int WPE, bool ACC32>
__global__ __launch_bounds__(WM_* WN_ * 64) __attribute__((amdgpu_waves_per_eu(WPE)))
void k_gemm_fp4(GemmFp4Args g, int tiles_m, int tiles_n, int64_t tiles_per_mat, GemmFin fin) {
  gemm_fp4_tile<MODE, WM_, WN_, TM, TN, ACC32>(g, blockIdx.x, tiles_m, tiles_n, tiles_per_mat, &fin);
}

// Several products of one mode per launch: each workgroup finds its product (uniform
// over the workgroup) from the cumulative workgroup counts.
template <int MODE, int WM_, int WN_, int TM, int TN, int WPE, bool ACC32>
__global__ __launch_bounds__(WM_* WN_ * 64) __attribute__((amdgpu_waves_per_eu(WPE)))
void k_gemm_fp4_multi(GemmFp4Batch gb) {
  int pi = 0;
  while (pi + 1 < gb.count && (int64_t)blockIdx.x >= gb.wg_end[pi]) ++pi;
  const int64_t wg = (int64_t)blockIdx.x - (pi > 0 ? gb.wg_end[pi - 1] : 0);
  gemm_fp4_tile<MODE, WM_, WN_, TM, TN, ACC32>(gb.p[pi], wg, gb.tiles_m[pi], gb.tiles_n[pi], gb.tiles_per_mat[pi],
                                              nullptr);
}

// Every configuration covers a 128 x 128 output tile with whole blocks per staging thread.
constexpr int kFp4Tile = 128;
template <class C>
constexpr bool fp4_cfg_ok() {
  return C::WM * C::TM * 32 == kFp4Tile && C::WN * C::TN * 32 == kFp4Tile &&
         (kFp4Tile * 4) % (C::WM * C::WN * 64) == 0;
}
static_assert(fp4_cfg_ok<Fp4Wide>() && fp4_cfg_ok<Fp4Narrow>(), "128 x 128 workgroup tiles (square: symmetric products)");
// resident workgroups of a full round: two per CU
constexpr int64_t kFp4Round = 2 * 256;

template <int MODE, class C, bool ACC32>
void launch_fp4_single(dim3 grid, hipStream_t st, const GemmFp4Args& g, int tm, int tn, int64_t per,
                       const GemmFin& f) {
  hipLaunchKernelGGL((k_gemm_fp4<MODE, C::WM, C::WN, C::TM, C::TN, C::WPE, ACC32>), grid, dim3(C::WM * C::WN * 64), 0,
                     st, g, tm, tn, per, f);
}
template <int MODE, class C, bool ACC32>
void launch_fp4_multi(dim3 grid, hipStream_t st, const GemmFp4Batch& gb) {
  hipLaunchKernelGGL((k_gemm_fp4_multi<MODE, C::WM, C::WN, C::TM, C::TN, C::WPE, ACC32>), grid,
                     dim3(C::WM * C::WN * 64), 0, st, gb);
}

// The kernel of one launch: mode, tile form and accumulation.
template <bool ACC32>
void launch_fp4_kernel(GemmMode mode, bool wide, dim3 grid, hipStream_t st, const GemmFp4Batch& gb,
                       const GemmFin& f) {
  if (gb.count == 1) {
    const GemmFp4Args& g = gb.p[0];
    const int tm = gb.tiles_m[0], tn = gb.tiles_n[0];
    const int64_t per = gb.tiles_per_mat[0];
    switch (mode) {
      case kModeGramA:
        if (wide) launch_fp4_single<kModeGramA, Fp4Wide, ACC32>(grid, st, g, tm, tn, per, f);
        else launch_fp4_single<kModeGramA, Fp4Narrow, ACC32>(grid, st, g, tm, tn, per, f);
        break;
      case kModeGramB: launch_fp4_single<kModeGramB, Fp4Narrow, ACC32>(grid, st, g, tm, tn, per, f); break;
      default:
        if (wide) launch_fp4_single<kModeUpdateX, Fp4Wide, ACC32>(grid, st, g, tm, tn, per, f);
        else launch_fp4_single<kModeUpdateX, Fp4Narrow, ACC32>(grid, st, g, tm, tn, per, f);
    }
    return;
  }
  if (mode == kModeGramA) {
    if (wide) launch_fp4_multi<kModeGramA, Fp4Wide, ACC32>(grid, st, gb);
    else launch_fp4_multi<kModeGramA, Fp4Narrow, ACC32>(grid, st, gb);
  } else {
    launch_fp4_multi<kModeGramB, Fp4Narrow, ACC32>(grid, st, gb);
  }
}

std::atomic<int> g_product_tiling{0};

int swap_product_tiling(int mode) { return g_product_tiling.exchange(mode); }

hipError_t launch_gemm_fp4_batch(GemmMode mode, const GemmFp4Args* list, int count, hipStream_t st,
                                 const GemmFin* fin) {
  constexpr int BM = kFp4Tile, BN = kFp4Tile;
  if (count < 1 || count > kMaxGemmProblems) return hipErrorInvalidValue;
  if (fin && fin->count > 0 && (count != 1 || mode != kModeUpdateX || fin->count != list[0].batch))
    return hipErrorInvalidValue;
  for (int i = 1; i < count; ++i)
    if (list[i].acc32 != list[0].acc32) return hipErrorInvalidValue;   // one accumulation per launch
  // longest contraction first: its tiles take the longest, the short ones fill the tail
  int order[kMaxGemmProblems];
  for (int i = 0; i < count; ++i) order[i] = i;
  for (int i = 1; i < count; ++i)
    for (int j = i; j > 0 && list[order[j]].K > list[order[j - 1]].K; --j) std::swap(order[j], order[j - 1]);
  GemmFp4Batch gb;
  gb.count = 0;
  int64_t total = 0;
  const bool sym = mode != kModeUpdateX;
  for (int i = 0; i < count; ++i) {
    const GemmFp4Args& g = list[order[i]];
    const int tiles_m = (int)((g.M + BM - 1) / BM), tiles_n = (int)((g.N + BN - 1) / BN);
    const int64_t per = sym ? (int64_t)tiles_m * (tiles_m + 1) / 2 : (int64_t)tiles_m * tiles_n;
    if (per * g.batch == 0) continue;
    const int k = gb.count++;
    gb.p[k] = g;
    gb.tiles_m[k] = tiles_m;
    gb.tiles_n[k] = tiles_n;
    gb.tiles_per_mat[k] = per;
    total += per * g.batch;
    gb.wg_end[k] = total;
  }
  if (gb.count == 0) return hipSuccess;
  const dim3 grid((uint32_t)total);
  const int forced = g_product_tiling.load(std::memory_order_relaxed);
  const bool wide = forced == 0 ? (total % kFp4Round == 0 || total >= kWideMinRounds * kFp4Round) : forced == 2;
  // several products per launch: the symmetric products only
  if (gb.count > 1 && ((fin && fin->count > 0) || mode == kModeUpdateX)) return hipErrorInvalidValue;
  GemmFin f;
  if (fin) f = *fin;
  if (gb.p[0].acc32) launch_fp4_kernel<true>(mode, wide, grid, st, gb, f);
  else launch_fp4_kernel<false>(mode, wide, grid, st, gb, f);
  return hipGetLastError();
}

}  // namespace fp4r
