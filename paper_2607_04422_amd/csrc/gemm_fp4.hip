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
#include "device.h"
#include "internal.h"

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

// LDS element (row, k) of a ROWS x 64 16-bit tile: 16-byte chunks XOR-swizzled by row.
FP4R_DEV int lds_idx(int row, int chunk) { return row * KS + ((chunk ^ (row & 7)) << 3); }

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
  uint2 codes[kPer];
  uint32_t scales[kPer];
};

template <int ROWS, int NT>
FP4R_DEV void fp4_load(const Fp4Operand& op, int64_t mat, int64_t rows, int64_t K, int64_t row0,
                       int stage, Fp4Stage<ROWS, NT>& s) {
  const int64_t nkb = K / 16;
#pragma unroll
  for (int j = 0; j < Fp4Stage<ROWS, NT>::kPer; ++j) {
    const int idx = threadIdx.x + NT * j;
    const int r = idx >> 2;
    const int64_t kb = (int64_t)stage * 4 + (idx & 3);
    const int64_t grow = row0 + r;
    if (grow < rows && kb < nkb) {
      s.codes[j] = *reinterpret_cast<const uint2*>(op.codes + mat * op.codes_bstride + grow * (K / 2) + kb * 8);
      s.scales[j] = op.scales[mat * op.scales_bstride + grow * nkb + kb];
    } else {
      s.codes[j] = make_uint2(0u, 0u);
      s.scales[j] = 0u;
    }
  }
}

template <int SEL>
FP4R_DEV f16x2 fp4_pair(uint32_t w, f16x2 s2) {
  // two E2M1 codes (low nibble first) -> two f16, then the exact product with the block scale
  const f16x2 q = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, SEL);
  return q * s2;
}

template <int ROWS, int NT>
FP4R_DEV void fp4_store(_Float16* lds, const Fp4Stage<ROWS, NT>& s) {
#pragma unroll
  for (int j = 0; j < Fp4Stage<ROWS, NT>::kPer; ++j) {
    const int idx = threadIdx.x + NT * j;
    const int r = idx >> 2, kb = idx & 3;
    const _Float16 sv = (_Float16)e4m3_value(s.scales[j]);
    const f16x2 s2 = {sv, sv};
    const uint32_t w[2] = {s.codes[j].x, s.codes[j].y};
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      f16x8 v;
      const f16x2 p0 = fp4_pair<0>(w[half], s2), p1 = fp4_pair<1>(w[half], s2);
      const f16x2 p2 = fp4_pair<2>(w[half], s2), p3 = fp4_pair<3>(w[half], s2);
      v[0] = p0[0]; v[1] = p0[1]; v[2] = p1[0]; v[3] = p1[1];
      v[4] = p2[0]; v[5] = p2[1]; v[6] = p3[0]; v[7] = p3[1];
      *reinterpret_cast<f16x8*>(lds + lds_idx(r, kb * 2 + half)) = v;
    }
  }
}

// ---------------------------------------------------------------------------
// Exact NVFP4 product.

#ifndef FP4R_FP4_WAVES_PER_EU
#define FP4R_FP4_WAVES_PER_EU 4
#endif
#ifndef FP4R_FP4_PIPELINE
#define FP4R_FP4_PIPELINE 0
#endif

template <int MODE, int WM_, int WN_, int TM, int TN>
__global__ __launch_bounds__(WM_* WN_ * 64) __attribute__((amdgpu_waves_per_eu(FP4R_FP4_WAVES_PER_EU)))
void k_gemm_fp4(GemmFp4Args g, int tiles_m, int tiles_n, int64_t tiles_per_mat) {
  constexpr int BM = WM_ * TM * 32, BN = WN_ * TN * 32, NT = WM_ * WN_ * 64;
  constexpr int kLdT = BN + 1;   // padded row of the FP32 output tile staged in LDS
  constexpr size_t kMainBytes = (size_t)2 * (BM + BN) * KS * sizeof(_Float16);
  constexpr size_t kEpiBytes = (size_t)BM * kLdT * sizeof(float);
  __shared__ __attribute__((aligned(16))) char smem[kMainBytes > kEpiBytes ? kMainBytes : kEpiBytes];
  _Float16(*lds_a)[BM * KS] = reinterpret_cast<_Float16(*)[BM * KS]>(smem);
  _Float16(*lds_b)[BN * KS] = reinterpret_cast<_Float16(*)[BN * KS]>(smem + 2 * BM * KS * sizeof(_Float16));
  constexpr bool kSym = MODE != kModeUpdateX;
  const int64_t mat = blockIdx.x / tiles_per_mat;
  int tm, tn;
  tile_coords(blockIdx.x % tiles_per_mat, tiles_m, tiles_n, kSym, tm, tn);
  const int64_t row0 = (int64_t)tm * BM, col0 = (int64_t)tn * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN_, wn = wave % WN_;
  const int64_t nkb = g.K / 16;
  const int nstages = (int)((nkb + 3) / 4);

  double acc[TM][TN][16];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0;

  Fp4Stage<BM, NT> sa;
  Fp4Stage<BN, NT> sb;
  fp4_load<BM, NT>(g.a, mat, g.M, g.K, row0, 0, sa);
  fp4_load<BN, NT>(g.b, mat, g.N, g.K, col0, 0, sb);
  fp4_store<BM, NT>(lds_a[0], sa);
  fp4_store<BN, NT>(lds_b[0], sb);
  __syncthreads();

  const f32x16 zero = {};
  for (int s = 0; s < nstages; ++s) {
    const int buf = s & 1;
    if (s + 1 < nstages) {
      fp4_load<BM, NT>(g.a, mat, g.M, g.K, row0, s + 1, sa);
      fp4_load<BN, NT>(g.b, mat, g.N, g.K, col0, s + 1, sb);
    }
    const _Float16* la = lds_a[buf];
    const _Float16* lb = lds_b[buf];
    const int kbs = (int)(nkb - (int64_t)s * 4 < 4 ? nkb - (int64_t)s * 4 : 4);
#if FP4R_FP4_PIPELINE
    // Software pipeline over the stage's (block, tile) jobs: the MFMA of job t+1
    // is in flight while the block sums of job t are folded into binary64.
    {
      constexpr int kJobs = TM * TN;
      f16x8 af[TM], bfr[TN];
      f32x16 pend;
      int pend_i = 0, pend_j = 0;
      bool have = false;
      for (int kb = 0; kb < kbs; ++kb) {
        const int chunk = kb * 2 + (lane >> 5);
#pragma unroll
        for (int i = 0; i < TM; ++i)
          af[i] = *reinterpret_cast<const f16x8*>(la + lds_idx((wm * TM + i) * 32 + (lane & 31), chunk));
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bfr[j] = *reinterpret_cast<const f16x8*>(lb + lds_idx((wn * TN + j) * 32 + (lane & 31), chunk));
#pragma unroll
        for (int t = 0; t < kJobs; ++t) {
          const int i = t / TN, j = t % TN;
          const f32x16 p = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[i], bfr[j], zero, 0, 0, 0);
          if (have) {
#pragma unroll
            for (int ii = 0; ii < TM; ++ii)
#pragma unroll
              for (int jj = 0; jj < TN; ++jj)
                if (ii == pend_i && jj == pend_j)
#pragma unroll
                  for (int e = 0; e < 16; ++e) acc[ii][jj][e] = acc[ii][jj][e] + (double)pend[e];
          }
          pend = p;
          pend_i = i;
          pend_j = j;
          have = true;
        }
      }
      if (have) {
#pragma unroll
        for (int ii = 0; ii < TM; ++ii)
#pragma unroll
          for (int jj = 0; jj < TN; ++jj)
            if (ii == pend_i && jj == pend_j)
#pragma unroll
              for (int e = 0; e < 16; ++e) acc[ii][jj][e] = acc[ii][jj][e] + (double)pend[e];
      }
    }
#else
    for (int kb = 0; kb < kbs; ++kb) {
      const int chunk = kb * 2 + (lane >> 5);
      f16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const f16x8*>(la + lds_idx((wm * TM + i) * 32 + (lane & 31), chunk));
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const f16x8*>(lb + lds_idx((wn * TN + j) * 32 + (lane & 31), chunk));
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
    if (s + 1 < nstages) {
      fp4_store<BM, NT>(lds_a[buf ^ 1], sa);
      fp4_store<BN, NT>(lds_b[buf ^ 1], sb);
    }
    __syncthreads();
  }

  // epilogue: binary64 formula, one rounding to binary32, staged through LDS
  // (the main loop's buffers are free after the last barrier)
  const double sga = (double)g.sc[mat].sg[g.slot_a], sgb = (double)g.sc[mat].sg[g.slot_b];
  const double alpha = sga * sgb;   // exact: product of two binary32 values
  const double ca = (double)g.ca, cb = (double)g.cb, cc = (double)g.cc;
  float* out = g.out + mat * g.out_bstride;
  const float* aux = g.aux ? g.aux + mat * g.out_bstride : nullptr;
  float* tile = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int rl = (wm * TM + i) * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        const int cl = (wn * TN + j) * 32 + (lane & 31);
        const int64_t r = row0 + rl, c = col0 + cl;
        float f = 0.0f;
        if (r < g.M && c < g.N) {
          double v = alpha * acc[i][j][e];
          if (MODE == kModeGramB) v = cb * (double)aux[r * g.N + c] + cc * v;
          if (MODE == kModeUpdateX) v = ca * (double)aux[r * g.N + c] + v;
          f = (float)v;
        }
        tile[rl * kLdT + cl] = f;
      }
  __syncthreads();
  // coalesced stores: rows of the tile, and (off-diagonal symmetric tiles) its transpose
  const bool mirror = kSym && tm != tn;
  constexpr int kSegs = BN / 16;                 // 16-float segments per row
  for (int idx = threadIdx.x; idx < BM * kSegs; idx += NT) {
    const int rl = idx / kSegs, q = idx % kSegs;
    const int64_t r = row0 + rl, c = col0 + 16 * q;
    if (r < g.M && c < g.N) {
      float4* dst = reinterpret_cast<float4*>(out + r * g.N + c);
#pragma unroll
      for (int k = 0; k < 4; ++k)
        dst[k] = make_float4(tile[rl * kLdT + 16 * q + 4 * k], tile[rl * kLdT + 16 * q + 4 * k + 1],
                             tile[rl * kLdT + 16 * q + 4 * k + 2], tile[rl * kLdT + 16 * q + 4 * k + 3]);
    }
    if (mirror) {
      // row cl of the mirrored tile = column cl of this tile
      const int cl = rl;
      const int64_t mr = col0 + cl, mc = row0 + 16 * q;
      if (mr < g.N && mc < g.M) {
        float4* dst = reinterpret_cast<float4*>(out + mr * g.N + mc);
#pragma unroll
        for (int k = 0; k < 4; ++k)
          dst[k] = make_float4(tile[(16 * q + 4 * k) * kLdT + cl], tile[(16 * q + 4 * k + 1) * kLdT + cl],
                               tile[(16 * q + 4 * k + 2) * kLdT + cl], tile[(16 * q + 4 * k + 3) * kLdT + cl]);
      }
    }
  }
  // rotated amaxes of the output: 16-column blocks of every row, and 16-row blocks
  // of every column (the mirrored tile's rows, or X_{k+1} along m)
  const bool do_rows = g.amax_row_slot >= 0;
  const bool do_cols = g.amax_col_slot >= 0 && (!kSym || mirror);
  float rmax = 0.0f, cmax = 0.0f;
  if (do_rows) {
    for (int idx = threadIdx.x; idx < BM * kSegs; idx += NT) {
      const int rl = idx / kSegs, q = idx % kSegs;
      float u[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) u[k] = tile[rl * kLdT + 16 * q + k];
      if (g.amax_rotate) rotate16(u, g.amax_mask);
#pragma unroll
      for (int k = 0; k < 16; ++k) rmax = fmaxf(rmax, fabsf(u[k]));
    }
  }
  if (do_cols) {
    constexpr int kRsegs = BM / 16;
    for (int idx = threadIdx.x; idx < BN * kRsegs; idx += NT) {
      const int cl = idx % BN, q = idx / BN;
      float u[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) u[k] = tile[(16 * q + k) * kLdT + cl];
      if (g.amax_rotate) rotate16(u, g.amax_mask);
#pragma unroll
      for (int k = 0; k < 16; ++k) cmax = fmaxf(cmax, fabsf(u[k]));
    }
  }
  if (do_rows) {
    const float w = warp_max(rmax);
    if (lane == 0) atomicMax(&g.sc[mat].amax[g.amax_row_slot], __float_as_uint(w));
  }
  if (do_cols) {
    const float w = warp_max(cmax);
    if (lane == 0) atomicMax(&g.sc[mat].amax[g.amax_col_slot], __float_as_uint(w));
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
