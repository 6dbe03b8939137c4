// Symmetric BF16 products of the plain Newton-Schulz comparison path on gfx950
// MFMA: the Gram of X and the Gram of A with the B epilogue, upper tiles only and
// mirrored, on bf16 operands with binary32 accumulation across the whole K loop
// (MFMA 32x32x16 bf16, accumulators in AGPRs).  Outputs are staged through LDS so
// that every global store (row-major and mirrored) is coalesced.  The update
// product of that path is a library GEMM (gemm_blaslt.cpp).
#include "device.h"
#include "internal.h"

namespace fp4r {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#ifndef FP4R_BF16_WAVES_M
#define FP4R_BF16_WAVES_M 4
#endif
#ifndef FP4R_BF16_WAVES_N
#define FP4R_BF16_WAVES_N 2
#endif
#ifndef FP4R_BF16_TM
#define FP4R_BF16_TM 2
#endif
#ifndef FP4R_BF16_TN
#define FP4R_BF16_TN 4
#endif

namespace {

constexpr int KS = 64;   // K per LDS stage

__device__ __forceinline__ int lds_idx(int row, int chunk) { return row * KS + ((chunk ^ (row & 7)) << 3); }

__device__ __forceinline__ void tile_coords(int64_t t, int tiles_m, int tiles_n, bool sym, int& tm, int& tn) {
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

template <int ROWS, int NT>
struct Stage {
  static constexpr int kPer = ROWS * 8 / NT;   // 16-byte chunks per thread per stage
  uint4 v[kPer];
};

template <int ROWS, int NT>
__device__ __forceinline__ void load_stage(const uint16_t* base, int64_t rows, int64_t K, int64_t row0,
                                           int stage, Stage<ROWS, NT>& s) {
#pragma unroll
  for (int q = 0; q < Stage<ROWS, NT>::kPer; ++q) {
    const int idx = threadIdx.x + NT * q;
    const int64_t grow = row0 + (idx >> 3);
    const int64_t k = (int64_t)stage * KS + (idx & 7) * 8;
    if (grow < rows && k < K)
      s.v[q] = *reinterpret_cast<const uint4*>(base + grow * K + k);
    else
      s.v[q] = make_uint4(0u, 0u, 0u, 0u);
  }
}

template <int ROWS, int NT>
__device__ __forceinline__ void store_stage(uint16_t* lds, const Stage<ROWS, NT>& s) {
#pragma unroll
  for (int q = 0; q < Stage<ROWS, NT>::kPer; ++q) {
    const int idx = threadIdx.x + NT * q;
    *reinterpret_cast<uint4*>(lds + lds_idx(idx >> 3, idx & 7)) = s.v[q];
  }
}

__device__ __forceinline__ uint16_t to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ float from_bf16(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// bf16 output tile [BM][BN] in LDS; 8-element groups XOR-swizzled by row.
template <int BN>
__device__ __forceinline__ int otile(int r, int c) { return r * BN + (c ^ ((r & 31) << 3)); }

}  // namespace

template <int MODE, int WM_, int WN_, int TM, int TN>
__global__ __launch_bounds__(WM_* WN_ * 64) void k_gemm_bf16(GemmBf16Args g, int tiles_m, int tiles_n,
                                                             int64_t tiles_per_mat) {
  constexpr int BM = WM_ * TM * 32, BN = WN_ * TN * 32, NT = WM_ * WN_ * 64;
  constexpr size_t kMain = (size_t)2 * (BM + BN) * KS * sizeof(uint16_t);
  constexpr size_t kEpi = (size_t)BM * BN * sizeof(uint16_t);
  __shared__ __attribute__((aligned(16))) char smem[kMain > kEpi ? kMain : kEpi];
  uint16_t(*lds_a)[BM * KS] = reinterpret_cast<uint16_t(*)[BM * KS]>(smem);
  uint16_t(*lds_b)[BN * KS] = reinterpret_cast<uint16_t(*)[BN * KS]>(smem + 2 * BM * KS * sizeof(uint16_t));
  static_assert(MODE == kModeGramA || MODE == kModeGramB, "symmetric products only");
  const int64_t mat = blockIdx.x / tiles_per_mat;
  int tm, tn;
  tile_coords(blockIdx.x % tiles_per_mat, tiles_m, tiles_n, true, tm, tn);
  const int64_t row0 = (int64_t)tm * BM, col0 = (int64_t)tn * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN_, wn = wave % WN_;
  const int nstages = (int)((g.K + KS - 1) / KS);
  const uint16_t* A = g.a + mat * g.a_bstride;
  const uint16_t* B = g.b + mat * g.b_bstride;

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};

  Stage<BM, NT> sa;
  Stage<BN, NT> sb;
  load_stage<BM, NT>(A, g.M, g.K, row0, 0, sa);
  load_stage<BN, NT>(B, g.N, g.K, col0, 0, sb);
  store_stage<BM, NT>(lds_a[0], sa);
  store_stage<BN, NT>(lds_b[0], sb);
  __syncthreads();
  for (int s = 0; s < nstages; ++s) {
    const int buf = s & 1;
    if (s + 1 < nstages) {
      load_stage<BM, NT>(A, g.M, g.K, row0, s + 1, sa);
      load_stage<BN, NT>(B, g.N, g.K, col0, s + 1, sb);
    }
    const uint16_t* la = lds_a[buf];
    const uint16_t* lb = lds_b[buf];
    const int64_t krem = g.K - (int64_t)s * KS;
    const int kbs = (int)(krem < KS ? krem / 16 : 4);
    for (int kb = 0; kb < kbs; ++kb) {
      const int chunk = kb * 2 + (lane >> 5);
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(la + lds_idx((wm * TM + i) * 32 + (lane & 31), chunk));
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(lb + lds_idx((wn * TN + j) * 32 + (lane & 31), chunk));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (s + 1 < nstages) {
      store_stage<BM, NT>(lds_a[buf ^ 1], sa);
      store_stage<BN, NT>(lds_b[buf ^ 1], sb);
    }
    __syncthreads();
  }

  // epilogue: binary32 formula, bf16 rounding, outputs staged in LDS
  uint16_t* tile = reinterpret_cast<uint16_t*>(smem);
  const uint16_t* aux16 = g.aux16 ? g.aux16 + mat * g.out16_bstride : nullptr;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int rl = (wm * TM + i) * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        const int cl = (wn * TN + j) * 32 + (lane & 31);
        const int64_t r = row0 + rl, c = col0 + cl;
        uint16_t h = 0;
        if (r < g.M && c < g.N) {
          float v = acc[i][j][e];
          if (MODE == kModeGramB) v = g.cb * from_bf16(aux16[r * g.N + c]) + g.cc * v;
          h = to_bf16(v);
        }
        tile[otile<BN>(rl, cl)] = h;
      }
  __syncthreads();
  uint16_t* o16 = g.out16 + mat * g.out16_bstride;
  // row-major bf16 output: 8 elements (16 bytes) per store
  constexpr int kGroups = BN / 8;
  for (int idx = threadIdx.x; idx < BM * kGroups; idx += NT) {
    const int rl = idx / kGroups, q = idx % kGroups;
    const int64_t r = row0 + rl, c = col0 + 8 * q;
    if (r < g.M && c < g.N)
      *reinterpret_cast<uint4*>(o16 + r * g.N + c) = *reinterpret_cast<const uint4*>(tile + otile<BN>(rl, 8 * q));
  }
  // the mirrored lower tile of an off-diagonal tile
  if (tm != tn) {
    uint16_t* ot = o16;
    const int64_t ldt = g.N;
    constexpr int kRGroups = BM / 8;
    for (int idx = threadIdx.x; idx < BN * kRGroups; idx += NT) {
      const int cl = idx / kRGroups, q = idx % kRGroups;
      const int64_t tr = col0 + cl, tc = row0 + 8 * q;
      if (tr < g.N && tc < g.M) {
        uint16_t v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = tile[otile<BN>(8 * q + k, cl)];
        uint4 w;
        w.x = v[0] | ((uint32_t)v[1] << 16);
        w.y = v[2] | ((uint32_t)v[3] << 16);
        w.z = v[4] | ((uint32_t)v[5] << 16);
        w.w = v[6] | ((uint32_t)v[7] << 16);
        *reinterpret_cast<uint4*>(ot + tr * ldt + tc) = w;
      }
    }
  }
}

hipError_t launch_gemm_bf16(GemmMode mode, const GemmBf16Args& g, hipStream_t st) {
  constexpr int WM_ = FP4R_BF16_WAVES_M, WN_ = FP4R_BF16_WAVES_N, TM = FP4R_BF16_TM, TN = FP4R_BF16_TN;
  constexpr int BM = WM_ * TM * 32, BN = WN_ * TN * 32, NT = WM_ * WN_ * 64;
  static_assert(BM == BN, "symmetric products need square tiles");
  static_assert((BM * 8) % NT == 0, "each thread stages whole 16-byte chunks");
  const int tiles_m = (int)((g.M + BM - 1) / BM), tiles_n = (int)((g.N + BN - 1) / BN);
  if (mode == kModeUpdateX || tiles_m != tiles_n) return hipErrorInvalidValue;
  const int64_t per = (int64_t)tiles_m * (tiles_m + 1) / 2;
  const dim3 grid((uint32_t)(per * g.batch));
  if (mode == kModeGramA)
    hipLaunchKernelGGL((k_gemm_bf16<kModeGramA, WM_, WN_, TM, TN>), grid, dim3(NT), 0, st, g, tiles_m, tiles_n, per);
  else
    hipLaunchKernelGGL((k_gemm_bf16<kModeGramB, WM_, WN_, TM, TN>), grid, dim3(NT), 0, st, g, tiles_m, tiles_n, per);
  return hipGetLastError();
}

}  // namespace fp4r
