// Internal launcher interface between the C ABI (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace fp4r {

// Device status bits (kept in the first word of every workspace).
constexpr uint32_t kStatusNonFinite = 1u;

// ---------------------------------------------------------------------------
// Matrix lists for the stages that read caller matrices (clipping, copies).
constexpr int kMaxChunk = 32;

struct MatDesc {
  const float* in;     // caller matrix, row-major
  float* out;          // caller output (copy-out stage) or nullptr
  int64_t rows, cols, ld_in, ld_out;
  int64_t lo;          // quantile order statistic index floor(q (N - 1))
  double frac;         // q (N - 1) - lo
  int64_t tile_begin;  // first flat block index of this matrix in a launch
};

struct MatChunk {
  MatDesc m[kMaxChunk];
  int count;
  int64_t total_tiles;
};

// Per-matrix scalars kept in the workspace (one struct per matrix).
// Amax records are maxima over many workgroups.  To keep same-address atomics
// few, each slot is spread over kAmaxSpread 64-byte lines (a workgroup adds its
// maximum to line (workgroup index mod kAmaxSpread)); readers take the maximum
// of the lines.
constexpr int kAmaxSpread = 8;
struct alignas(64) AmaxLine {
  uint32_t v[16];        // slot k in v[k] (bit patterns of non-negative binary32)
};

struct MatScalars {
  AmaxLine amax[kAmaxSpread];   // slots: X along n / along m (two pairs, alternating by step), A, B
  float sg[6];           // tensor scales derived from amax
  float tau;             // clip threshold (+inf without clipping)
  float inv_norm;        // 1 / (||X'||_F + eps)
  uint32_t sel_prefix[2];  // radix select state for ranks lo and lo + 1
  uint32_t sel_rank[2];
};

// Record a non-negative maximum in amax slot `slot` (line chosen by `spread`),
// and read a slot back.
__device__ inline void amax_record(MatScalars* s, int slot, uint32_t spread, float v) {
  atomicMax(&s->amax[spread % kAmaxSpread].v[slot], __float_as_uint(v));
}
__device__ inline uint32_t amax_read(const MatScalars& s, int slot) {
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < kAmaxSpread; ++i) m = m > s.amax[i].v[slot] ? m : s.amax[i].v[slot];
  return m;
}

// amax / tensor-scale slots.  The X slots alternate between steps so that the
// update product of step k can record the amaxes of X_{k+1} while step k still
// reads those of X_k.
constexpr int kSlotXn = 0, kSlotXm = 1, kSlotA = 4, kSlotB = 5;
// Quantized-state AdamW: the first moment's new tensor scale lives in slot 0 and the
// previous one is saved in sg[kSlotPrevState] by the step's first pass.
constexpr int kSlotPrevState = 1;
constexpr int kNumSlots = 6;

// Radix select histogram: [2 ranks][2048 bins] per matrix.
constexpr int kHistBins = 2048;
constexpr int kPrepRowsPerBlock = 8;

// ---------------------------------------------------------------------------
// Launchers (all asynchronous on `st`; return hipSuccess or the launch error).

hipError_t launch_fill_u32(uint32_t* p, uint32_t value, int64_t n, hipStream_t st);

// Quantile of |x| per matrix in the chunk; writes sc[i].tau (ranks lo, lo+1).
// hist: chunk.count * 2 * kHistBins words of scratch.  status: device word.
// With psum / pcnt (chunk.total_tiles doubles / words of scratch) it also writes
// sc[i].inv_norm = fl32(1/(||clamp(M, tau)|| + eps)), as launch_inv_norm does.
hipError_t launch_clip_threshold(const MatChunk& ch, MatScalars* sc, uint32_t* hist,
                                 uint32_t* status, hipStream_t st, double* psum = nullptr,
                                 uint32_t* pcnt = nullptr, float eps = 0.0f);

// *out = 0, or -4 (non-finite input seen) from the status word *status.
hipError_t launch_status_out(const uint32_t* status, int32_t* out, hipStream_t st);

// Frobenius norm of the clipped matrices: sc[i].inv_norm = fl32(1/(||.|| + eps)).
// partial: chunk.total_tiles doubles of scratch.  A NaN or infinite entry sets
// kStatusNonFinite in *status.
hipError_t launch_inv_norm(const MatChunk& ch, MatScalars* sc, double* partial, float eps,
                           uint32_t* status, hipStream_t st);

// Canonical copy: X_b (m x n, m = min(rows, cols)) = fl32(clamp(M, tau) * inv_norm),
// transposed when rows > cols.  x: base of the group's canonical buffer, matrix b
// of the chunk at x + (first + b) * x_bstride.  Also records the amaxes of X_b
// rotated along n and along m (Hadamard signs `mask`) in slots slot_n, slot_m.
hipError_t launch_prep_copy(const MatChunk& ch, MatScalars* sc, float* x, int64_t x_bstride,
                            uint32_t mask, bool rotate, int slot_n, int slot_m, hipStream_t st);

// Copy-out: caller out (rows x cols) from canonical X (transposed when rows > cols).
hipError_t launch_copy_out(const MatChunk& ch, const float* x, int64_t x_bstride,
                           hipStream_t st);

// Uniform batch view of FP32 matrices.
struct Batch {
  const float* x;
  int64_t batch, rows, cols, ld, bstride;
};

// NVFP4 output view (axis 1: rows x cols/2 codes; axis 0: cols x rows/2 codes).
struct QOut {
  uint8_t* codes;
  uint8_t* scales;
  int64_t codes_bstride, scales_bstride;
  // optional (axis 1 only, K = cols a multiple of 64): chain bound records, the
  // largest rho over each 16 rows per 64-element stage, [rows/16][K/64]
  float* rhog = nullptr;
  int64_t rhog_bstride = 0;
  // stage-major layout (the products' operands; axis-1 encoders only): per matrix
  // codes [ceil(K/64)][rows][32 bytes] and scales [ceil(K/64)][rows][4 bytes], so
  // that one 64-element stage of consecutive rows is contiguous; otherwise row-major
  int tiled = 0;
};

// Bytes of one matrix's codes / scales in the stage-major layout (rows rows, K
// contraction elements; a last partial stage is padded).
__host__ __device__ inline int64_t tiled_code_bytes(int64_t rows, int64_t K) { return (K + 63) / 64 * rows * 32; }
__host__ __device__ inline int64_t tiled_scale_bytes(int64_t rows, int64_t K) { return (K + 63) / 64 * rows * 4; }

// Copy of stage-major codes and scales (batch matrices of rows x K) into the
// row-major layout (codes rows x K/2, scales rows x K/16 per matrix); a null
// output is skipped.
hipError_t launch_untile_nvfp4(const uint8_t* codes, const uint8_t* scales, int64_t batch, int64_t rows,
                               int64_t K, uint8_t* out_codes, uint8_t* out_scales, hipStream_t st);

// amax over rotated 16-blocks along `axis`; atomically maxes into
// amax slot `slot` of sc[b].  tau: clamp each element to +-sc[b].tau first when clip != 0.
hipError_t launch_amax(const Batch& in, int axis, uint32_t sign_mask, bool rotate, bool clip,
                       MatScalars* sc, int slot, uint32_t* status, hipStream_t st);

// Encode with the tensor scale derived from amax slot `slot` of sc[b]; writes sc[b].sg[slot]
// and, when tensor_scale != nullptr, tensor_scale[b].
hipError_t launch_encode(const Batch& in, int axis, uint32_t sign_mask, bool rotate, bool clip,
                         bool adaptive46, MatScalars* sc, int slot, const QOut& out,
                         float* tensor_scale, hipStream_t st);

// launch_encode along rows (axis 1, no clipping, no chain records) with the element
// magnitudes rounded stochastically (fp4root_momentum_update); draws from `sr_key`.
hipError_t launch_encode_sr(const Batch& in, uint32_t sign_mask, bool rotate, bool adaptive46,
                            MatScalars* sc, int slot, const QOut& out, float* tensor_scale,
                            uint64_t sr_key, hipStream_t st);

// First-moment update of a batch of contiguous rows x cols matrices (matrix
// stride rows*cols): m = fl32(b1 decode(previous state) + b2 g) (previous state
// read only when has_prev, decoded with prev_mask), amax of m rotated with `mask`
// into amax slot 0 of sc[b]; non-finite g sets the status word.
hipError_t launch_mom_update(const float* g, float* m, int64_t batch, int64_t rows, int64_t cols,
                             const uint8_t* codes, const uint8_t* scales, const float* prev_sg,
                             bool has_prev, uint32_t prev_mask, uint32_t mask, bool rotate, float b1,
                             float b2, MatScalars* sc, uint32_t* status, hipStream_t st);

// Parameter update W <- bf16(fl32(fl32(W c1) - fl32(c2 O))) over `count` contiguous
// elements (a multiple of 8; W and O 16-byte aligned).
hipError_t launch_apply_update(uint16_t* w, const float* o, int64_t count, float c1, float c2, hipStream_t st);

// Second pass of a quantized-state AdamW step on a flat parameter of n elements:
// re-derive m_t from g and the unchanged previous first-moment state and encode it
// in place (stochastically when sr), tensor scale from amax slot 0 of sc[0].
hipError_t launch_mom_encode(const float* g, uint8_t* codes, uint8_t* scales, int64_t n, bool has_prev,
                             uint32_t prev_mask, uint32_t mask, bool rotate, bool adaptive, bool sr, float b1,
                             float b2, MatScalars* sc, float* tensor_scale, uint64_t sr_key, hipStream_t st);

// First pass of a quantized-state AdamW step over a flat parameter of n elements (a
// multiple of 256): see k_qadamw.  It forms this step's first moment m_t from the
// previous first-moment state (read only) and g, records its rotated amax in slot 0
// of sc[0], saves the previous tensor scale in sc[0].sg[kSlotPrevState], and
// writes m_t to m_out when that is not null.
struct QAdamWLaunch {
  uint16_t* w;
  const float* g;
  float* m_out;
  const uint8_t* mcodes;
  const uint8_t* mscales;
  const float* m_prev_sg;
  float b1, c1m;
  MatScalars* sc;
  uint8_t* vcodes;
  uint16_t* vscales;
  uint16_t* vmeans;
  int64_t n;
  bool has_prev, rotate, adaptive;
  uint32_t prev_mask, mask;
  float b2, c2, bc1, bc2, eps, lr, c1w;
  uint32_t* status;
};
hipError_t launch_qadamw(const QAdamWLaunch& p, hipStream_t st);

// Both quantisations of X (m x n, row stride n) from one read: qX along n into
// qx (slot_n), qXt along m into qxt (slot_m, stored transposed).
// reset_mask: amax slots of every matrix set to zero by the launch (for the
// products that run after it; never slot_n or slot_m), as launch_reset_scalars does.
hipError_t launch_encode_x2(const float* x, int64_t batch, int64_t m, int64_t n, int64_t x_bstride,
                            uint32_t sign_mask, bool rotate, bool adaptive46, MatScalars* sc,
                            int slot_n, int slot_m, const QOut& qx, const QOut& qxt, hipStream_t st,
                            uint32_t reset_mask = 0);

// ---------------------------------------------------------------------------
// GEMMs (all operands K-contiguous: C[i][j] = sum_k A[i][k] B[j][k]).

enum GemmMode { kModeGramA = 0, kModeGramB = 1, kModeUpdateX = 2 };

struct Fp4Operand {
  const uint8_t* codes;   // stage-major: [ceil(K/64)][rows][32 bytes] (QOut::tiled)
  const uint8_t* scales;  // stage-major: [ceil(K/64)][rows][4 bytes]
  int64_t codes_bstride, scales_bstride;
  const float* rhog = nullptr;  // [rows/16][K/64] chain bound records; null: no chaining
  int64_t rhog_bstride = 0;
};

struct GemmFp4Args {
  Fp4Operand a, b;
  int64_t M, N, K, batch;
  MatScalars* sc;         // tensor scales per matrix (and amax records written by the epilogue)
  int slot_a, slot_b;
  // Epilogue amax of the output rotated with `amax_mask`: 16-column blocks into
  // slot amax_row_slot, 16-row blocks into amax_col_slot (symmetric products:
  // the mirrored lower tiles' row blocks); -1 disables.
  int amax_row_slot, amax_col_slot;
  uint32_t amax_mask;
  int amax_rotate;        // 0: amax of the plain values (no Hadamard)
  float* out;             // FP32 [M][N] per matrix (ld = N)
  int64_t out_bstride;
  const float* aux;       // kModeGramB: A (may equal out); kModeUpdateX: X_k (may equal out)
  float ca, cb, cc;
  // 0: exact products (binary32 rounding of the exact value, chained groups folded
  // into binary64); 1: one binary32 MFMA accumulation over the whole contraction
  // (every product of a launch takes the same value)
  int acc32 = 0;
};

// kModeUpdateX, last step: when count > 0 the output goes to the callers' matrices
// instead of `out`: matrix b to out[b] with row stride ld[b], transposed
// (out[b][c][r] = X[r][c]) when tall[b].
struct GemmFin {
  int count = 0;
  float* out[kMaxChunk] = {};
  int64_t ld[kMaxChunk] = {};
  uint8_t tall[kMaxChunk] = {};
};

// NVFP4 product with exact block sums accumulated in binary64.
// kModeGramA / kModeGramB compute upper-triangle tiles only and mirror them.
// Several products of one mode in one launch (up to kMaxGemmProblems): the
// workgroups of product i follow those of product i - 1, so short products fill
// the last, partly occupied round of a long one.
constexpr int kMaxGemmProblems = 4;
struct GemmFp4Batch {
  GemmFp4Args p[kMaxGemmProblems];
  int32_t tiles_m[kMaxGemmProblems], tiles_n[kMaxGemmProblems];
  int64_t tiles_per_mat[kMaxGemmProblems];
  int64_t wg_end[kMaxGemmProblems];   // cumulative workgroup counts
  int32_t count;
};

// count products of one mode (1 <= count <= kMaxGemmProblems; more than one for the
// symmetric products only) in one launch, the products with the longest contraction
// first; fin (host, may be null) routes the output of a single update product to the
// callers' matrices.
hipError_t launch_gemm_fp4_batch(GemmMode mode, const GemmFp4Args* list, int count, hipStream_t st,
                                 const GemmFin* fin = nullptr);
// Tile form of the NVFP4 products (0: chosen per launch, 1: narrow, 2: wide; see
// fp4root_set_product_tiling); returns the previous value.
int swap_product_tiling(int mode);

struct GemmBf16Args {
  const uint16_t* a;      // bf16 [M][K] per matrix
  const uint16_t* b;      // bf16 [N][K] per matrix
  int64_t a_bstride, b_bstride;
  int64_t M, N, K, batch;
  uint16_t* out16;        // bf16 [M][N] (ld = N)
  int64_t out16_bstride;
  const uint16_t* aux16;  // kModeGramB: bf16 A (may equal out16)
  float cb, cc;
};

// Symmetric BF16 products of the comparison path with FP32 accumulation
// (kModeGramA: X X^T; kModeGramB: b A + c A A^T).
hipError_t launch_gemm_bf16(GemmMode mode, const GemmBf16Args& g, hipStream_t st);

// Update product of the BF16 path through hipBLASLt: X <- a X + B16 Xb for a batch
// (B16 [m][m] bf16 with matrix stride m*m, Xb [m][n] bf16 with stride m*n, X [m][n]
// FP32 with stride x_bstride), FP32 accumulation; ws: ws_bytes of device scratch.
hipError_t launch_bf16_update_blaslt(const uint16_t* b16, const uint16_t* xb, float* x, int64_t batch, int64_t m,
                                     int64_t n, int64_t x_bstride, float a, void* ws, size_t ws_bytes,
                                     hipStream_t st);

// Xb = bf16(X) (round to nearest even) for a batch of m x n FP32 matrices with
// matrix stride x_bstride; Xb contiguous (stride m*n).
hipError_t launch_cast_bf16(const float* x, int64_t batch, int64_t m, int64_t n, int64_t x_bstride,
                            uint16_t* xb, hipStream_t st);

// Zero the amax slots selected by `slot_mask` (bit i = slot i) of n scalar
// records; `full` also resets every tensor scale, tau (+inf) and inv_norm (1).
hipError_t launch_reset_scalars(MatScalars* sc, int64_t n, uint32_t slot_mask, bool full, hipStream_t st);

// out[i] = sc[i].tau (which = 0) or sc[i].sg[slot] (which = 1).
hipError_t launch_export_scalar(const MatScalars* sc, int64_t n, int which, int slot, float* out,
                                hipStream_t st);

}  // namespace fp4r
