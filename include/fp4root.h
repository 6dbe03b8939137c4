/*
 * fp4root -- NVFP4 Newton-Schulz orthogonalisation ("Q-Root") on AMD gfx950.
 *
 * C ABI of libfp4root.so.  Every entry point takes plain pointers and sizes;
 * device pointers are HIP device memory, host pointers are ordinary memory.
 * `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *
 * The method (paper: "Full-Stack FP4", Section 3.4 and its display equation;
 * Section 2 "NVFP4 format" and "Root optimizer"):
 *   - momentum M (rows x cols, FP32) is clipped at its 0.99 quantile of |M|
 *     (Section 3.4 "p99 outlier clipping"; Table 8 "Root quantile ratio 0.99"),
 *     oriented so the short side comes first (X = M^T when rows > cols) and
 *     divided by its Frobenius norm plus eps;
 *   - S Newton-Schulz steps X <- a X + b (X X^T) X + c (X X^T)^2 X run with every
 *     matrix product on NVFP4 operands:
 *         qX = Q1x16(X H), A = qX qX^T, qA = Q1x16(A H),
 *         B = b A + c qA qA^T, qB = Q1x16(B H), qXt = Q16x1(H^T X),
 *         X <- a X + qB qXt
 *     with H a fresh random 16x16 Hadamard transform per step, RTN rounding
 *     and adaptive 4/6 block scaling;
 *   - the result is returned in the input's orientation.
 *
 * NVFP4 tensor layout produced by fp4root_quantize (Section 2 "NVFP4 format"):
 *   codes:  one 4-bit code per element, bit 3 = sign, bits 0-2 = E2M1 magnitude
 *           index into {0, 0.5, 1, 1.5, 2, 3, 4, 6}; two codes per byte, element
 *           2j in the low nibble;
 *   scales: one E4M3FN byte (OCP FP8, bias 7, max 448) per 16-element block;
 *   tensor_scale: one FP32 s_g per matrix; decode x = code * scale * s_g.
 *   The quantiser's readings where the paper is silent: s_g = amax/2688 over the
 *   rotated matrix; block scale E4M3_RNE(min(bmax / (M s_g), 448)) for M = 6, and
 *   also M = 4 with adaptive 4/6 (kept iff its float64 squared error over the
 *   block is strictly smaller); element code E2M1_RNE(min(|u| / (s s_g), 6)).
 *
 * Products are evaluated exactly: each 16-element block product is exact in
 * FP32 and blocks are accumulated in FP64, so each product is the binary32
 * rounding of its (binary64) exact value.
 *
 * Errors: argument, shape and workspace errors are returned synchronously and
 * nothing is launched.  Non-finite input values are detected on the device and
 * recorded in a status word inside the workspace; read it with
 * fp4root_device_status().  The library allocates no device memory: every
 * buffer is the caller's, the workspace included.  Calls are asynchronous with
 * respect to the host; concurrent calls must use distinct workspaces.
 */
#ifndef FP4ROOT_H
#define FP4ROOT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
enum {
  FP4ROOT_OK = 0,
  FP4ROOT_ERR_INVALID_ARG = -1, /* null pointer, bad count, bad flag or parameter */
  FP4ROOT_ERR_SHAPE = -2,       /* a dimension is not a positive multiple of 16 or exceeds 2^21, more than 2^36 elements, or strides too small */
  FP4ROOT_ERR_WORKSPACE = -3,   /* workspace null or smaller than the size query returned */
  FP4ROOT_ERR_NONFINITE = -4,   /* (device status) a NaN or Inf was met in an input */
  FP4ROOT_ERR_HIP = -5,         /* a HIP runtime call failed */
  FP4ROOT_ERR_UNSUPPORTED = -6  /* a combination the library does not implement */
};

/* Flags. */
enum {
  FP4ROOT_F_CLIP = 1u,        /* clip at the clip_quantile of |M| before anything else        */
  FP4ROOT_F_HADAMARD = 2u,    /* apply the random 16x16 Hadamard rotation (Section 3.4)      */
  FP4ROOT_F_ADAPTIVE46 = 4u,  /* adaptive 4/6 block scaling (Section 3.4)                    */
  FP4ROOT_F_BF16_PATH = 8u,   /* plain BF16 Newton-Schulz instead of NVFP4 (comparison path) */
  FP4ROOT_F_STOCHASTIC = 16u, /* stochastic rounding of element codes (momentum state only)  */
  FP4ROOT_F_FP32_ACCUM = 32u, /* NVFP4 products accumulate in binary32 (MFMA order) instead of
                                 exactly; see fp4root_orthogonalize                            */
  FP4ROOT_F_DEFAULT = 7u      /* CLIP | HADAMARD | ADAPTIVE46: the paper's route             */
};

/* One matrix of a batched orthogonalisation.  in/out are device pointers to
 * row-major FP32 matrices of rows x cols with leading dimensions ld_in/ld_out
 * (in elements, >= cols).  in and out may be the same buffer with the same ld. */
typedef struct {
  const float* in;
  float* out;
  int64_t rows, cols, ld_in, ld_out;
} fp4root_matrix;

/* Newton-Schulz configuration (host memory). */
typedef struct {
  int32_t steps;        /* number of NS steps S (>= 0); the paper uses 5 (Section 2)       */
  const float* coeffs;  /* host array of steps*3 floats (a_k, b_k, c_k), or NULL for the
                           library's default table, chosen per matrix by aspect ratio     */
  uint32_t flags;       /* FP4ROOT_F_*                                                     */
  float clip_quantile;  /* quantile ratio q in [0, 1]; the paper's value is 0.99          */
  float eps;            /* Frobenius normalisation guard; 1e-7                             */
  uint64_t seed;        /* seed of the per-step Hadamard signs (SplitMix64 output k+1)     */
} fp4root_ns_config;

/* Optional per-step export of intermediates (device pointers, caller-owned; any
 * member may be NULL to skip it).  Layouts as for fp4root_quantize; A and B are
 * FP32 m x m row-major per matrix, batch stride m*m. */
typedef struct {
  uint8_t *qx_codes, *qx_scales;    float* qx_sg;    /* Q1x16(X H):   m x n/2, m x n/16 */
  uint8_t *qxt_codes, *qxt_scales;  float* qxt_sg;   /* Q16x1(H^T X): n x m/2, n x m/16 */
  float* A;                                          /* qX qX^T                         */
  uint8_t *qa_codes, *qa_scales;    float* qa_sg;    /* Q1x16(A H):   m x m/2, m x m/16 */
  float* B;                                          /* b A + c qA qA^T                 */
  uint8_t *qb_codes, *qb_scales;    float* qb_sg;    /* Q1x16(B H)                      */
} fp4root_ns_trace;

/* ---- size queries (host only, no GPU work) -------------------------------- */

/* Workspace bytes fp4root_quantize needs for this batch (at least 256). */
size_t fp4root_quantize_workspace(int64_t batch, int64_t rows, int64_t cols, uint32_t flags);

/* Workspace bytes fp4root_ns_step needs for a batch of m x n matrices. */
size_t fp4root_ns_step_workspace(int64_t batch, int64_t m, int64_t n, uint32_t flags);

/* Workspace bytes fp4root_orthogonalize needs for this matrix list and config.
 * Returns 0 when the arguments are invalid (the call would fail with an error). */
size_t fp4root_orthogonalize_workspace(const fp4root_matrix* mats, int64_t count,
                                       const fp4root_ns_config* cfg);

/* ---- the three operations ------------------------------------------------- */

/* NVFP4 quantiser (Section 2 "NVFP4 format"; Section 3.4, all quantisations RTN
 * with adaptive 4/6; clipping of Section 3.4 when FP4ROOT_F_CLIP is set).
 *   x:     device, batch matrices of rows x cols FP32, row stride ld, matrix
 *          stride batch_stride (elements);
 *   axis:  1 = blocks of 16 along a row (Q1x16); codes are batch x rows x cols/2
 *          bytes, scales batch x rows x cols/16;
 *          0 = blocks of 16 down a column (Q16x1), stored transposed: codes
 *          batch x cols x rows/2, scales batch x cols x rows/16;
 *   flags: FP4ROOT_F_CLIP | FP4ROOT_F_HADAMARD | FP4ROOT_F_ADAPTIVE46;
 *   clip_quantile: used with FP4ROOT_F_CLIP (threshold per matrix);
 *   seed, step: the Hadamard signs are those of NS step `step` under `seed`;
 *   codes, scales, tensor_scale (batch floats): device outputs;
 *   clip_threshold: optional device output (batch floats) of the thresholds, or NULL.
 * rows and cols must be multiples of 16. */
int fp4root_quantize(const float* x, int64_t batch, int64_t rows, int64_t cols, int64_t ld,
                     int64_t batch_stride, int axis, uint32_t flags, float clip_quantile,
                     uint64_t seed, int32_t step, uint8_t* codes, uint8_t* scales,
                     float* tensor_scale, float* clip_threshold, void* ws, size_t ws_bytes,
                     void* stream);

/* fp4root_quantize without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation).  The same arguments and results as fp4root_quantize; its scratch is
 * a fixed array in the library (about 0.7 MB per GPU, kept until the process ends)
 * that covers up to 256 matrices per call.  A larger batch returns
 * FP4ROOT_ERR_WORKSPACE before any work.
 *   status: optional device int32 that receives 0, or FP4ROOT_ERR_NONFINITE when a
 *           NaN or Inf was seen (the workspace query fp4root_device_status has no
 *           workspace to read here), or NULL.
 * The scratch of the current device is used, so the stream must belong to it.
 * Every call on a GPU shares that GPU's scratch: calls that overlap on one GPU
 * (different streams or threads) race.  No device memory is allocated or freed. */
int fp4root_quantize_noalloc(const float* x, int64_t batch, int64_t rows, int64_t cols, int64_t ld,
                             int64_t batch_stride, int axis, uint32_t flags, float clip_quantile,
                             uint64_t seed, int32_t step, uint8_t* codes, uint8_t* scales,
                             float* tensor_scale, float* clip_threshold, int32_t* status, void* stream);

/* One NVFP4 Newton-Schulz step (Section 3.4 display equation), in place.
 *   x: device, batch matrices m x n FP32, rows contiguous (row stride n), matrix
 *      stride batch_stride >= m*n; any m, n that are multiples of 16 (m <= n is
 *      the efficient orientation: the Gram matrix is m x m);
 *   a, b, c: this step's coefficients; flags: HADAMARD | ADAPTIVE46 | BF16_PATH |
 *   FP32_ACCUM (not with BF16_PATH); seed, step: select the Hadamard signs; trace:
 *   optional export, or NULL. */
int fp4root_ns_step(float* x, int64_t batch, int64_t m, int64_t n, int64_t batch_stride,
                    float a, float b, float c, uint32_t flags, uint64_t seed, int32_t step,
                    const fp4root_ns_trace* trace, void* ws, size_t ws_bytes, void* stream);

/* Batched NVFP4 Root orthogonalisation of `count` matrices (Section 3.4):
 * clip, orient short side first, normalise, cfg->steps NS steps, write back in
 * the input orientation.  Matrices of equal (short, long) shape are batched
 * into the same kernel launches.
 * Products: by default every product of the iteration is the binary32 rounding of
 * its exact value (exact block products chained where provably exact, binary64
 * accumulation), so the result equals the binary64-accumulating reference.  With
 * FP4ROOT_F_FP32_ACCUM (not with FP4ROOT_F_BF16_PATH) each product instead
 * accumulates its exact 16-element block products in one binary32 MFMA accumulator
 * over the whole contraction, as tensor-core NVFP4 products accumulate in FP32: the
 * quantisers are unchanged, each product is within the binary32 accumulation bound
 * of its exact value, and the rounding differences then grow through the
 * re-quantisations of later steps, so the output no longer equals the reference. */
int fp4root_orthogonalize(const fp4root_matrix* mats, int64_t count,
                          const fp4root_ns_config* cfg, void* ws, size_t ws_bytes,
                          void* stream);

/* ---- NVFP4 first-moment state ------------------------------------------------ */

/* Workspace bytes fp4root_momentum_update needs (at least 256), or 0 for a bad shape. */
size_t fp4root_momentum_workspace(int64_t batch, int64_t rows, int64_t cols);

/* One optimizer step of the first moment kept in NVFP4 (Section 3.3: the first
 * moment is stored in NVFP4 after 16-element Hadamard mixing, with stochastic
 * rounding and adaptive 4/6 scaling; Section 2 "AdamW optimizer" for the update
 * m_t = b1 m_{t-1} + (1 - b1) g_t; Section 3.4 feeds m_t to the NVFP4 Root
 * iteration).  For each of `batch` matrices of rows x cols:
 *   1. step > 0: m_hat = decode of the state S_{step-1}: u = fl32(q s s_g), then
 *      the inverse rotation (diag(d) H_16 / 4)^-1 = (H_16 / 4) diag(d) in binary32
 *      (butterfly strides 1, 2, 4, 8, then * 1/4, then the signs) with the signs
 *      of step - 1; step = 0: m_hat = 0 and the state is not read;
 *   2. m_t = fl32(b1 m_hat + b2 g) with b1 = beta, b2 = fl32(1 - beta), the
 *      products exact and their sum rounded once in binary64;
 *   3. m_t is written to `m` (FP32): the input of fp4root_orthogonalize;
 *   4. S_step = the NVFP4 record of m_t along rows, exactly as fp4root_quantize
 *      makes it (axis 1, rotation with the signs of step `step` when
 *      FP4ROOT_F_HADAMARD, 4/6 choice by the round-to-nearest errors when
 *      FP4ROOT_F_ADAPTIVE46), except that with FP4ROOT_F_STOCHASTIC each
 *      magnitude rounds stochastically with the chosen scale r = fl32(s s_g):
 *      with x = |u| / r exact and lo <= x < hi neighbours on the E2M1 grid, it
 *      rounds up to hi iff rho 2^-24 < (x - lo) / (hi - lo) (x >= 6 gives 6,
 *      r = 0 gives 0, the sign bit is kept), rho = 24 bits of SplitMix64 output
 *      floor(e / 2) + 1 of state SplitMix64(seed ^ 0x5352, step + 1) (bits 40..63
 *      for even e, 16..39 for odd e), for the element at flat index
 *      e = (b rows + i) cols + j.
 * Signs d of step t: bit i of SplitMix64 output t + 1 of state `seed` set means
 * d_i = -1 (the rule of the NS steps).
 *   g, m:   device, batch x rows x cols FP32, contiguous (row stride cols, matrix
 *           stride rows*cols), 16-byte aligned; m may equal g;
 *   codes, scales, tensor_scale: device, the state in the layout of
 *           fp4root_quantize (batch x rows x cols/2 bytes, batch x rows x cols/16
 *           bytes, batch floats), read (step > 0) and then overwritten;
 *   beta:   in [0, 1]; flags: FP4ROOT_F_HADAMARD | FP4ROOT_F_ADAPTIVE46 |
 *           FP4ROOT_F_STOCHASTIC; step >= 0.
 * rows and cols must be multiples of 16.  A NaN or Inf in g is recorded in the
 * workspace status (fp4root_device_status). */
int fp4root_momentum_update(const float* g, float* m, int64_t batch, int64_t rows, int64_t cols,
                            uint8_t* codes, uint8_t* scales, float* tensor_scale, float beta,
                            uint32_t flags, uint64_t seed, int32_t step, void* ws, size_t ws_bytes,
                            void* stream);

/* ---- the Root step around the orthogonalisation ------------------------------ */

/* Parameter update with the orthogonalised momentum O as the direction (Section 2
 * "Root optimizer"), decoupled weight decay (training setup: weight decay 0.1) and
 * BF16 master weights (Section 3.3: no FP32 master copy):
 *   W <- bf16(fl32(fl32(W c1) - fl32(c2 O))),  c1 = fl32(1 - fl32(lr wd)),  c2 = fl32(lr scale),
 * bf16() the round-to-nearest-even BF16 of a binary32 value.
 *   w: device BF16 bit patterns, updated in place; o: device FP32; both `count`
 *      contiguous elements, 16-byte aligned; count >= 0 a multiple of 8;
 *   lr, wd, scale: finite. */
int fp4root_apply_update(uint16_t* w, const float* o, int64_t count, float lr, float wd, float scale,
                         void* stream);

/* One parameter of a Root step: device pointers to contiguous row-major rows x cols
 * matrices (16-byte aligned), rows and cols multiples of 16. */
typedef struct {
  uint16_t* w;            /* BF16 weights, updated in place                               */
  const float* g;         /* FP32 gradient                                                */
  float* m;               /* FP32 scratch: receives m_t, then the orthogonalised O        */
  uint8_t* m_codes;       /* first-moment state, layout of fp4root_momentum_update (batch 1) */
  uint8_t* m_scales;
  float* m_tensor_scale;
  int64_t rows, cols;
  float scale;            /* update scale s of this parameter; 0 selects the default
                           * fl32(sqrt(max(1, rows / cols))) (Muon's shape factor)         */
} fp4root_param;

typedef struct {
  float lr, wd, beta;       /* learning rate, decoupled weight decay, first-moment beta1   */
  uint32_t momentum_flags;  /* FP4ROOT_F_HADAMARD | FP4ROOT_F_ADAPTIVE46 | FP4ROOT_F_STOCHASTIC */
  uint64_t momentum_seed;   /* parameter p uses seed momentum_seed + p                      */
  int32_t step;             /* optimizer step t >= 0                                        */
} fp4root_root_config;

/* Workspace bytes fp4root_root_step needs, or 0 for invalid parameters. */
size_t fp4root_root_step_workspace(const fp4root_param* params, int64_t count, const fp4root_ns_config* ns);

/* One Root optimizer step over `count` parameters (host arrays; device buffers):
 * for each parameter p, fp4root_momentum_update of g into m and its state (batch 1,
 * seed momentum_seed + p); then one fp4root_orthogonalize of every m in place with
 * `ns` (the p99 clipping, normalisation and NVFP4 NS steps); then
 * fp4root_apply_update of w with m and the parameter's scale.  A NaN or Inf in a
 * gradient reaches m and is reported by fp4root_device_status(ws): the status word is
 * cleared once per call and kept across the stages.  Every argument of every
 * parameter is checked before the first launch (FP4ROOT_ERR_INVALID_ARG for a null
 * or misaligned pointer, a negative or non-finite scale, ...), so an error leaves
 * all states unchanged. */
int fp4root_root_step(const fp4root_param* params, int64_t count, const fp4root_root_config* rc,
                      const fp4root_ns_config* ns, void* ws, size_t ws_bytes, void* stream);

/* ---- quantized-state AdamW ------------------------------------------------------ */

/* Workspace bytes fp4root_qadamw_update needs for a parameter of n elements, or 0. */
size_t fp4root_qadamw_workspace(int64_t n);

/* One quantized-state AdamW step of a flat parameter of n elements (Section 3.3:
 * both moments stored in NVFP4; Section 2 "AdamW optimizer" moments; BF16 master
 * weights).  n is a positive multiple of 256 (tiles of 256, blocks of 16), at most
 * 2^25, or a multiple of 4096 up to 2^29.
 *   1. the first moment exactly as fp4root_momentum_update on a row-major view with
 *      rows of a multiple of 16 elements (its blocks, draws and codes follow the flat
 *      index, so the view does not change the state); m_t is written to m when m
 *      is not NULL (the step itself does not need it: a second pass re-derives m_t
 *      from g and the previous state to encode the new one)
 *      (flags FP4ROOT_F_HADAMARD | FP4ROOT_F_ADAPTIVE46 | FP4ROOT_F_STOCHASTIC, seed,
 *      step); this step's binary32 m_t is left in m;
 *   2. the second moment: decode of the previous state (step > 0): u = q s (s the
 *      BF16 block scale), the inverse rotation with the signs of step - 1, + the BF16
 *      tile mean, squared (binary32); v_t = fl32(b2 v_hat + fl32(1 - b2) fl32(g g)),
 *      products exact, one binary64 rounding; the new state: y = sqrt(v_t), BF16 tile
 *      mean bf16(fl32(S / 256)) of the binary64 tile sum S (each 16-element block
 *      summed in element order, then the 16 block sums pairwise: a binary tree),
 *      residual fl32(y - mean), rotation with the signs of step, block scale
 *      bf16(fl32(bmax / M)) for M = 6 (and 4 with adaptive 4/6, chosen by the
 *      round-to-nearest binary64 error), E2M1 round-to-nearest codes;
 *   3. W <- bf16(fl32(fl32(W c1) - fl32(lr upd))), c1 = fl32(1 - fl32(lr wd)),
 *      upd = fl32(fl32(m_t / bc1) / fl32(fl32(sqrt(fl32(v_t / bc2))) + eps)),
 *      bc_i = fl32(1 - beta_i^(step+1)) (the power by repeated binary64
 *      multiplication), IEEE division and square root.
 *   w: device BF16 bit patterns [n] (in place); g: device FP32 [n]; m: device FP32
 *   [n] (receives m_t) or NULL, never g (the second pass reads g again); m_codes [n/2], m_scales [n/16], m_tensor_scale [1]: the
 *   first-moment state; v_codes [n/2], v_scales [n/16] (BF16), v_means [n/256]
 *   (BF16): the second-moment state; states are read (step > 0) and overwritten.
 *   All device buffers 16-byte aligned except the state arrays (8-byte codes).
 * A NaN or Inf in g is reported through fp4root_device_status(ws). */
int fp4root_qadamw_update(uint16_t* w, const float* g, float* m, int64_t n, uint8_t* m_codes,
                          uint8_t* m_scales, float* m_tensor_scale, uint8_t* v_codes, uint16_t* v_scales,
                          uint16_t* v_means, float lr, float wd, float beta1, float beta2, float eps,
                          uint32_t flags, uint64_t seed, int32_t step, void* ws, size_t ws_bytes,
                          void* stream);

/* ---- helpers --------------------------------------------------------------- */

/* The library's default per-step coefficients for a rows x cols matrix:
 * writes steps*3 floats to out3 (host).  The paper uses Root's shape-dependent
 * coefficients without printing them; this table is this library's own fit,
 * keyed by the aspect ratio round(long/short) clamped to [1, 4]. */
int fp4root_default_coeffs(int64_t rows, int64_t cols, int32_t steps, float* out3);

/* Waits for `stream`, then returns FP4ROOT_OK or the first device-detected error
 * recorded in the workspace `ws` by the last call that used it. */
int fp4root_device_status(const void* ws, void* stream);

/* Static description of a return code. */
const char* fp4root_status_string(int status);

/* Library version as major*10000 + minor*100 + patch. */
int fp4root_version(void);

/* ---- product tiling (tests and tuning) --------------------------------------
 * The NVFP4 products cover each 128 x 128 output tile with four waves of 64 x 64
 * outputs ("wide") or eight waves of 32 x 64 ("narrow").  By default (mode 0) the
 * Gram of qX and the update product take the wide form for a launch that fills
 * whole rounds of resident workgroups (two per CU) or at least four rounds, the
 * narrow form otherwise; the Gram with the B epilogue always takes the narrow one.
 * Mode 1 forces the narrow form everywhere, mode 2 the wide form for the Gram of
 * qX and the update product.  Every product is exact, so outputs are bit for bit
 * the same in every mode; only the time changes.  The setting is process-wide and
 * applies to launches issued after the call (calls on other threads race with it).
 * Returns the previous mode, or FP4ROOT_ERR_INVALID_ARG for a mode outside 0..2. */
int fp4root_set_product_tiling(int mode);

/* ---- kernel timing for measurement harnesses -------------------------------
 * While enabled, each matrix-product kernel the library launches is bracketed
 * by two HIP events recorded on the stream it is launched on.  Kernel ids:
 * 0 = Gram product A = qX qX^T, 1 = Gram product with the B epilogue,
 * 2 = update product X <- a X + qB qXt^T (for the BF16 path: the same three
 * products on bf16 operands).  Not for production use: recording costs a few
 * microseconds per launch. */
int fp4root_timer_enable(int on);

/* Waits for the recorded launches of `kernel` (-1 = all) and returns their
 * summed kernel time in milliseconds, their number and their algorithmic FLOP
 * (symmetric products: m(m+1)k; others: 2mnk; per matrix). */
int fp4root_timer_read(int kernel, double* ms, int64_t* launches, double* flop);

/* Drops every record (keeps the events for reuse). */
int fp4root_timer_reset(void);

#ifdef __cplusplus
}
#endif

#endif /* FP4ROOT_H */
