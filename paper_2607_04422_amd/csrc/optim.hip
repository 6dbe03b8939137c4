// The parameter update around the orthogonalised momentum (Section 2 "Root
// optimizer"; weight decay of the training setup; BF16 master weights, Section 3.3).
//   W <- bf16(fl32(fl32(W c1) - fl32(c2 O))),  c1 = fl32(1 - fl32(lr wd)),  c2 = fl32(lr s)
// HBM-bound: 2 B (W) + 4 B (O) read and 2 B (W) written per element; each thread
// moves eight elements with 16-byte accesses.
#include "device.h"
#include "internal.h"

namespace fp4r {

__global__ __launch_bounds__(256) void k_apply_update(uint16_t* w, const float* o, int64_t n8, float c1,
                                                      float c2) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n8; i += stride) {
    const uint4 wv = reinterpret_cast<const uint4*>(w)[i];
    const float4 o0 = reinterpret_cast<const float4*>(o)[2 * i];
    const float4 o1 = reinterpret_cast<const float4*>(o)[2 * i + 1];
    const float ov[8] = {o0.x, o0.y, o0.z, o0.w, o1.x, o1.y, o1.z, o1.w};
    const uint32_t ww[4] = {wv.x, wv.y, wv.z, wv.w};
    uint32_t out[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float w0 = __uint_as_float(ww[k] << 16), w1 = __uint_as_float(ww[k] & 0xFFFF0000u);
      const float a0 = w0 * c1, b0 = c2 * ov[2 * k];
      const float a1 = w1 * c1, b1 = c2 * ov[2 * k + 1];
      out[k] = (uint32_t)bf16_rne(a0 - b0) | ((uint32_t)bf16_rne(a1 - b1) << 16);
    }
    reinterpret_cast<uint4*>(w)[i] = make_uint4(out[0], out[1], out[2], out[3]);
  }
}

hipError_t launch_apply_update(uint16_t* w, const float* o, int64_t count, float c1, float c2, hipStream_t st) {
  const int64_t n8 = count / 8;
  if (n8 <= 0) return hipSuccess;
  const int64_t blocks = (n8 + 255) / 256;
  const uint32_t grid = (uint32_t)(blocks < (1 << 20) ? blocks : (1 << 20));
  hipLaunchKernelGGL(k_apply_update, dim3(grid), dim3(256), 0, st, w, o, n8, c1, c2);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Quantized-state AdamW (Section 3.3; Section 2 "AdamW optimizer" moments), first
// pass.  One thread per 16-element block of a flat parameter, so a row of 16 lanes
// holds one 256-element tile (the parameter length is a multiple of 256 and lanes
// past the end form whole rows, which compute on a clamped block and store nothing).
// Per block: this step's first moment m_t from the previous first-moment state and
// g (mom_block; its rotated amax goes to amax slot 0 for the second pass, which
// re-derives m_t and encodes it); decode the previous second-moment state (u = q s, the inverse
// rotation, + tile mean, squared), v_t = fl32(b2 v_hat + c2 fl32(g g)) (exact
// products, one binary64 rounding), y = sqrt(v_t); the tile sum of y in binary64
// (each block in element order, then the 16 block sums pairwise by DPP
// butterflies: lanes l, l^1, then l^2, then the mirrored half and the mirrored
// row, each partner sum formed identically in both lanes); the BF16 tile mean,
// the residual, the rotation and the BF16-scale quantiser; then the AdamW update
// of the BF16 weights from this step's binary32 m_t and v_t.
template <int CTRL>
FP4R_DEV double dpp_d(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = dpp_u<CTRL>((uint32_t)b), hi = dpp_u<CTRL>((uint32_t)(b >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

struct QAdamWArgs {
  uint16_t* w;
  const float* g;
  float* m_out;            // optional: this step's binary32 first moment
  const uint8_t* mcodes;   // previous first-moment state (read only here)
  const uint8_t* mscales;
  const float* m_prev_sg;
  float b1, c1m;
  MatScalars* sc;
  uint8_t* vcodes;         // [N/2]
  uint16_t* vscales;       // [N/16] BF16
  uint16_t* vmeans;        // [N/256] BF16
  int64_t nblk;
  int has_prev, rotate, adaptive;
  uint32_t prev_mask, mask;
  float b2, c2, bc1, bc2, eps, lr, c1w;
  uint32_t* status;
};

__global__ __launch_bounds__(256) void k_qadamw(QAdamWArgs a) {
  __shared__ float red[4];
  const int64_t blk0 = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const bool live = blk0 < a.nblk;
  const int64_t blk = live ? blk0 : a.nblk - 1;
  const int64_t e0 = blk * 16;
  const float m_prev_sg = a.has_prev ? a.m_prev_sg[0] : 0.0f;
  if (blk0 == 0) a.sc->sg[kSlotPrevState] = m_prev_sg;   // for the second pass
  float g[16], m[16], vh[16];
  {
    const float4* gp = reinterpret_cast<const float4*>(a.g + e0);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 x = gp[q];
      g[4 * q] = x.x; g[4 * q + 1] = x.y; g[4 * q + 2] = x.z; g[4 * q + 3] = x.w;
    }
  }
  bool ok = true;
#pragma unroll
  for (int i = 0; i < 16; ++i) ok = ok && ((__float_as_uint(g[i]) & 0x7F800000u) != 0x7F800000u);
  if (live && !ok) atomicOr(a.status, kStatusNonFinite);
  // this step's first moment, and the rotated amax of it for the second pass
  mom_block(g, a.mcodes, a.mscales, e0, m_prev_sg, a.has_prev != 0, a.prev_mask, a.rotate != 0, a.b1, a.c1m, m);
  if (live && a.m_out) {
    float4* mo = reinterpret_cast<float4*>(a.m_out + e0);
#pragma unroll
    for (int q = 0; q < 4; ++q) mo[q] = make_float4(m[4 * q], m[4 * q + 1], m[4 * q + 2], m[4 * q + 3]);
  }
  {
    float amax = 0.0f;
    if (a.rotate) {
      float t[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) t[i] = m[i];
      amax = 0.25f * rot16_absmax4(t, a.mask);
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) amax = fmaxf(amax, fabsf(m[i]));
    }
    if (!live || !ok) amax = 0.0f;
    amax = warp_max(amax);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
    __syncthreads();
    if (threadIdx.x == 0)
      amax_record(a.sc, 0, blockIdx.x, fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3])));
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) vh[i] = 0.0f;
  if (a.has_prev) {
    const uint2 cw = *reinterpret_cast<const uint2*>(a.vcodes + e0 / 2);
    const float s = bf16_value(a.vscales[blk]);
    const float mu = bf16_value(a.vmeans[blk >> 4]);
    const uint32_t wd[2] = {cw.x, cw.y};
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      float2 q;
      switch (k & 3) {
        case 0: q = __builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd[k >> 2], 1.0f, 0)); break;
        case 1: q = __builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd[k >> 2], 1.0f, 1)); break;
        case 2: q = __builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd[k >> 2], 1.0f, 2)); break;
        default: q = __builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd[k >> 2], 1.0f, 3)); break;
      }
      vh[2 * k] = q.x * s;          // exact
      vh[2 * k + 1] = q.y * s;
    }
    if (a.rotate) unrotate16(vh, a.prev_mask);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float y = vh[i] + mu;
      vh[i] = y * y;
    }
  }
  float v[16], y[16];
  double bs = 0.0;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const float gg = g[i] * g[i];
    v[i] = (float)__builtin_fma((double)a.b2, (double)vh[i], (double)a.c2 * (double)gg);
    y[i] = __builtin_sqrtf(v[i]);
    bs += (double)y[i];
  }
  bs = bs + dpp_d<0xB1>(bs);    // lanes l, l ^ 1
  bs = bs + dpp_d<0x4E>(bs);    // l ^ 2
  bs = bs + dpp_d<0x141>(bs);   // the other quad of the half-row
  bs = bs + dpp_d<0x140>(bs);   // the other half of the row
  const uint32_t mu_bits = bf16_rne((float)(bs * (1.0 / 256.0)));
  const float mu = bf16_value(mu_bits);
  float u[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) u[i] = y[i] - mu;
  if (a.rotate) rotate16(u, a.mask);
  uint32_t sbits;
  uint64_t codes;
  quant_block_bf16(u, a.adaptive != 0, sbits, codes);
  // AdamW on the BF16 weights with this step's moments
  const uint4* wp = reinterpret_cast<const uint4*>(a.w + e0);
  const uint4 w0 = wp[0], w1 = wp[1];
  const uint32_t ww[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
  uint32_t out[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    uint32_t pair = 0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int i = 2 * k + h;
      const float wv = __uint_as_float(h ? (ww[k] & 0xFFFF0000u) : (ww[k] << 16));
      const float mh = m[i] / a.bc1;
      const float den = __builtin_sqrtf(v[i] / a.bc2) + a.eps;
      const float upd = mh / den;
      const float t0 = wv * a.c1w, t1 = a.lr * upd;
      pair |= (uint32_t)bf16_rne(t0 - t1) << (16 * h);
    }
    out[k] = pair;
  }
  if (live) {
    uint4* wo = reinterpret_cast<uint4*>(a.w + e0);
    wo[0] = make_uint4(out[0], out[1], out[2], out[3]);
    wo[1] = make_uint4(out[4], out[5], out[6], out[7]);
    *reinterpret_cast<uint2*>(a.vcodes + e0 / 2) = make_uint2((uint32_t)codes, (uint32_t)(codes >> 32));
    a.vscales[blk] = (uint16_t)sbits;
    if ((blk & 15) == 0) a.vmeans[blk >> 4] = (uint16_t)mu_bits;
  }
}

hipError_t launch_qadamw(const QAdamWLaunch& p, hipStream_t st) {
  QAdamWArgs a;
  a.w = p.w; a.g = p.g; a.m_out = p.m_out; a.mcodes = p.mcodes; a.mscales = p.mscales; a.m_prev_sg = p.m_prev_sg;
  a.b1 = p.b1; a.c1m = p.c1m; a.sc = p.sc;
  a.vcodes = p.vcodes; a.vscales = p.vscales; a.vmeans = p.vmeans;
  a.nblk = p.n / 16;
  a.has_prev = p.has_prev; a.rotate = p.rotate; a.adaptive = p.adaptive;
  a.prev_mask = p.prev_mask; a.mask = p.mask;
  a.b2 = p.b2; a.c2 = p.c2; a.bc1 = p.bc1; a.bc2 = p.bc2; a.eps = p.eps; a.lr = p.lr; a.c1w = p.c1w;
  a.status = p.status;
  if (a.nblk <= 0) return hipSuccess;
  const dim3 grid((uint32_t)((a.nblk + 255) / 256));
  hipLaunchKernelGGL(k_qadamw, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace fp4r
