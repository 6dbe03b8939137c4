// Bandwidth-bound stages of the NVFP4 Newton-Schulz path on gfx950:
// p99 clipping threshold (exact radix select), Frobenius normalisation,
// canonical copies, and the fused rotate + amax / rotate + encode quantiser.
//
// Paper: Section 2 ("NVFP4 format", "Root optimizer"), Section 3.4 (p99
// clipping, NVFP4 NS iteration, RTN + adaptive 4/6), Table 8 (quantile 0.99).
#include "device.h"
#include "internal.h"

namespace fp4r {

// ---------------------------------------------------------------------------
__global__ void k_fill_u32(uint32_t* p, uint32_t v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

hipError_t launch_fill_u32(uint32_t* p, uint32_t value, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(k_fill_u32, dim3((uint32_t)blocks), dim3(256), 0, st, p, value, n);
  return hipGetLastError();
}

FP4R_DEV int find_matrix(const MatChunk& ch, int64_t tile) {
  int mi = 0;
  for (int i = 1; i < ch.count; ++i)
    if (ch.m[i].tile_begin <= tile) mi = i;
  return mi;
}

// ---------------------------------------------------------------------------
// Clip threshold: tau = fl32(v[lo] + f (v[lo+1] - v[lo])) over the sorted |M|,
// found with a three-pass radix select on the binary32 bit patterns (31-bit keys,
// digits of 11, 10 and 10 bits).  Both ranks are tracked in the same passes.
//
// The last pass can also give the Frobenius norm of clamp(M, tau): by then the
// 21-bit key prefixes p0 <= p1 of v[lo] and v[lo+1] are known, tau lies between
// the two, and no element lies strictly between them, so an element whose prefix
// is below p0 is not clipped (its square goes into a binary64 partial of the
// block), one above p1 is clipped to tau (it is only counted), and the elements
// with prefix p0 or p1 are exactly the pass's histograms (a key is the bit
// pattern of |x|), which the select step sums in bin order once tau is known.

__global__ void k_clip_init(MatChunk ch, MatScalars* sc) {
  const int i = threadIdx.x;
  if (i >= ch.count) return;
  const MatDesc& d = ch.m[i];
  const int64_t n = d.rows * d.cols;
  MatScalars& s = sc[i];
  s.sel_prefix[0] = s.sel_prefix[1] = 0;
  s.sel_rank[0] = (uint32_t)d.lo;
  s.sel_rank[1] = (uint32_t)(d.lo + 1 < n ? d.lo + 1 : d.lo);
}

__global__ __launch_bounds__(256) void k_radix_hist(MatChunk ch, const MatScalars* sc,
                                                    uint32_t* hist, uint32_t* status, int pass,
                                                    double* psum, uint32_t* pcnt) {
  __shared__ uint32_t h[2][kHistBins];
  __shared__ double red[256];
  __shared__ uint32_t above_all;
  for (int i = threadIdx.x; i < 2 * kHistBins; i += 256) (&h[0][0])[i] = 0;
  __syncthreads();
  const int64_t tile = blockIdx.x;
  const int mi = find_matrix(ch, tile);
  const MatDesc& d = ch.m[mi];
  const int64_t r0 = (tile - d.tile_begin) * kPrepRowsPerBlock;
  const int64_t r1 = r0 + kPrepRowsPerBlock < d.rows ? r0 + kPrepRowsPerBlock : d.rows;
  const uint32_t p0 = sc[mi].sel_prefix[0], p1 = sc[mi].sel_prefix[1];
  const bool two = pass > 0 && p0 != p1;
  const int pshift = pass == 1 ? 20 : 10;
  const bool norm = pass == 2 && psum != nullptr;
  double acc = 0.0;     // squares of the elements below prefix p0, in this thread's order
  uint32_t above = 0;   // elements above prefix p1
  if (threadIdx.x == 0) above_all = 0;
  bool bad = false;
  // The block's rows as one sequence of 16-byte quads (row r, quad c), thread t taking
  // quads t, t + 256, ...; four loads are issued before any is used.
  const uint32_t c4 = (uint32_t)(d.cols / 4);
  const uint32_t nq = (uint32_t)(r1 - r0) * c4;
  uint32_t rr = threadIdx.x / c4, cc = threadIdx.x - rr * c4;   // position of quad threadIdx.x
  auto step = [&]() {   // advance by 256 quads
    cc += 256u;
    while (cc >= c4) {
      cc -= c4;
      ++rr;
    }
  };
  for (uint32_t q0 = threadIdx.x; q0 < nq; q0 += 1024u) {
    float4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      v[u] = q0 + 256u * u < nq ? reinterpret_cast<const float4*>(d.in + (r0 + rr) * d.ld_in)[cc]
                                : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      step();
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (q0 + 256u * u >= nq) break;
      const float e[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t key = __float_as_uint(e[j]) & 0x7FFFFFFFu;
        if (key >= 0x7F800000u) { bad = true; continue; }
        uint32_t digit;
        if (pass == 0) {
          atomicAdd(&h[0][key >> 20], 1u);
          continue;
        }
        digit = pass == 1 ? ((key >> 10) & 1023u) : (key & 1023u);
        const uint32_t pre = key >> pshift;
        if (pre == p0) atomicAdd(&h[0][digit], 1u);
        if (two && pre == p1) atomicAdd(&h[1][digit], 1u);
        if (norm) {
          if (pre < p0) {
            const double x = (double)e[j];
            acc = acc + x * x;
          } else if (pre > p1) {
            ++above;
          }
        }
      }
    }
  }
  if (bad) atomicOr(status, kStatusNonFinite);
  if (norm) {
    red[threadIdx.x] = acc;
    if (above) atomicAdd(&above_all, above);
  }
  __syncthreads();
  if (norm) {
    for (int off = 128; off > 0; off >>= 1) {   // fixed-order tree
      if ((int)threadIdx.x < off) red[threadIdx.x] = red[threadIdx.x] + red[threadIdx.x + off];
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      psum[tile] = red[0];
      pcnt[tile] = above_all;
    }
  }
  const int nb = pass == 0 ? 2048 : 1024;
  for (int b = threadIdx.x; b < nb; b += 256) {
    if (h[0][b]) atomicAdd(&hist[(mi * 2 + 0) * kHistBins + b], h[0][b]);
    if (two && h[1][b]) atomicAdd(&hist[(mi * 2 + 1) * kHistBins + b], h[1][b]);
  }
}

__global__ __launch_bounds__(256) void k_radix_select(MatChunk ch, MatScalars* sc, uint32_t* hist,
                                                      int pass, const double* psum, const uint32_t* pcnt,
                                                      float eps) {
  __shared__ uint32_t part[256];
  __shared__ uint32_t found_prefix[2], found_rank[2];
  __shared__ double red[256];
  __shared__ unsigned long long above_all;
  const int mi = blockIdx.x;
  const int t = threadIdx.x;
  MatScalars& s = sc[mi];
  const int nb = pass == 0 ? 2048 : 1024;
  const int per = nb / 256;
  const bool two = pass > 0 && s.sel_prefix[0] != s.sel_prefix[1];
  for (int rr = 0; rr < 2; ++rr) {
    const uint32_t* hh = hist + (mi * 2 + (two ? rr : 0)) * kHistBins;
    uint32_t local = 0;
    for (int j = 0; j < per; ++j) local += hh[t * per + j];
    part[t] = local;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {   // inclusive Hillis-Steele scan
      const uint32_t add = t >= off ? part[t - off] : 0u;
      __syncthreads();
      part[t] += add;
      __syncthreads();
    }
    const uint32_t incl = part[t];
    const uint32_t excl = incl - local;
    const uint32_t target = s.sel_rank[rr];
    if (target >= excl && target < incl) {   // exactly one thread owns the target rank
      uint32_t cum = excl;
      for (int j = 0; j < per; ++j) {
        const uint32_t c = hh[t * per + j];
        if (target < cum + c) {
          const uint32_t bin = (uint32_t)(t * per + j);
          found_prefix[rr] = pass == 0 ? bin : ((s.sel_prefix[rr] << 10) | bin);
          found_rank[rr] = target - cum;
          break;
        }
        cum += c;
      }
    }
    __syncthreads();
  }
  if (pass == 2 && psum) {
    // ||clamp(M, tau)||^2 in a fixed order: the blocks' partials below p0, the
    // elements of the two prefixes from the histograms (bin order), the elements
    // above p1 at tau^2 each
    const MatDesc& d = ch.m[mi];
    const double v0 = (double)__uint_as_float(found_prefix[0]);
    const double v1 = (double)__uint_as_float(found_prefix[1]);
    const float tau = (float)__dadd_rn(v0, __dmul_rn(d.frac, __dsub_rn(v1, v0)));
    if (t == 0) above_all = 0;
    const int64_t nt = (d.rows + kPrepRowsPerBlock - 1) / kPrepRowsPerBlock;
    double below = 0.0;
    unsigned long long above = 0;
    for (int64_t i = t; i < nt; i += 256) {
      below = below + psum[d.tile_begin + i];
      above += pcnt[d.tile_begin + i];
    }
    double cand = 0.0;
    for (int rr = 0; rr < (two ? 2 : 1); ++rr) {
      const uint32_t* hh = hist + (mi * 2 + rr) * kHistBins;
      for (int j = 0; j < 4; ++j) {
        const uint32_t bin = (uint32_t)(4 * t + j), c = hh[bin];
        if (c) {
          const double x = (double)fminf(__uint_as_float((s.sel_prefix[rr] << 10) | bin), tau);
          cand = cand + (double)c * (x * x);
        }
      }
    }
    __syncthreads();
    atomicAdd(&above_all, above);
    red[t] = below;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
      if (t < off) red[t] = red[t] + red[t + off];
      __syncthreads();
    }
    const double sum_below = red[0];
    __syncthreads();
    red[t] = cand;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
      if (t < off) red[t] = red[t] + red[t + off];
      __syncthreads();
    }
    if (t == 0) {
      const double tt = (double)tau * (double)tau;
      const double total = __dadd_rn(__dadd_rn(sum_below, red[0]), __dmul_rn((double)above_all, tt));
      const double nu = __dsqrt_rn(total);
      s.inv_norm = (float)__ddiv_rn(1.0, __dadd_rn(nu, (double)eps));
    }
    __syncthreads();
  }
  for (int b = t; b < 2 * kHistBins; b += 256) hist[mi * 2 * kHistBins + b] = 0u;
  if (t == 0) {
    s.sel_prefix[0] = found_prefix[0];
    s.sel_prefix[1] = found_prefix[1];
    s.sel_rank[0] = found_rank[0];
    s.sel_rank[1] = found_rank[1];
    if (pass == 2) {
      const double v0 = (double)__uint_as_float(found_prefix[0]);
      const double v1 = (double)__uint_as_float(found_prefix[1]);
      const double f = ch.m[mi].frac;
      s.tau = (float)__dadd_rn(v0, __dmul_rn(f, __dsub_rn(v1, v0)));
    }
  }
}

hipError_t launch_clip_threshold(const MatChunk& ch, MatScalars* sc, uint32_t* hist,
                                 uint32_t* status, hipStream_t st, double* psum, uint32_t* pcnt,
                                 float eps) {
  hipError_t e = launch_fill_u32(hist, 0u, (int64_t)ch.count * 2 * kHistBins, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_clip_init, dim3(1), dim3(kMaxChunk), 0, st, ch, sc);
  for (int pass = 0; pass < 3; ++pass) {
    hipLaunchKernelGGL(k_radix_hist, dim3((uint32_t)ch.total_tiles), dim3(256), 0, st, ch, sc,
                       hist, status, pass, psum, pcnt);
    hipLaunchKernelGGL(k_radix_select, dim3(ch.count), dim3(256), 0, st, ch, sc, hist, pass,
                       (const double*)psum, (const uint32_t*)pcnt, eps);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Frobenius norm of clamp(M, tau): per-block binary64 partials in a fixed
// order, then one fixed-order sum per matrix (deterministic).

__global__ __launch_bounds__(256) void k_sumsq(MatChunk ch, const MatScalars* sc, double* partial,
                                               uint32_t* status) {
  __shared__ double red[256];
  const int64_t tile = blockIdx.x;
  const int mi = find_matrix(ch, tile);
  const MatDesc& d = ch.m[mi];
  const float tau = sc[mi].tau;
  const int64_t r0 = (tile - d.tile_begin) * kPrepRowsPerBlock;
  const int64_t r1 = r0 + kPrepRowsPerBlock < d.rows ? r0 + kPrepRowsPerBlock : d.rows;
  double acc = 0.0;
  bool bad = false;   // a NaN or infinite entry (the clamp would hide a NaN)
  for (int64_t r = r0; r < r1; ++r) {
    const float4* row = reinterpret_cast<const float4*>(d.in + r * d.ld_in);
    for (int64_t c = threadIdx.x; c < d.cols / 4; c += 256) {
      const float4 v = row[c];
      const float e[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        bad |= !(fabsf(e[j]) <= 3.40282347e38f);
        const double x = (double)fminf(fmaxf(e[j], -tau), tau);
        acc = acc + x * x;
      }
    }
  }
  if (__builtin_amdgcn_ballot_w64(bad) != 0 && (threadIdx.x & 63) == 0) atomicOr(status, kStatusNonFinite);
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off) red[threadIdx.x] = red[threadIdx.x] + red[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[tile] = red[0];
}

__global__ __launch_bounds__(256) void k_norm_final(MatChunk ch, MatScalars* sc, const double* partial,
                                                    float eps) {
  __shared__ double red[256];
  const int mi = blockIdx.x;
  const MatDesc& d = ch.m[mi];
  const int64_t nt = (d.rows + kPrepRowsPerBlock - 1) / kPrepRowsPerBlock;
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < nt; i += 256) acc = acc + partial[d.tile_begin + i];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off) red[threadIdx.x] = red[threadIdx.x] + red[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double nu = __dsqrt_rn(red[0]);
    sc[mi].inv_norm = (float)__ddiv_rn(1.0, __dadd_rn(nu, (double)eps));
  }
}

// The status code of a call (0, or FP4ROOT_ERR_NONFINITE = -4 when a NaN or Inf
// was seen) from its device status word, into a caller's device word.
__global__ void k_status_out(const uint32_t* status, int32_t* out) {
  if (threadIdx.x == 0) *out = (*status & kStatusNonFinite) ? -4 : 0;
}

hipError_t launch_status_out(const uint32_t* status, int32_t* out, hipStream_t st) {
  hipLaunchKernelGGL(k_status_out, dim3(1), dim3(64), 0, st, status, out);
  return hipGetLastError();
}

hipError_t launch_inv_norm(const MatChunk& ch, MatScalars* sc, double* partial, float eps,
                           uint32_t* status, hipStream_t st) {
  hipLaunchKernelGGL(k_sumsq, dim3((uint32_t)ch.total_tiles), dim3(256), 0, st, ch, sc, partial, status);
  hipLaunchKernelGGL(k_norm_final, dim3(ch.count), dim3(256), 0, st, ch, sc, partial, eps);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Tiled copies through LDS (64 x 64 tiles, coalesced on both sides).

constexpr int kT = 64;

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Block-wide max of non-negative floats; thread 0 returns the result.
FP4R_DEV float block_max_256(float v, float* red) {
  v = warp_max(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

// Prep: canonical X = fl32(clamp(M) * inv) (transposed when rows > cols), staged
// through a 64 x 64 LDS tile that also yields the amaxes of X rotated along n
// (16-column blocks) and along m (16-row blocks) for the first NS step.
__global__ __launch_bounds__(256) void k_prep_copy(MatChunk ch, MatScalars* sc, float* xbase,
                                                   int64_t x_bstride, uint32_t mask, int rotate,
                                                   int slot_n, int slot_m) {
  __shared__ float tile[kT][kT + 1];
  __shared__ float red[4];
  const int64_t t = blockIdx.x;
  const int mi = find_matrix(ch, t);
  const MatDesc& d = ch.m[mi];
  const bool tall = d.rows > d.cols;
  const int64_t xm = tall ? d.cols : d.rows, xn = tall ? d.rows : d.cols;   // canonical m x n
  const uint32_t tcols = (uint32_t)cdiv(xn, kT), tt = (uint32_t)(t - d.tile_begin);
  const int64_t xr0 = (int64_t)(tt / tcols) * kT, xc0 = (int64_t)(tt % tcols) * kT;   // canonical tile origin
  float* X = xbase + (int64_t)mi * x_bstride;
  const float tau = sc[mi].tau;
  const float inv = sc[mi].inv_norm;
  // tile[i][j] = canonical X[xr0 + i][xc0 + j]; 16-byte accesses of M and X (rows of
  // both are 16-byte aligned and m, n are multiples of 16): thread -> four quads
  // v = threadIdx.x + 256 k, row v / 16 of the tile, columns 4 (v % 16) .. + 3
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int v = (int)threadIdx.x + 256 * k, i = v >> 4, q = v & 15;
    if (!tall) {
      const int64_t r = xr0 + i, c = xc0 + 4 * q;
      if (r < xm && c < xn) {
        float4 a = *reinterpret_cast<const float4*>(d.in + r * d.ld_in + c);
        a.x = fminf(fmaxf(a.x, -tau), tau) * inv;
        a.y = fminf(fmaxf(a.y, -tau), tau) * inv;
        a.z = fminf(fmaxf(a.z, -tau), tau) * inv;
        a.w = fminf(fmaxf(a.w, -tau), tau) * inv;
        *reinterpret_cast<float4*>(X + r * xn + c) = a;
        tile[i][4 * q] = a.x; tile[i][4 * q + 1] = a.y; tile[i][4 * q + 2] = a.z; tile[i][4 * q + 3] = a.w;
      }
    } else {
      // M row xc0 + i, M columns xr0 + 4q .. + 3  ->  X rows xr0 + 4q .. + 3, column xc0 + i
      const int64_t r = xc0 + i, c = xr0 + 4 * q;
      if (r < d.rows && c < d.cols) {
        const float4 a = *reinterpret_cast<const float4*>(d.in + r * d.ld_in + c);
        tile[4 * q][i] = fminf(fmaxf(a.x, -tau), tau) * inv;
        tile[4 * q + 1][i] = fminf(fmaxf(a.y, -tau), tau) * inv;
        tile[4 * q + 2][i] = fminf(fmaxf(a.z, -tau), tau) * inv;
        tile[4 * q + 3][i] = fminf(fmaxf(a.w, -tau), tau) * inv;
      }
    }
  }
  __syncthreads();
  if (tall) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int v = (int)threadIdx.x + 256 * k, i = v >> 4, q = v & 15;
      const int64_t r = xr0 + i, c = xc0 + 4 * q;
      if (r < xm && c < xn)
        *reinterpret_cast<float4*>(X + r * xn + c) =
            make_float4(tile[i][4 * q], tile[i][4 * q + 1], tile[i][4 * q + 2], tile[i][4 * q + 3]);
    }
  }
  // rotated amaxes: thread -> one 16-column block and one 16-row block of the tile
  float mr = 0.0f, mc = 0.0f;
  {
    const int i = threadIdx.x >> 2, b = threadIdx.x & 3;
    if (xr0 + i < xm && xc0 + 16 * b < xn) {
      float u[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) u[k] = tile[i][16 * b + k];
      if (rotate) {
        mr = 0.25f * rot16_absmax4(u, mask);
      } else {
#pragma unroll
        for (int k = 0; k < 16; ++k) mr = fmaxf(mr, fabsf(u[k]));
      }
    }
  }
  {
    const int j = threadIdx.x & 63, b = threadIdx.x >> 6;
    if (xc0 + j < xn && xr0 + 16 * b < xm) {
      float u[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) u[k] = tile[16 * b + k][j];
      if (rotate) {
        mc = 0.25f * rot16_absmax4(u, mask);
      } else {
#pragma unroll
        for (int k = 0; k < 16; ++k) mc = fmaxf(mc, fabsf(u[k]));
      }
    }
  }
  const float br = block_max_256(mr, red);
  __syncthreads();
  const float bc = block_max_256(mc, red);
  if (threadIdx.x == 0) {
    amax_record(&sc[mi], slot_n, blockIdx.x, br);
    amax_record(&sc[mi], slot_m, blockIdx.x, bc);
  }
}

// Copy-out: caller M (rows x cols) from canonical X (transposed back when tall).
__global__ __launch_bounds__(256) void k_copy_out(MatChunk ch, const float* xbase, int64_t x_bstride) {
  __shared__ float tile[kT][kT + 1];
  const int64_t t = blockIdx.x;
  const int mi = find_matrix(ch, t);
  const MatDesc& d = ch.m[mi];
  const bool tall = d.rows > d.cols;
  const uint32_t tcols = (uint32_t)cdiv(d.cols, kT), tt = (uint32_t)(t - d.tile_begin);
  const int64_t br = (int64_t)(tt / tcols) * kT, bc = (int64_t)(tt % tcols) * kT;   // tile origin in M coordinates
  const float* X = xbase + (int64_t)mi * x_bstride;
  const int64_t xld = tall ? d.rows : d.cols;
  // 16-byte accesses (see k_prep_copy): thread -> quads v = threadIdx.x + 256 k,
  // row v / 16 of the tile, columns 4 (v % 16) .. + 3
  if (!tall) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int v = (int)threadIdx.x + 256 * k, i = v >> 4, q = v & 15;
      const int64_t r = br + i, c = bc + 4 * q;
      if (r < d.rows && c < d.cols)
        *reinterpret_cast<float4*>(d.out + r * d.ld_out + c) = *reinterpret_cast<const float4*>(X + r * xld + c);
    }
    return;
  }
  // X row bc + i, X columns br + 4q .. + 3  ->  M rows br + 4q .. + 3, column bc + i
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int v = (int)threadIdx.x + 256 * k, i = v >> 4, q = v & 15;
    const int64_t c = bc + i, r = br + 4 * q;
    if (r < d.rows && c < d.cols) {
      const float4 a = *reinterpret_cast<const float4*>(X + c * xld + r);
      tile[4 * q][i] = a.x; tile[4 * q + 1][i] = a.y; tile[4 * q + 2][i] = a.z; tile[4 * q + 3][i] = a.w;
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int v = (int)threadIdx.x + 256 * k, i = v >> 4, q = v & 15;
    const int64_t r = br + i, c = bc + 4 * q;
    if (r < d.rows && c < d.cols)
      *reinterpret_cast<float4*>(d.out + r * d.ld_out + c) =
          make_float4(tile[i][4 * q], tile[i][4 * q + 1], tile[i][4 * q + 2], tile[i][4 * q + 3]);
  }
}

hipError_t launch_prep_copy(const MatChunk& ch, MatScalars* sc, float* x, int64_t x_bstride,
                            uint32_t mask, bool rotate, int slot_n, int slot_m, hipStream_t st) {
  hipLaunchKernelGGL(k_prep_copy, dim3((uint32_t)ch.total_tiles), dim3(256), 0, st, ch, sc, x,
                     x_bstride, mask, (int)rotate, slot_n, slot_m);
  return hipGetLastError();
}

hipError_t launch_copy_out(const MatChunk& ch, const float* x, int64_t x_bstride, hipStream_t st) {
  hipLaunchKernelGGL(k_copy_out, dim3((uint32_t)ch.total_tiles), dim3(256), 0, st, ch, x, x_bstride);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// The rotation ahead of the quantiser: with a tensor scale of at least 2^-40 the
// factor 1/4 is left to the quantiser's scales (returns kf = 4, see quant_block);
// otherwise the block is rotated in full (kf = 1).
FP4R_DEV float rotate_for_quant(float (&u)[16], uint32_t mask, int rotate, float sg) {
  if (!rotate) return 1.0f;
  hadamard16(u, mask);
  if (sg >= 0x1p-40f) return 4.0f;
  quarter16(u);
  return 1.0f;
}

// Quantiser: one thread per 16-element block.  Axis 1: blocks along a row,
// consecutive threads take consecutive blocks of a row (contiguous 64-byte
// reads).  Axis 0: blocks down a column, consecutive threads take consecutive
// columns (each of the 16 loads is a contiguous 256-byte wave access).

template <int AXIS>
FP4R_DEV void block_pos(const Batch& in, int64_t g, int64_t& r, int64_t& c) {
  if (AXIS == 1) {
    const int64_t nbr = in.cols / 16;
    r = g / nbr;
    c = (g % nbr) * 16;
  } else {
    c = g % in.cols;
    r = (g / in.cols) * 16;
  }
}

template <int AXIS>
FP4R_DEV bool load_block_at(const Batch& in, int64_t b, int64_t r, int64_t c, float (&u)[16]) {
  const float* x = in.x + b * in.bstride;
  if (AXIS == 1) {
    const float4* p = reinterpret_cast<const float4*>(x + r * in.ld + c);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 v = p[q];
      u[4 * q] = v.x; u[4 * q + 1] = v.y; u[4 * q + 2] = v.z; u[4 * q + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) u[i] = x[(r + i) * in.ld + c];
  }
  bool ok = true;
#pragma unroll
  for (int i = 0; i < 16; ++i) ok = ok && ((__float_as_uint(u[i]) & 0x7F800000u) != 0x7F800000u);
  return ok;
}

template <int AXIS>
__global__ __launch_bounds__(256) void k_amax(Batch in, uint32_t mask, int rotate, int clip,
                                              MatScalars* sc, int slot, uint32_t* status) {
  __shared__ float red[4];
  const int64_t b = blockIdx.y;
  const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t nblk = in.rows * in.cols / 16;
  float m = 0.0f;
  if (g < nblk) {
    float u[16];
    int64_t r, c;
    block_pos<AXIS>(in, g, r, c);
    const bool ok = load_block_at<AXIS>(in, b, r, c, u);
    if (!ok) atomicOr(status, kStatusNonFinite);
    if (clip) {
      const float tau = sc[b].tau;
#pragma unroll
      for (int i = 0; i < 16; ++i) u[i] = fminf(fmaxf(u[i], -tau), tau);
    }
    if (rotate) {
      m = 0.25f * rot16_absmax4(u, mask);
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) m = fmaxf(m, fabsf(u[i]));
    }
    if (!ok) m = 0.0f;
  }
  m = warp_max(m);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    const float mm = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    amax_record(&sc[b], slot, blockIdx.x, mm);
  }
}

// E2M1 magnitude of index 0..7 (the hardware decode of the code, exact).
FP4R_DEV double e2m1_grid(uint32_t idx) {
  return (double)__builtin_bit_cast(float2, __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(idx, 1.0f, 0)).x;
}

// Stochastic rounding of one block's magnitudes (the first-moment state; see
// fp4root_momentum_update): u holds kf times the rotated block, `scale` is the
// chosen E4M3 code and `rtn` the round-to-nearest codes with that scale; element
// e0 + i takes 24 bits of SplitMix64 output (e0 + i) / 2 + 1 of `key` (two elements
// per output, see below).  With x = |u| / r exact
// (r = fl32(s s_g)), the floor grid point of x is the nearest one or the one
// below it (the round-to-nearest quotient is within one ulp of x), and
// rho (hi - lo) r < (|u| - lo r) 2^24 is exact in binary64 (every term has at
// most 48 significant bits; |u| - lo r is a difference of numbers within a factor 2).
FP4R_DEV uint64_t sr_block_codes(const float (&u)[16], float kf, uint32_t scale, float sg, uint64_t rtn,
                                 uint64_t key, uint64_t e0) {
  const float r = e4m3_value(scale) * sg;
  if (!(r > 0.0f)) return rtn & 0x8888888888888888ull;   // magnitudes 0, signs kept
  const double rd = (double)r;
  // element e0 + i takes 24 bits of SplitMix64 output (e0 + i) / 2 + 1 (e0 is even):
  // bits 40..63 for even i, bits 16..39 for odd i
  const uint64_t z0 = key + 0x9E3779B97F4A7C15ull * (e0 / 2 + 1);
  uint64_t zk = 0;
  uint64_t out = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    if ((i & 1) == 0) zk = splitmix64_mix(z0 + 0x9E3779B97F4A7C15ull * (uint64_t)(i / 2));
    const float ui = kf == 1.0f ? u[i] : u[i] * 0.25f;
    const double a = (double)fabsf(ui);
    const uint32_t c = (uint32_t)(rtn >> (4 * i)) & 15u;
    uint32_t idx = c & 7u;
    double lo = e2m1_grid(idx);
    if (idx > 0 && lo * rd > a) {
      --idx;
      lo = e2m1_grid(idx);
    }
    if (idx < 7) {
      const double hi = e2m1_grid(idx + 1);
      const uint32_t rho = (uint32_t)(zk >> ((i & 1) ? 16 : 40)) & 0xFFFFFFu;
      if ((double)rho * (hi - lo) * rd < (a - lo * rd) * 16777216.0) ++idx;
    }
    out |= (uint64_t)((c & 8u) | idx) << (4 * i);
  }
  return out;
}

template <int AXIS, bool SR = false>
__global__ __launch_bounds__(256) void k_encode(Batch in, uint32_t mask, int rotate, int clip,
                                                int adaptive, MatScalars* sc, int slot, QOut out,
                                                float* tensor_scale, uint64_t sr_key = 0) {
  const int64_t b = blockIdx.y;
  const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t nblk = in.rows * in.cols / 16;
  const float sg = tensor_scale_from_amax(amax_read(sc[b], slot));
  if (g == 0) {
    sc[b].sg[slot] = sg;
    if (tensor_scale) tensor_scale[b] = sg;
  }
  // With chain records (axis 1, cols a multiple of 64) each wave takes 16 rows x
  // one 64-column stage: lane 4i + k holds block k of row i, so the stage bound
  // of a row and the record over the 16 rows reduce within the wave.
  const bool want_rho = AXIS == 1 && out.rhog != nullptr;
  if (g >= nblk) return;   // nblk is a multiple of 64 when records are requested: whole waves leave
  int64_t r = 0, c = 0;
  if (want_rho) {
    // the wave index is uniform (waves never straddle a 256-thread group), so the
    // division by the stage count is scalar work
    const uint32_t nst = (uint32_t)(in.cols / 64);
    const uint32_t wv = __builtin_amdgcn_readfirstlane((uint32_t)(g >> 6));
    const uint32_t rg = wv / nst, st = wv - rg * nst;
    const int lane = (int)(threadIdx.x & 63);
    r = (int64_t)rg * 16 + (lane >> 2);
    c = ((int64_t)st * 4 + (lane & 3)) * 16;
  } else {
    block_pos<AXIS>(in, g, r, c);
  }
  {
    float u[16];
    load_block_at<AXIS>(in, b, r, c, u);
    if (clip) {
      const float tau = sc[b].tau;
#pragma unroll
      for (int i = 0; i < 16; ++i) u[i] = fminf(fmaxf(u[i], -tau), tau);
    }
    const float kf = rotate_for_quant(u, mask, rotate, sg);
    uint32_t scale;
    uint64_t codes;
    uint32_t n2;
    quant_block(u, sg, adaptive != 0, scale, codes, n2, want_rho, kf);
    if constexpr (SR)
      codes = sr_block_codes(u, kf, scale, sg, codes, sr_key, (uint64_t)((b * in.rows + r) * in.cols + c));
    if (want_rho) {
      const float rho = wave_max_pos(quad_stage_rho(n2, block_exp(scale)));
      if ((threadIdx.x & 63) == 0)
        out.rhog[b * out.rhog_bstride + (r / 16) * (in.cols / 64) + c / 64] = rho;
    }
    int64_t code_off, scale_off;
    if (AXIS == 1 && out.tiled) {   // stage-major: [cols/64][rows][32 B], [cols/64][rows][4 B]
      code_off = ((c / 64) * in.rows + r) * 32 + (c % 64) / 2;
      scale_off = ((c / 64) * in.rows + r) * 4 + (c % 64) / 16;
    } else if (AXIS == 1) {   // [rows][cols/2], [rows][cols/16]
      code_off = r * (in.cols / 2) + c / 2;
      scale_off = r * (in.cols / 16) + c / 16;
    } else {           // transposed: [cols][rows/2], [cols][rows/16]
      code_off = c * (in.rows / 2) + r / 2;
      scale_off = c * (in.rows / 16) + r / 16;
    }
    *reinterpret_cast<uint2*>(out.codes + b * out.codes_bstride + code_off) =
        make_uint2((uint32_t)codes, (uint32_t)(codes >> 32));
    out.scales[b * out.scales_bstride + scale_off] = (uint8_t)scale;
  }
}

// Both quantisations of X from one read: a 64 x 64 tile is staged in LDS; each
// thread encodes one 16-column block (qX, along n) and one 16-row block (qXt,
// along m, written transposed).
// Eight waves per SIMD (64 VGPRs and 24 bytes of scratch per lane) rather than the
// six its 73 registers would allow: the extra waves cover part of its LDS and
// memory waits (about 2.5 % less time per launch).
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(8))) void k_encode_x2(const float* x, int64_t m, int64_t n, int64_t x_bstride,
                                                   uint32_t mask, int rotate, int adaptive, MatScalars* sc,
                                                   int slot_n, int slot_m, QOut qx, QOut qxt, uint32_t reset_mask) {
  // rows padded to 68 floats: 16-byte row slices for the row blocks.  gfx950 serves
  // a 128-bit LDS read 16 lanes per cycle over 64 banks and a 128-bit write 8 lanes
  // per cycle over 32 banks: the 16 lanes of one read (4 rows x 4 slices) and 64
  // consecutive columns of one row fall in distinct banks, and so do the 8 lanes of
  // one write (2 rows x 4 slices) because lanes with bit 1 of q set store their
  // four slices in the order k ^ 2
  __shared__ __align__(16) float tile[kT][kT + 4];
  const int64_t b = blockIdx.y;
  const uint32_t tn = (uint32_t)cdiv(n, kT);   // tiles per row of tiles (grid.x < 2^32)
  const int64_t r0 = (int64_t)(blockIdx.x / tn) * kT, c0 = (int64_t)(blockIdx.x % tn) * kT;
  const float* X = x + b * x_bstride;
  const float sgn = tensor_scale_from_amax(amax_read(sc[b], slot_n));
  const float sgm = tensor_scale_from_amax(amax_read(sc[b], slot_m));
  if (blockIdx.x == 0) {
    if (threadIdx.x == 0) {
      sc[b].sg[slot_n] = sgn;
      sc[b].sg[slot_m] = sgm;
    }
    // amax slots the next kernels record into (this kernel reads only slot_n, slot_m)
    if (threadIdx.x < kAmaxSpread * kNumSlots) {
      const int line = (int)threadIdx.x / kNumSlots, slot = (int)threadIdx.x % kNumSlots;
      if ((reset_mask >> slot) & 1u) sc[b].amax[line].v[slot] = 0u;
    }
  }
  {
    const int i = threadIdx.x >> 2, q = threadIdx.x & 3;   // row i, 16 columns at 16 q
    if (r0 + i < m && c0 + 16 * q < n) {
      const float4* p = reinterpret_cast<const float4*>(X + (r0 + i) * n + c0 + 16 * q);
      float4* t = reinterpret_cast<float4*>(&tile[i][16 * q]);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int kk = k ^ (q & 2);
        t[kk] = p[kk];
      }
    }
  }
  __syncthreads();
  {
    const int i = threadIdx.x >> 2, q = threadIdx.x & 3;
    const int64_t r = r0 + i, c = c0 + 16 * q;
    uint32_t n2 = 0, e = 15;
    if (r < m && c < n) {
      float u[16];
      const float4* t = reinterpret_cast<const float4*>(&tile[i][16 * q]);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float4 v = t[k];
        u[4 * k] = v.x; u[4 * k + 1] = v.y; u[4 * k + 2] = v.z; u[4 * k + 3] = v.w;
      }
      const float kf = rotate_for_quant(u, mask, rotate, sgn);
      uint32_t scale;
      uint64_t codes;
      quant_block(u, sgn, adaptive != 0, scale, codes, n2, qx.rhog != nullptr, kf);
      e = block_exp(scale);
      const int64_t oc = qx.tiled ? ((c0 / 64) * m + r) * 32 + 8 * q : r * (n / 2) + c / 2;
      const int64_t os = qx.tiled ? ((c0 / 64) * m + r) * 4 + q : r * (n / 16) + c / 16;
      *reinterpret_cast<uint2*>(qx.codes + b * qx.codes_bstride + oc) = make_uint2((uint32_t)codes, (uint32_t)(codes >> 32));
      qx.scales[b * qx.scales_bstride + os] = (uint8_t)scale;
    }
    // chain record of this wave's 16 rows for the tile's 64-column stage: lanes
    // 4i .. 4i + 3 hold row i's four blocks (blocks past the edge count as zero)
    if (qx.rhog) {
      const float rho = wave_max_pos(quad_stage_rho(n2, e));
      if ((threadIdx.x & 63) == 0 && r0 + 16 * (threadIdx.x >> 6) < m)
        qx.rhog[b * qx.rhog_bstride + ((r0 / 16) + (threadIdx.x >> 6)) * (n / 64) + c0 / 64] = rho;
    }
  }
  {
    const int j = threadIdx.x & 63, q = threadIdx.x >> 6;   // column j, 16 rows at 16 q
    const int64_t c = c0 + j, r = r0 + 16 * q;
    uint32_t n2 = 0, e = 15;
    if (r < m && c < n) {
      float u[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) u[k] = tile[16 * q + k][j];
      const float kf = rotate_for_quant(u, mask, rotate, sgm);
      uint32_t scale;
      uint64_t codes;
      quant_block(u, sgm, adaptive != 0, scale, codes, n2, qxt.rhog != nullptr, kf);
      e = block_exp(scale);
      const int64_t oc = qxt.tiled ? ((r0 / 64) * n + c) * 32 + 8 * q : c * (m / 2) + r / 2;
      const int64_t os = qxt.tiled ? ((r0 / 64) * n + c) * 4 + q : c * (m / 16) + r / 16;
      *reinterpret_cast<uint2*>(qxt.codes + b * qxt.codes_bstride + oc) = make_uint2((uint32_t)codes, (uint32_t)(codes >> 32));
      qxt.scales[b * qxt.scales_bstride + os] = (uint8_t)scale;
    }
    if (qxt.rhog) {
      // the stage's four blocks of column j sit in the four waves: exchange in LDS
      // (the tile is no longer read once every thread has passed the barrier),
      // then wave 0 reduces each 16 columns (16 rows of qXt) to a record
      __syncthreads();
      uint32_t* xn = reinterpret_cast<uint32_t*>(&tile[0][0]);
      xn[q * 64 + j] = n2;
      xn[256 + q * 64 + j] = e;
      __syncthreads();
      if (q == 0) {
        uint32_t qn[4], qe[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          qn[k] = xn[k * 64 + j];
          qe[k] = xn[256 + k * 64 + j];
        }
        const float rho = row16_max_pos(stage_rho(qn, qe));
        if ((j & 15) == 0 && c < n)
          qxt.rhog[b * qxt.rhog_bstride + (c / 16) * (m / 64) + r0 / 64] = rho;
      }
    }
  }
}

// One thread per (row, stage) of a matrix: 32 code bytes and 4 scale bytes from the
// stage-major layout to the row-major one (a last partial stage copies its blocks only).
__global__ __launch_bounds__(256) void k_untile_nvfp4(const uint8_t* codes, const uint8_t* scales, int64_t rows,
                                                       int64_t K, uint8_t* out_codes, uint8_t* out_scales) {
  const int64_t b = blockIdx.y;
  const int64_t nst = (K + 63) / 64;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= rows * nst) return;
  const int64_t st = t / rows, r = t % rows;
  const int nb = (int)(K / 16 - 4 * st < 4 ? K / 16 - 4 * st : 4);   // blocks in this stage
  const uint8_t* sc = codes + b * tiled_code_bytes(rows, K) + (st * rows + r) * 32;
  const uint8_t* ss = scales + b * tiled_scale_bytes(rows, K) + (st * rows + r) * 4;
  uint8_t* dc = out_codes ? out_codes + b * rows * (K / 2) + r * (K / 2) + st * 32 : nullptr;
  uint8_t* ds = out_scales ? out_scales + b * rows * (K / 16) + r * (K / 16) + st * 4 : nullptr;
  for (int k = 0; k < nb; ++k) {
    if (out_codes) *reinterpret_cast<uint2*>(dc + 8 * k) = *reinterpret_cast<const uint2*>(sc + 8 * k);
    if (out_scales) ds[k] = ss[k];
  }
}

hipError_t launch_untile_nvfp4(const uint8_t* codes, const uint8_t* scales, int64_t batch, int64_t rows,
                               int64_t K, uint8_t* out_codes, uint8_t* out_scales, hipStream_t st) {
  const int64_t n = rows * ((K + 63) / 64);
  if (n == 0 || batch == 0) return hipSuccess;
  if (K % 16 != 0) return hipErrorInvalidValue;
  const dim3 grid((uint32_t)((n + 255) / 256), (uint32_t)batch);
  hipLaunchKernelGGL(k_untile_nvfp4, grid, dim3(256), 0, st, codes, scales, rows, K, out_codes, out_scales);
  return hipGetLastError();
}

hipError_t launch_encode_x2(const float* x, int64_t batch, int64_t m, int64_t n, int64_t x_bstride,
                            uint32_t sign_mask, bool rotate, bool adaptive46, MatScalars* sc,
                            int slot_n, int slot_m, const QOut& qx, const QOut& qxt, hipStream_t st,
                            uint32_t reset_mask) {
  if (reset_mask & ((1u << slot_n) | (1u << slot_m))) return hipErrorInvalidValue;
  const dim3 grid((uint32_t)(cdiv(m, kT) * cdiv(n, kT)), (uint32_t)batch);
  hipLaunchKernelGGL(k_encode_x2, grid, dim3(256), 0, st, x, m, n, x_bstride, sign_mask, (int)rotate,
                     (int)adaptive46, sc, slot_n, slot_m, qx, qxt, reset_mask);
  return hipGetLastError();
}

hipError_t launch_amax(const Batch& in, int axis, uint32_t sign_mask, bool rotate, bool clip,
                       MatScalars* sc, int slot, uint32_t* status, hipStream_t st) {
  const int64_t nblk = in.rows * in.cols / 16;
  const dim3 grid((uint32_t)((nblk + 255) / 256), (uint32_t)in.batch);
  if (axis == 1)
    hipLaunchKernelGGL(k_amax<1>, grid, dim3(256), 0, st, in, sign_mask, (int)rotate, (int)clip, sc,
                       slot, status);
  else
    hipLaunchKernelGGL(k_amax<0>, grid, dim3(256), 0, st, in, sign_mask, (int)rotate, (int)clip, sc,
                       slot, status);
  return hipGetLastError();
}

hipError_t launch_encode(const Batch& in, int axis, uint32_t sign_mask, bool rotate, bool clip,
                         bool adaptive46, MatScalars* sc, int slot, const QOut& out,
                         float* tensor_scale, hipStream_t st) {
  // chain records: row blocks over whole 64-column stages; the stage-major layout: row blocks
  if (out.rhog && (axis != 1 || in.cols % 64 != 0 || in.rows % 16 != 0)) return hipErrorInvalidValue;
  if (out.tiled && axis != 1) return hipErrorInvalidValue;
  const int64_t nblk = in.rows * in.cols / 16;
  const dim3 grid((uint32_t)((nblk + 255) / 256), (uint32_t)in.batch);
  if (axis == 1)
    hipLaunchKernelGGL((k_encode<1, false>), grid, dim3(256), 0, st, in, sign_mask, (int)rotate, (int)clip,
                       (int)adaptive46, sc, slot, out, tensor_scale, (uint64_t)0);
  else
    hipLaunchKernelGGL((k_encode<0, false>), grid, dim3(256), 0, st, in, sign_mask, (int)rotate, (int)clip,
                       (int)adaptive46, sc, slot, out, tensor_scale, (uint64_t)0);
  return hipGetLastError();
}

hipError_t launch_encode_sr(const Batch& in, uint32_t sign_mask, bool rotate, bool adaptive46,
                            MatScalars* sc, int slot, const QOut& out, float* tensor_scale,
                            uint64_t sr_key, hipStream_t st) {
  if (out.rhog) return hipErrorInvalidValue;
  const int64_t nblk = in.rows * in.cols / 16;
  const dim3 grid((uint32_t)((nblk + 255) / 256), (uint32_t)in.batch);
  hipLaunchKernelGGL((k_encode<1, true>), grid, dim3(256), 0, st, in, sign_mask, (int)rotate, 0,
                     (int)adaptive46, sc, slot, out, tensor_scale, sr_key);
  return hipGetLastError();
}


// ---------------------------------------------------------------------------
// First-moment update: one thread per 16-element row block of a contiguous
// matrix.  Decodes the previous NVFP4 state (one rounding of q s s_g, then the
// inverse rotation), forms m = fl32(b1 m_hat + b2 g) (exact products, one binary64
// rounding, then binary32), writes m and records the amax of m rotated with
// `mask` (the tensor scale of the next state) in amax slot 0.
__global__ __launch_bounds__(256) void k_mom_update(const float* g, float* m, int64_t rows, int64_t cols,
                                                    const uint8_t* codes, const uint8_t* scales,
                                                    const float* prev_sg, int has_prev, uint32_t prev_mask,
                                                    uint32_t mask, int rotate, float b1, float b2,
                                                    MatScalars* sc, uint32_t* status) {
  __shared__ float red[4];
  const int64_t b = blockIdx.y;
  const int64_t blk = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t nblk = rows * cols / 16;
  float amax = 0.0f;
  if (blk < nblk) {
    const int64_t e0 = b * rows * cols + blk * 16;
    float x[16];
    const float4* gp = reinterpret_cast<const float4*>(g + e0);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 v = gp[q];
      x[4 * q] = v.x; x[4 * q + 1] = v.y; x[4 * q + 2] = v.z; x[4 * q + 3] = v.w;
    }
    bool ok = true;
#pragma unroll
    for (int i = 0; i < 16; ++i) ok = ok && ((__float_as_uint(x[i]) & 0x7F800000u) != 0x7F800000u);
    if (!ok) atomicOr(status, kStatusNonFinite);
    float mv[16];
    mom_block(x, codes, scales, e0, has_prev ? prev_sg[b] : 0.0f, has_prev, prev_mask, rotate, b1, b2, mv);
    float4* mp = reinterpret_cast<float4*>(m + e0);
#pragma unroll
    for (int q = 0; q < 4; ++q) mp[q] = make_float4(mv[4 * q], mv[4 * q + 1], mv[4 * q + 2], mv[4 * q + 3]);
    if (rotate) {
      amax = 0.25f * rot16_absmax4(mv, mask);
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) amax = fmaxf(amax, fabsf(mv[i]));
    }
    if (!ok) amax = 0.0f;
  }
  amax = warp_max(amax);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
  __syncthreads();
  if (threadIdx.x == 0) {
    const float mm = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    amax_record(&sc[b], 0, blockIdx.x, mm);
  }
}

// Re-encode the first moment of a flat parameter (batch 1, n elements) in place,
// recomputing m_t = fl32(b1 decode(old state) + b2 g) exactly as mom_block does:
// the quantized-state AdamW step's second pass (its first pass recorded the rotated
// amax of m_t in slot 0 and saved the previous tensor scale in sg[kSlotPrevState]).
// Each thread reads and writes only its own block of the state.
template <bool SR>
__global__ __launch_bounds__(256) void k_mom_encode(const float* g, uint8_t* codes, uint8_t* scales,
                                                    int64_t nblk, int has_prev, uint32_t prev_mask,
                                                    uint32_t mask, int rotate, int adaptive, float b1, float b2,
                                                    MatScalars* sc, float* tensor_scale, uint64_t sr_key) {
  const int64_t blk = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const float sg = tensor_scale_from_amax(amax_read(sc[0], 0));
  if (blk == 0) {
    sc[0].sg[0] = sg;
    tensor_scale[0] = sg;
  }
  if (blk >= nblk) return;
  const int64_t e0 = blk * 16;
  float x[16];
  const float4* gp = reinterpret_cast<const float4*>(g + e0);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 v = gp[q];
    x[4 * q] = v.x; x[4 * q + 1] = v.y; x[4 * q + 2] = v.z; x[4 * q + 3] = v.w;
  }
  float u[16];
  mom_block(x, codes, scales, e0, sc[0].sg[kSlotPrevState], has_prev != 0, prev_mask, rotate != 0, b1, b2, u);
  const float kf = rotate_for_quant(u, mask, rotate, sg);
  uint32_t scale, n2;
  uint64_t c;
  quant_block(u, sg, adaptive != 0, scale, c, n2, false, kf);
  if constexpr (SR) c = sr_block_codes(u, kf, scale, sg, c, sr_key, (uint64_t)e0);
  *reinterpret_cast<uint2*>(codes + e0 / 2) = make_uint2((uint32_t)c, (uint32_t)(c >> 32));
  scales[blk] = (uint8_t)scale;
}

hipError_t launch_mom_encode(const float* g, uint8_t* codes, uint8_t* scales, int64_t n, bool has_prev,
                             uint32_t prev_mask, uint32_t mask, bool rotate, bool adaptive, bool sr, float b1,
                             float b2, MatScalars* sc, float* tensor_scale, uint64_t sr_key, hipStream_t st) {
  const int64_t nblk = n / 16;
  const dim3 grid((uint32_t)((nblk + 255) / 256));
  if (sr)
    hipLaunchKernelGGL(k_mom_encode<true>, grid, dim3(256), 0, st, g, codes, scales, nblk, (int)has_prev, prev_mask,
                       mask, (int)rotate, (int)adaptive, b1, b2, sc, tensor_scale, sr_key);
  else
    hipLaunchKernelGGL(k_mom_encode<false>, grid, dim3(256), 0, st, g, codes, scales, nblk, (int)has_prev, prev_mask,
                       mask, (int)rotate, (int)adaptive, b1, b2, sc, tensor_scale, sr_key);
  return hipGetLastError();
}

hipError_t launch_mom_update(const float* g, float* m, int64_t batch, int64_t rows, int64_t cols,
                             const uint8_t* codes, const uint8_t* scales, const float* prev_sg,
                             bool has_prev, uint32_t prev_mask, uint32_t mask, bool rotate, float b1,
                             float b2, MatScalars* sc, uint32_t* status, hipStream_t st) {
  const int64_t nblk = rows * cols / 16;
  const dim3 grid((uint32_t)((nblk + 255) / 256), (uint32_t)batch);
  hipLaunchKernelGGL(k_mom_update, grid, dim3(256), 0, st, g, m, rows, cols, codes, scales, prev_sg,
                     (int)has_prev, prev_mask, mask, (int)rotate, b1, b2, sc, status);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// BF16 comparison path: Xb = bf16(X) and Xbt = bf16(X)^T (round to nearest even).


// Xb = bf16(X): four elements per thread, 16-byte reads and 8-byte writes.
__global__ __launch_bounds__(256) void k_cast_bf16(const float* x, int64_t mn, int64_t x_bstride, uint16_t* xb) {
  const int64_t b = blockIdx.y;
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i >= mn) return;
  const float4 v = *reinterpret_cast<const float4*>(x + b * x_bstride + i);
  uint2 o;
  o.x = (uint32_t)bf16_rne(v.x) | ((uint32_t)bf16_rne(v.y) << 16);
  o.y = (uint32_t)bf16_rne(v.z) | ((uint32_t)bf16_rne(v.w) << 16);
  *reinterpret_cast<uint2*>(xb + b * mn + i) = o;
}

hipError_t launch_cast_bf16(const float* x, int64_t batch, int64_t m, int64_t n, int64_t x_bstride,
                            uint16_t* xb, hipStream_t st) {
  // rows are contiguous with row stride n, so each matrix is m*n consecutive floats
  // (m*n and x_bstride are multiples of 4)
  const int64_t mn = m * n;
  if (batch == 0 || mn == 0) return hipSuccess;
  const dim3 grid((uint32_t)((mn / 4 + 255) / 256), (uint32_t)batch);
  hipLaunchKernelGGL(k_cast_bf16, grid, dim3(256), 0, st, x, mn, x_bstride, xb);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Small per-matrix scalar kernels.

__global__ void k_reset_scalars(MatScalars* sc, int64_t n, uint32_t slot_mask, int full) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  MatScalars& s = sc[i];
#pragma unroll
  for (int k = 0; k < kNumSlots; ++k)
    if ((slot_mask >> k) & 1u)
#pragma unroll
      for (int l = 0; l < kAmaxSpread; ++l) s.amax[l].v[k] = 0u;
  if (full) {
#pragma unroll
    for (int k = 0; k < kNumSlots; ++k) s.sg[k] = 0.0f;
    s.tau = __uint_as_float(0x7F800000u);   // +inf: clamping is the identity
    s.inv_norm = 1.0f;
  }
}

hipError_t launch_reset_scalars(MatScalars* sc, int64_t n, uint32_t slot_mask, bool full, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_reset_scalars, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, st, sc, n,
                     slot_mask, (int)full);
  return hipGetLastError();
}

__global__ void k_export_scalar(const MatScalars* sc, int64_t n, int which, int slot, float* out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  out[i] = which == 0 ? sc[i].tau : sc[i].sg[slot];
}

hipError_t launch_export_scalar(const MatScalars* sc, int64_t n, int which, int slot, float* out,
                                hipStream_t st) {
  if (n <= 0 || !out) return hipSuccess;
  hipLaunchKernelGGL(k_export_scalar, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, st, sc, n,
                     which, slot, out);
  return hipGetLastError();
}

}  // namespace fp4r
