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

}  // namespace fp4r
