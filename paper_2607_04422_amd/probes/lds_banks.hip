// LDS bank-conflict calibration for gfx950: known 16-byte access patterns, one
// kernel each, for reading the SQ_LDS_BANK_CONFLICT counter against
// SQ_INSTS_LDS.  Standalone program (not part of the library):
//
//   hipcc --offload-arch=gfx950 -O3 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       paper_2607_04422_amd/probes/lds_banks.hip -o lds_banks
//   rocprofv3 --pmc SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT --output-format csv -d OUT -o run -- ./lds_banks
//
// Patterns, as the 16-byte slot index of each lane l (slot s at byte 16 s):
//   reads   R0: s = l             R1: s = 2 l
//   writes  W0: s = l             W1: s = 2 l
//           W2: s = (l & 7) + 16 (l >> 3)        W3: s = 16 (l & 3) + (l >> 2)
//   the product kernel's decode stores (row t / 4, block t % 4 of thread t, both
//   16-byte halves) with the earlier block offsets {0, 128, 272, 400} bytes (W4)
//   and the current ones {0, 16, 64, 80} (W5).
// What the counter showed: R0, W0, W2 and W5 conflict-free; R1 3.9 conflict
// cycles per instruction; W1 and W4 8.0; W3 24.0.  So reads are served 16 lanes
// per cycle over 64 banks (slot mod 16) and writes 8 lanes per cycle over 32
// banks (slot mod 8).  Every access stays inside the 64 KiB dynamic LDS block.
#include <hip/hip_runtime.h>

#include <cstdio>

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
constexpr int kLdsBytes = 64 * 1024;
constexpr int kIters = 1024;

__device__ __forceinline__ int decode_store_off(int t, int half, bool current) {
  const int r = t >> 2, kb = t & 3;
  const int base = current ? 32 * 128 * kb + 16 * ((kb & 1) + 4 * (kb >> 1)) : 32 * 128 * kb + 128 * kb + 16 * (kb >> 1);
  return base + r * 32 + ((half ^ ((r >> 2) & 1) ^ ((r >> 3) & 1)) << 4);
}

// byte offset of lane l (thread t of the block) for pattern P; below 32 KiB
__device__ __forceinline__ int pattern_off(int P, int t, int it) {
  const int l = t & 63, w = t >> 6;
  switch (P) {
    case 0: return 1024 * w + 16 * l;
    case 1: return 2048 * w + 32 * l;
    case 2: return 4096 * w + 16 * ((l & 7) + 16 * (l >> 3));
    case 3: return 4096 * w + 16 * (16 * (l & 3) + (l >> 2));
    case 4: return decode_store_off(t, it & 1, false);
    default: return decode_store_off(t, it & 1, true);
  }
}

template <int P>
__global__ __launch_bounds__(512) void k_read(float* out) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  for (int i = threadIdx.x; i < kLdsBytes / 4; i += 512) reinterpret_cast<float*>(lds)[i] = (float)i;
  __syncthreads();
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int it = 0; it < kIters; ++it) {
    acc += *reinterpret_cast<const f32x4*>(lds + pattern_off(P, threadIdx.x, it));
    asm volatile("" ::: "memory");
  }
  out[blockIdx.x * 512 + threadIdx.x] = acc[0] + acc[1] + acc[2] + acc[3];
}

template <int P>
__global__ __launch_bounds__(512) void k_write(float* out) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  f32x4 v = {(float)threadIdx.x, 1.0f, 2.0f, 3.0f};
  for (int it = 0; it < kIters; ++it) {
    *reinterpret_cast<f32x4*>(lds + pattern_off(P, threadIdx.x, it)) = v;
    v[0] += 1.0f;
    asm volatile("" ::: "memory");
  }
  __syncthreads();
  out[blockIdx.x * 512 + threadIdx.x] = reinterpret_cast<const float*>(lds)[threadIdx.x];
}

template <typename K>
bool launch(K kernel, float* out, int blocks) {
  if (hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes) != hipSuccess)
    return false;
  hipLaunchKernelGGL(kernel, dim3(blocks), dim3(512), kLdsBytes, 0, out);
  return hipDeviceSynchronize() == hipSuccess;
}

}  // namespace

int main() {
  const int blocks = 512;
  float* out = nullptr;
  if (hipMalloc(&out, (size_t)blocks * 512 * sizeof(float)) != hipSuccess) return 1;
  const bool ok = launch(k_read<0>, out, blocks) && launch(k_read<1>, out, blocks) && launch(k_write<0>, out, blocks) &&
                  launch(k_write<1>, out, blocks) && launch(k_write<2>, out, blocks) &&
                  launch(k_write<3>, out, blocks) && launch(k_write<4>, out, blocks) && launch(k_write<5>, out, blocks);
  (void)hipFree(out);
  std::printf("lds_banks %s\n", ok ? "done" : "failed");
  return ok ? 0 : 2;
}
