// Inner loops of the two NVFP4 -> MFMA bridge candidates on gfx950, registers only
// (no memory traffic, no decode), timed as kernels.  Standalone program (not part of
// the library):
//
//   hipcc --offload-arch=gfx950 -O3 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       paper_2607_04422_amd/probes/bridge_candidates.hip -o bridge_candidates
//   rocprofv3 --kernel-trace --stats --output-format csv -d OUT -o run -- ./bridge_candidates
//
// Every wave owns two 32x32 output tiles (as the product kernels do) and runs kStages
// 64-element stages of four 16-element NVFP4 blocks:
//   k_f16_only        f16 MFMA 32x32x16 per block, chained over the whole loop (the MFMA
//                     roofline of this loop shape: no fold, not exact);
//   k_f16_fold<false> the library's bridge: f16 MFMA per block, blocks of a stage chained
//                     in one binary32 register, folded into binary64 once per stage;
//   k_f16_fold<true>  the same with a binary64 fold after every block (a stage whose chain
//                     bound fails);
//   k_fp4<true>       the second candidate: the FP4 MFMA 32x32x64 (E8M0 scales at 1.0) on
//                     one 16-element block padded to 64 with zero codes, then the block sum
//                     times s_a s_b added to an FP32 accumulator (one multiply for the
//                     per-row scale product and one fma per output and block);
//   k_fp4<false>      the padded FP4 MFMA alone, chained.
// Useful work per block and tile is 2 x 32 x 32 x 16 FLOP in every kernel.  Operands are
// kept in registers and marked as changing every block, so no MFMA is hoisted.
#include <hip/hip_runtime.h>

#include <cstdio>

namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

constexpr int kStages = 1024;
constexpr int kThreads = 512;

template <typename T>
__device__ __forceinline__ void touch(T& v) {
  asm volatile("" : "+v"(v));
}

__device__ __forceinline__ float fold_out(const double (&acc)[2][16]) {
  double s = 0.0;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[t][e];
  return (float)s;
}

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void k_f16_only(float* out) {
  f16x8 a, b0, b1;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (_Float16)(float)((threadIdx.x + e) & 7);
    b0[e] = (_Float16)(float)((threadIdx.x * 3 + e) & 7);
    b1[e] = (_Float16)(float)((threadIdx.x * 5 + e) & 7);
  }
  f32x16 p0 = {}, p1 = {};
  for (int s = 0; s < kStages; ++s) {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      touch(a);
      touch(b0);
      touch(b1);
      p0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b0, p0, 0, 0, 0);
      p1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b1, p1, 0, 0, 0);
    }
  }
  float r = 0.0f;
#pragma unroll
  for (int e = 0; e < 16; ++e) r += p0[e] + p1[e];
  out[blockIdx.x * kThreads + threadIdx.x] = r;
}

template <bool PER_BLOCK>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void k_f16_fold(float* out) {
  f16x8 a, b0, b1;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (_Float16)(float)((threadIdx.x + e) & 7);
    b0[e] = (_Float16)(float)((threadIdx.x * 3 + e) & 7);
    b1[e] = (_Float16)(float)((threadIdx.x * 5 + e) & 7);
  }
  const f32x16 zero = {};
  double acc[2][16];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[t][e] = 0.0;
  for (int s = 0; s < kStages; ++s) {
    f32x16 p0, p1;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      touch(a);
      touch(b0);
      touch(b1);
      const bool fresh = PER_BLOCK || kb == 0;
      p0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b0, fresh ? zero : p0, 0, 0, 0);
      p1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b1, fresh ? zero : p1, 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);   // as the product kernels: folds after their MFMAs
      if (PER_BLOCK || kb == 3) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          acc[0][e] += (double)p0[e];
          acc[1][e] += (double)p1[e];
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  out[blockIdx.x * kThreads + threadIdx.x] = fold_out(acc);
}

template <bool SCALE>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void k_fp4(float* out) {
  // A and B operands of the FP4 MFMA: 32 x 64 codes, 16 bytes per lane; one 16-element
  // block of codes and zeros elsewhere (lanes hold 32 consecutive K of one row: the
  // block's lanes carry codes, the padding lanes zero)
  i32x8 a = {}, b0 = {}, b1 = {};
  const int live = (threadIdx.x & 63) < 32 ? 1 : 0;
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    a[e] = live * (int)(0x21436587u ^ threadIdx.x);
    b0[e] = live * (int)(0x12345678u ^ (threadIdx.x * 3));
    b1[e] = live * (int)(0x76543210u ^ (threadIdx.x * 5));
  }
  // per-lane row scales s_a of its 16 outputs and the column scale s_b, changed per block
  float sa[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) sa[e] = 1.0f + 0.125f * (float)((threadIdx.x + e) & 7);
  float sb0 = 1.5f, sb1 = 1.25f;
  const f32x16 zero = {};
  f32x16 acc0 = {}, acc1 = {};
  for (int s = 0; s < kStages; ++s) {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      touch(a);
      touch(b0);
      touch(b1);
      const f32x16 q0 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b0, SCALE ? zero : acc0, 4, 4, 0, 127, 0, 127);
      const f32x16 q1 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b1, SCALE ? zero : acc1, 4, 4, 0, 127, 0, 127);
      if (SCALE) {
        touch(sb0);
        touch(sb1);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          acc0[e] = __builtin_fmaf(sa[e] * sb0, q0[e], acc0[e]);
          acc1[e] = __builtin_fmaf(sa[e] * sb1, q1[e], acc1[e]);
        }
      } else {
        acc0 = q0;
        acc1 = q1;
      }
    }
  }
  float r = 0.0f;
#pragma unroll
  for (int e = 0; e < 16; ++e) r += acc0[e] + acc1[e];
  out[blockIdx.x * kThreads + threadIdx.x] = r;
}

}  // namespace

int main() {
  const int blocks = 2048;   // 8 workgroups of 8 waves per CU over 256 CUs
  float* out = nullptr;
  if (hipMalloc(&out, (size_t)blocks * kThreads * sizeof(float)) != hipSuccess) return 1;
  bool ok = true;
  for (int rep = 0; rep < 3 && ok; ++rep) {
    hipLaunchKernelGGL(k_f16_only, dim3(blocks), dim3(kThreads), 0, 0, out);
    hipLaunchKernelGGL(k_f16_fold<false>, dim3(blocks), dim3(kThreads), 0, 0, out);
    hipLaunchKernelGGL(k_f16_fold<true>, dim3(blocks), dim3(kThreads), 0, 0, out);
    hipLaunchKernelGGL(k_fp4<true>, dim3(blocks), dim3(kThreads), 0, 0, out);
    hipLaunchKernelGGL(k_fp4<false>, dim3(blocks), dim3(kThreads), 0, 0, out);
    ok = hipDeviceSynchronize() == hipSuccess;
  }
  (void)hipFree(out);
  const double flop = (double)blocks * (kThreads / 64) * kStages * 4 * 2 * (2.0 * 32 * 32 * 16);
  std::printf("bridge_candidates %s: useful FLOP per launch %.6e\n", ok ? "done" : "failed", flop);
  return ok ? 0 : 2;
}
