// Update product of the BF16 comparison path through hipBLASLt:
//   X <- a X + B16 Xb   (B16 m x m symmetric bf16, Xb = bf16(X) m x n, X FP32),
// FP32 accumulation and FP32 output, batched with strides.  The symmetric Gram
// products of that path stay in this library (they compute the upper tiles only);
// the plain update product is a library GEMM.
//
// Column-major view used by hipBLASLt: the row-major m x n matrices Xb and X are
// column-major n x m (leading dimension n), so D = A B with A = Xb (n x m),
// B = B16 (m x m; symmetric, so its layout does not matter) and C = D = X.
#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include <map>
#include <mutex>
#include <tuple>

#include "internal.h"

namespace fp4r {

namespace {
struct Plan {
  hipblasLtMatmulDesc_t desc = nullptr;
  hipblasLtMatrixLayout_t la = nullptr, lb = nullptr, lc = nullptr;
  hipblasLtMatmulAlgo_t algo{};
};

std::mutex g_mu;
std::map<int, hipblasLtHandle_t> g_handles;
std::map<std::tuple<int, int64_t, int64_t, int64_t, int64_t, size_t>, Plan> g_plans;

bool layout(hipblasLtMatrixLayout_t* l, hipDataType t, int64_t rows, int64_t cols, int64_t ld, int32_t batch,
            int64_t stride) {
  if (hipblasLtMatrixLayoutCreate(l, t, (uint64_t)rows, (uint64_t)cols, ld) != HIPBLAS_STATUS_SUCCESS) return false;
  return hipblasLtMatrixLayoutSetAttribute(*l, HIPBLASLT_MATRIX_LAYOUT_BATCH_COUNT, &batch, sizeof(batch)) ==
             HIPBLAS_STATUS_SUCCESS &&
         hipblasLtMatrixLayoutSetAttribute(*l, HIPBLASLT_MATRIX_LAYOUT_STRIDED_BATCH_OFFSET, &stride,
                                           sizeof(stride)) == HIPBLAS_STATUS_SUCCESS;
}

// The handle and plan of this device and shape (created on first use and kept
// until the process ends, like the library's code objects).
const Plan* plan_for(int64_t batch, int64_t m, int64_t n, int64_t x_bstride, size_t ws_bytes) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  std::lock_guard<std::mutex> lk(g_mu);
  auto key = std::make_tuple(dev, batch, m, n, x_bstride, ws_bytes);
  auto it = g_plans.find(key);
  if (it != g_plans.end()) return &it->second;
  hipblasLtHandle_t& h = g_handles[dev];
  if (!h && hipblasLtCreate(&h) != HIPBLAS_STATUS_SUCCESS) {
    h = nullptr;
    return nullptr;
  }
  Plan p;
  if (hipblasLtMatmulDescCreate(&p.desc, HIPBLAS_COMPUTE_32F, HIP_R_32F) != HIPBLAS_STATUS_SUCCESS) return nullptr;
  const hipblasOperation_t op = HIPBLAS_OP_N;
  hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSA, &op, sizeof(op));
  hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSB, &op, sizeof(op));
  const int32_t b32 = (int32_t)batch;
  if (!layout(&p.la, HIP_R_16BF, n, m, n, b32, m * n) || !layout(&p.lb, HIP_R_16BF, m, m, m, b32, m * m) ||
      !layout(&p.lc, HIP_R_32F, n, m, n, b32, x_bstride))
    return nullptr;
  hipblasLtMatmulPreference_t pref = nullptr;
  if (hipblasLtMatmulPreferenceCreate(&pref) != HIPBLAS_STATUS_SUCCESS) return nullptr;
  const uint64_t wsb = ws_bytes;
  hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &wsb, sizeof(wsb));
  hipblasLtMatmulHeuristicResult_t res{};
  int found = 0;
  const hipblasStatus_t hs =
      hipblasLtMatmulAlgoGetHeuristic(h, p.desc, p.la, p.lb, p.lc, p.lc, pref, 1, &res, &found);
  hipblasLtMatmulPreferenceDestroy(pref);
  if (hs != HIPBLAS_STATUS_SUCCESS || found < 1) return nullptr;
  p.algo = res.algo;
  return &g_plans.emplace(key, p).first->second;
}
}  // namespace

hipError_t launch_bf16_update_blaslt(const uint16_t* b16, const uint16_t* xb, float* x, int64_t batch, int64_t m,
                                     int64_t n, int64_t x_bstride, float a, void* ws, size_t ws_bytes,
                                     hipStream_t st) {
  if (batch == 0) return hipSuccess;
  const Plan* p = plan_for(batch, m, n, x_bstride, ws_bytes);
  if (!p) return hipErrorNotSupported;
  hipblasLtHandle_t h;
  {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_mu);
    h = g_handles[dev];
  }
  const float alpha = 1.0f, beta = a;
  const hipblasStatus_t s = hipblasLtMatmul(h, p->desc, &alpha, xb, p->la, b16, p->lb, &beta, x, p->lc, x, p->lc,
                                            &p->algo, ws, ws_bytes, st);
  return s == HIPBLAS_STATUS_SUCCESS ? hipSuccess : hipErrorLaunchFailure;
}

}  // namespace fp4r
