// Plain GEMMs of the block stack (the MLP and the linear layers around the
// Physics-Attention layer) on hipBLASLt: row-major D[m,n] = alpha op(A) op(B)
// + beta C (+ a bias broadcast over rows), C = D unless given.  hipBLASLt is
// column-major, so the product is issued as D^T = op(B)^T op(A)^T on the
// same buffers.
#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include <cstdint>
#include <cstring>
#include <map>
#include <mutex>
#include <tuple>

#include "pa_internal.h"

namespace pa {
namespace {

std::mutex g_mu;
hipblasLtHandle_t g_handle[64] = {};

// One hipBLASLt handle per device, created on first use (the library's
// only allocation of its own; it lives until the process ends).
hipblasStatus_t handle_for_current_device(hipblasLtHandle_t* h) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return HIPBLAS_STATUS_INVALID_VALUE;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_handle[dev]) {
    hipblasStatus_t s = hipblasLtCreate(&g_handle[dev]);
    if (s != HIPBLAS_STATUS_SUCCESS) return s;
  }
  *h = g_handle[dev];
  return HIPBLAS_STATUS_SUCCESS;
}

hipDataType hip_type(int dtype) { return dtype == 1 ? HIP_R_16BF : HIP_R_32F; }

// Heuristic choice cached per problem (shape, types, transposes, bias).
using Key = std::tuple<int, int, int64_t, int64_t, int64_t, int, int, int, int, bool, int>;
std::map<Key, hipblasLtMatmulAlgo_t> g_algo;

struct Descs {
  hipblasLtMatmulDesc_t op = nullptr;
  hipblasLtMatrixLayout_t a = nullptr, b = nullptr, d = nullptr;
  hipblasLtMatmulPreference_t pref = nullptr;
  ~Descs() {
    if (pref) hipblasLtMatmulPreferenceDestroy(pref);
    if (d) hipblasLtMatrixLayoutDestroy(d);
    if (b) hipblasLtMatrixLayoutDestroy(b);
    if (a) hipblasLtMatrixLayoutDestroy(a);
    if (op) hipblasLtMatmulDescDestroy(op);
  }
};

}  // namespace

int gemm(const Gemm& g, hipStream_t st) {
  hipblasLtHandle_t h;
  hipblasStatus_t s = handle_for_current_device(&h);
  if (s != HIPBLAS_STATUS_SUCCESS) return (int)s;
  Descs d;
#define PA_LT(call)                                  \
  do {                                               \
    hipblasStatus_t s_ = (call);                     \
    if (s_ != HIPBLAS_STATUS_SUCCESS) return (int)s_; \
  } while (0)
  // column-major operands: first = stored B, second = stored A
  const hipblasOperation_t op1 = g.transB ? HIPBLAS_OP_T : HIPBLAS_OP_N;
  const hipblasOperation_t op2 = g.transA ? HIPBLAS_OP_T : HIPBLAS_OP_N;
  PA_LT(hipblasLtMatmulDescCreate(&d.op, HIPBLAS_COMPUTE_32F, HIP_R_32F));
  int32_t o1 = op1, o2 = op2;
  PA_LT(hipblasLtMatmulDescSetAttribute(d.op, HIPBLASLT_MATMUL_DESC_TRANSA, &o1, sizeof o1));
  PA_LT(hipblasLtMatmulDescSetAttribute(d.op, HIPBLASLT_MATMUL_DESC_TRANSB, &o2, sizeof o2));
  if (g.bias) {
    uint32_t epi = HIPBLASLT_EPILOGUE_BIAS;
    int32_t bt = HIP_R_32F;
    PA_LT(hipblasLtMatmulDescSetAttribute(d.op, HIPBLASLT_MATMUL_DESC_EPILOGUE, &epi, sizeof epi));
    PA_LT(hipblasLtMatmulDescSetAttribute(d.op, HIPBLASLT_MATMUL_DESC_BIAS_DATA_TYPE, &bt, sizeof bt));
    const void* bp = g.bias;
    PA_LT(hipblasLtMatmulDescSetAttribute(d.op, HIPBLASLT_MATMUL_DESC_BIAS_POINTER, &bp, sizeof bp));
  }
  // stored B: row-major (transB ? [n,k] : [k,n]) = column-major (transB ? [k x n] : [n x k])
  if (g.transB)
    PA_LT(hipblasLtMatrixLayoutCreate(&d.a, hip_type(g.tb), g.k, g.n, g.k));
  else
    PA_LT(hipblasLtMatrixLayoutCreate(&d.a, hip_type(g.tb), g.n, g.k, g.n));
  // stored A: row-major (transA ? [k,m] : [m,k]) = column-major (transA ? [m x k] : [k x m])
  if (g.transA)
    PA_LT(hipblasLtMatrixLayoutCreate(&d.b, hip_type(g.ta), g.m, g.k, g.m));
  else
    PA_LT(hipblasLtMatrixLayoutCreate(&d.b, hip_type(g.ta), g.k, g.m, g.k));
  PA_LT(hipblasLtMatrixLayoutCreate(&d.d, hip_type(g.td), g.n, g.m, g.n));

  int dev = 0;
  (void)hipGetDevice(&dev);
  const Key key{dev, (int)g.transA * 2 + (int)g.transB, g.m, g.n, g.k, g.ta, g.tb, g.td,
                g.beta != 0.f ? 1 : 0, g.bias != nullptr, (int)(g.ws_bytes >> 20)};
  hipblasLtMatmulAlgo_t algo;
  bool have = false;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_algo.find(key);
    if (it != g_algo.end()) {
      algo = it->second;
      have = true;
    }
  }
  if (!have) {
    PA_LT(hipblasLtMatmulPreferenceCreate(&d.pref));
    uint64_t wmax = g.ws_bytes;
    PA_LT(hipblasLtMatmulPreferenceSetAttribute(d.pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES,
                                                &wmax, sizeof wmax));
    hipblasLtMatmulHeuristicResult_t res[1];
    int n = 0;
    PA_LT(hipblasLtMatmulAlgoGetHeuristic(h, d.op, d.a, d.b, d.d, d.d, d.pref, 1, res, &n));
    if (n < 1 || res[0].state != HIPBLAS_STATUS_SUCCESS) return (int)HIPBLAS_STATUS_NOT_SUPPORTED;
    algo = res[0].algo;
    std::lock_guard<std::mutex> lk(g_mu);
    g_algo[key] = algo;
  }
  const float alpha = g.alpha, beta = g.beta;
  PA_LT(hipblasLtMatmul(h, d.op, &alpha, g.B, d.a, g.A, d.b, &beta, g.Cin ? g.Cin : g.D, d.d,
                        g.D, d.d, &algo, g.ws, g.ws_bytes, st));
#undef PA_LT
  return 0;
}

}  // namespace pa
