// Internal launch interface between the C-ABI layer (pa_api.cpp) and the
// kernels (pa_stream.hip, pa_small.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pa {

struct StreamLaunch {
  const void* x = nullptr;
  const void* G = nullptr;
  const void* dY = nullptr;
  const void* img = nullptr;
  void* out = nullptr;
  float* tau_out = nullptr;
  const float* dW = nullptr;
  const float* dtau = nullptr;
  float* partials = nullptr;
  int64_t N = 0;
  int M = 0;
  int rec = 0;
  int P = 1;
  double tb = 0.0;  // tau0 + b_t
  float tau_min = 0.f;
  bool states = false;
  bool deslice = false;
};

// Streaming passes (pass = pa::Pass).  dtype: 0 fp32, 1 bf16.
hipError_t launch_stream(int pass, int dtype, int C, int MB, const StreamLaunch& L,
                         hipStream_t st);
// Waves per block of a pass at this shape (0 = shape not served).
int stream_waves(int pass, int dtype, int C, int MB);

// Table image for a pass, written into `img` (device).
struct PrepArgs {
  int pass = 0;
  int dtype = 0;
  int C = 0, M = 0, MB = 0;
  float eps = 0.f;
  const void* A = nullptr;    // [C,M] dtype
  const float* b = nullptr;   // [M]
  const void* a = nullptr;    // [C] dtype
  const float* Sp = nullptr;  // [M,C]  (kDeslice, kSliceBwd deslice term)
  const float* num = nullptr; // [M,C]  (kSliceBwd states term)
  const float* den = nullptr; // [M]
  const float* dS = nullptr;  // [M,C]
  void* img = nullptr;
};
hipError_t launch_prep(const PrepArgs& p, hipStream_t st);
// Bytes of the table image of a pass.
size_t image_bytes(int pass, int dtype, int C, int MB);

// out[k] = sum_{p < P} partials[p * rec + k] (k < rec), in order p = 0..P-1,
// scattered into up to 6 destination segments.
struct Segments {
  float* dst[6];
  int64_t len[6];
  int n;
};
hipError_t launch_reduce(const float* partials, int P, int64_t rec, const Segments& seg,
                         hipStream_t st);

// S = num / max(den, eps)
hipError_t launch_states(const float* num, const float* den, float* S, int M, int C, float eps,
                         hipStream_t st);

// Small dense products for the token attention (fp32):
//   out[i][j] = beta*out[i][j] + sum_k A(i,k) B(k,j) (+ bias[j]),
//   A(i,k) = A[i*sai + k*sak], B(k,j) = B[k*sbk + j*sbj].
struct Gemm {
  const float* A; int64_t sai, sak;
  const float* B; int64_t sbk, sbj;
  const float* bias;
  float* out; int64_t ldo;
  int rows, cols, K;
  int accumulate;
};
hipError_t launch_gemm(const Gemm& g, hipStream_t st);
// Column sums: out[j] = sum_i in[i*ld + j], i < rows.
hipError_t launch_colsum(const float* in, int rows, int cols, int64_t ld, float* out,
                         hipStream_t st);
// Per-head attention core: P_h = softmax(Q_h K_h^T * scale), O_h = P_h V_h.
hipError_t launch_attn_core(const float* Q, const float* K, const float* V, float* P, float* O,
                            int M, int C, int H, hipStream_t st);
// Per-head attention backward core: from dO, P, Q, K, V -> dQ, dK, dV.
hipError_t launch_attn_core_bwd(const float* Q, const float* K, const float* V,
                                const float* P, const float* dO, float* dQ, float* dK,
                                float* dV, int M, int C, int H, hipStream_t st);

}  // namespace pa
