// Token side of the layer in double precision (gfx950), used for fp32
// storage.  Attention among the M <= 64 states (Eq. 2) and its backward are
// tiny products whose results feed the slice backward through the
// differences s'_j - s'_k of nearly equal tokens: an fp32 rounding error of
// 1e-7 in S' moves dA by about 1e-5 at the synthetic workloads' shapes.  So
// for fp32 storage every token-side value is formed in double and rounded
// once, when it leaves as an fp32 output (S', dS, the parameter gradients).
//
//   k_mm64        batches of small products out = sum_t op(A_t) op(B_t) + b
//                 (operands fp32 or fp64 with arbitrary strides, "ones"
//                 operands for column sums), 32 x 32 output tiles, K chunks
//                 staged in LDS, fp64 FMAs
//   k_core64      per head: P = softmax(Q_h K_h^T / sqrt(D)), O_h = P V_h
//   k_core64_bwd  per head: P recomputed, dP = dO_h V_h^T,
//                 dE = P o (dP - rowsum(dP o P)), dQ_h, dK_h, dV_h (and O_h)
#include "pa_internal.h"

namespace pa {

namespace {

constexpr int kT = 32;          // output tile edge and K chunk
constexpr int kMMThreads = 256; // 16 x 16 threads, 2 x 2 outputs each

__device__ __forceinline__ double opnd_at(const Opnd64& o, int64_t i, int64_t k) {
  if (!o.p) return 1.0;
  const int64_t e = i * o.rs + k * o.cs;
  return o.dbl ? static_cast<const double*>(o.p)[e] : (double)static_cast<const float*>(o.p)[e];
}

// One 32 x 32 tile (tile index blockIdx.x) of product q.
__device__ __forceinline__ void mm64_tile(const MM64& q) {
  __shared__ double as[kT][kT + 1];  // [row][k]
  __shared__ double bs[kT][kT + 1];  // [k][col]
  const int tc = (q.cols + kT - 1) / kT;
  const int tiles = tc * ((q.rows + kT - 1) / kT);
  if ((int)blockIdx.x >= tiles) return;
  const int i0 = (blockIdx.x / tc) * kT, j0 = (blockIdx.x % tc) * kT;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  double acc[2][2] = {{0.0, 0.0}, {0.0, 0.0}};
  for (int t = 0; t < q.nt; ++t) {
    const Opnd64 A = q.A[t], B = q.B[t];
    const int K = q.K[t];
    // consecutive threads walk the operand's unit-stride dimension
    const bool a_k_fast = A.cs == 1 || !A.p, b_j_fast = B.cs == 1 || !B.p;
    for (int k0 = 0; k0 < K; k0 += kT) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = threadIdx.x + kMMThreads * u;  // < 1024 = kT * kT
        const int hi = e >> 5, lo = e & 31;
        {
          const int i = a_k_fast ? hi : lo, k = a_k_fast ? lo : hi;
          const bool in = i0 + i < q.rows && k0 + k < K;
          as[i][k] = in ? opnd_at(A, i0 + i, k0 + k) : 0.0;
        }
        {
          const int k = b_j_fast ? hi : lo, j = b_j_fast ? lo : hi;
          const bool in = k0 + k < K && j0 + j < q.cols;
          bs[k][j] = in ? opnd_at(B, k0 + k, j0 + j) : 0.0;
        }
      }
      __syncthreads();
#pragma unroll 8
      for (int k = 0; k < kT; ++k) {
        const double a0 = as[2 * ty][k], a1 = as[2 * ty + 1][k];
        const double b0 = bs[k][2 * tx], b1 = bs[k][2 * tx + 1];
        acc[0][0] = fma(a0, b0, acc[0][0]);
        acc[0][1] = fma(a0, b1, acc[0][1]);
        acc[1][0] = fma(a1, b0, acc[1][0]);
        acc[1][1] = fma(a1, b1, acc[1][1]);
      }
      __syncthreads();
    }
  }
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int i = i0 + 2 * ty + a, j = j0 + 2 * tx + b;
      if (i >= q.rows || j >= q.cols) continue;
      const double v = acc[a][b] + (q.bias ? (double)q.bias[j] : 0.0);
      const int64_t o = (int64_t)i * q.ld + j;
      if (q.out_dbl)
        static_cast<double*>(q.out)[o] = v;
      else
        static_cast<float*>(q.out)[o] = (float)v;
    }
}

// The product of a batch is chosen with constant indices (a run-time index
// into the by-value argument array would copy the arguments to scratch).
__global__ void __launch_bounds__(kMMThreads) k_mm64(MM64Batch b) {
  switch (blockIdx.y) {
#define PA_MM64_CASE(I) \
    case I:             \
      if (I < b.n) mm64_tile(b.p[I]); \
      break;
    PA_MM64_CASE(0) PA_MM64_CASE(1) PA_MM64_CASE(2) PA_MM64_CASE(3) PA_MM64_CASE(4)
    PA_MM64_CASE(5) PA_MM64_CASE(6) PA_MM64_CASE(7) PA_MM64_CASE(8)
#undef PA_MM64_CASE
    default:
      break;
  }
}

constexpr int kCoreThreads = 256;

// P = softmax(Q_h K_h^T * scale) of head h into ps ([M][M + 1], LDS).
__device__ __forceinline__ void core64_probs(const double* Q, const double* K, int M, int C,
                                             int off, int D, double* ps) {
  const int MS = M + 1;
  const double scale = 1.0 / sqrt((double)D);
  for (int e = threadIdx.x; e < M * M; e += kCoreThreads) {
    const int r = e / M, c = e - r * M;
    const double* q = Q + (int64_t)r * C + off;
    const double* k = K + (int64_t)c * C + off;
    double s = 0.0;
    for (int d = 0; d < D; ++d) s = fma(q[d], k[d], s);
    ps[r * MS + c] = s * scale;
  }
  __syncthreads();
  // one thread per row: max, exponentials, sum, normalisation
  for (int r = threadIdx.x; r < M; r += kCoreThreads) {
    double* row = ps + r * MS;
    double mx = row[0];
    for (int c = 1; c < M; ++c) mx = fmax(mx, row[c]);
    double sum = 0.0;
    for (int c = 0; c < M; ++c) {
      const double e = exp(row[c] - mx);
      row[c] = e;
      sum += e;
    }
    const double inv = 1.0 / sum;
    for (int c = 0; c < M; ++c) row[c] *= inv;
  }
  __syncthreads();
}

// O_h = P V_h (rows of O at stride C, columns off .. off + D).
template <typename TO>
__device__ __forceinline__ void core64_pv(const double* ps, const double* V, int M, int C, int off,
                                          int D, TO* O) {
  const int MS = M + 1;
  for (int e = threadIdx.x; e < M * D; e += kCoreThreads) {
    const int r = e / D, d = e - r * D;
    double s = 0.0;
    for (int c = 0; c < M; ++c) s = fma(ps[r * MS + c], V[(int64_t)c * C + off + d], s);
    O[(int64_t)r * C + off + d] = (TO)s;
  }
}

template <typename TO>
__global__ void __launch_bounds__(kCoreThreads) k_core64(const double* Q, const double* K,
                                                         const double* V, TO* O, int M, int C,
                                                         int H) {
  extern __shared__ __attribute__((aligned(16))) double dsm[];
  const int D = C / H, off = blockIdx.x * D;
  core64_probs(Q, K, M, C, off, D, dsm);
  core64_pv(dsm, V, M, C, off, D, O);
}

template <typename TD>
__global__ void __launch_bounds__(kCoreThreads) k_core64_bwd(const double* Q, const double* K,
                                                             const double* V, const TD* dO,
                                                             double* dQ, double* dK, double* dV,
                                                             double* O, int M, int C, int H) {
  extern __shared__ __attribute__((aligned(16))) double dsm[];
  const int D = C / H, off = blockIdx.x * D, MS = M + 1;
  double* ps = dsm;           // P  [M][M+1]
  double* es = dsm + M * MS;  // dP, then dE
  core64_probs(Q, K, M, C, off, D, ps);
  if (O) core64_pv(ps, V, M, C, off, D, O);
  for (int e = threadIdx.x; e < M * M; e += kCoreThreads) {
    const int r = e / M, c = e - r * M;
    double s = 0.0;
    for (int d = 0; d < D; ++d)
      s = fma((double)dO[(int64_t)r * C + off + d], V[(int64_t)c * C + off + d], s);
    es[r * MS + c] = s;
  }
  __syncthreads();
  for (int r = threadIdx.x; r < M; r += kCoreThreads) {
    double rs = 0.0;
    for (int c = 0; c < M; ++c) rs = fma(es[r * MS + c], ps[r * MS + c], rs);
    for (int c = 0; c < M; ++c) es[r * MS + c] = ps[r * MS + c] * (es[r * MS + c] - rs);
  }
  __syncthreads();
  const double scale = 1.0 / sqrt((double)D);
  for (int e = threadIdx.x; e < M * D; e += kCoreThreads) {
    const int r = e / D, d = e - r * D;
    double sq = 0.0, sk = 0.0, sv = 0.0;
    for (int c = 0; c < M; ++c) {
      const int64_t cd = (int64_t)c * C + off + d;
      sq = fma(es[r * MS + c], K[cd], sq);
      sk = fma(es[c * MS + r], Q[cd], sk);
      sv = fma(ps[c * MS + r], (double)dO[cd], sv);
    }
    const int64_t rd = (int64_t)r * C + off + d;
    dQ[rd] = scale * sq;
    dK[rd] = scale * sk;
    dV[rd] = sv;
  }
}

size_t core64_lds(int M, bool bwd) { return (size_t)(bwd ? 2 : 1) * M * (M + 1) * sizeof(double); }

bool core64_ok(int M, int C, int H) { return M >= 1 && M <= 64 && H >= 1 && C % H == 0; }

}  // namespace

hipError_t launch_mm64(const MM64Batch& b, hipStream_t st) {
  if (b.n < 1 || b.n > kMM64Max) return hipErrorInvalidValue;
  int tiles = 0;
  for (int i = 0; i < b.n; ++i) {
    const MM64& q = b.p[i];
    if (q.rows < 1 || q.cols < 1 || q.nt < 1 || q.nt > 3 || !q.out || q.ld < q.cols)
      return hipErrorInvalidValue;
    for (int t = 0; t < q.nt; ++t)
      if (q.K[t] < 1) return hipErrorInvalidValue;
    const int n = ((q.rows + kT - 1) / kT) * ((q.cols + kT - 1) / kT);
    tiles = n > tiles ? n : tiles;
  }
  hipLaunchKernelGGL(k_mm64, dim3(tiles, b.n), dim3(kMMThreads), 0, st, b);
  return hipGetLastError();
}

hipError_t launch_core64(const double* Q, const double* K, const double* V, void* O, bool O_dbl,
                         int M, int C, int H, hipStream_t st) {
  if (!Q || !K || !V || !O || !core64_ok(M, C, H)) return hipErrorInvalidValue;
  if (O_dbl)
    hipLaunchKernelGGL(k_core64<double>, dim3(H), dim3(kCoreThreads), core64_lds(M, false), st,
                       Q, K, V, static_cast<double*>(O), M, C, H);
  else
    hipLaunchKernelGGL(k_core64<float>, dim3(H), dim3(kCoreThreads), core64_lds(M, false), st,
                       Q, K, V, static_cast<float*>(O), M, C, H);
  return hipGetLastError();
}

hipError_t launch_core64_bwd(const double* Q, const double* K, const double* V, const void* dO,
                             bool dO_dbl, double* dQ, double* dK, double* dV, double* O, int M,
                             int C, int H, hipStream_t st) {
  if (!Q || !K || !V || !dO || !dQ || !dK || !dV || !core64_ok(M, C, H))
    return hipErrorInvalidValue;
  if (dO_dbl)
    hipLaunchKernelGGL(k_core64_bwd<double>, dim3(H), dim3(kCoreThreads), core64_lds(M, true), st,
                       Q, K, V, static_cast<const double*>(dO), dQ, dK, dV, O, M, C, H);
  else
    hipLaunchKernelGGL(k_core64_bwd<float>, dim3(H), dim3(kCoreThreads), core64_lds(M, true), st,
                       Q, K, V, static_cast<const float*>(dO), dQ, dK, dV, O, M, C, H);
  return hipGetLastError();
}

}  // namespace pa
