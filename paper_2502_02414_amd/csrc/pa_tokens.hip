// Token side of the layer (gfx950): attention among the M <= 64 physical
// states (Eq. 2) and its backward.  These products are tiny (M x C by C x C
// at most); what costs is latency, so every block stages its operands in
// LDS with one round of coalesced loads and then computes from LDS.
//   k_proj    out_p = In_p op(W_p) + b_p  (op = W or W^T; or the sum over p)
//   k_outer   out_p = S^T dX_p            (weight gradients, K = M)
//   k_colsum  out_p = 1^T dX_p            (bias gradients)
//   k_attn_core / k_attn_core_bwd: one block per head h (channels
//             [hD, hD + D)): P_h = softmax(Q_h K_h^T / sqrt(D)), O_h = P_h V_h
//             and its backward.
#include "pa_device.hpp"
#include "pa_internal.h"

namespace pa {

constexpr int kThreads = 256;  // every token-side kernel runs 256 threads

// Stage n elements with all of a thread's loads in flight before its
// stores: ld(e) must be valid for every e < n (callers clamp), st(e, v)
// writes element e.
template <int NB, typename Ld, typename St>
__device__ __forceinline__ void staged(int n, Ld&& ld, St&& st) {
  for (int base = threadIdx.x; base < n; base += NB * kThreads) {
    float v[NB];
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const int e = base + u * kThreads;
      v[u] = ld(e < n ? e : n - 1);
    }
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const int e = base + u * kThreads;
      if (e < n) st(e, v[u]);
    }
  }
}

// ---------------------------------------------------------------------------
// k_proj: 32 output columns per block; rows are the M tokens.
// ---------------------------------------------------------------------------
template <int U>  // rows per thread: token rows rg + 8u, u < U (M <= 8U)
__global__ void __launch_bounds__(256) k_proj(Proj q) {
  extern __shared__ __attribute__((aligned(16))) float sm[];
  const int M = q.M, Cin = q.Cin, Cout = q.Cout;
  constexpr int MP = 8 * U;                 // rows padded with zeros
  float* in_s = sm;                         // [MP][Cin + 1]
  float* w_s = sm + MP * (Cin + 1);         // [Cin][33]
  const int j0 = blockIdx.x * 32;
  const int jj = threadIdx.x & 31, rg = threadIdx.x >> 5;  // 8 row groups
  float acc[U];
#pragma unroll
  for (int u = 0; u < U; ++u) acc[u] = 0.f;
  const int p0 = q.sum ? 0 : blockIdx.y, p1 = q.sum ? q.n : blockIdx.y + 1;
  for (int p = p0; p < p1; ++p) {
    const float* in = q.in[p];
    const float* W = q.W[p];
    const int nin = M * Cin;
    staged<16>(MP * Cin, [&](int e) { return in[e < nin ? e : nin - 1]; },
               [&](int e, float v) {
                 const int r = e / Cin, k = e - r * Cin;
                 in_s[r * (Cin + 1) + k] = r < M ? v : 0.f;
               });
    if (!q.transW) {
      // op(W)[k][j] = W[k][j], W is [Cin][Cout]
      staged<16>(32 * Cin, [&](int e) { return W[(int64_t)(e >> 5) * Cout + j0 + (e & 31)]; },
                 [&](int e, float v) { w_s[(e >> 5) * 33 + (e & 31)] = v; });
    } else {
      // op(W)[k][j] = W[j][k], W is [Cout][Cin]
      staged<16>(32 * Cin, [&](int e) { return W[(int64_t)j0 * Cin + e]; },
                 [&](int e, float v) {
                   const int c = e / Cin, k = e - c * Cin;
                   w_s[k * 33 + c] = v;
                 });
    }
    __syncthreads();
    const float* ip = in_s + rg * (Cin + 1);
#pragma unroll 8
    for (int k = 0; k < Cin; ++k) {
      const float wv = w_s[k * 33 + jj];
#pragma unroll
      for (int u = 0; u < U; ++u) acc[u] += ip[8 * u * (Cin + 1) + k] * wv;
    }
    __syncthreads();
    if (!q.sum) {
      const float bj = q.b[p] ? q.b[p][j0 + jj] : 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = rg + 8 * u;
        if (r < M) q.out[p][(int64_t)r * Cout + j0 + jj] = acc[u] + bj;
        acc[u] = 0.f;
      }
    }
  }
  if (q.sum) {
    const float bj = q.b[0] ? q.b[0][j0 + jj] : 0.f;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = rg + 8 * u;
      if (r < M) q.out[0][(int64_t)r * Cout + j0 + jj] = acc[u] + bj;
    }
  }
}

hipError_t launch_proj(const Proj& q, hipStream_t st) {
  if (q.n < 1 || q.n > 3 || q.M < 1 || q.M > 64 || q.Cin < 1 || q.Cout % 32) return hipErrorInvalidValue;
  for (int p = 0; p < q.n; ++p)
    if (!q.in[p] || !q.W[p] || (!q.sum && !q.out[p])) return hipErrorInvalidValue;
  if (q.sum && !q.out[0]) return hipErrorInvalidValue;
  const int U = (q.M + 7) / 8;
  const size_t lds = ((size_t)8 * U * (q.Cin + 1) + (size_t)q.Cin * 33) * sizeof(float);
  if (lds > 160 * 1024) return hipErrorInvalidConfiguration;
  dim3 grid(q.Cout / 32, q.sum ? 1 : q.n);
  switch (U) {
#define PA_U(u) case u: hipLaunchKernelGGL(k_proj<u>, grid, dim3(256), lds, st, q); break;
    PA_U(1) PA_U(2) PA_U(3) PA_U(4) PA_U(5) PA_U(6) PA_U(7) PA_U(8)
#undef PA_U
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// k_outer: out_p[i][j] = sum_r S[r][i] dX_p[r][j]; 32 x 32 outputs per block.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) k_outer(Outer q) {
  __shared__ float a_s[64][33], b_s[64][33];
  const int M = q.M, C = q.C;
  const int j0 = blockIdx.x * 32, i0 = blockIdx.y * 32, p = blockIdx.z;
  const float* dX = q.dX[p];
  staged<8>(M * 32, [&](int e) { return q.S[(int64_t)(e >> 5) * C + i0 + (e & 31)]; },
            [&](int e, float v) { a_s[e >> 5][e & 31] = v; });
  staged<8>(M * 32, [&](int e) { return dX[(int64_t)(e >> 5) * C + j0 + (e & 31)]; },
            [&](int e, float v) { b_s[e >> 5][e & 31] = v; });
  __syncthreads();
  const int jj = threadIdx.x & 31, ig = threadIdx.x >> 5;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int r = 0; r < M; ++r) {
    const float bv = b_s[r][jj];
#pragma unroll
    for (int u = 0; u < 4; ++u) acc[u] += a_s[r][ig + 8 * u] * bv;
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) q.out[p][(int64_t)(i0 + ig + 8 * u) * C + j0 + jj] = acc[u];
}

hipError_t launch_outer(const Outer& q, hipStream_t st) {
  if (!q.S || q.n < 1 || q.n > 3 || q.M < 1 || q.M > 64 || q.C % 32) return hipErrorInvalidValue;
  for (int p = 0; p < q.n; ++p)
    if (!q.dX[p] || !q.out[p]) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_outer, dim3(q.C / 32, q.C / 32, q.n), dim3(256), 0, st, q);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// k_colsum: out_p[j] = sum_r in_p[r][j].
// ---------------------------------------------------------------------------
__global__ void k_colsum(ColSum q) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x, p = blockIdx.y;
  if (j >= q.C || !q.out[p]) return;
  float s = 0.f;
#pragma unroll 8
  for (int r = 0; r < q.M; ++r) s += q.in[p][(int64_t)r * q.C + j];
  q.out[p][j] = s;
}

hipError_t launch_colsum(const ColSum& q, hipStream_t st) {
  if (q.n < 1 || q.n > 3 || q.M < 1) return hipErrorInvalidValue;
  for (int p = 0; p < q.n; ++p)
    if (!q.in[p]) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_colsum, dim3((q.C + 255) / 256, q.n), dim3(256), 0, st, q);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Attention core, one block per head.  Q_h, K_h, V_h (and dO_h) are staged
// in LDS when they fit (always for D <= 64); otherwise read from global.
// ---------------------------------------------------------------------------
static size_t core_lds(int M, int D, int nmat) {
  return ((size_t)nmat * M * (D + 1) + 2 * (size_t)M * (M + 1)) * sizeof(float);
}

template <bool STAGE>
__global__ void __launch_bounds__(256) k_attn_core(const float* Q, const float* K, const float* V,
                                                   float* P, float* O, int M, int C, int H) {
  extern __shared__ __attribute__((aligned(16))) float sm[];
  const int h = blockIdx.x, D = C / H, off = h * D, DS = D + 1;
  float* sp = sm;                            // [M][M+1]
  float* qs = sm + M * (M + 1);              // [M][D+1] x 3
  float* ks = qs + M * DS;
  float* vs = ks + M * DS;
  if (STAGE) {
    auto src = [&](const float* X) {
      return [=](int e) { const int r = e / D; return X[r * C + off + (e - r * D)]; };
    };
    auto dst = [&](float* Y) {
      return [=](int e, float v) { const int r = e / D; Y[r * DS + (e - r * D)] = v; };
    };
    staged<8>(M * D, src(Q), dst(qs));
    staged<8>(M * D, src(K), dst(ks));
    staged<8>(M * D, src(V), dst(vs));
    __syncthreads();
  }
  auto q_ = [&](int r, int d) { return STAGE ? qs[r * DS + d] : Q[r * C + off + d]; };
  auto k_ = [&](int r, int d) { return STAGE ? ks[r * DS + d] : K[r * C + off + d]; };
  auto v_ = [&](int r, int d) { return STAGE ? vs[r * DS + d] : V[r * C + off + d]; };
  const float scale = 1.0f / sqrtf((float)D);
  for (int e = threadIdx.x; e < M * M; e += blockDim.x) {
    const int r = e / M, c = e - r * M;
    float s = 0.f;
    for (int d = 0; d < D; ++d) s += q_(r, d) * k_(c, d);
    sp[r * (M + 1) + c] = s * scale;
  }
  __syncthreads();
  for (int r = threadIdx.x; r < M; r += blockDim.x) {
    float mx = -INFINITY;
    for (int c = 0; c < M; ++c) mx = fmaxf(mx, sp[r * (M + 1) + c]);
    float sum = 0.f;
    for (int c = 0; c < M; ++c) {
      const float e = expf(sp[r * (M + 1) + c] - mx);
      sp[r * (M + 1) + c] = e;
      sum += e;
    }
    const float inv = 1.0f / sum;
    for (int c = 0; c < M; ++c) sp[r * (M + 1) + c] *= inv;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < M * M; e += blockDim.x) {
    const int r = e / M, c = e - r * M;
    P[(int64_t)h * M * M + e] = sp[r * (M + 1) + c];
  }
  for (int e = threadIdx.x; e < M * D; e += blockDim.x) {
    const int r = e / D, d = e - r * D;
    float s = 0.f;
    for (int c = 0; c < M; ++c) s += sp[r * (M + 1) + c] * v_(c, d);
    O[r * C + off + d] = s;
  }
}

hipError_t launch_attn_core(const float* Q, const float* K, const float* V, float* P, float* O,
                            int M, int C, int H, hipStream_t st) {
  if (!Q || !K || !V || !P || !O || M < 1 || M > 64 || H < 1 || C % H) return hipErrorInvalidValue;
  const int D = C / H;
  const size_t lds = core_lds(M, D, 3);
  if (lds <= 150 * 1024)
    hipLaunchKernelGGL(k_attn_core<true>, dim3(H), dim3(256), lds, st, Q, K, V, P, O, M, C, H);
  else
    hipLaunchKernelGGL(k_attn_core<false>, dim3(H), dim3(256), core_lds(M, 0, 0), st, Q, K, V, P,
                       O, M, C, H);
  return hipGetLastError();
}

template <bool STAGE>
__global__ void __launch_bounds__(256) k_attn_core_bwd(const float* Q, const float* K,
                                                       const float* V, const float* P,
                                                       const float* dO, float* dQ, float* dK,
                                                       float* dV, int M, int C, int H) {
  extern __shared__ __attribute__((aligned(16))) float sm[];
  const int h = blockIdx.x, D = C / H, off = h * D, DS = D + 1, MS = M + 1;
  float* sp = sm;                 // P   [M][M+1]
  float* se = sp + M * MS;        // dE  [M][M+1]
  float* qs = se + M * MS;        // [M][D+1] x 4
  float* ks = qs + M * DS;
  float* vs = ks + M * DS;
  float* os = vs + M * DS;
  const float* Ph = P + (int64_t)h * M * M;
  staged<8>(M * M, [&](int e) { return Ph[e]; },
            [&](int e, float v) { const int r = e / M; sp[r * MS + (e - r * M)] = v; });
  if (STAGE) {
    auto src = [&](const float* X) {
      return [=](int e) { const int r = e / D; return X[r * C + off + (e - r * D)]; };
    };
    auto dst = [&](float* Y) {
      return [=](int e, float v) { const int r = e / D; Y[r * DS + (e - r * D)] = v; };
    };
    staged<8>(M * D, src(Q), dst(qs));
    staged<8>(M * D, src(K), dst(ks));
    staged<8>(M * D, src(V), dst(vs));
    staged<8>(M * D, src(dO), dst(os));
  }
  __syncthreads();
  auto q_ = [&](int r, int d) { return STAGE ? qs[r * DS + d] : Q[r * C + off + d]; };
  auto k_ = [&](int r, int d) { return STAGE ? ks[r * DS + d] : K[r * C + off + d]; };
  auto v_ = [&](int r, int d) { return STAGE ? vs[r * DS + d] : V[r * C + off + d]; };
  auto o_ = [&](int r, int d) { return STAGE ? os[r * DS + d] : dO[r * C + off + d]; };
  const float scale = 1.0f / sqrtf((float)D);
  // dP = dO_h V_h^T
  for (int e = threadIdx.x; e < M * M; e += blockDim.x) {
    const int r = e / M, c = e - r * M;
    float s = 0.f;
    for (int d = 0; d < D; ++d) s += o_(r, d) * v_(c, d);
    se[r * MS + c] = s;
  }
  __syncthreads();
  // dE = P o (dP - rowsum(dP o P))
  for (int r = threadIdx.x; r < M; r += blockDim.x) {
    float rs = 0.f;
    for (int c = 0; c < M; ++c) rs += se[r * MS + c] * sp[r * MS + c];
    for (int c = 0; c < M; ++c) se[r * MS + c] = sp[r * MS + c] * (se[r * MS + c] - rs);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < M * D; e += blockDim.x) {
    const int r = e / D, d = e - r * D;
    float sv = 0.f, sq = 0.f, sk = 0.f;
    for (int c = 0; c < M; ++c) {
      sv += sp[c * MS + r] * o_(c, d);
      sq += se[r * MS + c] * k_(c, d);
      sk += se[c * MS + r] * q_(c, d);
    }
    dV[r * C + off + d] = sv;
    dQ[r * C + off + d] = scale * sq;
    dK[r * C + off + d] = scale * sk;
  }
}

hipError_t launch_attn_core_bwd(const float* Q, const float* K, const float* V,
                                const float* P, const float* dO, float* dQ, float* dK,
                                float* dV, int M, int C, int H, hipStream_t st) {
  if (!Q || !K || !V || !P || !dO || !dQ || !dK || !dV || M < 1 || M > 64 || H < 1 || C % H)
    return hipErrorInvalidValue;
  const int D = C / H;
  const size_t lds = core_lds(M, D, 4);
  if (lds <= 150 * 1024)
    hipLaunchKernelGGL(k_attn_core_bwd<true>, dim3(H), dim3(256), lds, st, Q, K, V, P, dO, dQ,
                       dK, dV, M, C, H);
  else
    hipLaunchKernelGGL(k_attn_core_bwd<false>, dim3(H), dim3(256), core_lds(M, 0, 0), st, Q, K,
                       V, P, dO, dQ, dK, dV, M, C, H);
  return hipGetLastError();
}

}  // namespace pa
