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
// k_proj: one block per 16 token rows x 32 output columns (of one product,
// or of the sum over products).  The block's rows of In (transposed to
// [k][row]) and its 32 columns of op(W) are staged in LDS; the 4 waves split
// K into quarters, each lane accumulating 2 rows x 4 columns, and the
// quarters are added in wave order.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) k_proj(Proj q) {
  extern __shared__ __attribute__((aligned(16))) float sm[];
  const int M = q.M, Cin = q.Cin, Cout = q.Cout;
  float* in_s = sm;               // [Cin][16]
  float* w_s = sm + Cin * 16;     // [Cin][32]
  float* red = w_s + Cin * 32;    // [4 waves][16][32]
  const int j0 = blockIdx.x * 32, r0 = blockIdx.y * 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int cg = lane & 7, rp = lane >> 3;  // columns 4cg..+3, rows 2rp, 2rp+1
  const int kq = Cin / 4, kb = wave * kq;
  float acc[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  const int p0 = q.sum ? 0 : blockIdx.z, p1 = q.sum ? q.n : blockIdx.z + 1;
  for (int p = p0; p < p1; ++p) {
    const float* in = q.in[p];
    const float* W = q.W[p];
    // In rows r0..r0+15 (zero past M; stored transposed) and 32 columns of
    // op(W), as float4 along the contiguous dimension: every load of the
    // thread is issued before its LDS stores (one memory round trip)
    const int ci4 = Cin / 4;
    float4 vi[4], vw[8];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = threadIdx.x + 256 * u;  // < 16 * ci4 = 4 Cin <= 1024
      const int r = e & 15, k4 = e >> 4;    // consecutive threads: consecutive LDS words
      const int rr = r0 + r < M ? r0 + r : M - 1;
      if (e < 16 * ci4) vi[u] = *reinterpret_cast<const float4*>(in + (int64_t)rr * Cin + 4 * k4);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = threadIdx.x + 256 * u;  // < 8 Cin <= 2048
      if (e < 8 * Cin) {
        if (!q.transW) {
          const int k = e >> 3, c4 = e & 7;  // W is [Cin][Cout]
          vw[u] = *reinterpret_cast<const float4*>(W + (int64_t)k * Cout + j0 + 4 * c4);
        } else {
          const int c = e & 31, k4 = e >> 5;  // W is [Cout][Cin]
          vw[u] = *reinterpret_cast<const float4*>(W + (int64_t)(j0 + c) * Cin + 4 * k4);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = threadIdx.x + 256 * u;
      if (e < 16 * ci4) {
        const int r = e & 15, k4 = e >> 4;
        const float4 v = r0 + r < M ? vi[u] : float4{0.f, 0.f, 0.f, 0.f};
        in_s[(4 * k4 + 0) * 16 + r] = v.x;
        in_s[(4 * k4 + 1) * 16 + r] = v.y;
        in_s[(4 * k4 + 2) * 16 + r] = v.z;
        in_s[(4 * k4 + 3) * 16 + r] = v.w;
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = threadIdx.x + 256 * u;
      if (e < 8 * Cin) {
        if (!q.transW) {
          const int k = e >> 3, c4 = e & 7;
          *reinterpret_cast<float4*>(w_s + k * 32 + 4 * c4) = vw[u];
        } else {
          const int c = e & 31, k4 = e >> 5;
          w_s[(4 * k4 + 0) * 32 + c] = vw[u].x;
          w_s[(4 * k4 + 1) * 32 + c] = vw[u].y;
          w_s[(4 * k4 + 2) * 32 + c] = vw[u].z;
          w_s[(4 * k4 + 3) * 32 + c] = vw[u].w;
        }
      }
    }
    __syncthreads();
#pragma unroll 4
    for (int k = kb; k < kb + kq; ++k) {
      const float2 iv = *reinterpret_cast<const float2*>(in_s + k * 16 + 2 * rp);
      const float4 wv = *reinterpret_cast<const float4*>(w_s + k * 32 + 4 * cg);
      acc[0][0] += iv.x * wv.x; acc[0][1] += iv.x * wv.y; acc[0][2] += iv.x * wv.z; acc[0][3] += iv.x * wv.w;
      acc[1][0] += iv.y * wv.x; acc[1][1] += iv.y * wv.y; acc[1][2] += iv.y * wv.z; acc[1][3] += iv.y * wv.w;
    }
    __syncthreads();  // the next product restages in_s / w_s
  }
  // K quarters -> one output, added in wave order
#pragma unroll
  for (int i = 0; i < 2; ++i)
    *reinterpret_cast<float4*>(red + (wave * 16 + 2 * rp + i) * 32 + 4 * cg) =
        float4{acc[i][0], acc[i][1], acc[i][2], acc[i][3]};
  __syncthreads();
  const int po = q.sum ? 0 : blockIdx.z;
  for (int e = threadIdx.x; e < 16 * 32; e += 256) {
    const int r = e >> 5, c = e & 31;
    if (r0 + r >= M) continue;
    const float v = ((red[e] + red[512 + e]) + red[1024 + e]) + red[1536 + e];
    const float bj = q.b[po] ? q.b[po][j0 + c] : 0.f;
    q.out[po][(int64_t)(r0 + r) * Cout + j0 + c] = v + bj;
  }
}

hipError_t launch_proj(const Proj& q, hipStream_t st) {
  // (Cin <= 256: the staging loads of k_proj cover 4 Cin and 8 Cin float4)
  if (q.n < 1 || q.n > 3 || q.M < 1 || q.M > 64 || q.Cin < 16 || q.Cin % 16 || q.Cin > 256 ||
      q.Cout % 32)
    return hipErrorInvalidValue;
  for (int p = 0; p < q.n; ++p)
    if (!q.in[p] || !q.W[p] || (!q.sum && !q.out[p])) return hipErrorInvalidValue;
  if (q.sum && !q.out[0]) return hipErrorInvalidValue;
  const size_t lds = ((size_t)q.Cin * 48 + 4 * 16 * 32) * sizeof(float);
  if (lds > 160 * 1024) return hipErrorInvalidConfiguration;
  dim3 grid(q.Cout / 32, (q.M + 15) / 16, q.sum ? 1 : q.n);
  hipLaunchKernelGGL(k_proj, grid, dim3(256), lds, st, q);
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
// The row softmax (and the backward's row sums) use G = 256 / Mp lanes per
// row (Mp = M rounded up to a power of two), reduced with lane shuffles.
// ---------------------------------------------------------------------------
static size_t core_lds(int M, int D, int nmat) {
  return ((size_t)nmat * M * (D + 1) + 2 * (size_t)M * (M + 1)) * sizeof(float);
}

// Stage nmat [M][D] blocks (columns [off, off + D) of [M][C] matrices) into
// LDS rows of stride DS: per round, each thread loads 4 elements of every
// matrix (one index division shared by the matrices) before storing them.
template <int NMAT>
__device__ __forceinline__ void stage_heads(const float* const (&src)[NMAT], float* const (&dst)[NMAT],
                                            int M, int D, int C, int off, int DS) {
  const int per = M * D;
  for (int base = threadIdx.x; base < per; base += 4 * kThreads) {
    float v[NMAT][4];
    int ri[4], di[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = base + u * kThreads;
      const int x = e < per ? e : per - 1;
      ri[u] = x / D;
      di[u] = x - ri[u] * D;
#pragma unroll
      for (int m = 0; m < NMAT; ++m) v[m][u] = src[m][(int64_t)ri[u] * C + off + di[u]];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (base + u * kThreads < per)
#pragma unroll
        for (int m = 0; m < NMAT; ++m) dst[m][ri[u] * DS + di[u]] = v[m][u];
  }
}

__device__ __forceinline__ int row_lanes(int M) {
  int mp = 1;
  while (mp < M) mp <<= 1;
  const int g = 256 / mp;  // a row's lanes stay inside one wave
  return g < 64 ? g : 64;  // 4 .. 64 (a power of two)
}

template <typename Op>
__device__ __forceinline__ float lanes_reduce(float v, int G, Op op) {
  for (int o = 1; o < G; o <<= 1) v = op(v, __shfl_xor(v, o));
  return v;
}

template <bool STAGE>
__global__ void __launch_bounds__(256) k_attn_core(const float* Q, const float* K, const float* V,
                                                   float* P, float* O, int M, int C, int H) {
  extern __shared__ __attribute__((aligned(16))) float sm[];
  const int h = blockIdx.x, D = C / H, off = h * D, DS = D + 1, MS = M + 1;
  float* sp = sm;                            // [M][M+1]
  float* qs = sm + 2 * M * MS;               // [M][D+1] x 3
  float* ks = qs + M * DS;
  float* vs = ks + M * DS;
  if (STAGE) {
    const float* src[3] = {Q, K, V};
    float* const dst[3] = {qs, ks, vs};
    stage_heads<3>(src, dst, M, D, C, off, DS);
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
    sp[r * MS + c] = s * scale;
  }
  __syncthreads();
  {
    // row r = tid / G, its columns c = lane-in-row + G j
    const int G = row_lanes(M), r = threadIdx.x / G, li = threadIdx.x - r * G;
    float mx = -INFINITY;
    if (r < M)
      for (int c = li; c < M; c += G) mx = fmaxf(mx, sp[r * MS + c]);
    mx = lanes_reduce(mx, G, [](float a, float b) { return fmaxf(a, b); });
    float sum = 0.f;
    if (r < M)
      for (int c = li; c < M; c += G) {
        const float e = expf(sp[r * MS + c] - mx);
        sp[r * MS + c] = e;
        sum += e;
      }
    sum = lanes_reduce(sum, G, [](float a, float b) { return a + b; });
    const float inv = 1.0f / sum;
    if (r < M)
      for (int c = li; c < M; c += G) sp[r * MS + c] *= inv;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < M * M; e += blockDim.x) {
    const int r = e / M, c = e - r * M;
    P[(int64_t)h * M * M + e] = sp[r * MS + c];
  }
  for (int e = threadIdx.x; e < M * D; e += blockDim.x) {
    const int r = e / D, d = e - r * D;
    float s = 0.f;
    for (int c = 0; c < M; ++c) s += sp[r * MS + c] * v_(c, d);
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
    const float* src[4] = {Q, K, V, dO};
    float* const dst[4] = {qs, ks, vs, os};
    stage_heads<4>(src, dst, M, D, C, off, DS);
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
  {
    const int G = row_lanes(M), r = threadIdx.x / G, li = threadIdx.x - r * G;
    float rs = 0.f;
    if (r < M)
      for (int c = li; c < M; c += G) rs += se[r * MS + c] * sp[r * MS + c];
    rs = lanes_reduce(rs, G, [](float a, float b) { return a + b; });
    if (r < M)
      for (int c = li; c < M; c += G) se[r * MS + c] = sp[r * MS + c] * (se[r * MS + c] - rs);
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
