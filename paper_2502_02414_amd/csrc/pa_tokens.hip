// Token side of the layer (gfx950): attention among the M <= 64 physical
// states (Eq. 2) and its backward.  These products are tiny (M x C by C x C
// at most); what costs is latency and the number of launches, so the layer's
// token step is one launch per head-parallel part:
//   k_head_fwd   per head h (channels [hD, hD + D)): Q_h, K_h, V_h = S W_h +
//                b_h, P_h = softmax(Q_h K_h^T / sqrt(D)), O_h = P_h V_h
//   k_head_bwd   per head: the same forward, then dV_h, dQ_h, dK_h
//   k_token_grads  dS = sum_p dX_p W_p^T, dW_p = A_p^T B_p, db_p = 1^T B_p,
//                every output tile of every product in one launch
// The head kernels run the projections (3 M x C x D contractions) on
// v_mfma_f32_16x16x4f32 from LDS and the core from LDS.  Shapes whose head
// does not fit on chip use the general kernels:
//   k_proj       out_p = In_p op(W_p) + b_p  (op = W or W^T; or the sum over p)
//   k_attn_core / k_attn_core_bwd  the core of one head from global Q, K, V
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
// or of the sum over products; the last block of columns may hold 16).  The
// block's rows of In (transposed to [k][row]) and its 32 columns of op(W)
// (zero past Cout) are staged in LDS; the 4 waves split K into quarters,
// each lane accumulating 2 rows x 4 columns, and the quarters are added in
// wave order.
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
          vw[u] = j0 + 4 * c4 < Cout
                      ? *reinterpret_cast<const float4*>(W + (int64_t)k * Cout + j0 + 4 * c4)
                      : float4{0.f, 0.f, 0.f, 0.f};
        } else {
          const int c = e & 31, k4 = e >> 5;  // W is [Cout][Cin]
          vw[u] = j0 + c < Cout
                      ? *reinterpret_cast<const float4*>(W + (int64_t)(j0 + c) * Cin + 4 * k4)
                      : float4{0.f, 0.f, 0.f, 0.f};
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
    if (r0 + r >= M || j0 + c >= Cout) continue;
    const float v = ((red[e] + red[512 + e]) + red[1024 + e]) + red[1536 + e];
    const float bj = q.b[po] ? q.b[po][j0 + c] : 0.f;
    q.out[po][(int64_t)(r0 + r) * Cout + j0 + c] = v + bj;
  }
}

hipError_t launch_proj(const Proj& q, hipStream_t st) {
  // (Cin <= 256: the staging loads of k_proj cover 4 Cin and 8 Cin float4)
  if (q.n < 1 || q.n > 3 || q.M < 1 || q.M > 64 || q.Cin < 16 || q.Cin % 16 || q.Cin > 256 ||
      q.Cout < 16 || q.Cout % 16)
    return hipErrorInvalidValue;
  for (int p = 0; p < q.n; ++p)
    if (!q.in[p] || !q.W[p] || (!q.sum && !q.out[p])) return hipErrorInvalidValue;
  if (q.sum && !q.out[0]) return hipErrorInvalidValue;
  const size_t lds = ((size_t)q.Cin * 48 + 4 * 16 * 32) * sizeof(float);
  if (lds > 160 * 1024) return hipErrorInvalidConfiguration;
  dim3 grid((q.Cout + 31) / 32, (q.M + 15) / 16, q.sum ? 1 : q.n);
  hipLaunchKernelGGL(k_proj, grid, dim3(256), lds, st, q);
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

// ---------------------------------------------------------------------------
// Fused per-head kernels.  One block of kHeadThreads per head.  Every
// contraction runs on v_mfma_f32_16x16x4f32 over 16 x 16 tiles.  Operand
// runs of 4 consecutive k are read as float4 (lane group g, step q:
// k = 16q + 4g .. +3, the same k on both sides, so the pairing is exact).
//   Projections: tiles (matrix m in {Q, K, V}, row tile mt, column tile nt),
//     wave w owning tiles w, w + kHeadWaves, ...; the contraction over C runs
//     in K chunks of KC: the chunk of S (rows >= M zero) and of the head's
//     columns of W_m, transposed (columns >= D zero), are staged in LDS with
//     one round of loads.  Q_h, K_h, V_h are then kept in LDS as zero-padded
//     [M16][D16 + 4] tiles (the core buffers alias the chunk buffers).
//   Core: wave mt owns query rows [16mt, 16mt + 16).  Its scores are formed
//     transposed (K_h Q_h^T), so that lane (r, g) holds row 16mt + r at
//     columns 16ct + 4g + i: the row softmax reduces in-lane and across the
//     four lane groups, and P is already the A operand of P V_h.
// ---------------------------------------------------------------------------
constexpr int kHeadThreads = 512;
constexpr int kHeadWaves = kHeadThreads / 64;
constexpr int kHeadTPW = 4;        // projection tiles per wave (at most)
constexpr int kHeadDO = 8;         // padded dO_h elements per thread (at most)

__device__ __forceinline__ f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
// acc += sum_i a[i] b[i] over the 4 k of a float4 run
__device__ __forceinline__ f32x4 mfma4x4(const f32x4& a, const f32x4& b, f32x4 c) {
  c = mfma4(a[0], b[0], c);
  c = mfma4(a[1], b[1], c);
  c = mfma4(a[2], b[2], c);
  return mfma4(a[3], b[3], c);
}

// A kernel-argument pointer as an opaque uniform register value: choosing
// among such values per lane stays a register select (an indexed read of the
// argument array would copy the arguments to scratch memory).
template <typename P> __device__ __forceinline__ P in_sreg(P p) {
  asm volatile("" : "+s"(p));
  return p;
}
struct Ptr3 {
  const float *p0, *p1, *p2;
  __device__ __forceinline__ const float* operator()(int m) const {
    return m == 0 ? p0 : m == 1 ? p1 : p2;
  }
};
__device__ __forceinline__ Ptr3 ptr3(const float* const (&v)[3]) {
  return {in_sreg(v[0]), in_sreg(v[1]), in_sreg(v[2])};
}

struct HeadTile { int m, mt, nt; };
__device__ __forceinline__ HeadTile head_tile(const HeadGeo& G, int t) {
  const int m = t / (G.MT * G.NT), rem = t - m * G.MT * G.NT;
  return {m, rem / G.NT, rem - (rem / G.NT) * G.NT};
}

// Projection tiles of the calling wave (tile j = wave + kHeadWaves j) in
// acc, with their biases in bias (lane (r, g): column 16 nt + r).
__device__ __forceinline__ void head_project(const HeadArgs& a, float* sm, f32x4 (&acc)[kHeadTPW],
                                             float (&bias)[kHeadTPW]) {
  const HeadGeo& G = a.geo;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int tid = threadIdx.x, off = blockIdx.x * G.D;
  float* s_ch = sm;                    // [M16][SR]
  float* w_ch = sm + G.M16 * G.SR;     // [3 D16][SR]
  const Ptr3 b = ptr3(a.b);
  int sa[kHeadTPW], sb[kHeadTPW];
#pragma unroll
  for (int j = 0; j < kHeadTPW; ++j) {
    acc[j] = zero4();
    const int t = wave + kHeadWaves * j;
    const HeadTile h = head_tile(G, t < G.T ? t : 0);
    sa[j] = (16 * h.mt + r) * G.SR + 4 * g;
    sb[j] = (h.m * G.D16 + 16 * h.nt + r) * G.SR + 4 * g;
    const int col = 16 * h.nt + r;
    const float* bm = b(h.m);
    bias[j] = (t < G.T && bm != nullptr && col < G.D) ? bm[off + col] : 0.f;
  }
  // KC and D16 are powers of two (C is, and D divides it): shifts, not
  // divisions.  Per round each thread has 4 S and 4 x 3 W float4 loads in
  // flight before its LDS stores.
  const int KC4 = G.KC / 4, D4 = G.D16 / 4;
  const int lKC4 = __builtin_ctz(KC4), lD4 = __builtin_ctz(D4);
  const int nS4 = G.M16 * KC4, nW4 = G.KC * D4;
  const int nmax = nS4 > nW4 ? nS4 : nW4;
  for (int k0 = 0; k0 < G.C; k0 += G.KC) {
    for (int base = tid; base < nmax; base += 4 * kHeadThreads) {
      float4 vs[4], vw[3][4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = base + u * kHeadThreads;
        const int es = e < nS4 ? e : nS4 - 1;
        const int row = es >> lKC4, c4 = es & (KC4 - 1);
        const int rr = row < G.M ? row : G.M - 1;
        vs[u] = *reinterpret_cast<const float4*>(a.S + rr * G.C + k0 + 4 * c4);
        const int ew = e < nW4 ? e : nW4 - 1;
        const int k = ew >> lD4, d4 = ew & (D4 - 1);
        const int dd = 4 * d4 < G.D ? 4 * d4 : 0;
#pragma unroll
        for (int m = 0; m < 3; ++m)
          vw[m][u] = *reinterpret_cast<const float4*>(a.W[m] + (k0 + k) * G.C + off + dd);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = base + u * kHeadThreads;
        if (e < nS4) {
          const int row = e >> lKC4, c4 = e & (KC4 - 1);
          const float4 v = row < G.M ? vs[u] : float4{0.f, 0.f, 0.f, 0.f};
          *reinterpret_cast<float4*>(s_ch + row * G.SR + 4 * c4) = v;
        }
        if (e < nW4) {
          const int k = e >> lD4, d4 = e & (D4 - 1);
          const bool valid = 4 * d4 < G.D;
#pragma unroll
          for (int m = 0; m < 3; ++m) {
            const float4 v = valid ? vw[m][u] : float4{0.f, 0.f, 0.f, 0.f};
            float* d = w_ch + (m * G.D16 + 4 * d4) * G.SR + k;
            d[0] = v.x;
            d[G.SR] = v.y;
            d[2 * G.SR] = v.z;
            d[3 * G.SR] = v.w;
          }
        }
      }
    }
    __syncthreads();
    // two K steps per round: the reads of both are issued before the MFMAs
    for (int q = 0; q < G.KC / 16; q += 2) {
      f32x4 x0[kHeadTPW], w0[kHeadTPW], x1[kHeadTPW], w1[kHeadTPW];
#pragma unroll
      for (int j = 0; j < kHeadTPW; ++j) {
        if (wave + kHeadWaves * j < G.T) {
          x0[j] = *reinterpret_cast<const f32x4*>(s_ch + sa[j] + 16 * q);
          w0[j] = *reinterpret_cast<const f32x4*>(w_ch + sb[j] + 16 * q);
          x1[j] = *reinterpret_cast<const f32x4*>(s_ch + sa[j] + 16 * q + 16);
          w1[j] = *reinterpret_cast<const f32x4*>(w_ch + sb[j] + 16 * q + 16);
        }
      }
#pragma unroll
      for (int j = 0; j < kHeadTPW; ++j)
        if (wave + kHeadWaves * j < G.T) acc[j] = mfma4x4(x0[j], w0[j], acc[j]);
#pragma unroll
      for (int j = 0; j < kHeadTPW; ++j)
        if (wave + kHeadWaves * j < G.T) acc[j] = mfma4x4(x1[j], w1[j], acc[j]);
    }
    __syncthreads();  // the chunk buffers are restaged, or become the core's
  }
}

// Projection tiles -> zero-padded Q_h, K_h, V_h tiles ([M16][QS] each at qkv).
__device__ __forceinline__ void head_store_qkv(const HeadGeo& G, const f32x4 (&acc)[kHeadTPW],
                                               const float (&bias)[kHeadTPW], float* qkv, int QS) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
#pragma unroll
  for (int j = 0; j < kHeadTPW; ++j) {
    const int t = wave + kHeadWaves * j;
    if (t >= G.T) continue;
    const HeadTile h = head_tile(G, t);
    const int col = 16 * h.nt + r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 16 * h.mt + 4 * g + i;
      qkv[(h.m * G.M16 + row) * QS + col] = (row < G.M && col < G.D) ? acc[j][i] + bias[j] : 0.f;
    }
  }
}

// Rows [16mt, 16mt + 16) of X Y^T, transposed: lane (r, g) of tile ct holds
// (X Y^T)[16mt + r][16ct + 4g + i] (X, Y: [M16][QS] tiles, K = D16).
__device__ __forceinline__ void head_rows_xyt(const float* X, const float* Y, int mt, int MT,
                                              int D16, int QS, f32x4 (&t)[4]) {
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
    t[ct] = zero4();
    if (ct < MT)
      for (int q = 0; q < D16 / 16; ++q) {
        const f32x4 y = *reinterpret_cast<const f32x4*>(Y + (16 * ct + r) * QS + 16 * q + 4 * g);
        const f32x4 x = *reinterpret_cast<const f32x4*>(X + (16 * mt + r) * QS + 16 * q + 4 * g);
        t[ct] = mfma4x4(y, x, t[ct]);
      }
  }
}

// Row softmax of the transposed score rows (columns >= M masked): P in place.
__device__ __forceinline__ void head_row_softmax(f32x4 (&p)[4], int MT, int M, float scale) {
  const int lane = threadIdx.x & 63, g = lane >> 4;
  float mx = -INFINITY;
#pragma unroll
  for (int ct = 0; ct < 4; ++ct)
    if (ct < MT)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool v = 16 * ct + 4 * g + i < M;
        p[ct][i] = v ? p[ct][i] * scale : -INFINITY;
        mx = fmaxf(mx, p[ct][i]);
      }
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  float sum = 0.f;
#pragma unroll
  for (int ct = 0; ct < 4; ++ct)
    if (ct < MT)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[ct][i] = expf(p[ct][i] - mx);
        sum += p[ct][i];
      }
  sum += __shfl_xor(sum, 16);
  sum += __shfl_xor(sum, 32);
  const float inv = 1.0f / sum;
#pragma unroll
  for (int ct = 0; ct < 4; ++ct)
    if (ct < MT) p[ct] *= inv;
}

// Tile (mt, dt) of A V: A in the transposed-row layout (tiles ct), V a
// [M16][QS] tile in LDS.  Result lane (r, g): row 16mt + 4g + i, column
// 16dt + r.
__device__ __forceinline__ f32x4 head_rows_times(const f32x4 (&A)[4], const float* V, int dt, int MT,
                                                 int QS) {
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  f32x4 o = zero4();
#pragma unroll
  for (int ct = 0; ct < 4; ++ct)
    if (ct < MT)
#pragma unroll
      for (int i = 0; i < 4; ++i) o = mfma4(A[ct][i], V[(16 * ct + 4 * g + i) * QS + 16 * dt + r], o);
  return o;
}

// Global store of a result tile (lane (r, g): row 16 rt + 4g + i, column
// 16 ct + r of the head's [M, D] block of dst).
__device__ __forceinline__ void head_put(float* dst, const f32x4& v, int rt, int ct, int M, int D,
                                         int C, int off, float scale) {
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int col = 16 * ct + r;
  if (col >= D) return;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 16 * rt + 4 * g + i;
    if (row < M) dst[row * C + off + col] = scale * v[i];
  }
}

__global__ void __launch_bounds__(kHeadThreads) k_head_fwd(HeadArgs a) {
  extern __shared__ __attribute__((aligned(16))) float sm[];
  const HeadGeo& G = a.geo;
  const int QS = G.D16 + 4, off = blockIdx.x * G.D, wave = threadIdx.x >> 6;
  f32x4 acc[kHeadTPW];
  float bias[kHeadTPW];
  head_project(a, sm, acc, bias);
  float* qs = sm;
  float* ks = qs + G.M16 * QS;
  float* vs = ks + G.M16 * QS;
  head_store_qkv(G, acc, bias, qs, QS);
  __syncthreads();
  if (wave < G.MT) {
    f32x4 p[4];
    head_rows_xyt(qs, ks, wave, G.MT, G.D16, QS, p);
    head_row_softmax(p, G.MT, G.M, 1.0f / sqrtf((float)G.D));
    for (int dt = 0; dt < G.NT; ++dt)
      head_put(a.O, head_rows_times(p, vs, dt, G.MT, QS), wave, dt, G.M, G.D, G.C, off, 1.f);
  }
}

__global__ void __launch_bounds__(kHeadThreads) k_head_bwd(HeadArgs a) {
  extern __shared__ __attribute__((aligned(16))) float sm[];
  const HeadGeo& G = a.geo;
  const int QS = G.D16 + 4, PS = G.M16 + 4, off = blockIdx.x * G.D, wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int C = G.C, M = G.M, D = G.D, MT = G.MT, NT = G.NT;
  // padded dO_h in registers first: its loads overlap the projections
  const int lD16 = __builtin_ctz(G.D16), nDO = G.M16 * G.D16;
  float dov[kHeadDO];
#pragma unroll
  for (int u = 0; u < kHeadDO; ++u) {
    const int e = threadIdx.x + u * kHeadThreads;
    const int x = e < nDO ? e : nDO - 1;
    const int row = x >> lD16, col = x & (G.D16 - 1);
    const int rr = row < M ? row : M - 1, cc = col < D ? col : D - 1;
    dov[u] = a.dO[rr * C + off + cc];
  }
  f32x4 acc[kHeadTPW];
  float bias[kHeadTPW];
  head_project(a, sm, acc, bias);
  float* qs = sm;
  float* ks = qs + G.M16 * QS;
  float* vs = ks + G.M16 * QS;
  float* os = vs + G.M16 * QS;  // dO_h
  float* ps = os + G.M16 * QS;  // P  [M16][PS]
  float* es = ps + G.M16 * PS;  // dE [M16][PS]
  head_store_qkv(G, acc, bias, qs, QS);
#pragma unroll
  for (int u = 0; u < kHeadDO; ++u) {
    const int e = threadIdx.x + u * kHeadThreads;
    if (e < nDO) {
      const int row = e >> lD16, col = e & (G.D16 - 1);
      os[row * QS + col] = (row < M && col < D) ? dov[u] : 0.f;
    }
  }
  __syncthreads();
  const float scale = 1.0f / sqrtf((float)D);
  if (wave < MT) {
    // P, dP = dO_h V_h^T and dE = P o (dP - rowsum(dP o P)) for the wave's
    // rows; then dQ_h = scale dE K_h (and O_h = P V_h when wanted)
    f32x4 p[4], e[4];
    head_rows_xyt(qs, ks, wave, MT, G.D16, QS, p);
    head_row_softmax(p, MT, M, scale);
    head_rows_xyt(os, vs, wave, MT, G.D16, QS, e);
    float rs = 0.f;
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
      if (ct < MT)
#pragma unroll
        for (int i = 0; i < 4; ++i) rs += e[ct][i] * p[ct][i];
    rs += __shfl_xor(rs, 16);
    rs += __shfl_xor(rs, 32);
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
      if (ct < MT)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          e[ct][i] = p[ct][i] * (e[ct][i] - rs);
          const int o = (16 * wave + r) * PS + 16 * ct + 4 * g + i;
          ps[o] = p[ct][i];
          es[o] = e[ct][i];
        }
    for (int dt = 0; dt < NT; ++dt) {
      head_put(a.dX[0], head_rows_times(e, ks, dt, MT, QS), wave, dt, M, D, C, off, scale);
      if (a.O) head_put(a.O, head_rows_times(p, vs, dt, MT, QS), wave, dt, M, D, C, off, 1.f);
    }
  }
  __syncthreads();
  // dK_h = scale dE^T Q_h and dV_h = P^T dO_h: tiles (which, key tile ct,
  // column tile dt) over the waves; K = the query rows
  for (int t = wave; t < 2 * MT * NT; t += kHeadWaves) {
    const int which = t / (MT * NT), rem = t - which * MT * NT;
    const int ct = rem / NT, dt = rem - ct * NT;
    const float* Am = which == 0 ? es : ps;
    const float* Bm = which == 0 ? qs : os;
    f32x4 o = zero4();
    for (int q = 0; q < MT; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * q + 4 * g + i;
        o = mfma4(Am[row * PS + 16 * ct + r], Bm[row * QS + 16 * dt + r], o);
      }
    head_put(which == 0 ? a.dX[1] : a.dX[2], o, ct, dt, M, D, C, off, which == 0 ? scale : 1.f);
  }
}

// Geometry of the fused head kernels, or false if the head does not fit.
static bool head_geo(int M, int C, int H, bool bwd, HeadGeo& G) {
  if (M < 1 || M > 64 || H < 1 || C % H || C < 16 || (C & (C - 1))) return false;
  G.M = M; G.C = C; G.H = H; G.D = C / H;  // C, and so D, a power of two
  if (G.D % 4) return false;
  G.M16 = (M + 15) / 16 * 16;
  G.D16 = (G.D + 15) / 16 * 16;
  G.MT = G.M16 / 16; G.NT = G.D16 / 16; G.T = 3 * G.MT * G.NT;
  if (G.T > kHeadWaves * kHeadTPW) return false;
  if (bwd && G.M16 * G.D16 > kHeadDO * kHeadThreads) return false;
  const int QS = G.D16 + 4, PS = G.M16 + 4;
  const size_t core = ((size_t)(bwd ? 4 : 3) * G.M16 * QS + (bwd ? 2 : 0) * (size_t)G.M16 * PS) * 4;
  const size_t cap = 150 * 1024;
  if (core > cap) return false;
  for (int kc = C; kc >= 32; kc /= 2) {
    const size_t chunk = ((size_t)G.M16 + 3 * (size_t)G.D16) * (kc + 4) * 4;
    if (chunk <= cap) {
      G.KC = kc;
      G.SR = kc + 4;
      G.lds = chunk > core ? chunk : core;
      return true;
    }
  }
  return false;
}

bool head_fits(int M, int C, int H) {
  HeadGeo G;
  return head_geo(M, C, H, false, G) && head_geo(M, C, H, true, G);
}

hipError_t launch_head(HeadArgs a, bool bwd, hipStream_t st) {
  if (!head_geo(a.geo.M, a.geo.C, a.geo.H, bwd, a.geo)) return hipErrorInvalidConfiguration;
  if (!a.S || !a.W[0] || !a.W[1] || !a.W[2]) return hipErrorInvalidValue;
  if (bwd ? (!a.dO || !a.dX[0] || !a.dX[1] || !a.dX[2]) : !a.O) return hipErrorInvalidValue;
  if (bwd)
    hipLaunchKernelGGL(k_head_bwd, dim3(a.geo.H), dim3(kHeadThreads), a.geo.lds, st, a);
  else
    hipLaunchKernelGGL(k_head_fwd, dim3(a.geo.H), dim3(kHeadThreads), a.geo.lds, st, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// k_token_grads: the parameter-side products of the token backward, all in
// one launch (256 threads per block, fp32 MFMA):
//   blocks [0, nSB): dS tiles (16 x 16) = sum_p X_p W_p^T, K = nS C split
//     over the 4 waves (each lane loads its operands as float4 runs of 4
//     consecutive k straight from global), the 4 partial tiles added in
//     wave order;
//   the rest: one 16 x 16 tile of dW_p = A_p^T B_p per wave (K = M), and for
//     the tiles of row 0 the column sums db_p of B_p.
// ---------------------------------------------------------------------------
constexpr int kGradQ = 12;  // dS K steps (of 16) per wave, at most (C <= 256, nS <= 3)

__global__ void __launch_bounds__(256) k_token_grads(GradArgs a) {
  __shared__ f32x4 red[4][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int M = a.M, C = a.C, CT = C / 16;
  const int nSB = a.nS ? ((M + 15) / 16) * CT : 0;
  if ((int)blockIdx.x < nSB) {
    const int rt = blockIdx.x / CT, ct = blockIdx.x - rt * CT;
    const int Q = a.nS * CT, q0 = wave * Q / 4, nq = (wave + 1) * Q / 4 - q0;
    const int row = 16 * rt + r, rr = row < M ? row : M - 1;
    f32x4 xa[kGradQ], wb[kGradQ];
#pragma unroll
    for (int i = 0; i < kGradQ; ++i) {
      if (i < nq) {
        const int q = q0 + i, p = q / CT, k = 16 * (q - p * CT) + 4 * g;
        const float* X = p == 0 ? a.X[0] : p == 1 ? a.X[1] : a.X[2];
        const float* W = p == 0 ? a.W[0] : p == 1 ? a.W[1] : a.W[2];
        xa[i] = *reinterpret_cast<const f32x4*>(X + (int64_t)rr * C + k);
        wb[i] = *reinterpret_cast<const f32x4*>(W + (int64_t)(16 * ct + r) * C + k);
      }
    }
    f32x4 acc = zero4();
#pragma unroll
    for (int i = 0; i < kGradQ; ++i) {
      if (i < nq) {
        const f32x4 x = row < M ? xa[i] : zero4();
        acc = mfma4(x[0], wb[i][0], acc);
        acc = mfma4(x[1], wb[i][1], acc);
        acc = mfma4(x[2], wb[i][2], acc);
        acc = mfma4(x[3], wb[i][3], acc);
      }
    }
    red[wave][lane] = acc;
    __syncthreads();
    if (wave == 0) {
      const f32x4 t = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int orow = 16 * rt + 4 * g + i;
        if (orow < M) a.dS[(int64_t)orow * C + 16 * ct + r] = t[i];
      }
    }
    return;
  }
  // dW / db tiles: wave -> (product p, row tile ct of channels of A, column tile jt)
  const int gw = ((int)blockIdx.x - nSB) * 4 + wave;
  const int p = gw / (CT * CT), tile = gw - p * CT * CT;
  if (p >= a.nO) return;
  const int ct = tile / CT, jt = tile - ct * CT;
  auto pick = [p](auto const (&v)[4]) { return p == 0 ? v[0] : p == 1 ? v[1] : p == 2 ? v[2] : v[3]; };
  float* dW = pick(a.dW);
  float* db = pick(a.db);
  const bool wantW = dW != nullptr, wantB = db != nullptr && ct == 0;
  if (!wantW && !wantB) return;
  const float* A = pick(a.A);
  const float* Bm = pick(a.B);
  const int S4 = (M + 3) / 4;  // K steps: k = 4 s + g
  float av[16], bv[16];
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    if (s < S4) {
      const int k = 4 * s + g, kk = k < M ? k : M - 1;
      av[s] = A[(int64_t)kk * C + 16 * ct + r];
      bv[s] = Bm[(int64_t)kk * C + 16 * jt + r];
    }
  }
  f32x4 acc = zero4();
  float cs = 0.f;
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    if (s < S4) {
      const bool v = 4 * s + g < M;
      const float x = v ? av[s] : 0.f, y = v ? bv[s] : 0.f;
      acc = mfma4(x, y, acc);
      cs += y;
    }
  }
  if (wantW) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      dW[(int64_t)(16 * ct + 4 * g + i) * C + 16 * jt + r] = acc[i];
  }
  if (wantB) {
    cs += __shfl_xor(cs, 16);
    cs += __shfl_xor(cs, 32);
    if (g == 0) db[16 * jt + r] = cs;
  }
}

hipError_t launch_token_grads(const GradArgs& a, hipStream_t st) {
  if (a.M < 1 || a.M > 64 || a.C < 16 || a.C % 16 || a.C > 256 || a.nS < 0 || a.nS > 3 ||
      a.nO < 0 || a.nO > 4)
    return hipErrorInvalidValue;
  if (a.nS && !a.dS) return hipErrorInvalidValue;
  for (int p = 0; p < a.nS; ++p)
    if (!a.X[p] || !a.W[p]) return hipErrorInvalidValue;
  for (int p = 0; p < a.nO; ++p)
    if (!a.A[p] || !a.B[p]) return hipErrorInvalidValue;
  const int CT = a.C / 16;
  const int nSB = a.nS ? ((a.M + 15) / 16) * CT : 0;
  const int nOB = (a.nO * CT * CT + 3) / 4;
  if (nSB + nOB == 0) return hipSuccess;
  hipLaunchKernelGGL(k_token_grads, dim3(nSB + nOB), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace pa
