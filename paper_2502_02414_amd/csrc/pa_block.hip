// Kernels of the block stack around the Physics-Attention layer (gfx950):
// a Transolver++ block is the Transformer block with Physics-Attention in
// place of attention (Section 3; Figure 2a), read as pre-norm with residual
// adds, x <- x + PA(LN(x)); x <- x + GELU(LN(x) W1 + b1) W2 + b2.
//   - LayerNorm over the C channels of a row, with the residual add that
//     precedes it fused (the sum is written once, in the storage dtype), and
//     its backward with the residual gradient added; the gain and bias
//     gradients are per-block partial sums added in block order;
//   - exact GELU (x Phi(x), erf) and its derivative, elementwise;
//   - column sums of a [N, C] matrix (the bias gradients of the linear
//     layers), deterministic;
//   - Algorithm 1's Project step x_proj = h Wp + bp folded into the slice
//     parameters and the states (the layer then runs on h), and the chain
//     rule of that folding.
// Row kernels hold 16 bytes of a row per lane (8 bf16 or 4 fp32 channels):
// L = C / E lanes per row, 64 / L rows per wave; row sums reduce across the
// L lanes with xor shuffles.
#include "pa_device.hpp"
#include "pa_internal.h"

namespace pa {
namespace {

template <typename T> struct Vec { static constexpr int E = 16 / (int)sizeof(T); };

template <typename T>
__device__ __forceinline__ void load16(const T* p, float (&v)[Vec<T>::E]) {
  const uint4 q = *reinterpret_cast<const uint4*>(p);
  if constexpr (sizeof(T) == 2) {
    const bf16x8 b = __builtin_bit_cast(bf16x8, q);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (float)b[e];
  } else {
    const f32x4 f = __builtin_bit_cast(f32x4, q);
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = f[e];
  }
}

template <typename T>
__device__ __forceinline__ void store16(T* p, const float (&v)[Vec<T>::E]) {
  if constexpr (sizeof(T) == 2) {
    bf16x8 b;
#pragma unroll
    for (int e = 0; e < 8; ++e) b[e] = (bf16)v[e];
    *reinterpret_cast<uint4*>(p) = __builtin_bit_cast(uint4, b);
  } else {
    f32x4 f;
#pragma unroll
    for (int e = 0; e < 4; ++e) f[e] = v[e];
    *reinterpret_cast<uint4*>(p) = __builtin_bit_cast(uint4, f);
  }
}

// Sum over the L lanes of a row group (L a power of two, groups aligned).
__device__ __forceinline__ float group_sum(float v, int L) {
  for (int o = 1; o < L; o <<= 1) v += __shfl_xor(v, o);
  return v;
}

// ---------------------------------------------------------------------------
// LayerNorm: s = x (+ r, rounded to the storage dtype; written to xs when
// given); y = (s - mean) rstd g + b with rstd = 1 / sqrt(var + eps), var the
// biased variance; mean and rstd [N] saved for the backward.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) k_ln_fwd(LayerNormArgs a) {
  constexpr int E = Vec<T>::E;
  const int L = a.C / E, rpw = 64 / L;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = ((int64_t)blockIdx.x * 4 + wave) * rpw + lane / L;
  const int c0 = (lane % L) * E;
  if (row >= a.N) return;  // whole row groups leave together (their shuffles stay within the group)
  const T* x = reinterpret_cast<const T*>(a.x) + row * a.C + c0;
  float v[E];
  load16<T>(x, v);
  if (a.r) {
    float rv[E];
    load16<T>(reinterpret_cast<const T*>(a.r) + row * a.C + c0, rv);
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = to_f<T>(from_f<T>(v[e] + rv[e]));
    if (a.xs) store16<T>(reinterpret_cast<T*>(a.xs) + row * a.C + c0, v);
  }
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) s += v[e];
  const float mean = group_sum(s, L) / (float)a.C;
  float q = 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) q += (v[e] - mean) * (v[e] - mean);
  const float rstd = 1.0f / sqrtf(group_sum(q, L) / (float)a.C + a.eps);
  float y[E];
#pragma unroll
  for (int e = 0; e < E; ++e)
    y[e] = (v[e] - mean) * rstd * (a.g ? a.g[c0 + e] : 1.f) + (a.b ? a.b[c0 + e] : 0.f);
  store16<T>(reinterpret_cast<T*>(a.y) + row * a.C + c0, y);
  if (lane % L == 0) {
    a.mean[row] = mean;
    a.rstd[row] = rstd;
  }
}

// Backward: with xhat = (s - mean) rstd and gh = dy g,
//   dx = rstd (gh - mean_c(gh) - xhat mean_c(gh xhat)) (+ dres),
// and per-block partial sums of dg = dy xhat, db = dy over the block's rows
// (rows [blockIdx.x * R, +R), each lane's rows in order, then the block's
// row slots in order), written as record [dg | db] of 2C floats.
template <typename T>
__global__ void __launch_bounds__(256) k_ln_bwd(LayerNormArgs a) {
  constexpr int E = Vec<T>::E;
  const int L = a.C / E, rpw = 64 / L, slots = 4 * rpw;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int slot = wave * rpw + lane / L;
  const int c0 = (lane % L) * E;
  const int64_t r0 = (int64_t)blockIdx.x * a.rows_per_block;
  const int64_t r1 = r0 + a.rows_per_block < a.N ? r0 + a.rows_per_block : a.N;
  float ag[E], ab[E];
#pragma unroll
  for (int e = 0; e < E; ++e) ag[e] = ab[e] = 0.f;
  // every lane of a row group runs the same number of iterations
  for (int64_t row = r0 + slot; row < r1; row += slots) {
    float v[E], dy[E];
    load16<T>(reinterpret_cast<const T*>(a.x) + row * a.C + c0, v);
    load16<T>(reinterpret_cast<const T*>(a.dy) + row * a.C + c0, dy);
    const float mean = a.mean[row], rstd = a.rstd[row];
    float xh[E], gh[E], sg = 0.f, sgx = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      xh[e] = (v[e] - mean) * rstd;
      gh[e] = dy[e] * (a.g ? a.g[c0 + e] : 1.f);
      sg += gh[e];
      sgx += gh[e] * xh[e];
      ag[e] += dy[e] * xh[e];
      ab[e] += dy[e];
    }
    const float mg = group_sum(sg, L) / (float)a.C, mgx = group_sum(sgx, L) / (float)a.C;
    float dx[E];
#pragma unroll
    for (int e = 0; e < E; ++e) dx[e] = rstd * (gh[e] - mg - xh[e] * mgx);
    if (a.dres) {
      float d2[E];
      load16<T>(reinterpret_cast<const T*>(a.dres) + row * a.C + c0, d2);
#pragma unroll
      for (int e = 0; e < E; ++e) dx[e] += d2[e];
    }
    store16<T>(reinterpret_cast<T*>(a.dx) + row * a.C + c0, dx);
  }
  if (!a.partials) return;
  extern __shared__ float red[];  // [slots][2C]
#pragma unroll
  for (int e = 0; e < E; ++e) {
    red[slot * 2 * a.C + c0 + e] = ag[e];
    red[slot * 2 * a.C + a.C + c0 + e] = ab[e];
  }
  __syncthreads();
  for (int k = threadIdx.x; k < 2 * a.C; k += blockDim.x) {
    float t = 0.f;
    for (int s2 = 0; s2 < slots; ++s2) t += red[s2 * 2 * a.C + k];
    a.partials[(int64_t)blockIdx.x * 2 * a.C + k] = t;
  }
}

// ---------------------------------------------------------------------------
// Exact GELU and its derivative, elementwise (n a multiple of E).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float gelu_f(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }
__device__ __forceinline__ float dgelu_f(float x) {
  const float cdf = 0.5f * (1.f + erff(x * 0.70710678118654752f));
  const float pdf = 0.39894228040143268f * expf(-0.5f * x * x);
  return cdf + x * pdf;
}

template <typename T>
__global__ void __launch_bounds__(256) k_gelu(int64_t n, const T* x, const T* dy, T* out) {
  constexpr int E = Vec<T>::E;
  const int64_t nv = n / E;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < nv;
       q += (int64_t)gridDim.x * blockDim.x) {
    float v[E], o[E];
    load16<T>(x + q * E, v);
    if (dy) {
      float d[E];
      load16<T>(dy + q * E, d);
#pragma unroll
      for (int e = 0; e < E; ++e) o[e] = d[e] * dgelu_f(v[e]);
    } else {
#pragma unroll
      for (int e = 0; e < E; ++e) o[e] = gelu_f(v[e]);
    }
    store16<T>(out + q * E, o);
  }
}

// ---------------------------------------------------------------------------
// Column sums of x [N, C]: block b sums rows [b R, (b + 1) R) in order into
// its record of C floats (threads over columns).
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) k_colsum(int64_t N, int C, int64_t R, const T* x,
                                                float* partials) {
  const int64_t r0 = (int64_t)blockIdx.x * R, r1 = r0 + R < N ? r0 + R : N;
  for (int c = threadIdx.x; c < C; c += blockDim.x) {
    float s = 0.f;
#pragma unroll 8
    for (int64_t r = r0; r < r1; ++r) s += to_f<T>(x[r * C + c]);
    partials[(int64_t)blockIdx.x * C + c] = s;
  }
}

// ---------------------------------------------------------------------------
// Algorithm 1's Project step folded (x_proj = h Wp + bp, Wp [C,C] in the
// x*W layout):
//   A' = Wp A,  b' = b + bp A,  a' = Wp a,  b_t' = bp.a   (added to b_t),
// so that the logits and temperature of x_proj are those of h under the
// primed parameters; and the states of x_proj are S_proj = S Wp + bp
// (each point's weights sum to 1).  Sums in fp32, fixed order.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(64) k_fold(FoldArgs f) {
  const int C = f.C, M = f.M, t = threadIdx.x;
  if ((int)blockIdx.x < C) {  // row c of A' (threads j < M) and a'[c] (thread M)
    const int c = blockIdx.x;
    for (int j = t; j <= M; j += blockDim.x) {
      float s = 0.f;
      if (j < M) {
        for (int k = 0; k < C; ++k) s += f.Wp[c * C + k] * f.A[k * M + j];
        reinterpret_cast<T*>(f.A_out)[c * M + j] = from_f<T>(s);
      } else {
        if (f.a)
          for (int k = 0; k < C; ++k) s += f.Wp[c * C + k] * f.a[k];
        reinterpret_cast<T*>(f.a_out)[c] = from_f<T>(s);
      }
    }
  } else {  // b' (threads j < M), b_t' (thread M)
    for (int j = t; j <= M; j += blockDim.x) {
      float s = 0.f;
      if (j < M) {
        s = f.b ? f.b[j] : 0.f;
        for (int k = 0; k < C; ++k) s += f.bp[k] * f.A[k * M + j];
        f.b_out[j] = s;
      } else {
        if (f.a)
          for (int k = 0; k < C; ++k) s += f.bp[k] * f.a[k];
        f.bt_out[0] = s;
      }
    }
  }
}

// S_proj [M,C] = S Wp + bp (block j, threads over the output channel k).
__global__ void __launch_bounds__(256) k_project_states(int M, int C, const float* S,
                                                        const float* Wp, const float* bp,
                                                        float* Sp) {
  const int j = blockIdx.x;
  for (int k = threadIdx.x; k < C; k += blockDim.x) {
    float s = bp[k];
    for (int c = 0; c < C; ++c) s += S[j * C + c] * Wp[c * C + k];
    Sp[j * C + k] = s;
  }
}

// Chain rule of the folding, from the gradients of the primed parameters
// (dA', db', da', db_t') and of the projected states dS_proj:
//   dWp[c,k] = sum_j dA'[c,j] A[k,j] + da'[c] a[k] + sum_j S[j,c] dSp[j,k]
//   dbp[k]   = sum_j db'[j] A[k,j] + db_t' a[k] + sum_j dSp[j,k]
//   dA[k,j]  = sum_c Wp[c,k] dA'[c,j] + bp[k] db'[j]
//   da[k]    = sum_c Wp[c,k] da'[c] + bp[k] db_t'
//   dS[j,c]  = sum_k dSp[j,k] Wp[c,k];  db = db', db_t = db_t'.
// Blocks [0, C): dWp row c; block C: dbp, db, db_t; blocks (C, 2C]: dA row
// k and da[k]; blocks (2C, 2C + M]: dS row j.
__global__ void __launch_bounds__(256) k_fold_grads(FoldGradArgs f) {
  const int C = f.C, M = f.M, t = threadIdx.x;
  const int bid = blockIdx.x;
  if (bid < C) {
    const int c = bid;
    for (int k = t; k < C; k += blockDim.x) {
      float s = 0.f;
      for (int j = 0; j < M; ++j) s += f.dAf[c * M + j] * f.A[k * M + j];
      if (f.a) s += f.daf[c] * f.a[k];
      for (int j = 0; j < M; ++j) s += f.S[j * C + c] * f.dSp[j * C + k];
      f.dWp[c * C + k] = s;
    }
  } else if (bid == C) {
    for (int k = t; k < C; k += blockDim.x) {
      float s = 0.f;
      for (int j = 0; j < M; ++j) s += f.dbf[j] * f.A[k * M + j];
      if (f.a) s += f.dbtf[0] * f.a[k];
      for (int j = 0; j < M; ++j) s += f.dSp[j * C + k];
      f.dbp[k] = s;
    }
    for (int j = t; j < M; j += blockDim.x)
      if (f.db) f.db[j] = f.dbf[j];
    if (t == 0 && f.dbt) f.dbt[0] = f.dbtf[0];
  } else if (bid <= 2 * C) {
    const int k = bid - C - 1;
    for (int j = t; j <= M; j += blockDim.x) {
      float s = 0.f;
      if (j < M) {
        for (int c = 0; c < C; ++c) s += f.Wp[c * C + k] * f.dAf[c * M + j];
        f.dA[k * M + j] = s + f.bp[k] * f.dbf[j];
      } else if (f.da) {
        for (int c = 0; c < C; ++c) s += f.Wp[c * C + k] * f.daf[c];
        f.da[k] = s + f.bp[k] * f.dbtf[0];
      }
    }
  } else if (f.dS) {
    const int j = bid - 2 * C - 1;
    for (int c = t; c < C; c += blockDim.x) {
      float s = 0.f;
      for (int k = 0; k < C; ++k) s += f.dSp[j * C + k] * f.Wp[c * C + k];
      f.dS[j * C + c] = s;
    }
  }
}

}  // namespace

hipError_t launch_layernorm(const LayerNormArgs& a, int dtype, bool bwd, hipStream_t st) {
  const int E = dtype == 1 ? 8 : 4;
  if (a.C % E || (a.C / E) > 64 || ((a.C / E) & (a.C / E - 1)) || a.N < 1) return hipErrorInvalidValue;
  const int rpb = 4 * (64 / (a.C / E));  // rows per block-iteration
  if (!bwd) {
    const int64_t blocks = (a.N + rpb - 1) / rpb;
    if (dtype == 1)
      hipLaunchKernelGGL(k_ln_fwd<bf16>, dim3((unsigned)blocks), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL(k_ln_fwd<float>, dim3((unsigned)blocks), dim3(256), 0, st, a);
  } else {
    const size_t lds = (size_t)rpb * 2 * a.C * sizeof(float);
    const int P = a.blocks;
    if (dtype == 1)
      hipLaunchKernelGGL(k_ln_bwd<bf16>, dim3(P), dim3(256), lds, st, a);
    else
      hipLaunchKernelGGL(k_ln_bwd<float>, dim3(P), dim3(256), lds, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_gelu(int64_t n, int dtype, const void* x, const void* dy, void* out,
                       hipStream_t st) {
  const int E = dtype == 1 ? 8 : 4;
  if (n < 1 || n % E) return hipErrorInvalidValue;
  const int64_t nv = n / E;
  const unsigned blocks = (unsigned)(nv / 256 + 1 < 8192 ? nv / 256 + 1 : 8192);
  if (dtype == 1)
    hipLaunchKernelGGL(k_gelu<bf16>, dim3(blocks), dim3(256), 0, st, n, (const bf16*)x,
                       (const bf16*)dy, (bf16*)out);
  else
    hipLaunchKernelGGL(k_gelu<float>, dim3(blocks), dim3(256), 0, st, n, (const float*)x,
                       (const float*)dy, (float*)out);
  return hipGetLastError();
}

hipError_t launch_colsum(int64_t N, int C, int dtype, const void* x, float* partials, int P,
                         hipStream_t st) {
  if (N < 1 || C < 1 || P < 1) return hipErrorInvalidValue;
  const int64_t R = (N + P - 1) / P;
  if (dtype == 1)
    hipLaunchKernelGGL(k_colsum<bf16>, dim3(P), dim3(256), 0, st, N, C, R, (const bf16*)x,
                       partials);
  else
    hipLaunchKernelGGL(k_colsum<float>, dim3(P), dim3(256), 0, st, N, C, R, (const float*)x,
                       partials);
  return hipGetLastError();
}

hipError_t launch_fold(const FoldArgs& f, int dtype, hipStream_t st) {
  if (f.C < 1 || f.M < 1 || !f.Wp || !f.bp || !f.A || !f.A_out || !f.a_out || !f.b_out || !f.bt_out)
    return hipErrorInvalidValue;
  if (dtype == 1)
    hipLaunchKernelGGL(k_fold<bf16>, dim3(f.C + 1), dim3(64), 0, st, f);
  else
    hipLaunchKernelGGL(k_fold<float>, dim3(f.C + 1), dim3(64), 0, st, f);
  return hipGetLastError();
}

hipError_t launch_project_states(int M, int C, const float* S, const float* Wp, const float* bp,
                                 float* Sp, hipStream_t st) {
  if (M < 1 || C < 1 || !S || !Wp || !bp || !Sp) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_project_states, dim3(M), dim3(256), 0, st, M, C, S, Wp, bp, Sp);
  return hipGetLastError();
}

hipError_t launch_fold_grads(const FoldGradArgs& f, hipStream_t st) {
  if (f.C < 1 || f.M < 1 || !f.Wp || !f.bp || !f.A || !f.S || !f.dSp || !f.dAf || !f.dbf ||
      !f.daf || !f.dbtf || !f.dWp || !f.dbp || !f.dA)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_fold_grads, dim3(2 * f.C + 1 + f.M), dim3(256), 0, st, f);
  return hipGetLastError();
}

}  // namespace pa
