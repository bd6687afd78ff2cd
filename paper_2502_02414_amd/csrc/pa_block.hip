// Kernels of the block stack around the Physics-Attention layer (gfx950):
// a Transolver++ block is the Transformer block with Physics-Attention in
// place of attention (Section 3; Figure 2a), read as pre-norm with residual
// adds, x <- x + PA(LN(x)); x <- x + GELU(LN(x) W1 + b1) W2 + b2.
//   - LayerNorm over the C channels of a row, with the residual add that
//     precedes it fused (the sum is written once, in the storage dtype), and
//     its backward with the residual gradient added; the gain and bias
//     gradients are per-block partial sums added in block order;
//   - GELU in its exact form, x Phi(x) with Phi the standard normal CDF
//     (device erf), and its derivative Phi(x) + x phi(x), elementwise;
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
// A wave takes kLnRows row groups (rpw rows each) per iteration of a
// grid-stride loop and issues all their loads before any arithmetic; rows
// past N re-read row N - 1 and are not stored.  The loop bounds and every
// shuffle are uniform within a row group.
// ---------------------------------------------------------------------------
constexpr int kLnRows = 4;

template <typename T>
__global__ void __launch_bounds__(256) k_ln_fwd(LayerNormArgs a) {
  constexpr int E = Vec<T>::E, R = kLnRows;
  const int L = a.C / E, rpw = 64 / L;
  const int lane = threadIdx.x & 63, sub = lane / L, c0 = (lane % L) * E;
  const int64_t gw = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t step = (int64_t)gridDim.x * 4 * R * rpw;
  const T* X = reinterpret_cast<const T*>(a.x);
  const T* Rr = reinterpret_cast<const T*>(a.r);
  // the lane's gains and biases, once (the stores below could alias them)
  float gv[E], bv[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    gv[e] = a.g ? a.g[c0 + e] : 1.f;
    bv[e] = a.b ? a.b[c0 + e] : 0.f;
  }
  for (int64_t base = gw * R * rpw; base < a.N; base += step) {
    float v[R][E];
    int64_t row[R];
#pragma unroll
    for (int k = 0; k < R; ++k) {
      row[k] = base + k * rpw + sub;
      load16<T>(X + (row[k] < a.N ? row[k] : a.N - 1) * a.C + c0, v[k]);
    }
    if (Rr) {
      float rv[R][E];
#pragma unroll
      for (int k = 0; k < R; ++k)
        load16<T>(Rr + (row[k] < a.N ? row[k] : a.N - 1) * a.C + c0, rv[k]);
#pragma unroll
      for (int k = 0; k < R; ++k) {
#pragma unroll
        for (int e = 0; e < E; ++e) v[k][e] = to_f<T>(from_f<T>(v[k][e] + rv[k][e]));
        if (a.xs && row[k] < a.N) store16<T>(reinterpret_cast<T*>(a.xs) + row[k] * a.C + c0, v[k]);
      }
    }
#pragma unroll
    for (int k = 0; k < R; ++k) {
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) s += v[k][e];
      const float mean = group_sum(s, L) / (float)a.C;
      float q = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) q += (v[k][e] - mean) * (v[k][e] - mean);
      const float rstd = 1.0f / sqrtf(group_sum(q, L) / (float)a.C + a.eps);
      float y[E];
#pragma unroll
      for (int e = 0; e < E; ++e)
        y[e] = (v[k][e] - mean) * rstd * gv[e] + bv[e];
      if (row[k] < a.N) {
        store16<T>(reinterpret_cast<T*>(a.y) + row[k] * a.C + c0, y);
        if (lane % L == 0) {
          a.mean[row[k]] = mean;
          a.rstd[row[k]] = rstd;
        }
      }
    }
  }
}

// Backward: with xhat = (s - mean) rstd and gh = dy g,
//   dx = rstd (gh - mean_c(gh) - xhat mean_c(gh xhat)) (+ dres),
// and per-block partial sums of dg = dy xhat, db = dy: each lane adds its
// rows in loop order, then the block's row slots are added in slot order,
// giving the block's record [dg | db] of 2C floats.  The rows a block
// handles are fixed by (N, C, grid), so the sums are deterministic.
template <typename T>
__global__ void __launch_bounds__(256) k_ln_bwd(LayerNormArgs a) {
  constexpr int E = Vec<T>::E, R = kLnRows;
  const int L = a.C / E, rpw = 64 / L, slots = 4 * rpw;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, sub = lane / L;
  const int slot = wave * rpw + sub, c0 = (lane % L) * E;
  const int64_t gw = (int64_t)blockIdx.x * 4 + wave;
  const int64_t step = (int64_t)gridDim.x * 4 * R * rpw;
  const T* X = reinterpret_cast<const T*>(a.x);
  const T* DY = reinterpret_cast<const T*>(a.dy);
  const T* DR = reinterpret_cast<const T*>(a.dres);
  float ag[E], ab[E], gv[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    ag[e] = ab[e] = 0.f;
    gv[e] = a.g ? a.g[c0 + e] : 1.f;
  }
  for (int64_t base = gw * R * rpw; base < a.N; base += step) {
    float v[R][E], dy[R][E], mean[R], rstd[R];
    int64_t row[R];
#pragma unroll
    for (int k = 0; k < R; ++k) {
      row[k] = base + k * rpw + sub;
      const int64_t rr = row[k] < a.N ? row[k] : a.N - 1;
      load16<T>(X + rr * a.C + c0, v[k]);
      load16<T>(DY + rr * a.C + c0, dy[k]);
      mean[k] = a.mean[rr];
      rstd[k] = a.rstd[rr];
    }
#pragma unroll
    for (int k = 0; k < R; ++k) {
      const bool ok = row[k] < a.N;
      float xh[E], gh[E], sg = 0.f, sgx = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        xh[e] = (v[k][e] - mean[k]) * rstd[k];
        gh[e] = dy[k][e] * gv[e];
        sg += gh[e];
        sgx += gh[e] * xh[e];
        if (ok) {
          ag[e] += dy[k][e] * xh[e];
          ab[e] += dy[k][e];
        }
      }
      const float mg = group_sum(sg, L) / (float)a.C, mgx = group_sum(sgx, L) / (float)a.C;
      float dx[E];
#pragma unroll
      for (int e = 0; e < E; ++e) dx[e] = rstd[k] * (gh[e] - mg - xh[e] * mgx);
      if (ok) {
        if (DR) {
          float d2[E];
          load16<T>(DR + row[k] * a.C + c0, d2);
#pragma unroll
          for (int e = 0; e < E; ++e) dx[e] += d2[e];
        }
        store16<T>(reinterpret_cast<T*>(a.dx) + row[k] * a.C + c0, dx);
      }
    }
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
// GELU, y = x Phi(x) with Phi(x) = (1 + erf(x / sqrt 2)) / 2 the standard
// normal CDF, and its derivative dy/dx = Phi(x) + x phi(x), phi(x) =
// exp(-x^2 / 2) / sqrt(2 pi); elementwise (n a multiple of E).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float gelu_f(float x) {
  return 0.5f * x * (1.f + erff(x * 0.7071067811865476f));
}
__device__ __forceinline__ float dgelu_f(float x) {
  const float Phi = 0.5f * (1.f + erff(x * 0.7071067811865476f));
  return fmaf(x * 0.3989422804014327f, expf(-0.5f * x * x), Phi);
}

template <typename T>
__global__ void __launch_bounds__(256) k_gelu(int64_t n, const T* x, const T* dy, T* out) {
  constexpr int E = Vec<T>::E, U = 2;  // U chunks of 16 bytes per thread and iteration
  const int64_t nv = n / E, stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t q0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q0 < nv; q0 += U * stride) {
    float v[U][E], d[U][E];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t q = q0 + u * stride < nv ? q0 + u * stride : q0;
      load16<T>(x + q * E, v[u]);
      if (dy) load16<T>(dy + q * E, d[u]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float o[E];
#pragma unroll
      for (int e = 0; e < E; ++e) o[e] = dy ? d[u][e] * dgelu_f(v[u][e]) : gelu_f(v[u][e]);
      if (q0 + u * stride < nv) store16<T>(out + (q0 + u * stride) * E, o);
    }
  }
}

// ---------------------------------------------------------------------------
// Column sums of x [N, C] (C / E <= 256 column groups of 16 bytes): block b
// sums rows [b R0, (b + 1) R0); thread t owns column group t % CG of every
// RL-th row (RL = 256 / CG row lanes), kLnRows rows' loads in flight; the
// row lanes are then added in order through LDS into the block's record of
// C floats.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) k_colsum(int64_t N, int C, int64_t R0, const T* x,
                                                float* partials) {
  constexpr int E = Vec<T>::E, U = kLnRows;
  const int CG = C / E, RL = 256 / CG;
  const int t = threadIdx.x, rl = t / CG, cg = t % CG;
  const int64_t r0 = (int64_t)blockIdx.x * R0, r1 = r0 + R0 < N ? r0 + R0 : N;
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  if (rl < RL) {
    for (int64_t r = r0 + rl; r < r1; r += (int64_t)RL * U) {
      float v[U][E];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t rr = r + (int64_t)u * RL;
        load16<T>(x + (rr < r1 ? rr : r1 - 1) * C + cg * E, v[u]);
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (r + (int64_t)u * RL < r1)
#pragma unroll
          for (int e = 0; e < E; ++e) acc[e] += v[u][e];
    }
  }
  extern __shared__ float red[];  // [RL][C]
  if (rl < RL)
#pragma unroll
    for (int e = 0; e < E; ++e) red[rl * C + cg * E + e] = acc[e];
  __syncthreads();
  for (int c = t; c < C; c += blockDim.x) {
    float s = 0.f;
    for (int k = 0; k < RL; ++k) s += red[k * C + c];
    partials[(int64_t)blockIdx.x * C + c] = s;
  }
}

// ---------------------------------------------------------------------------
// Algorithm 1's Project step folded (x_proj = h Wp + bp, Wp [C,C] in the
// x*W layout):
//   A' = Wp A,  b' = b + bp A,  a' = Wp a,  b_t' = bp.a   (added to b_t),
// so that the logits and temperature of x_proj are those of h under the
// primed parameters; and the states of x_proj are S_proj = S Wp + bp
// (each point's weights sum to 1).  Sums in fp64, fixed order, rounded once:
// with fp32 storage the projected states feed the token attention, whose
// backward amplifies their rounding (see the double-precision token side).
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(64) k_fold(FoldArgs f) {
  const int C = f.C, M = f.M, t = threadIdx.x;
  if ((int)blockIdx.x < C) {  // row c of A' (threads j < M) and a'[c] (thread M)
    const int c = blockIdx.x;
    for (int j = t; j <= M; j += blockDim.x) {
      double s = 0.0;
      if (j < M) {
        for (int k = 0; k < C; ++k) s += (double)f.Wp[c * C + k] * f.A[k * M + j];
        reinterpret_cast<T*>(f.A_out)[c * M + j] = from_f<T>((float)s);
      } else {
        if (f.a)
          for (int k = 0; k < C; ++k) s += (double)f.Wp[c * C + k] * f.a[k];
        reinterpret_cast<T*>(f.a_out)[c] = from_f<T>((float)s);
      }
    }
  } else {  // b' (threads j < M), b_t' (thread M)
    for (int j = t; j <= M; j += blockDim.x) {
      double s = 0.0;
      if (j < M) {
        s = f.b ? f.b[j] : 0.0;
        for (int k = 0; k < C; ++k) s += (double)f.bp[k] * f.A[k * M + j];
        f.b_out[j] = (float)s;
      } else {
        if (f.a)
          for (int k = 0; k < C; ++k) s += (double)f.bp[k] * f.a[k];
        f.bt_out[0] = (float)s;
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
    double s = bp[k];
    for (int c = 0; c < C; ++c) s += (double)S[j * C + c] * Wp[c * C + k];
    Sp[j * C + k] = (float)s;
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
      double s = 0.0;
      for (int j = 0; j < M; ++j) s += (double)f.dAf[c * M + j] * f.A[k * M + j];
      if (f.a) s += (double)f.daf[c] * f.a[k];
      for (int j = 0; j < M; ++j) s += (double)f.S[j * C + c] * f.dSp[j * C + k];
      f.dWp[c * C + k] = (float)s;
    }
  } else if (bid == C) {
    for (int k = t; k < C; k += blockDim.x) {
      double s = 0.0;
      for (int j = 0; j < M; ++j) s += (double)f.dbf[j] * f.A[k * M + j];
      if (f.a) s += (double)f.dbtf[0] * f.a[k];
      for (int j = 0; j < M; ++j) s += f.dSp[j * C + k];
      f.dbp[k] = (float)s;
    }
    for (int j = t; j < M; j += blockDim.x)
      if (f.db) f.db[j] = f.dbf[j];
    if (t == 0 && f.dbt) f.dbt[0] = f.dbtf[0];
  } else if (bid <= 2 * C) {
    const int k = bid - C - 1;
    for (int j = t; j <= M; j += blockDim.x) {
      double s = 0.0;
      if (j < M) {
        for (int c = 0; c < C; ++c) s += (double)f.Wp[c * C + k] * f.dAf[c * M + j];
        f.dA[k * M + j] = (float)(s + (double)f.bp[k] * f.dbf[j]);
      } else if (f.da) {
        for (int c = 0; c < C; ++c) s += (double)f.Wp[c * C + k] * f.daf[c];
        f.da[k] = (float)(s + (double)f.bp[k] * f.dbtf[0]);
      }
    }
  } else if (f.dS) {
    const int j = bid - 2 * C - 1;
    for (int c = t; c < C; c += blockDim.x) {
      double s = 0.0;
      for (int k = 0; k < C; ++k) s += (double)f.dSp[j * C + k] * f.Wp[c * C + k];
      f.dS[j * C + c] = (float)s;
    }
  }
}

}  // namespace

int layernorm_blocks(int64_t N, int C, int dtype, bool bwd) {
  const int E = dtype == 1 ? 8 : 4;
  const int rpw = 64 / (C / E);
  const int64_t per_block = (int64_t)4 * kLnRows * rpw;  // rows per block iteration
  const int64_t need = (N + per_block - 1) / per_block;
  const int64_t cap = bwd ? kLnPartials : 2048;
  return (int)(need < cap ? need : cap);
}

hipError_t launch_layernorm(const LayerNormArgs& a, int dtype, bool bwd, hipStream_t st) {
  const int E = dtype == 1 ? 8 : 4;
  if (a.C % E || (a.C / E) > 64 || ((a.C / E) & (a.C / E - 1)) || a.N < 1) return hipErrorInvalidValue;
  const int blocks = layernorm_blocks(a.N, a.C, dtype, bwd);
  if (bwd && a.partials && a.blocks != blocks) return hipErrorInvalidValue;
  if (!bwd) {
    if (dtype == 1)
      hipLaunchKernelGGL(k_ln_fwd<bf16>, dim3(blocks), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL(k_ln_fwd<float>, dim3(blocks), dim3(256), 0, st, a);
  } else {
    const size_t lds = (size_t)4 * (64 / (a.C / E)) * 2 * a.C * sizeof(float);
    if (dtype == 1)
      hipLaunchKernelGGL(k_ln_bwd<bf16>, dim3(blocks), dim3(256), lds, st, a);
    else
      hipLaunchKernelGGL(k_ln_bwd<float>, dim3(blocks), dim3(256), lds, st, a);
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

int colsum_blocks(int64_t N) { return (int)(N < kLnPartials ? N : kLnPartials); }

hipError_t launch_colsum(int64_t N, int C, int dtype, const void* x, float* partials, int P,
                         hipStream_t st) {
  const int E = dtype == 1 ? 8 : 4;
  if (N < 1 || C < E || C % E || C / E > 256 || P != colsum_blocks(N)) return hipErrorInvalidValue;
  const int64_t R0 = (N + P - 1) / P;
  const size_t lds = (size_t)(256 / (C / E)) * C * sizeof(float);
  if (dtype == 1)
    hipLaunchKernelGGL(k_colsum<bf16>, dim3(P), dim3(256), lds, st, N, C, R0, (const bf16*)x,
                       partials);
  else
    hipLaunchKernelGGL(k_colsum<float>, dim3(P), dim3(256), lds, st, N, C, R0, (const float*)x,
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
