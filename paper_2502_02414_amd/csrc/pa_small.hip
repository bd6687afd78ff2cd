// Small kernels around the streaming passes (gfx950):
//   - the per-call table image (logits table [A^T ; a], deslice table S'^T,
//     backward table [dnum | S'], biases, dden) in the exact byte layout the
//     streaming kernels copy into LDS;
//   - the ordered reduction of per-block partial-sum records (the partial
//     sums of Section 4.2, here over point chunks of one GPU);
//   - the states s_j = num_j / max(den_j, eps) (Eq. 1);
//   - token attention among the M states and its backward (Eq. 2), built
//     from a small fp32 product kernel and a per-head core kernel.  These
//     work on M <= 64 tokens and are latency-bound, not throughput-bound.
#include "pa_device.hpp"
#include "pa_internal.h"
#include "pa_layout.h"

namespace pa {

// ---------------------------------------------------------------------------
// Table image
// ---------------------------------------------------------------------------
struct PrepGeo {
  int C, M, MB, M16, SZ;
  int TROW, SROW, WROW, OFF_L, OFF_2;
};

static PrepGeo prep_geo(int dtype, int C, int M, int MB) {
  PrepGeo g;
  g.C = C; g.M = M; g.MB = MB; g.M16 = 16 * MB; g.SZ = dtype == 1 ? 2 : 4;
  g.TROW = C * g.SZ + 16;
  g.SROW = g.M16 * g.SZ + 16;
  g.WROW = 2 * C * g.SZ + 16;
  g.OFF_L = (2 * g.M16 + 2 * C) * 4;  // header: bias, dden, cN, cS
  g.OFF_2 = g.OFF_L + (MB + 1) * 16 * g.TROW;
  return g;
}

size_t image_bytes(int pass, int dtype, int C, int MB) {
  PrepGeo g = prep_geo(dtype, C, 16 * MB, MB);
  if (pass == kDeslice) return (size_t)g.OFF_2 + (size_t)C * g.SROW;
  if (pass == kSliceBwd || pass == kWeightsBwd) return (size_t)g.OFF_2 + (size_t)g.M16 * g.WROW;
  return (size_t)g.OFF_2;
}

template <typename T>
__global__ void k_prep(PrepGeo g, PrepArgs p) {
  char* img = reinterpret_cast<char*>(p.img);
  const T* A = reinterpret_cast<const T*>(p.A);
  const T* av = reinterpret_cast<const T*>(p.a);
  const int C = g.C, M = g.M, M16 = g.M16;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t nth = (int64_t)gridDim.x * blockDim.x;
  const bool states = p.dS != nullptr && p.pass == kSliceBwd;
  const bool desl = p.Sp != nullptr && (p.pass == kSliceBwd || p.pass == kDeslice);

  // header: bias[M16]; the backward pass's dden, cN, cS come from
  // k_prep_center (run first); other passes get zeros
  float* hdr = reinterpret_cast<float*>(img);
  for (int64_t j = tid; j < M16; j += nth) hdr[j] = (j < M && p.b) ? p.b[j] : 0.f;
  if (p.pass != kSliceBwd)
    for (int64_t k = tid; k < M16 + 2 * C; k += nth) hdr[M16 + k] = 0.f;
  // logits table: rows j < M16: A[:, j] (0 beyond M); rows M16..M16+15: a
  const int64_t nL = (int64_t)(M16 + 16) * C;
  for (int64_t k = tid; k < nL; k += nth) {
    const int j = (int)(k / C), c = (int)(k - (int64_t)j * C);
    T v;
    if (j < M16)
      v = j < M ? A[(int64_t)c * M + j] : from_f<T>(0.f);
    else
      v = av ? av[c] : from_f<T>(0.f);
    *reinterpret_cast<T*>(img + g.OFF_L + j * g.TROW + c * g.SZ) = v;
  }
  if (p.pass == kDeslice) {
    // S'^T: row c, column j
    const int64_t nS = (int64_t)C * M16;
    for (int64_t k = tid; k < nS; k += nth) {
      const int c = (int)(k / M16), j = (int)(k - (int64_t)c * M16);
      const float v = (j < M) ? p.Sp[j * C + c] : 0.f;
      *reinterpret_cast<T*>(img + g.OFF_2 + c * g.SROW + j * g.SZ) = from_f<T>(v);
    }
  }
  if (p.pass == kSliceBwd || p.pass == kWeightsBwd) {
    // row j: (dnum_j | s'_j)
    const int64_t nW = (int64_t)M16 * 2 * C;
    for (int64_t k = tid; k < nW; k += nth) {
      const int j = (int)(k / (2 * C)), cc = (int)(k - (int64_t)j * 2 * C);
      // rows centred by cN / cS: a shift common to all slices leaves the
      // softmax backward unchanged and keeps the small differences between
      // nearly equal tokens out of the rounding
      float v = 0.f;
      if (j < M) {
        if (cc < C) {
          if (states) {
            const float d = p.den[j] >= p.eps ? p.den[j] : p.eps;
            v = p.dS[j * C + cc] / d - hdr[2 * M16 + cc];
          }
        } else if (desl) {
          v = p.Sp[j * C + (cc - C)] - hdr[2 * M16 + C + (cc - C)];
        }
      }
      *reinterpret_cast<T*>(img + g.OFF_2 + j * g.WROW + cc * g.SZ) = from_f<T>(v);
    }
  }
}

// Backward header: dden_j (chain rule of Eq. 1; 0 when den_j < eps) and
// the centres cN, cS, cD of dnum_j, s'_j, dden_j over slices.  Any centre
// common to all slices leaves the softmax backward unchanged; the mean
// weighted by den_j (the slices' share of the points) keeps a slice with a
// tiny or floored denominator -- whose dnum_j = dS_j / max(den_j, eps) can
// be huge -- from dragging the centre away from the rows that carry weight.
// Without the states term den is not given and cS is the plain mean.  The
// header stores dden_j - cD.  One block.
__global__ void k_prep_center(PrepGeo g, PrepArgs p) {
  __shared__ float sdd[64], sw[64];
  float* hdr = reinterpret_cast<float*>(p.img);
  const int C = g.C, M = g.M, M16 = g.M16;
  const bool states = p.dS != nullptr;
  const bool desl = p.Sp != nullptr;
  for (int j = threadIdx.x; j < 64; j += blockDim.x) {
    float dd = 0.f;
    if (states && j < M && p.den[j] >= p.eps) {
      const float d = p.den[j];
      float s = 0.f;
      for (int c = 0; c < C; ++c) s += p.dS[j * C + c] * (p.num[j * C + c] / d);
      dd = -s / d;
    }
    sdd[j] = dd;
    sw[j] = j < M ? (states ? fmaxf(p.den[j], 0.f) : 1.f) : 0.f;
  }
  __syncthreads();
  float wsum = 0.f;
  for (int j = 0; j < M; ++j) wsum += sw[j];
  const float inv = wsum > 0.f ? 1.0f / wsum : 0.f;
  for (int c = threadIdx.x; c < C; c += blockDim.x) {
    float sn = 0.f, ss = 0.f;
    for (int j = 0; j < M; ++j) {
      if (states) {
        const float d = p.den[j] >= p.eps ? p.den[j] : p.eps;
        sn += sw[j] * (p.dS[j * C + c] / d);
      }
      if (desl) ss += sw[j] * p.Sp[j * C + c];
    }
    hdr[2 * M16 + c] = sn * inv;
    hdr[2 * M16 + C + c] = ss * inv;
  }
  float cD = 0.f;
  for (int j = 0; j < M; ++j) cD += sw[j] * sdd[j];
  cD *= inv;
  for (int j = threadIdx.x; j < M16; j += blockDim.x) hdr[M16 + j] = j < M ? sdd[j] - cD : 0.f;
}

hipError_t launch_prep(const PrepArgs& p, hipStream_t st) {
  if (!p.img || !p.A) return hipErrorInvalidValue;
  if (p.pass == kDeslice && !p.Sp) return hipErrorInvalidValue;
  if (p.pass == kSliceBwd && p.dS && (!p.num || !p.den)) return hipErrorInvalidValue;
  PrepGeo g = prep_geo(p.dtype, p.C, p.M, p.MB);
  if (p.pass == kSliceBwd) {
    hipLaunchKernelGGL(k_prep_center, dim3(1), dim3(256), 0, st, g, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int blocks = 64;
  if (p.dtype == 1)
    hipLaunchKernelGGL(k_prep<bf16>, dim3(blocks), dim3(256), 0, st, g, p);
  else
    hipLaunchKernelGGL(k_prep<float>, dim3(blocks), dim3(256), 0, st, g, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Ordered reduction of partial records
// ---------------------------------------------------------------------------
__global__ void k_reduce(const float* __restrict__ parts, int P, int64_t rec, Segments seg) {
  __shared__ float sh[4][64];
  const int kk = threadIdx.x & 63, pg = threadIdx.x >> 6;
  const int64_t k = (int64_t)blockIdx.x * 64 + kk;
  float s = 0.f;
  if (k < rec)
    for (int p = pg; p < P; p += 4) s += parts[(int64_t)p * rec + k];
  sh[pg][kk] = s;
  __syncthreads();
  if (pg == 0 && k < rec) {
    const float tot = (sh[0][kk] + sh[1][kk]) + (sh[2][kk] + sh[3][kk]);
    int64_t off = k;
    for (int i = 0; i < seg.n; ++i) {
      if (off < seg.len[i]) {
        if (seg.dst[i]) seg.dst[i][off] = tot;
        break;
      }
      off -= seg.len[i];
    }
  }
}

hipError_t launch_reduce(const float* partials, int P, int64_t rec, const Segments& seg,
                         hipStream_t st) {
  if (!partials || P < 1 || rec < 1) return hipErrorInvalidValue;
  const int blocks = (int)((rec + 63) / 64);
  hipLaunchKernelGGL(k_reduce, dim3(blocks), dim3(256), 0, st, partials, P, rec, seg);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// States
// ---------------------------------------------------------------------------
__global__ void k_states(const float* num, const float* den, float* S, int M, int C, float eps) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= (int64_t)M * C) return;
  const int j = (int)(k / C);
  const float d = den[j] >= eps ? den[j] : eps;
  S[k] = num[k] / d;
}

hipError_t launch_states(const float* num, const float* den, float* S, int M, int C, float eps,
                         hipStream_t st) {
  if (!num || !den || !S) return hipErrorInvalidValue;
  const int64_t n = (int64_t)M * C;
  hipLaunchKernelGGL(k_states, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, num, den, S,
                     M, C, eps);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Small fp32 products (token side)
// ---------------------------------------------------------------------------
__global__ void k_gemm(Gemm g) {
  // one 16x16 output tile per block, one output per thread, K in chunks of 16
  __shared__ float sa[16][17], sb[16][17];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int i = blockIdx.y * 16 + ty, j = blockIdx.x * 16 + tx;
  float acc = 0.f;
  for (int k0 = 0; k0 < g.K; k0 += 16) {
    const int ka = k0 + tx, kb = k0 + ty;
    const int ia = blockIdx.y * 16 + ty, jb = blockIdx.x * 16 + tx;
    sa[ty][tx] = (ia < g.rows && ka < g.K) ? g.A[ia * g.sai + ka * g.sak] : 0.f;
    sb[ty][tx] = (kb < g.K && jb < g.cols) ? g.B[kb * g.sbk + jb * g.sbj] : 0.f;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) acc += sa[ty][kk] * sb[kk][tx];
    __syncthreads();
  }
  if (i < g.rows && j < g.cols) {
    if (g.bias) acc += g.bias[j];
    float* o = g.out + (int64_t)i * g.ldo + j;
    *o = g.accumulate ? *o + acc : acc;
  }
}

hipError_t launch_gemm(const Gemm& g, hipStream_t st) {
  if (!g.A || !g.B || !g.out || g.rows < 1 || g.cols < 1 || g.K < 1) return hipErrorInvalidValue;
  dim3 grid((g.cols + 15) / 16, (g.rows + 15) / 16);
  hipLaunchKernelGGL(k_gemm, grid, dim3(256), 0, st, g);
  return hipGetLastError();
}

__global__ void k_colsum(const float* in, int rows, int cols, int64_t ld, float* out) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= cols) return;
  float s = 0.f;
  for (int i = 0; i < rows; ++i) s += in[(int64_t)i * ld + j];
  out[j] = s;
}

hipError_t launch_colsum(const float* in, int rows, int cols, int64_t ld, float* out,
                         hipStream_t st) {
  if (!in || !out) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_colsum, dim3((cols + 255) / 256), dim3(256), 0, st, in, rows, cols, ld,
                     out);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Attention core, one block per head (M <= 64).
// ---------------------------------------------------------------------------
__global__ void k_attn_core(const float* Q, const float* K, const float* V, float* P, float* O,
                            int M, int C, int H) {
  __shared__ float sp[64][65];
  const int h = blockIdx.x, D = C / H, off = h * D;
  const float scale = 1.0f / sqrtf((float)D);
  for (int e = threadIdx.x; e < M * M; e += blockDim.x) {
    const int r = e / M, c = e - r * M;
    float s = 0.f;
    for (int d = 0; d < D; ++d) s += Q[r * C + off + d] * K[c * C + off + d];
    sp[r][c] = s * scale;
  }
  __syncthreads();
  for (int r = threadIdx.x; r < M; r += blockDim.x) {
    float mx = -INFINITY;
    for (int c = 0; c < M; ++c) mx = fmaxf(mx, sp[r][c]);
    float sum = 0.f;
    for (int c = 0; c < M; ++c) {
      const float e = expf(sp[r][c] - mx);
      sp[r][c] = e;
      sum += e;
    }
    const float inv = 1.0f / sum;
    for (int c = 0; c < M; ++c) sp[r][c] *= inv;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < M * M; e += blockDim.x) {
    const int r = e / M, c = e - r * M;
    P[(int64_t)h * M * M + e] = sp[r][c];
  }
  for (int e = threadIdx.x; e < M * D; e += blockDim.x) {
    const int r = e / D, d = e - r * D;
    float s = 0.f;
    for (int c = 0; c < M; ++c) s += sp[r][c] * V[c * C + off + d];
    O[r * C + off + d] = s;
  }
}

hipError_t launch_attn_core(const float* Q, const float* K, const float* V, float* P, float* O,
                            int M, int C, int H, hipStream_t st) {
  if (!Q || !K || !V || !P || !O || M < 1 || M > 64 || H < 1 || C % H) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_attn_core, dim3(H), dim3(256), 0, st, Q, K, V, P, O, M, C, H);
  return hipGetLastError();
}

__global__ void k_attn_core_bwd(const float* Q, const float* K, const float* V, const float* P,
                                const float* dO, float* dQ, float* dK, float* dV, int M, int C,
                                int H) {
  __shared__ float sp[64][65];
  __shared__ float se[64][65];
  const int h = blockIdx.x, D = C / H, off = h * D;
  const float scale = 1.0f / sqrtf((float)D);
  const float* Ph = P + (int64_t)h * M * M;
  for (int e = threadIdx.x; e < M * M; e += blockDim.x) {
    const int r = e / M, c = e - r * M;
    sp[r][c] = Ph[e];
    float s = 0.f;  // dP = dO_h V_h^T
    for (int d = 0; d < D; ++d) s += dO[r * C + off + d] * V[c * C + off + d];
    se[r][c] = s;
  }
  __syncthreads();
  for (int r = threadIdx.x; r < M; r += blockDim.x) {
    float rs = 0.f;
    for (int c = 0; c < M; ++c) rs += se[r][c] * sp[r][c];
    for (int c = 0; c < M; ++c) se[r][c] = sp[r][c] * (se[r][c] - rs);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < M * D; e += blockDim.x) {
    const int r = e / D, d = e - r * D;
    float sv = 0.f, sq = 0.f, sk = 0.f;
    for (int c = 0; c < M; ++c) {
      sv += sp[c][r] * dO[c * C + off + d];
      sq += se[r][c] * K[c * C + off + d];
      sk += se[c][r] * Q[c * C + off + d];
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
  hipLaunchKernelGGL(k_attn_core_bwd, dim3(H), dim3(256), 0, st, Q, K, V, P, dO, dQ, dK, dV, M,
                     C, H);
  return hipGetLastError();
}

}  // namespace pa
