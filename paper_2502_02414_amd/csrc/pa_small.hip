// Small kernels around the streaming passes (gfx950):
//   - the per-call table image (logits table [A^T ; a], deslice table S'^T,
//     backward table [dnum | S'], biases, dden) in the exact byte layout the
//     streaming kernels copy into LDS (rows of the logits and backward tables
//     padded as in pa_layout.h);
//   - the ordered reduction of per-block partial-sum records (the partial
//     sums of Section 4.2, here over point chunks of one GPU);
//     with the states s_j = num_j / max(den_j, eps) (Eq. 1) formed there;
// (token attention lives in pa_tokens.hip).
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
  g.TROW = C * g.SZ + 32;
  g.SROW = g.M16 * g.SZ + 16;
  g.WROW = 2 * C * g.SZ + 32;
  g.OFF_L = (3 * g.M16 + 3 * C) * 4;  // header: bias, dden, cN, cS, sw, a
  g.OFF_2 = g.OFF_L + (g.M16 + 1) * g.TROW;
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
  // padded slices j >= M get bias -inf: their softmax weight is exactly 0
  for (int64_t j = tid; j < M16; j += nth) hdr[j] = j < M ? (p.b ? p.b[j] : 0.f) : -INFINITY;
  if (p.pass != kSliceBwd)
    for (int64_t k = tid; k < 2 * M16 + 2 * C; k += nth) hdr[M16 + k] = 0.f;
  for (int64_t c = tid; c < C; c += nth) hdr[3 * M16 + 2 * C + c] = av ? to_f<T>(av[c]) : 0.f;
  // logits table: rows j < M16: A[:, j] (0 beyond M); row M16: a
  const int64_t nL = (int64_t)(M16 + 1) * C;
#pragma unroll 4
  for (int64_t k = tid; k < nL; k += nth) {
    const int j = (int)(k / C), c = (int)(k - (int64_t)j * C);
    T v;
    if (j < M16)
      v = j < M ? A[(int64_t)c * M + j] : from_f<T>(0.f);
    else
      v = av ? av[c] : from_f<T>(0.f);
    *reinterpret_cast<T*>(img + g.OFF_L + lds_off(j, c * g.SZ, g.TROW)) = v;
  }
  if (p.pass == kDeslice) {
    // S'^T: row c, column j
    const int64_t nS = (int64_t)C * M16;
#pragma unroll 4
    for (int64_t k = tid; k < nS; k += nth) {
      const int c = (int)(k / M16), j = (int)(k - (int64_t)c * M16);
      const float v = (j < M) ? p.Sp[j * C + c] : 0.f;
      *reinterpret_cast<T*>(img + g.OFF_2 + c * g.SROW + j * g.SZ) = from_f<T>(v);
    }
  }
  if (p.pass == kSliceBwd || p.pass == kWeightsBwd) {
    // row j: (dnum_j | s'_j)
    const int64_t nW = (int64_t)M16 * 2 * C;
#pragma unroll 4
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
      *reinterpret_cast<T*>(img + g.OFF_2 + lds_off(j, cc * g.SZ, g.WROW)) = from_f<T>(v);
    }
  }
}

// Backward header: dden_j (chain rule of Eq. 1; 0 when den_j < eps), the
// normalised slice weights sw_j = den_j / sum den, and the centres cN, cS of
// dnum_j, s'_j over slices.  Any centre common to all slices leaves the
// softmax backward unchanged; the mean weighted by den_j (the slices' share
// of the points) keeps a slice with a tiny or floored denominator -- whose
// dnum_j = dS_j / max(den_j, eps) can be huge -- from dragging the centre
// away from the rows that carry weight.  Without the states term den is not
// given and the weights are uniform.  Blocks [0, M) reduce dden_j over C;
// the others compute the centres of 256 channels each.
__global__ void k_prep_center(PrepGeo g, PrepArgs p) {
  __shared__ float red[256];
  float* hdr = reinterpret_cast<float*>(p.img);
  const int C = g.C, M = g.M, M16 = g.M16;
  const bool states = p.dS != nullptr;
  const bool desl = p.Sp != nullptr;
  if ((int)blockIdx.x < M) {
    const int j = blockIdx.x;
    float s = 0.f;
    if (states && p.den[j] >= p.eps) {
      const float d = p.den[j];
      for (int c = threadIdx.x; c < C; c += 256) s += p.dS[j * C + c] * (p.num[j * C + c] / d);
    }
    red[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      const float dd = (states && p.den[j] >= p.eps) ? -red[0] / p.den[j] : 0.f;
      hdr[M16 + j] = dd;
      float wsum = 0.f;
#pragma unroll 8
      for (int k = 0; k < M; ++k) wsum += states ? fmaxf(p.den[k], 0.f) : 1.f;
      hdr[2 * M16 + 2 * C + j] = (states ? fmaxf(p.den[j], 0.f) : 1.f) / wsum;
    }
    if (j == 0)
      for (int k = M + threadIdx.x; k < M16; k += blockDim.x) {
        hdr[M16 + k] = 0.f;
        hdr[2 * M16 + 2 * C + k] = 0.f;
      }
    return;
  }
  const int c = (blockIdx.x - M) * blockDim.x + threadIdx.x;
  if (c >= C) return;
  float wsum = 0.f, sn = 0.f, ss = 0.f;
  // weights and values for 8 slices at a time, loads first
  for (int j0 = 0; j0 < M; j0 += 8) {
    float wj[8], dv[8], sv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = j0 + u < M ? j0 + u : M - 1;
      wj[u] = states ? p.den[j] : 1.f;
      dv[u] = states ? p.dS[j * C + c] : 0.f;
      sv[u] = desl ? p.Sp[j * C + c] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (j0 + u >= M) break;
      const float w = states ? fmaxf(wj[u], 0.f) : 1.f;
      const float d = wj[u] >= p.eps ? wj[u] : p.eps;
      wsum += w;
      sn += w * (dv[u] / d);
      ss += w * sv[u];
    }
  }
  const float inv = wsum > 0.f ? 1.0f / wsum : 0.f;
  hdr[2 * M16 + c] = sn * inv;
  hdr[2 * M16 + C + c] = ss * inv;
}

hipError_t launch_prep(const PrepArgs& p, hipStream_t st) {
  if (!p.img || !p.A) return hipErrorInvalidValue;
  if (p.pass == kDeslice && !p.Sp) return hipErrorInvalidValue;
  if (p.pass == kSliceBwd && p.dS && (!p.num || !p.den)) return hipErrorInvalidValue;
  PrepGeo g = prep_geo(p.dtype, p.C, p.M, p.MB);
  if (p.pass == kSliceBwd) {
    hipLaunchKernelGGL(k_prep_center, dim3(p.M + (p.C + 255) / 256), dim3(256), 0, st, g, p);
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
// Ordered reduction of partial records (and the states of Eq. 1)
// ---------------------------------------------------------------------------
// Fixed-order sum of the 16 group sums of one column.
__device__ __forceinline__ float group_total(const double (&t16)[16]) {
  double t[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) t[q] = t16[2 * q] + t16[2 * q + 1];
  return (float)(((t[0] + t[1]) + (t[2] + t[3])) + ((t[4] + t[5]) + (t[6] + t[7])));
}

__global__ void k_reduce(const float* __restrict__ parts, int P, int64_t rec, Segments seg) {
  // 16 record columns x 16 partial groups per block: each thread adds every
  // 16th partial (few dependent loads per thread), then the 16 group sums
  // are added in a fixed tree order.  The sums are formed in fp64: the
  // records are signed partial sums (gradients) whose total can be far
  // smaller than the sum of their magnitudes.  A block of numerator columns
  // (16 columns of one slice j, as 16 divides C) also forms den_j, in the
  // same order as den_j's own block, for the states.
  __shared__ double sh[17][16];
  const int kk = threadIdx.x & 15, pg = threadIdx.x >> 4;
  const int64_t k0 = (int64_t)blockIdx.x * 16, k = k0 + kk;
  const bool states = seg.S != nullptr && k0 < seg.nS;
  double acc = 0.0;
  if (k < rec) {
#pragma unroll 8
    for (int p = pg; p < P; p += 16) acc += (double)parts[(int64_t)p * rec + k];
  }
  sh[kk][pg] = acc;
  if (states && kk == 0) {
    const int64_t dc = seg.den_col + k0 / seg.C;
    double ad = 0.0;
#pragma unroll 8
    for (int p = pg; p < P; p += 16) ad += (double)parts[(int64_t)p * rec + dc];
    sh[16][pg] = ad;
  }
  __syncthreads();
  if (pg == 0 && k < rec) {
    const float tot = group_total(sh[kk]);
    int64_t off = k;
    for (int i = 0; i < seg.n; ++i) {
      if (off < seg.len[i]) {
        if (seg.dst[i]) seg.dst[i][off] = tot;
        if (seg.dst2[i]) seg.dst2[i][off] = tot;
        break;
      }
      off -= seg.len[i];
    }
    if (states && k < seg.nS) {
      const float den = group_total(sh[16]);
      seg.S[k] = tot / (den >= seg.eps ? den : seg.eps);
    }
  }
}

hipError_t launch_reduce(const float* partials, int P, int64_t rec, const Segments& seg,
                         hipStream_t st) {
  if (!partials || P < 1 || rec < 1) return hipErrorInvalidValue;
  if (seg.S && (seg.C < 16 || seg.C % 16 || seg.nS > rec || seg.den_col < 0 ||
                seg.den_col + seg.nS / seg.C > rec))
    return hipErrorInvalidValue;
  const int blocks = (int)((rec + 15) / 16);
  hipLaunchKernelGGL(k_reduce, dim3(blocks), dim3(256), 0, st, partials, P, rec, seg);
  return hipGetLastError();
}

}  // namespace pa
