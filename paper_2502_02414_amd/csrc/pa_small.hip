// Small kernels around the streaming passes (gfx950):
//   - the per-call table image (logits table [A^T ; a], deslice table S'^T,
//     backward table [dnum | S'] with its centres, biases, dden) in the exact
//     byte layout the streaming kernels copy into LDS (rows of the logits and
//     backward tables padded as in pa_layout.h), one launch per call;
//   - the ordered reduction of per-block partial-sum records (the partial
//     sums of Section 4.2, here over point chunks of one GPU);
//     with the states s_j = num_j / max(den_j, eps) (Eq. 1) formed there;
// (token attention lives in pa_tokens.hip).
#include <type_traits>

#include "pa_device.hpp"
#include "pa_internal.h"
#include "pa_layout.h"

namespace pa {

// ---------------------------------------------------------------------------
// Table image
// ---------------------------------------------------------------------------
struct PrepGeo {
  int C, M, MB, M16, SZ;  // C: the tables' width (the parameters' cr <= C channels, zeros beyond)
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
  if (pass == kDeslice || pass == kDesliceW) return (size_t)g.OFF_2 + (size_t)C * g.SROW;
  if (pass == kDesliceBwdW) return 0;
  if (pass == kSliceBwd || pass == kWeightsBwd) return (size_t)g.OFF_2 + (size_t)g.M16 * g.WROW;
  return (size_t)g.OFF_2;
}

// The backward header and table (kSliceBwd, kWeightsBwd), block `bid` of
// M + ceil(2C/256):
//   blocks [0, M): dden_j (chain rule of Eq. 1; 0 when den_j < eps), reduced
//     over C in a fixed tree, and sw_j = w_j / sum w;
//   the others: one column cc of the backward table per thread (dnum for
//     cc < C, s' beyond), its centre cN[c] / cS[c] and its M16 rows.
// Any centre common to all slices leaves the softmax backward unchanged;
// the mean weighted by w_j = max(den_j, 0) (the slices' share of the points)
// keeps a slice with a tiny or floored denominator -- whose dnum_j =
// dS_j / max(den_j, eps) can be huge -- from dragging the centre away from
// the rows that carry weight, and keeps the small differences between nearly
// equal rows out of the rounding.  Without the states term den is not given
// and the weights are uniform; kWeightsBwd has neither term (zeros).
template <typename T>
__device__ __forceinline__ void prep_back(const PrepGeo& g, const PrepArgs& p, int bid,
                                          float* red) {
  char* img = reinterpret_cast<char*>(p.img);
  float* hdr = reinterpret_cast<float*>(img);
  const int C = g.C, M = g.M, M16 = g.M16, cr = p.cr;
  const bool states = p.dS != nullptr && p.pass == kSliceBwd;
  const bool desl = p.Sp != nullptr && p.pass == kSliceBwd;
  if (bid < M) {
    const int j = bid;
    // loads first: den_j, row j of dS and num (one element per thread for
    // C <= 256), and in wave 0 the weights w_k (one slice per lane)
    const float dj = states ? p.den[j] : 1.f;
    float s = 0.f;
    for (int c = threadIdx.x; c < cr; c += 256) {
      const float dv = states ? p.dS[j * cr + c] : 0.f, nv = states ? p.num[j * cr + c] : 0.f;
      s += dv * (nv / dj);
    }
    const int k = threadIdx.x < 64 ? (int)threadIdx.x : 0;
    const float wk = k < M ? (states ? fmaxf(p.den[k < M ? k : 0], 0.f) : 1.f) : 0.f;
    const bool live = states && dj >= p.eps;
    red[threadIdx.x] = live ? s : 0.f;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
      __syncthreads();
    }
    float wsum = wk;  // wave 0: fixed-order butterfly over the slices
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) wsum += __shfl_xor(wsum, o);
    if (threadIdx.x == 0) {
      hdr[M16 + j] = live ? -red[0] / dj : 0.f;
      hdr[2 * M16 + 2 * C + j] = (states ? fmaxf(dj, 0.f) : 1.f) / wsum;
    }
    if (j == 0)
      for (int q = M + threadIdx.x; q < M16; q += blockDim.x) {
        hdr[M16 + q] = 0.f;
        hdr[2 * M16 + 2 * C + q] = 0.f;
      }
    return;
  }
  // per slice (once per block, in LDS): the weight w_j and 1 / max(den_j, eps)
  float* wl = red;
  float* rl = red + 64;
  if (threadIdx.x < 64) {
    const int j = threadIdx.x < M ? (int)threadIdx.x : M - 1;
    const float dj = states ? p.den[j] : 1.f;
    wl[threadIdx.x] = states ? fmaxf(dj, 0.f) : 1.f;
    rl[threadIdx.x] = 1.0f / (dj >= p.eps ? dj : p.eps);
  }
  __syncthreads();
  const int cc = (bid - M) * blockDim.x + threadIdx.x;
  if (cc >= 2 * C) return;
  const bool first = cc < C;
  const int c = first ? cc : cc - C;
  // (columns c >= cr are padding: zero rows, centre 0)
  const bool on = (first ? states : desl) && c < cr;
  const int cl = c < cr ? c : 0;
  // the column's values, all loads issued at once (M <= 64)
  float v[64];
#pragma unroll
  for (int j = 0; j < 64; ++j) {
    const int jj = j < M ? j : M - 1;
    v[j] = on ? (first ? p.dS[jj * cr + cl] : p.Sp[jj * cr + cl]) : 0.f;
  }
  float wsum = 0.f, sum = 0.f;
#pragma unroll
  for (int j = 0; j < 64; ++j) {
    if (j < M) {
      if (first) v[j] *= rl[j];  // dnum_j
      wsum += wl[j];
      sum += wl[j] * v[j];
    }
  }
  const float ctr = on && wsum > 0.f ? sum * (1.0f / wsum) : 0.f;
  hdr[2 * M16 + cc] = ctr;  // cN[c] (cc < C), then cS[c]
#pragma unroll
  for (int j = 0; j < 64; ++j)
    if (j < M16)
      *reinterpret_cast<T*>(img + g.OFF_2 + lds_off(j, cc * g.SZ, g.WROW)) =
          from_f<T>(on && j < M ? v[j] - ctr : 0.f);
}

// The table image of a pass: for the backward passes the blocks
// [0, M + ceil(2C/256)) build the backward header and table (prep_back),
// the rest (grid-stride) the bias and a header, the logits table [A^T ; a]
// and, for kDeslice, S'^T.
// The deslice table S'^T (row c, column j; columns j >= M zero) at OFF_2.
template <typename T>
__device__ __forceinline__ void prep_deslice_table(const PrepGeo& g, const PrepArgs& p, char* img,
                                                   int64_t tid, int64_t nth) {
  const int C = g.C, M = g.M, M16 = g.M16, cr = p.cr;
  const int64_t nS = (int64_t)C * M16;
#pragma unroll 4
  for (int64_t k = tid; k < nS; k += nth) {
    const int c = (int)(k / M16), j = (int)(k - (int64_t)c * M16);
    const float v = (j < M && c < cr) ? p.Sp[j * cr + c] : 0.f;
    *reinterpret_cast<T*>(img + g.OFF_2 + c * g.SROW + j * g.SZ) = from_f<T>(v);
  }
}

// A per-head batch builds head blockIdx.y's image from its parameters and
// states at the batch's byte strides (a stride of 0: shared by the heads).
template <typename Q>
__device__ __forceinline__ Q* head_at(Q* q, int64_t stride) {
  using B = typename std::conditional<std::is_const<Q>::value, const char*, char*>::type;
  return q ? reinterpret_cast<Q*>(reinterpret_cast<B>(q) + (int64_t)blockIdx.y * stride) : q;
}

template <typename T>
__global__ void __launch_bounds__(256) k_prep(PrepGeo g, PrepArgs p) {
  __shared__ float red[256];
  if (gridDim.y > 1) {
    p.A = head_at(p.A, p.hs_A);
    p.b = head_at(p.b, p.hs_b);
    p.a = head_at(p.a, p.hs_a);
    p.Sp = head_at(p.Sp, p.hs_Sp);
    p.num = head_at(p.num, p.hs_num);
    p.den = head_at(p.den, p.hs_den);
    p.dS = head_at(p.dS, p.hs_dS);
    p.img = head_at(p.img, p.hs_img);
  }
  const bool back = p.pass == kSliceBwd || p.pass == kWeightsBwd;
  const int nback = back ? g.M + (2 * g.C + 255) / 256 : 0;
  if ((int)blockIdx.x < nback) {
    prep_back<T>(g, p, blockIdx.x, red);
    return;
  }
  char* img = reinterpret_cast<char*>(p.img);
  const T* A = reinterpret_cast<const T*>(p.A);
  const T* av = reinterpret_cast<const T*>(p.a);
  const int C = g.C, M = g.M, M16 = g.M16, cr = p.cr;
  const int64_t tid = (int64_t)(blockIdx.x - nback) * blockDim.x + threadIdx.x;
  const int64_t nth = (int64_t)(gridDim.x - nback) * blockDim.x;

  float* hdr = reinterpret_cast<float*>(img);
  if (p.pass == kDesliceW) {  // the stored-weights deslice: its S'^T table only
    prep_deslice_table<T>(g, p, img, tid, nth);
    return;
  }
  // padded slices j >= M get bias -inf: their softmax weight is exactly 0
  for (int64_t j = tid; j < M16; j += nth) hdr[j] = j < M ? (p.b ? p.b[j] : 0.f) : -INFINITY;
  if (!back)
    for (int64_t k = tid; k < 2 * M16 + 2 * C; k += nth) hdr[M16 + k] = 0.f;  // dden, cN, cS, sw
  for (int64_t c = tid; c < C; c += nth)
    hdr[3 * M16 + 2 * C + c] = av && c < cr ? to_f<T>(av[c]) : 0.f;
  // logits table: rows j < M16: A[:, j] (0 beyond M); row M16: a (columns
  // c >= cr: 0)
  const int64_t nL = (int64_t)(M16 + 1) * C;
#pragma unroll 4
  for (int64_t k = tid; k < nL; k += nth) {
    const int j = (int)(k / C), c = (int)(k - (int64_t)j * C);
    T v;
    if (c >= cr)
      v = from_f<T>(0.f);
    else if (j < M16)
      v = j < M ? A[(int64_t)c * M + j] : from_f<T>(0.f);
    else
      v = av ? av[c] : from_f<T>(0.f);
    *reinterpret_cast<T*>(img + g.OFF_L + lds_off(j, c * g.SZ, g.TROW)) = v;
  }
  if (p.pass == kDeslice) prep_deslice_table<T>(g, p, img, tid, nth);
}

hipError_t launch_prep(const PrepArgs& p, hipStream_t st) {
  if (!p.img || (!p.A && p.pass != kDesliceW)) return hipErrorInvalidValue;
  if (p.cr < 16 || p.cr > p.C || p.cr % 16) return hipErrorInvalidValue;
  if ((p.pass == kDeslice || p.pass == kDesliceW) && !p.Sp) return hipErrorInvalidValue;
  if (p.pass == kSliceBwd && p.dS && (!p.num || !p.den)) return hipErrorInvalidValue;
  PrepGeo g = prep_geo(p.dtype, p.C, p.M, p.MB);
  const bool back = p.pass == kSliceBwd || p.pass == kWeightsBwd;
  if (p.heads < 1 || p.heads > kMaxHeads) return hipErrorInvalidValue;
  const int blocks = 64 + (back ? p.M + (2 * p.C + 255) / 256 : 0);
  if (p.dtype == 1)
    hipLaunchKernelGGL(k_prep<bf16>, dim3(blocks, p.heads), dim3(256), 0, st, g, p);
  else
    hipLaunchKernelGGL(k_prep<float>, dim3(blocks, p.heads), dim3(256), 0, st, g, p);
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
  // head blockIdx.y of a per-head batch (0 otherwise): its records and
  // destinations at the batch's strides, applied where they are used (the
  // argument struct is only read: writing its arrays would copy it to scratch)
  parts = head_at(parts, seg.hs_parts);
  float* const S = head_at(seg.S, seg.hs_S);
  const int kk = threadIdx.x & 15, pg = threadIdx.x >> 4;
  const int64_t k0 = (int64_t)blockIdx.x * 16, k = k0 + kk;
  const bool states = S != nullptr && k0 < seg.nS;
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
        if (seg.dst[i]) head_at(seg.dst[i], seg.hs_dst[i])[off] = tot;
        if (seg.dst2[i]) head_at(seg.dst2[i], seg.hs_dst2[i])[off] = tot;
        break;
      }
      off -= seg.len[i];
    }
    if (states && k < seg.nS) {
      const float den = group_total(sh[16]);
      S[k] = tot / (den >= seg.eps ? den : seg.eps);
    }
  }
}

hipError_t launch_reduce(const float* partials, int P, int64_t rec, const Segments& seg,
                         hipStream_t st) {
  if (!partials || P < 1 || rec < 1) return hipErrorInvalidValue;
  if (seg.S && (seg.C < 16 || seg.C % 16 || seg.nS > rec || seg.den_col < 0 ||
                seg.den_col + seg.nS / seg.C > rec))
    return hipErrorInvalidValue;
  const int heads = seg.heads > 1 ? seg.heads : 1;
  if (heads > kMaxHeads) return hipErrorInvalidValue;
  const int blocks = (int)((rec + 15) / 16);
  hipLaunchKernelGGL(k_reduce, dim3(blocks, heads), dim3(256), 0, st, partials, P, rec, seg);
  return hipGetLastError();
}

}  // namespace pa
