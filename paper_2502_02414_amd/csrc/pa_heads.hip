// Kernels of the per-head slicing layout (gfx950).  With per-head slicing
// the C channels split into H contiguous blocks of D = C / H; each head runs
// the layer's streaming passes on its own block, stored head-major [H, N, D]
// so that a head's rows are contiguous, and the token attention of all heads
// runs as one H-head call on the heads' states side by side, [M, H*D], with
// the shared D x D token projections laid on the block diagonal.
//   - relayout between the point-major [R, H, D] and head-major [H, R, D]
//     layouts, 16 bytes per lane: plain copies, HBM-bound (each byte read
//     once and written once);
//   - a shared parameter expanded to every head (block-diagonal matrix or
//     H copies of a vector), and the reverse sum over the heads (the
//     gradient of a shared parameter), in head order, in double precision.
#include "pa_device.hpp"
#include "pa_internal.h"

namespace pa {
namespace {

// One 16-byte vector per lane, grid-stride.  i runs over the point-major
// layout [R, H, VPR] (VPR vectors of a head's D elements); the head-major
// position of the same vector is (h R + r) VPR + v.
__global__ __launch_bounds__(256) void k_relayout(int64_t R, int H, int VPR, int to_heads,
                                                  const uint4* __restrict__ src,
                                                  uint4* __restrict__ dst) {
  const int64_t total = R * H * VPR;
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += step) {
    const int64_t v = i % VPR;
    const int64_t rh = i / VPR;
    const int64_t h = rh % H;
    const int64_t r = rh / H;
    const int64_t j = (h * R + r) * VPR + v;
    if (to_heads)
      dst[j] = src[i];
    else
      dst[i] = src[j];
  }
}

__global__ __launch_bounds__(256) void k_expand(int H, int64_t L, int blockdiag,
                                                const float* __restrict__ src,
                                                float* __restrict__ dst) {
  const int64_t total = blockdiag ? (int64_t)H * L * H * L : (int64_t)H * L;
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += step) {
    if (blockdiag) {
      const int64_t C = (int64_t)H * L;
      const int64_t row = i / C, col = i % C;
      dst[i] = row / L == col / L ? src[(row % L) * L + col % L] : 0.f;
    } else {
      dst[i] = src[i % L];
    }
  }
}

// The sum over the heads of one parameter's gradient (grid-stride over its
// elements), in head order in double precision.
__device__ __forceinline__ void head_sum(int H, int64_t L, int blockdiag,
                                         const float* __restrict__ src, float* __restrict__ dst) {
  const int64_t total = blockdiag ? L * L : L;
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += step) {
    double s = 0.0;
    if (blockdiag) {
      const int64_t C = (int64_t)H * L;
      const int64_t a = i / L, b = i % L;
      for (int h = 0; h < H; ++h) s += (double)src[(h * L + a) * C + h * L + b];
    } else {
      for (int h = 0; h < H; ++h) s += (double)src[h * L + i];
    }
    dst[i] = (float)s;
  }
}

__global__ __launch_bounds__(256) void k_head_sum(int H, int64_t L, int blockdiag,
                                                  const float* __restrict__ src,
                                                  float* __restrict__ dst) {
  head_sum(H, L, blockdiag, src, dst);
}

// Item blockIdx.y of a batch: selected case by case (a run-time index into
// the by-value argument array would copy the arguments to scratch memory).
__global__ __launch_bounds__(256) void k_head_sum_batch(int H, HeadSumBatch b) {
  HeadSumItem t;
  switch (blockIdx.y) {
    case 0: t = b.it[0]; break;
    case 1: t = b.it[1]; break;
    case 2: t = b.it[2]; break;
    case 3: t = b.it[3]; break;
    case 4: t = b.it[4]; break;
    case 5: t = b.it[5]; break;
    case 6: t = b.it[6]; break;
    default: t = b.it[7]; break;
  }
  head_sum(H, t.L, t.blockdiag, t.src, t.dst);
}

unsigned grid_for(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return (unsigned)(b < 8192 ? (b > 0 ? b : 1) : 8192);
}

}  // namespace

hipError_t launch_heads_relayout(int64_t R, int H, int D, int dtype, int to_heads,
                                 const void* src, void* dst, hipStream_t st) {
  const int64_t rowb = (int64_t)D * (dtype == 1 ? 2 : 4);
  if (R < 1 || H < 1 || D < 1 || rowb % 16 || !src || !dst) return hipErrorInvalidValue;
  const int VPR = (int)(rowb / 16);
  hipLaunchKernelGGL(k_relayout, dim3(grid_for(R * H * VPR)), dim3(256), 0, st, R, H, VPR,
                     to_heads, (const uint4*)src, (uint4*)dst);
  return hipGetLastError();
}

hipError_t launch_heads_expand(int H, int64_t L, int blockdiag, const float* src, float* dst,
                               hipStream_t st) {
  if (H < 1 || L < 1 || !src || !dst) return hipErrorInvalidValue;
  const int64_t n = blockdiag ? (int64_t)H * L * H * L : (int64_t)H * L;
  hipLaunchKernelGGL(k_expand, dim3(grid_for(n)), dim3(256), 0, st, H, L, blockdiag, src, dst);
  return hipGetLastError();
}

hipError_t launch_heads_sum_batch(int H, const HeadSumBatch& b, hipStream_t st) {
  static_assert(kHeadSumMax == 8, "k_head_sum_batch selects among 8 items");
  if (H < 1 || b.n < 1 || b.n > kHeadSumMax) return hipErrorInvalidValue;
  unsigned blocks = 1;
  for (int i = 0; i < b.n; ++i) {
    const HeadSumItem& t = b.it[i];
    if (t.L < 1 || !t.src || !t.dst) return hipErrorInvalidValue;
    const unsigned g = grid_for(t.blockdiag ? t.L * t.L : t.L);
    blocks = g > blocks ? g : blocks;
  }
  hipLaunchKernelGGL(k_head_sum_batch, dim3(blocks, b.n), dim3(256), 0, st, H, b);
  return hipGetLastError();
}

hipError_t launch_heads_sum(int H, int64_t L, int blockdiag, const float* src, float* dst,
                            hipStream_t st) {
  if (H < 1 || L < 1 || !src || !dst) return hipErrorInvalidValue;
  const int64_t n = blockdiag ? L * L : L;
  hipLaunchKernelGGL(k_head_sum, dim3(grid_for(n)), dim3(256), 0, st, H, L, blockdiag, src, dst);
  return hipGetLastError();
}

}  // namespace pa
