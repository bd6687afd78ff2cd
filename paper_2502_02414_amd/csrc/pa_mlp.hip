// The first product of a block's MLP with its activation in one kernel
// (bf16 storage, gfx950): the feed-forward layer of the Transformer block
// that Physics-Attention sits in (Figure 2a; the block stack of Table 5's
// industrial model), x2 = x1 + GELU(h W1 + b1) W2 + b2 with h = LN2(x1).
//
//   forward:   G[n, f]  = GELU(u[n, f]),             u = h W1 + b1
//   backward:  dU[n, f] = (dY W2^T)[n, f] GELU'(u[n, f])
//
// The pre-activation u is never stored: the forward writes only GELU(u)
// (which the second product and the weight gradient of W2 read), and the
// backward recomputes u from h (K = C channels: a cheap contraction next to
// the [N, 4C] tensors it saves writing and reading).  Both contractions run
// on v_mfma_f32_16x16x32_bf16 with fp32 accumulation; the activation is
// applied to the fp32 accumulator and rounded to bf16 once.
//
// A block of four waves (eight in the backward, whose two products double
// the weights staged per chunk) takes 32 points per wave (two 16-point MFMA
// tiles) and walks the F = 4C output columns in chunks of FC: each chunk of
// the weights ([F, K] rows: W1 transposed, or W2 as it is) is staged in LDS
// once for the block, with the next chunk's loads in flight in registers;
// each wave keeps its points' K-long rows of h (and dY) in registers as the
// MFMA B operand for the whole column walk; results go through a
// wave-private LDS staging tile so that every global store is a 16-byte,
// row-contiguous access.
#include "pa_internal.h"
#include "pa_stream.hpp"

namespace pa {

namespace {

// Phi(x) and exp(-x^2 / 2) from the rational approximation of erf of
// Abramowitz and Stegun (formula 7.1.26; absolute error below 1.5e-7):
//   erf(z) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-z^2),
//   t = 1 / (1 + p z),  z = |x| / sqrt(2) >= 0.
// Phi(x) = (1 + erf(x / sqrt 2)) / 2 is then 1 - q for x >= 0 and q for
// x < 0, q = (a1 t + ... + a5 t^5) exp(-x^2 / 2) / 2, with no cancellation
// in the lower tail.  Far below bf16's rounding step, which is what the
// results are stored in.
struct Gauss {
  float Phi, e;
};
__device__ __forceinline__ Gauss gauss(float x) {
  const float z = fabsf(x) * 0.70710678118654752f;
  const float t = fast_rcp(fmaf(0.3275911f, z, 1.f));
  float p = fmaf(t, 0.5f * 1.061405429f, 0.5f * -1.453152027f);
  p = fmaf(t, p, 0.5f * 1.421413741f);
  p = fmaf(t, p, 0.5f * -0.284496736f);
  p = fmaf(t, p, 0.5f * 0.254829592f);
  p *= t;
  const float e = fast_exp2(-kLog2e * z * z);
  const float q = p * e;
  return {x >= 0.f ? 1.f - q : q, e};
}
// GELU(x) = x Phi(x); GELU'(x) = Phi(x) + x phi(x), phi(x) = exp(-x^2/2) / sqrt(2 pi).
__device__ __forceinline__ float gelu_ap(float x) { return x * gauss(x).Phi; }
__device__ __forceinline__ float dgelu_ap(float x) {
  const Gauss g = gauss(x);
  return fmaf(x * 0.3989422804014327f, g.e, g.Phi);
}

#ifndef PA_MLP_WPAD
#define PA_MLP_WPAD 32
#endif

template <int K, int FC, int PT, int NW, bool BWD>
struct MlpGeo {
  static constexpr int WAVES = NW;
  static constexpr int PW = 16 * PT;           // points per wave (PT 16-point MFMA tiles)
  static constexpr int PTS = PW * WAVES;       // points per block
  static constexpr int NM = BWD ? 2 : 1;       // weight matrices per chunk
  static constexpr int WROW = K * 2 + PA_MLP_WPAD;  // chunk row in LDS (bytes, padded)
  static constexpr int WMAT = FC * WROW;       // one matrix's chunk
  static constexpr int SROW = FC * 2 + 16;     // staging row (bytes)
  static constexpr int OFF_S = NM * WMAT;      // staging tiles, one per wave
  static constexpr int SWAVE = PW * SROW;
  static constexpr int LDS = OFF_S + WAVES * SWAVE;
  static constexpr int RCH = K * 2 / 16;       // 16-byte chunks of a weight row
  static constexpr int MCH = FC * RCH;         // ... of one matrix's chunk
  static constexpr int WCH = NM * MCH / (64 * WAVES);  // per thread
  static constexpr int KS = K / 32;            // K32 steps
  static constexpr int CT = FC / 16;           // 16-column tiles per chunk
  static constexpr int OCH = FC * 2 / 16;      // 16-byte chunks of a staged row
  static_assert(NM * MCH == WCH * 64 * WAVES, "weight chunk must split evenly over the block");
  static_assert(PW * OCH % 64 == 0, "staged rows must split evenly over a wave");
};

struct MlpArgs {
  int64_t N;
  int F;
  const bf16* X;    // [N, K]: h
  const bf16* DY;   // [N, K]: the MLP output's gradient (backward)
  const bf16* W1T;  // [F, K]: W1 transposed
  const bf16* W2;   // [F, K] (backward)
  const float* b1;  // [F]
  bf16* out;        // [N, F]: GELU(u), or dU
};

template <int K, int FC, int PT, int NW, bool BWD>
__global__ void __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2)))
k_mlp_up(MlpArgs a) {
  using Gm = MlpGeo<K, FC, PT, NW, BWD>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int wave = threadIdx.x >> 6, lane = lane_id(), r = lane & 15, g = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * Gm::PTS + Gm::PW * wave;  // the wave's first point
  const int F = a.F, nch = F / FC;

  // the weight chunk of columns [c FC, c FC + FC): matrix m's rows, 16
  // bytes per load, this thread's WCH of them
  auto wsrc = [&](int e) {
    const int m = Gm::NM == 2 ? e / Gm::MCH : 0;
    const int q = e - m * Gm::MCH, row = q / Gm::RCH, cc = q - row * Gm::RCH;
    return std::pair<int, int>(m, row * Gm::RCH + cc);
  };
  uint4 wpre[Gm::WCH];
  auto wload = [&](int c) {
#pragma unroll
    for (int j = 0; j < Gm::WCH; ++j) {
      const int e = threadIdx.x + 64 * NW * j;
      const auto mq = wsrc(e);
      const bf16* W = mq.first ? a.W2 : a.W1T;
      wpre[j] = ld_global16<false>(reinterpret_cast<const char*>(W + (int64_t)c * FC * K) +
                                   16 * mq.second);
    }
  };
  auto wstore = [&]() {
#pragma unroll
    for (int j = 0; j < Gm::WCH; ++j) {
      const int e = threadIdx.x + 64 * NW * j;
      const auto mq = wsrc(e);
      const int row = mq.second / Gm::RCH, cc = mq.second - row * Gm::RCH;
      *reinterpret_cast<uint4*>(smem + mq.first * Gm::WMAT + row * Gm::WROW + 16 * cc) = wpre[j];
    }
  };

  // the wave's rows of h (and dY) as MFMA B fragments: lane (r, g) holds
  // row n0 + 16 pt + r, channels 32 s + 8 g .. + 7 (rows past N read row
  // N - 1; their results are not stored)
  K32<bf16> xf[PT][Gm::KS], yf[BWD ? PT : 1][BWD ? Gm::KS : 1];
#pragma unroll
  for (int pt = 0; pt < PT; ++pt) {
    const int64_t n = n0 + 16 * pt + r;
    const int64_t nn = n < a.N ? n : a.N - 1;
#pragma unroll
    for (int s = 0; s < Gm::KS; ++s) {
      const uint32_t off = (uint32_t)(32 * s + 8 * g) * 2;
      xf[pt][s].v = __builtin_bit_cast(
          bf16x8, ld_global16<true>(reinterpret_cast<const char*>(a.X + nn * K) + off));
      if constexpr (BWD)
        yf[pt][s].v = __builtin_bit_cast(
            bf16x8, ld_global16<true>(reinterpret_cast<const char*>(a.DY + nn * K) + off));
    }
  }
  wload(0);

  char* stg = smem + Gm::OFF_S + wave * Gm::SWAVE;
  for (int c = 0; c < nch; ++c) {
    block_sync();  // every wave is done with chunk c - 1
    wstore();
    block_sync();
    wload(c + 1 < nch ? c + 1 : c);  // (the last chunk again: no branch around the loads)

    // accumulators [column tile][point tile]: acc = X W1 (forward) or
    // dY W2^T (backward); accu = X W1 (backward)
    f32x4 acc[Gm::CT][PT], accu[BWD ? Gm::CT : 1][PT];
#pragma unroll
    for (int ct = 0; ct < Gm::CT; ++ct)
#pragma unroll
      for (int pt = 0; pt < PT; ++pt) {
        acc[ct][pt] = zero4();
        if constexpr (BWD) accu[ct][pt] = zero4();
      }
#pragma unroll
    for (int s = 0; s < Gm::KS; ++s) {
#pragma unroll
      for (int ct = 0; ct < Gm::CT; ++ct) {
        const int ro = (16 * ct + r) * Gm::WROW + 64 * s + 16 * g;
        K32<bf16> w1;
        ld_k32(w1, smem + ro);
        if constexpr (BWD) {
          K32<bf16> w2;
          ld_k32(w2, smem + Gm::WMAT + ro);
#pragma unroll
          for (int pt = 0; pt < PT; ++pt) {
            acc[ct][pt] = mma32(w2, yf[pt][s], acc[ct][pt]);
            accu[ct][pt] = mma32(w1, xf[pt][s], accu[ct][pt]);
          }
        } else {
#pragma unroll
          for (int pt = 0; pt < PT; ++pt) acc[ct][pt] = mma32(w1, xf[pt][s], acc[ct][pt]);
        }
      }
    }

    // epilogue: lane (r, g) holds column c FC + 16 ct + 4 g + i of point
    // n0 + 16 pt + r; staged as bf16 rows of the wave's points
#pragma unroll
    for (int ct = 0; ct < Gm::CT; ++ct) {
      const f32x4 bias = *reinterpret_cast<const f32x4*>(a.b1 + c * FC + 16 * ct + 4 * g);
#pragma unroll
      for (int pt = 0; pt < PT; ++pt) {
        bf16x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if constexpr (BWD)
            o[i] = (bf16)(acc[ct][pt][i] * dgelu_ap(accu[ct][pt][i] + bias[i]));
          else
            o[i] = (bf16)gelu_ap(acc[ct][pt][i] + bias[i]);
        }
        *reinterpret_cast<bf16x4*>(stg + (16 * pt + r) * Gm::SROW + (16 * ct + 4 * g) * 2) = o;
      }
    }
    wave_sync();
    // the staged rows to memory: 16-byte row-contiguous stores
#pragma unroll
    for (int j = 0; j < Gm::PW * Gm::OCH / 64; ++j) {
      const int q = lane + 64 * j, row = q / Gm::OCH, cc = q - row * Gm::OCH;
      const uint4 v = *reinterpret_cast<const uint4*>(stg + row * Gm::SROW + 16 * cc);
      const int64_t n = n0 + row;
      if (n < a.N)
        st_global16(reinterpret_cast<char*>(a.out + n * F + (int64_t)c * FC) + 16 * cc, v);
    }
  }
}

// W [K, F] -> WT [F, K] (bf16), 32 x 32 tiles through LDS.
__global__ void __launch_bounds__(256) k_transpose_bf16(int K, int F, const bf16* W, bf16* WT) {
  __shared__ bf16 t[32][33];
  const int f0 = blockIdx.x * 32, k0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int y = ty; y < 32; y += 8) {
    const int k = k0 + y, f = f0 + tx;
    t[y][tx] = (k < K && f < F) ? W[(int64_t)k * F + f] : (bf16)0.f;
  }
  __syncthreads();
  for (int y = ty; y < 32; y += 8) {
    const int f = f0 + y, k = k0 + tx;
    if (f < F && k < K) WT[(int64_t)f * K + k] = t[tx][y];
  }
}

template <int K, int FC, int PT, int NW, bool BWD>
hipError_t launch_k(const MlpArgs& a, hipStream_t st) {
  using Gm = MlpGeo<K, FC, PT, NW, BWD>;
  const int64_t blocks = (a.N + Gm::PTS - 1) / Gm::PTS;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((k_mlp_up<K, FC, PT, NW, BWD>), dim3((unsigned)blocks), dim3(64 * NW),
                     Gm::LDS, st, a);
  return hipGetLastError();
}

}  // namespace

bool mlp_up_served(int K, int F) {
  return (K == 64 || K == 128 || K == 256) && F >= 64 && F % 64 == 0;
}

hipError_t launch_mlp_up(int64_t N, int K, int F, const void* X, const void* W1, const float* b1,
                         const void* DY, const void* W2, void* out, void* W1T, hipStream_t st) {
  if (N < 1 || !mlp_up_served(K, F) || !X || !W1 || !b1 || !out || !W1T) return hipErrorInvalidValue;
  if (DY && !W2) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_transpose_bf16, dim3((F + 31) / 32, (K + 31) / 32), dim3(256), 0, st, K, F,
                     (const bf16*)W1, (bf16*)W1T);
  MlpArgs a{N, F, (const bf16*)X, (const bf16*)DY, (const bf16*)W1T, (const bf16*)W2, b1,
            (bf16*)out};
  const bool bwd = DY != nullptr;
  switch (K) {
    case 64: return bwd ? launch_k<64, 32, 2, 8, true>(a, st) : launch_k<64, 64, 2, 4, false>(a, st);
    case 128:
      return bwd ? launch_k<128, 32, 2, 8, true>(a, st) : launch_k<128, 64, 2, 4, false>(a, st);
    default:
      return bwd ? launch_k<256, 32, 2, 8, true>(a, st) : launch_k<256, 64, 2, 4, false>(a, st);
  }
}

}  // namespace pa
