// Streaming passes over the N points of one Physics-Attention layer (gfx950).
//
// Every pass recomputes the slice weights of a 16-point tile on chip:
//   logits  l = x A + b  and  t = tau0 + b_t + x.a   (one MFMA contraction
//           over C against the table [A^T ; a a ... a], Eq. 3 and Eq. 4)
//   w       = softmax_j((l + g) / max(t, tau_min))    (Eq. 4, in registers)
// and then does its own contraction:
//   kAggregate   num = W^T x, den = 1^T W        (Eq. 1; Section 4.2 partials)
//   kDeslice     y = W S'                         (deslice, Section 3)
//   kDesliceBwd  dS' = W^T dY                     (chain rule of the deslice)
//   kWeights     W, tau written out               (diagnostics)
//   kSliceBwd    dx, dA, db, da, db_t             (chain rule of Eq. 1, 3, 4)
//   kWeightsBwd  same, from an explicit dW
//
// Work split: a block has WAVES wavefronts; the grid has P = num_chunks(N)
// blocks; global wave w owns the contiguous tile range
// [T*w/(P*WAVES), T*(w+1)/(P*WAVES)) of the T = ceil(N/16) tiles.  Each wave
// streams its tiles independently (no block barrier inside the loop).  A
// tile's rows are loaded from HBM in 16-byte chunks (1 KB contiguous per wave
// instruction) into registers, written to a wave-private LDS tile at the top
// of the iteration, and the next tile's loads are issued into the same
// registers right away, so they have a whole tile of work to land.  All MFMA
// operands are then read from LDS (16-byte row reads, or ds_read_b64_tr_b16
// for the transposed operand of the contractions over points).  Sums over
// points are accumulated in registers, reduced across the block's waves in
// LDS in wave order and written as one fp32 record per block; a separate
// kernel adds the P records in block order.
#pragma once

#include "pa_device.hpp"
#include "pa_internal.h"
#include "pa_layout.h"

namespace pa {

struct StreamArgs {
  const void* x;
  const void* G;
  const void* dY;        // kDesliceBwd, kSliceBwd (deslice term)
  const void* img;       // table image (workspace)
  void* out;             // y, dx (dtype) or W (fp32)
  float* tau_out;        // kWeights (nullable)
  const float* dW;       // kWeightsBwd
  const float* dtau;     // kWeightsBwd (nullable)
  float* partials;       // [P][rec]
  int64_t N;
  int M;
  int rec;               // floats per record
  double tb;             // tau0 + b_t (exact sum of the two fp32 values)
  float tau_min;
  int flags;
};

enum Flags { kHasG = 1, kStatesTerm = 2, kDesliceTerm = 4 };

__device__ __forceinline__ uint4 ld_global16(const void* p) {
  return *reinterpret_cast<const uint4*>(p);
}

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---------------------------------------------------------------------------
// Point tiles: HBM -> registers -> swizzled LDS
// ---------------------------------------------------------------------------
// Rows [p0, p0+16) of a [N,C] tensor are 16*C*SZ contiguous bytes; lane l
// holds 16-byte chunks q = l + 64k.  Rows >= N are zero.
template <typename T, int C>
struct TileRegs {
  static constexpr int RCH = C * (int)sizeof(T) / 16;  // chunks per row
  static constexpr int NCH = 16 * RCH / 64;            // chunks per lane
  uint4 c[NCH];
};

template <typename T, int C>
__device__ __forceinline__ void load_tile(TileRegs<T, C>& R, const T* base, int64_t p0,
                                          int64_t N) {
  constexpr int RCH = TileRegs<T, C>::RCH;
  const int lane = lane_id();
  const char* src = reinterpret_cast<const char*>(base + p0 * C);
#pragma unroll
  for (int k = 0; k < TileRegs<T, C>::NCH; ++k) {
    const int q = lane + 64 * k;
    R.c[k] = (p0 + q / RCH < N) ? ld_global16(src + 16 * q) : uint4{0, 0, 0, 0};
  }
}

template <typename T, int C>
__device__ __forceinline__ void store_tile(char* tile, const TileRegs<T, C>& R) {
  constexpr int RCH = TileRegs<T, C>::RCH;
  constexpr int ROW = C * (int)sizeof(T) + 32;
  const int lane = lane_id();
#pragma unroll
  for (int k = 0; k < TileRegs<T, C>::NCH; ++k) {
    const int q = lane + 64 * k;
    const int row = q / RCH, cc = q - row * RCH;
    *reinterpret_cast<uint4*>(tile + swz(row, 16 * cc, ROW)) = R.c[k];
  }
}

// The Gumbel rows of a tile: 16*M elements, contiguous in G.  GCH 16-byte
// chunks per lane cover the largest tile (M = 16*MB).  In LDS each row has
// stride GROW = 16*MB*sz + 16 bytes (only the first M elements are used).
template <typename T, int MB>
struct GRegs {
  static constexpr int BYTES = 16 * 16 * MB * (int)sizeof(T);
  static constexpr int GCH = (BYTES / 16 + 63) / 64;
  uint4 c[GCH];
};

template <typename T, int MB>
__device__ __forceinline__ void load_g(GRegs<T, MB>& gr, const T* G, int64_t p0, int64_t N,
                                       int M, bool hasG) {
  const int lane = lane_id();
  const int nchunk = M * (int)sizeof(T);  // (16 rows * M * sz) / 16
  const int64_t nvalid = N - p0 < 16 ? N - p0 : 16;
  const char* base = reinterpret_cast<const char*>(G + p0 * M);
#pragma unroll
  for (int k = 0; k < GRegs<T, MB>::GCH; ++k) {
    const int q = lane + 64 * k;
    uint4 v{0, 0, 0, 0};
    if (hasG && q < nchunk) {
      if (nvalid == 16) {
        v = ld_global16(base + 16 * q);
      } else {
        // tail tile: element-wise, only elements of valid rows
        const int64_t nel = nvalid * M;
        const T* e = reinterpret_cast<const T*>(base + 16 * q);
        const int64_t e0 = (int64_t)q * 16 / (int)sizeof(T);
        T tmp[16 / sizeof(T)];
#pragma unroll
        for (int u = 0; u < (int)(16 / sizeof(T)); ++u)
          tmp[u] = (e0 + u < nel) ? e[u] : from_f<T>(0.f);
        v = *reinterpret_cast<uint4*>(tmp);
      }
    }
    gr.c[k] = v;
  }
}

template <typename T, int MB>
__device__ __forceinline__ void store_g(char* gt, const GRegs<T, MB>& gr, int M) {
  constexpr int SZ = (int)sizeof(T);
  constexpr int GROW = 16 * MB * SZ + 16;
  const int lane = lane_id();
  const int nchunk = M * SZ;
  const int rch = (M * SZ) / 16;  // chunks per row when rows are 16-byte multiples
#pragma unroll
  for (int k = 0; k < GRegs<T, MB>::GCH; ++k) {
    const int q = lane + 64 * k;
    if (q >= nchunk) continue;
    if ((M * SZ) % 16 == 0) {
      const int row = q / rch, cc = q - row * rch;
      *reinterpret_cast<uint4*>(gt + row * GROW + 16 * cc) = gr.c[k];
    } else {
      const T* e = reinterpret_cast<const T*>(&gr.c[k]);
#pragma unroll
      for (int u = 0; u < 16 / SZ; ++u) {
        const int el = q * (16 / SZ) + u, row = el / M, col = el - row * M;
        *reinterpret_cast<T*>(gt + row * GROW + col * SZ) = e[u];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// LDS operand reads
// ---------------------------------------------------------------------------
// K32 fragment of row `row`, elements [col, col+8) of a swizzled array.
template <typename T>
__device__ __forceinline__ void ld_k32s(K32<T>& f, const char* base, int row, int col, int RB) {
  if constexpr (sizeof(T) == 2) {
    f.v = *reinterpret_cast<const bf16x8*>(base + swz(row, 2 * col, RB));
  } else {
    f.lo = *reinterpret_cast<const f32x4*>(base + swz(row, 4 * col, RB));
    f.hi = *reinterpret_cast<const f32x4*>(base + swz(row, 4 * col + 16, RB));
  }
}

// Transposed K16 fragment: lane (r,g) element i = arr[row0 + 4g + i][col0 + r]
// (row stride RB bytes; swizzled or plain).  bf16 uses ds_read_b64_tr_b16:
// within each 16-lane group, lane 4a+e receives element e of the 8-byte
// chunks addressed by lanes a, a+4, a+8, a+12, so lane k addresses row
// row0 + 4g + k/4, columns col0 + 4 (k%4) .. +3.  fp32 reads the four
// elements one by one.
template <typename T, bool SWZ>
__device__ __forceinline__ void ld_k16_t(K16<T>& f, const char* base, int RB, int row0,
                                         int col0) {
  const int r = lane_id() & 15, g = lane_id() >> 4;
  if constexpr (sizeof(T) == 2) {
    typedef __bf16 bf16x4v __attribute__((__vector_size__(4 * sizeof(__bf16))));
    const int row = row0 + 4 * g + (r >> 2), bcol = (col0 + 4 * (r & 3)) * 2;
    const char* p = base + (SWZ ? swz(row, bcol, RB) : row * RB + bcol);
    bf16x4v v = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (__attribute__((address_space(3))) bf16x4v*)(p));
    f.v = __builtin_bit_cast(bf16x4, v);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = row0 + 4 * g + i, bcol = (col0 + r) * 4;
      f.v[i] = *reinterpret_cast<const float*>(base + (SWZ ? swz(row, bcol, RB) : row * RB + bcol));
    }
  }
}

// Four consecutive elements [col, col+4) of a swizzled row, as floats.
template <typename T>
__device__ __forceinline__ void ld4s(float (&v)[4], const char* base, int row, int col, int RB) {
  if constexpr (sizeof(T) == 2) {
    const bf16x4 q = *reinterpret_cast<const bf16x4*>(base + swz(row, 2 * col, RB));
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = (float)q[i];
  } else {
    const f32x4 q = *reinterpret_cast<const f32x4*>(base + swz(row, 4 * col, RB));
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = q[i];
  }
}

template <typename T>
__device__ __forceinline__ float lds_elem(const char* base, int idx) {
  return to_f<T>(reinterpret_cast<const T*>(base)[idx]);
}

// ---------------------------------------------------------------------------
// Logits and temperature: one contraction over C against the logits table.
//   PS layout (SP = false): D[point][slice]; lane (r,g) holds point 4g+i,
//                           slice 16nb+r.
//   SP layout (SP = true):  D[slice][point]; lane (r,g) holds slice
//                           16nb+4g+i, point r.
// bf16: block nb = MB is the temperature block (every row of the table is
// a), so every lane receives x.a for its point(s).
// ---------------------------------------------------------------------------
template <typename T, int C, int MB, bool SP>
__device__ __forceinline__ void logits(typename LAcc<T, SP>::v (&acc)[MB + 1], const char* xt,
                                       const char* tabL) {
  using G_ = Geo<sizeof(T), C, MB>;
  using V = typename LAcc<T, SP>::v;
  constexpr int NT = sizeof(T) == 2 ? MB + 1 : MB;
  const int r = lane_id() & 15, g = lane_id() >> 4;
  const int ra = SP ? a_row<V>(r) : r;  // table row supplied by this lane
#pragma unroll
  for (int nb = 0; nb <= MB; ++nb) acc[nb] = zero_acc<V>();
#pragma unroll
  for (int s = 0; s < C / 32; ++s) {
    K32<T> xa;
    ld_k32s<T>(xa, xt, r, 32 * s + 8 * g, G_::XT_ROW);
#pragma unroll
    for (int nb = 0; nb < NT; ++nb) {
      K32<T> t;
      ld_k32s<T>(t, tabL, nb * 16 + ra, 32 * s + 8 * g, G_::TROW);
      acc[nb] = SP ? mma_acc(t, xa, acc[nb]) : mma_acc(xa, t, acc[nb]);
    }
  }
}

// Unclamped temperature t = tau0 + b_t + x.a of the lane's own point (row r
// of the tile).  bf16 storage: the MFMA temperature block (fp32 accumulate).
// fp32 storage: the products x_c a_c are exact in fp64 and are summed in
// fp64, because t can sit just above tau_min after cancellation (tau0 vs
// x.a) and the backward scales with 1/tau^2; an fp32 sum would lose about
// 1e-5 of tau there.
template <typename T, int C, int MB, typename V>
__device__ __forceinline__ float temperature_own(const V (&acc)[MB + 1], const char* xt,
                                                 const char* tabL, double tb) {
  using G_ = Geo<sizeof(T), C, MB>;
  if constexpr (sizeof(T) == 2) {
    return (float)((double)acc[MB][0] + tb);
  } else {
    const int r = lane_id() & 15, g = lane_id() >> 4;
    double s = 0.0;
#pragma unroll
    for (int q = 0; q < C / 32; ++q) {
      K32<float> xa, av;
      ld_k32s<float>(xa, xt, r, 32 * q + 8 * g, G_::XT_ROW);
      ld_k32s<float>(av, tabL, 16 * MB, 32 * q + 8 * g, G_::TROW);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s = fma((double)xa.lo[e], (double)av.lo[e], s);
        s = fma((double)xa.hi[e], (double)av.hi[e], s);
      }
    }
    s = s + __shfl_xor(s, 16);
    s = s + __shfl_xor(s, 32);
    return (float)(tb + s);
  }
}

// PS layout: temperatures of points 4g+i (i = 0..3).
template <typename T, int C, int MB, typename V>
__device__ __forceinline__ void temperature_ps(const V (&acc)[MB + 1], const char* xt,
                                               const char* tabL, double tb, float (&t)[4]) {
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int i = 0; i < 4; ++i) t[i] = (float)((double)acc[MB][i] + tb);
  } else {
    const float own = temperature_own<T, C, MB, V>(acc, xt, tabL, tb);
    const int g = lane_id() >> 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) t[i] = __shfl(own, 4 * g + i);
  }
}

// Softmax over slices, PS layout.  u = l + b + g (the noisy logit), m its
// row maximum; the base-2 exponent zs = (u - m) log2(e) / tau is formed
// after the shift, so its error is relative to u - m (not to u / tau, which
// is large when tau is clamped); w = 2^zs / sum.  Invalid slices (j >= M)
// and points beyond N get w = 0.  The Gumbel values are read transposed
// from the padded G tile (rows 4g+i, column 16nb+r).
template <typename T, int MB, typename V>
__device__ __forceinline__ void softmax_ps(const V (&acc)[MB + 1], const char* gt,
                                           const float (&bias)[MB], int M, bool hasG,
                                           const float (&t)[4], float tau_min, int nvalid,
                                           float (&w)[MB][4], float (&tau)[4]) {
  using R = decltype(acc[0][0] + 0.f);
  constexpr int GROW = 16 * MB * (int)sizeof(T) + 16;
  const int r = lane_id() & 15, g = lane_id() >> 4;
  R u[MB][4];
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) {
    const int j = 16 * nb + r;
    const bool valid = j < M;
    K16<T> gv;
    if (hasG)
      ld_k16_t<T, false>(gv, gt, GROW, 0, 16 * nb);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float gg = (hasG && valid) ? k16_elem(gv, i) : 0.f;
      u[nb][i] = valid ? (R)acc[nb][i] + (R)bias[nb] + (R)gg : (R)-INFINITY;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    tau[i] = fmaxf(t[i], tau_min);
    const R k = (R)(kLog2e / tau[i]);
    float m = (float)u[0][i];
#pragma unroll
    for (int nb = 1; nb < MB; ++nb) m = fmaxf(m, (float)u[nb][i]);
    m = row16_max(m);
    float e[MB], s = 0.f;
#pragma unroll
    for (int nb = 0; nb < MB; ++nb) {
      e[nb] = fast_exp2((float)((u[nb][i] - (R)m) * k));
      s += e[nb];
    }
    s = row16_sum(s);
    const float inv = 1.0f / s;
    const bool pv = (4 * g + i) < nvalid;
#pragma unroll
    for (int nb = 0; nb < MB; ++nb) w[nb][i] = pv ? e[nb] * inv : 0.f;
  }
}

// Softmax over slices, SP layout (the lane's point is r).  Also returns the
// shifted base-2 exponents zs (the natural logit is zs ln 2 + const) for
// the temperature gradient.  The Gumbel values are four consecutive
// elements of row r of the G tile.
template <typename T, int MB, typename V>
__device__ __forceinline__ void softmax_sp(const V (&acc)[MB + 1], const char* gt,
                                           const float (&bias)[MB][4], int M, bool hasG, float t,
                                           float tau_min, int nvalid, float (&w)[MB][4],
                                           float (&zs)[MB][4], float& tau) {
  using R = decltype(acc[0][0] + 0.f);
  constexpr int SZ = (int)sizeof(T);
  constexpr int GROW = 16 * MB * SZ + 16;
  const int r = lane_id() & 15, g = lane_id() >> 4;
  tau = fmaxf(t, tau_min);
  const R k = (R)(kLog2e / tau);
  R u[MB][4];
  float m = -INFINITY;
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) {
    float gv[4] = {0.f, 0.f, 0.f, 0.f};
    if (hasG) {
      const char* p = gt + r * GROW + (16 * nb + 4 * g) * SZ;
      if constexpr (SZ == 2) {
        const bf16x4 q = *reinterpret_cast<const bf16x4*>(p);
#pragma unroll
        for (int i = 0; i < 4; ++i) gv[i] = (float)q[i];
      } else {
        const f32x4 q = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
        for (int i = 0; i < 4; ++i) gv[i] = q[i];
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = 16 * nb + 4 * g + i;
      const bool valid = j < M;
      u[nb][i] = valid ? (R)acc[nb][i] + (R)bias[nb][i] + (R)gv[i] : (R)-INFINITY;
      m = fmaxf(m, (float)u[nb][i]);
    }
  }
  m = groups_max(m);
  float s = 0.f;
  float e[MB][4];
#pragma unroll
  for (int nb = 0; nb < MB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      zs[nb][i] = (float)((u[nb][i] - (R)m) * k);
      e[nb][i] = fast_exp2(zs[nb][i]);
      s += e[nb][i];
    }
  s = groups_sum(s);
  const float inv = 1.0f / s;
  const bool pv = r < nvalid;
#pragma unroll
  for (int nb = 0; nb < MB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) w[nb][i] = pv ? e[nb][i] * inv : 0.f;
}

// Copy the table image from global memory into LDS (all threads).
__device__ __forceinline__ void copy_image(char* lds, const void* img, int bytes) {
  const uint4* src = reinterpret_cast<const uint4*>(img);
  uint4* dst = reinterpret_cast<uint4*>(lds);
  for (int q = threadIdx.x; q < bytes / 16; q += blockDim.x) dst[q] = src[q];
}

__device__ __forceinline__ void tile_range(int64_t N, int waves, int64_t& t0, int64_t& t1) {
  const int64_t tiles = (N + 15) / 16;
  const int64_t tw = (int64_t)gridDim.x * waves;
  const int64_t gw = (int64_t)blockIdx.x * waves + (threadIdx.x >> 6);
  t0 = tiles * gw / tw;
  t1 = tiles * (gw + 1) / tw;
}

// Ordered (wave 0, 1, ...) sum of per-wave register partials into an LDS
// region; `put(first)` writes (first) or adds this wave's values.
template <typename Put>
__device__ __forceinline__ void block_ordered_reduce(int waves, Put put) {
  const int wave = threadIdx.x >> 6;
  for (int w = 0; w < waves; ++w) {
    if (wave == w) put(w == 0);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// kAggregate and kDesliceBwd (PS layout): W^T x (with den) or W^T dY.
// ---------------------------------------------------------------------------
template <typename T, int C, int MB, bool BWD>
__global__ void __launch_bounds__((64 * Geo<sizeof(T), C, MB>::waves(BWD ? kDesliceBwd : kAggregate)))
k_aggregate(StreamArgs a) {
  using G_ = Geo<sizeof(T), C, MB>;
  constexpr int PASS = BWD ? kDesliceBwd : kAggregate;
  constexpr int WAVES = G_::waves(PASS);
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int wave = threadIdx.x >> 6, r = lane_id() & 15, g = lane_id() >> 4;
  const bool hasG = a.flags & kHasG;

  copy_image(smem, a.img, G_::img_bytes(PASS));
  __syncthreads();
  const char* tabL = smem + G_::OFF_L;
  char* wreg = smem + G_::img_bytes(PASS) + wave * G_::wave_bytes(PASS);
  char* xt = wreg;                          // x tile (logits)
  char* yt = BWD ? wreg + G_::XT : wreg;    // tile contracted over points
  char* gt = wreg + (BWD ? 2 : 1) * G_::XT; // Gumbel rows

  float bias[MB];
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) bias[nb] = reinterpret_cast<const float*>(smem)[16 * nb + r];

  f32x4 acc[MB][G_::CB];
#pragma unroll
  for (int nb = 0; nb < MB; ++nb)
#pragma unroll
    for (int cb = 0; cb < G_::CB; ++cb) acc[nb][cb] = zero4();
  float den[MB];
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) den[nb] = 0.f;

  const T* X = reinterpret_cast<const T*>(a.x);
  const T* Y = reinterpret_cast<const T*>(a.dY);
  const T* Gp = reinterpret_cast<const T*>(a.G);
  int64_t t0, t1;
  tile_range(a.N, WAVES, t0, t1);

  TileRegs<T, C> xr, yr;
  GRegs<T, MB> gr;
  if (t0 < t1) {
    load_tile<T, C>(xr, X, t0 * 16, a.N);
    if constexpr (BWD) load_tile<T, C>(yr, Y, t0 * 16, a.N);
    load_g<T, MB>(gr, Gp, t0 * 16, a.N, a.M, hasG);
  }
  for (int64_t t = t0; t < t1; ++t) {
    const int64_t p0 = t * 16;
    const int nvalid = (int)(a.N - p0 < 16 ? a.N - p0 : 16);
    wave_sync();
    store_tile<T, C>(xt, xr);
    if constexpr (BWD) store_tile<T, C>(yt, yr);
    store_g<T, MB>(gt, gr, a.M);
    wave_sync();
    if (t + 1 < t1) {
      load_tile<T, C>(xr, X, p0 + 16, a.N);
      if constexpr (BWD) load_tile<T, C>(yr, Y, p0 + 16, a.N);
      load_g<T, MB>(gr, Gp, p0 + 16, a.N, a.M, hasG);
    }

    typename LAcc<T, false>::v lg[MB + 1];
    logits<T, C, MB, false>(lg, xt, tabL);
    float w[MB][4], tau[4], tt[4];
    temperature_ps<T, C, MB>(lg, xt, tabL, a.tb, tt);
    softmax_ps<T, MB>(lg, gt, bias, a.M, hasG, tt, a.tau_min, nvalid, w, tau);

    K16<T> wt[MB];
#pragma unroll
    for (int nb = 0; nb < MB; ++nb) {
      set_k16(wt[nb], w[nb][0], w[nb][1], w[nb][2], w[nb][3]);
      if (!BWD)
        den[nb] += (k16_elem(wt[nb], 0) + k16_elem(wt[nb], 1)) +
                   (k16_elem(wt[nb], 2) + k16_elem(wt[nb], 3));
    }
#pragma unroll
    for (int cb = 0; cb < G_::CB; ++cb) {
      K16<T> xb;
      ld_k16_t<T, true>(xb, yt, G_::XT_ROW, 0, 16 * cb);
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) acc[nb][cb] = mma16(wt[nb], xb, acc[nb][cb]);
    }
  }

  // den: lane (r,g) holds slice 16nb+r summed over its points -> sum groups
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) den[nb] = groups_sum(den[nb]);

  __syncthreads();  // every wave is done with the tables and tiles
  float* red = reinterpret_cast<float*>(smem);  // [M16][C] then den [M16]
  block_ordered_reduce(WAVES, [&](bool first) {
#pragma unroll
    for (int nb = 0; nb < MB; ++nb)
#pragma unroll
      for (int cb = 0; cb < G_::CB; ++cb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float* d = red + (16 * nb + 4 * g + i) * C + 16 * cb + r;
          *d = first ? acc[nb][cb][i] : *d + acc[nb][cb][i];
        }
    if (!BWD && g == 0)
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) {
        float* d = red + G_::M16 * C + 16 * nb + r;
        *d = first ? den[nb] : *d + den[nb];
      }
  });
  float* rec = a.partials + (int64_t)blockIdx.x * a.rec;
  const int MC = a.M * C;
  for (int k = threadIdx.x; k < MC; k += blockDim.x) rec[k] = red[k];
  if (!BWD)
    for (int j = threadIdx.x; j < a.M; j += blockDim.x) rec[MC + j] = red[G_::M16 * C + j];
}

// ---------------------------------------------------------------------------
// kDeslice (SP layout): y = W S'.
// ---------------------------------------------------------------------------
template <typename T, int C, int MB>
__global__ void __launch_bounds__((64 * Geo<sizeof(T), C, MB>::waves(kDeslice))) k_deslice(StreamArgs a) {
  using G_ = Geo<sizeof(T), C, MB>;
  constexpr int WAVES = G_::waves(kDeslice);
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int wave = threadIdx.x >> 6, r = lane_id() & 15, g = lane_id() >> 4;
  const bool hasG = a.flags & kHasG;

  copy_image(smem, a.img, G_::img_bytes(kDeslice));
  __syncthreads();
  const char* tabL = smem + G_::OFF_L;
  const char* tabS = smem + G_::OFF_2;
  char* xt = smem + G_::img_bytes(kDeslice) + wave * G_::wave_bytes(kDeslice);
  char* gt = xt + G_::XT;

  float bias[MB][4];
#pragma unroll
  for (int nb = 0; nb < MB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      bias[nb][i] = reinterpret_cast<const float*>(smem)[16 * nb + 4 * g + i];

  const T* X = reinterpret_cast<const T*>(a.x);
  const T* Gp = reinterpret_cast<const T*>(a.G);
  T* Y = reinterpret_cast<T*>(a.out);
  int64_t t0, t1;
  tile_range(a.N, WAVES, t0, t1);

  TileRegs<T, C> xr;
  GRegs<T, MB> gr;
  if (t0 < t1) {
    load_tile<T, C>(xr, X, t0 * 16, a.N);
    load_g<T, MB>(gr, Gp, t0 * 16, a.N, a.M, hasG);
  }
  for (int64_t t = t0; t < t1; ++t) {
    const int64_t p0 = t * 16;
    const int nvalid = (int)(a.N - p0 < 16 ? a.N - p0 : 16);
    wave_sync();
    store_tile<T, C>(xt, xr);
    store_g<T, MB>(gt, gr, a.M);
    wave_sync();
    if (t + 1 < t1) {
      load_tile<T, C>(xr, X, p0 + 16, a.N);
      load_g<T, MB>(gr, Gp, p0 + 16, a.N, a.M, hasG);
    }

    typename LAcc<T, true>::v lg[MB + 1];
    logits<T, C, MB, true>(lg, xt, tabL);
    float w[MB][4], zs[MB][4], tau;
    const float tt = temperature_own<T, C, MB>(lg, xt, tabL, a.tb);
    softmax_sp<T, MB>(lg, gt, bias, a.M, hasG, tt, a.tau_min, nvalid, w, zs, tau);

    K16<T> wb[MB];
#pragma unroll
    for (int nb = 0; nb < MB; ++nb) set_k16(wb[nb], w[nb][0], w[nb][1], w[nb][2], w[nb][3]);
    const bool pv = r < nvalid;
    T* yrow = Y + (p0 + r) * C + 4 * g;
#pragma unroll
    for (int cb = 0; cb < G_::CB; ++cb) {
      f32x4 d = zero4();
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) {
        K16<T> sa;
        ld_k16(sa, tabS + (16 * cb + r) * G_::SROW + (16 * nb + 4 * g) * (int)sizeof(T));
        d = mma16(sa, wb[nb], d);
      }
      if (pv) {
        if constexpr (sizeof(T) == 2) {
          bf16x4 o;
          o[0] = (bf16)d[0]; o[1] = (bf16)d[1]; o[2] = (bf16)d[2]; o[3] = (bf16)d[3];
          *reinterpret_cast<bf16x4*>(yrow + 16 * cb) = o;
        } else {
          *reinterpret_cast<f32x4*>(yrow + 16 * cb) = d;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// kWeights (PS layout): W [N,M] fp32 and tau [N] written out.
// ---------------------------------------------------------------------------
template <typename T, int C, int MB>
__global__ void __launch_bounds__((64 * Geo<sizeof(T), C, MB>::waves(kWeights))) k_weights(StreamArgs a) {
  using G_ = Geo<sizeof(T), C, MB>;
  constexpr int WAVES = G_::waves(kWeights);
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int wave = threadIdx.x >> 6, r = lane_id() & 15, g = lane_id() >> 4;
  const bool hasG = a.flags & kHasG;

  copy_image(smem, a.img, G_::img_bytes(kWeights));
  __syncthreads();
  const char* tabL = smem + G_::OFF_L;
  char* xt = smem + G_::img_bytes(kWeights) + wave * G_::wave_bytes(kWeights);
  char* gt = xt + G_::XT;
  float bias[MB];
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) bias[nb] = reinterpret_cast<const float*>(smem)[16 * nb + r];

  const T* X = reinterpret_cast<const T*>(a.x);
  const T* Gp = reinterpret_cast<const T*>(a.G);
  float* W = reinterpret_cast<float*>(a.out);
  int64_t t0, t1;
  tile_range(a.N, WAVES, t0, t1);
  TileRegs<T, C> xr;
  GRegs<T, MB> gr;
  for (int64_t t = t0; t < t1; ++t) {
    const int64_t p0 = t * 16;
    load_tile<T, C>(xr, X, p0, a.N);
    load_g<T, MB>(gr, Gp, p0, a.N, a.M, hasG);
    const int nvalid = (int)(a.N - p0 < 16 ? a.N - p0 : 16);
    wave_sync();
    store_tile<T, C>(xt, xr);
    store_g<T, MB>(gt, gr, a.M);
    wave_sync();
    typename LAcc<T, false>::v lg[MB + 1];
    logits<T, C, MB, false>(lg, xt, tabL);
    float w[MB][4], tau[4], tt[4];
    temperature_ps<T, C, MB>(lg, xt, tabL, a.tb, tt);
    softmax_ps<T, MB>(lg, gt, bias, a.M, hasG, tt, a.tau_min, nvalid, w, tau);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = 4 * g + i;
      if (p < nvalid) {
#pragma unroll
        for (int nb = 0; nb < MB; ++nb) {
          const int j = 16 * nb + r;
          if (j < a.M) W[(p0 + p) * a.M + j] = w[nb][i];
        }
        if (r == 0 && a.tau_out) a.tau_out[p0 + p] = tau[i];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// kSliceBwd / kWeightsBwd (SP layout, with a PS transpose for dA).
//   dw   = [dY Sp^T] + [x dnum^T] + dden    (kSliceBwd)   or  dW (kWeightsBwd)
//   dz   = w (dw - <w, dw>)
//   dl   = dz / tau;  dtau = dtau_in - <dz, z> / tau;  dt = dtau if t > tau_min
//   dx   = W dnum + A dl + a dt   (W dnum only with the states term)
//   dA  += x^T dl,  db += 1^T dl,  da += x^T dt,  db_t += 1^T dt
// The backward table rows hold dnum_j - cN and s'_j - cS (a shift common to
// all slices, which the softmax backward does not see); the header's dden is
// centred here by its den-weighted mean cD.
// ---------------------------------------------------------------------------
template <typename T, int C, int MB, int PASS>
__global__ void __launch_bounds__((64 * Geo<sizeof(T), C, MB>::waves(PASS))) k_slice_bwd(StreamArgs a) {
  using G_ = Geo<sizeof(T), C, MB>;
  constexpr int WAVES = G_::waves(PASS);
  constexpr int M16 = G_::M16;
  constexpr int SROWF = M16 + 1;  // dl transpose row stride (floats)
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int wave = threadIdx.x >> 6, r = lane_id() & 15, g = lane_id() >> 4;
  const bool hasG = a.flags & kHasG;
  const bool states = (PASS == kSliceBwd) && (a.flags & kStatesTerm);
  const bool deslice = (PASS == kSliceBwd) && (a.flags & kDesliceTerm);

  copy_image(smem, a.img, G_::img_bytes(PASS));
  __syncthreads();
  const float* hdr = reinterpret_cast<const float*>(smem);
  const float* dden_tab = hdr + M16;
  const float* cN = hdr + 2 * M16;
  const char* tabL = smem + G_::OFF_L;
  const char* tabW = smem + G_::OFF_2;
  char* wreg = smem + G_::img_bytes(PASS) + wave * G_::wave_bytes(PASS);
  char* xt = wreg;
  char* yt = wreg + G_::XT;  // dY tile (kSliceBwd only)
  char* gt = wreg + (PASS == kSliceBwd ? 2 : 1) * G_::XT;
  float* scr = reinterpret_cast<float*>(gt + G_::GT);  // [16][M16+1]
  float* scr_dt = scr + 16 * SROWF;                     // [16]

  // dden_j centred by its den-weighted mean (a shift common to all slices)
  float cD = 0.f;
  {
    const float* sw = hdr + 2 * M16 + 2 * C;
    for (int j = 0; j < a.M; ++j) cD += sw[j] * dden_tab[j];
  }
  float bias[MB][4], dden[MB][4];
#pragma unroll
  for (int nb = 0; nb < MB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = 16 * nb + 4 * g + i;
      bias[nb][i] = hdr[j];
      dden[nb][i] = j < a.M ? dden_tab[j] - cD : 0.f;
    }

  f32x4 dA[G_::CB][MB];
  float da[G_::CB];
#pragma unroll
  for (int cb = 0; cb < G_::CB; ++cb) {
    da[cb] = 0.f;
#pragma unroll
    for (int nb = 0; nb < MB; ++nb) dA[cb][nb] = zero4();
  }
  float db[MB];
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) db[nb] = 0.f;
  float dbt = 0.f;

  const T* X = reinterpret_cast<const T*>(a.x);
  const T* Y = reinterpret_cast<const T*>(a.dY);
  const T* Gp = reinterpret_cast<const T*>(a.G);
  T* DX = reinterpret_cast<T*>(a.out);
  int64_t t0, t1;
  tile_range(a.N, WAVES, t0, t1);

  TileRegs<T, C> xr, yr;
  GRegs<T, MB> gr;
  if (t0 < t1) {
    load_tile<T, C>(xr, X, t0 * 16, a.N);
    if (deslice) load_tile<T, C>(yr, Y, t0 * 16, a.N);
    load_g<T, MB>(gr, Gp, t0 * 16, a.N, a.M, hasG);
  }
  for (int64_t t = t0; t < t1; ++t) {
    const int64_t p0 = t * 16;
    const int nvalid = (int)(a.N - p0 < 16 ? a.N - p0 : 16);
    const bool pv = r < nvalid;
    wave_sync();
    store_tile<T, C>(xt, xr);
    if (deslice) store_tile<T, C>(yt, yr);
    store_g<T, MB>(gt, gr, a.M);
    wave_sync();
    if (t + 1 < t1) {
      load_tile<T, C>(xr, X, p0 + 16, a.N);
      if (deslice) load_tile<T, C>(yr, Y, p0 + 16, a.N);
      load_g<T, MB>(gr, Gp, p0 + 16, a.N, a.M, hasG);
    }

    typename LAcc<T, true>::v lg[MB + 1];
    logits<T, C, MB, true>(lg, xt, tabL);
    float w[MB][4], zs[MB][4], tau;
    const float tt = temperature_own<T, C, MB>(lg, xt, tabL, a.tb);
    softmax_sp<T, MB>(lg, gt, bias, a.M, hasG, tt, a.tau_min, nvalid, w, zs, tau);

    // dw in the SP layout
    float dw[MB][4];
    if constexpr (PASS == kSliceBwd) {
      using V = typename LAcc<T, true>::v;
      V acc[MB];
      const int ra = a_row<V>(r);
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) acc[nb] = zero_acc<V>();
      if (states) {
#pragma unroll
        for (int s = 0; s < G_::XF; ++s) {
          K32<T> xa;
          ld_k32s<T>(xa, xt, r, 32 * s + 8 * g, G_::XT_ROW);
#pragma unroll
          for (int nb = 0; nb < MB; ++nb) {
            K32<T> tw;
            ld_k32s<T>(tw, tabW, 16 * nb + ra, 32 * s + 8 * g, G_::WROW);
            acc[nb] = mma_acc(tw, xa, acc[nb]);
          }
        }
      }
      if (deslice) {
#pragma unroll
        for (int s = 0; s < G_::XF; ++s) {
          K32<T> ya;
          ld_k32s<T>(ya, yt, r, 32 * s + 8 * g, G_::XT_ROW);
#pragma unroll
          for (int nb = 0; nb < MB; ++nb) {
            K32<T> tw;
            ld_k32s<T>(tw, tabW, 16 * nb + ra, C + 32 * s + 8 * g, G_::WROW);
            acc[nb] = mma_acc(tw, ya, acc[nb]);
          }
        }
      }
#pragma unroll
      for (int nb = 0; nb < MB; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i) dw[nb][i] = (float)(acc[nb][i] + dden[nb][i]);
    } else {
#pragma unroll
      for (int nb = 0; nb < MB; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int j = 16 * nb + 4 * g + i;
          dw[nb][i] = (pv && j < a.M) ? a.dW[(p0 + r) * a.M + j] : 0.f;
        }
    }

    // softmax backward, dz = w (dw - <w, dw>), with <w, dw> compensated by a
    // second pass over the residuals (rows can be nearly one-hot, where the
    // difference is tiny next to dw), then the temperature chain.  The
    // exponents zs are shifted by a per-point constant, which <dz, zs> does
    // not see because sum_j dz_j = 0.
    float wdw = 0.f;
#pragma unroll
    for (int nb = 0; nb < MB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) wdw += w[nb][i] * dw[nb][i];
    wdw = groups_sum(wdw);
    float res = 0.f;
#pragma unroll
    for (int nb = 0; nb < MB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) res += w[nb][i] * (dw[nb][i] - wdw);
    res = groups_sum(res);
    const float rtau = 1.0f / tau;
    float dl[MB][4];
    float zdz = 0.f;
#pragma unroll
    for (int nb = 0; nb < MB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float dz = w[nb][i] * ((dw[nb][i] - wdw) - res);
        dl[nb][i] = dz * rtau;
        if (w[nb][i] != 0.f) zdz += dz * zs[nb][i];
      }
    zdz = groups_sum(zdz);
    float dtau = -kLn2 * zdz * rtau;
    if (PASS == kWeightsBwd && a.dtau != nullptr && pv) dtau += a.dtau[p0 + r];
    const float dt = (pv && tt > a.tau_min) ? dtau : 0.f;

    // dx = [W | dl] [dnum - cN ; A^T] + a dt + cN   (SP: D[channel][point])
    K16<T> wb[MB], lb[MB];
#pragma unroll
    for (int nb = 0; nb < MB; ++nb) {
      set_k16(wb[nb], w[nb][0], w[nb][1], w[nb][2], w[nb][3]);
      set_k16(lb[nb], dl[nb][0], dl[nb][1], dl[nb][2], dl[nb][3]);
    }
    T* dxrow = DX + (p0 + r) * C + 4 * g;
#pragma unroll
    for (int cb = 0; cb < G_::CB; ++cb) {
      f32x4 d = zero4();
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) {
        K16<T> ta;  // A^T rows of the logits table, read transposed
        ld_k16_t<T, true>(ta, tabL, G_::TROW, 16 * nb, 16 * cb);
        d = mma16(ta, lb[nb], d);
        if (states) {
          K16<T> tn;  // (dnum_j - cN) rows of the backward table, transposed
          ld_k16_t<T, true>(tn, tabW, G_::WROW, 16 * nb, 16 * cb);
          d = mma16(tn, wb[nb], d);
        }
      }
      // + a dt (a is any row of the temperature block of the logits table),
      // + cN: the table rows hold dnum_j - cN, and sum_j w_j = 1
      float av[4];
      ld4s<T>(av, tabL, 16 * MB, 16 * cb + 4 * g, G_::TROW);
#pragma unroll
      for (int i = 0; i < 4; ++i) d[i] += av[i] * dt;
      if (states) {
        const f32x4 cn = *reinterpret_cast<const f32x4*>(cN + 16 * cb + 4 * g);
#pragma unroll
        for (int i = 0; i < 4; ++i) d[i] += cn[i];
      }
      if (pv) {
        if constexpr (sizeof(T) == 2) {
          bf16x4 o;
          o[0] = (bf16)d[0]; o[1] = (bf16)d[1]; o[2] = (bf16)d[2]; o[3] = (bf16)d[3];
          *reinterpret_cast<bf16x4*>(dxrow + 16 * cb) = o;
        } else {
          *reinterpret_cast<f32x4*>(dxrow + 16 * cb) = d;
        }
      }
    }

    // parameter gradients: transpose dl (and dt) to the PS layout
#pragma unroll
    for (int nb = 0; nb < MB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) scr[r * SROWF + 16 * nb + 4 * g + i] = dl[nb][i];
    if (g == 0) scr_dt[r] = dt;
    wave_sync();
    float dlp[MB][4], dtp[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      dtp[i] = scr_dt[4 * g + i];
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) dlp[nb][i] = scr[(4 * g + i) * SROWF + 16 * nb + r];
    }
    K16<T> lp[MB];
#pragma unroll
    for (int nb = 0; nb < MB; ++nb) {
      set_k16(lp[nb], dlp[nb][0], dlp[nb][1], dlp[nb][2], dlp[nb][3]);
      db[nb] += (dlp[nb][0] + dlp[nb][1]) + (dlp[nb][2] + dlp[nb][3]);
    }
    if (g == 0) dbt += dt;
#pragma unroll
    for (int cb = 0; cb < G_::CB; ++cb) {
      K16<T> xa;
      ld_k16_t<T, true>(xa, xt, G_::XT_ROW, 0, 16 * cb);
      da[cb] += (k16_elem(xa, 0) * dtp[0] + k16_elem(xa, 1) * dtp[1]) +
                (k16_elem(xa, 2) * dtp[2] + k16_elem(xa, 3) * dtp[3]);
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) dA[cb][nb] = mma16(xa, lp[nb], dA[cb][nb]);
    }
  }

  // lane partials -> wave totals
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) db[nb] = groups_sum(db[nb]);
#pragma unroll
  for (int cb = 0; cb < G_::CB; ++cb) da[cb] = groups_sum(da[cb]);
  dbt = row16_sum(dbt);  // only g == 0 lanes carry values; sum their row

  __syncthreads();
  float* red = reinterpret_cast<float*>(smem);  // dA [C][M16], db [M16], da [C], dbt
  block_ordered_reduce(WAVES, [&](bool first) {
#pragma unroll
    for (int cb = 0; cb < G_::CB; ++cb)
#pragma unroll
      for (int nb = 0; nb < MB; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float* d = red + (16 * cb + 4 * g + i) * M16 + 16 * nb + r;
          *d = first ? dA[cb][nb][i] : *d + dA[cb][nb][i];
        }
    if (g == 0) {
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) {
        float* d = red + C * M16 + 16 * nb + r;
        *d = first ? db[nb] : *d + db[nb];
      }
#pragma unroll
      for (int cb = 0; cb < G_::CB; ++cb) {
        float* d = red + C * M16 + M16 + 16 * cb + r;
        *d = first ? da[cb] : *d + da[cb];
      }
      if (r == 0) {
        float* d = red + C * M16 + M16 + C;
        *d = first ? dbt : *d + dbt;
      }
    }
  });
  float* rec = a.partials + (int64_t)blockIdx.x * a.rec;
  const int M = a.M;
  for (int k = threadIdx.x; k < C * M; k += blockDim.x) {
    const int c = k / M, j = k - c * M;
    rec[k] = red[c * M16 + j];
  }
  for (int j = threadIdx.x; j < M; j += blockDim.x) rec[C * M + j] = red[C * M16 + j];
  for (int c = threadIdx.x; c < C; c += blockDim.x) rec[C * M + M + c] = red[C * M16 + M16 + c];
  if (threadIdx.x == 0) rec[C * M + M + C] = red[C * M16 + M16 + C];
}

// ---------------------------------------------------------------------------
// Launch of one pass, dispatched over dtype, C and slice blocks.  Each pass
// is instantiated in its own translation unit (pa_stream_<pass>.hip).
// ---------------------------------------------------------------------------
template <int PASS, typename T, int C, int MB>
static hipError_t launch_t(const StreamArgs& a, int P, hipStream_t st) {
  using G_ = Geo<sizeof(T), C, MB>;
  if constexpr (!G_::fits(PASS)) {
    return hipErrorInvalidConfiguration;
  } else {
    const int threads = 64 * G_::waves(PASS);
    const size_t lds = (size_t)G_::lds_bytes(PASS);
    if constexpr (PASS == kAggregate)
      hipLaunchKernelGGL((k_aggregate<T, C, MB, false>), dim3(P), dim3(threads), lds, st, a);
    else if constexpr (PASS == kDesliceBwd)
      hipLaunchKernelGGL((k_aggregate<T, C, MB, true>), dim3(P), dim3(threads), lds, st, a);
    else if constexpr (PASS == kDeslice)
      hipLaunchKernelGGL((k_deslice<T, C, MB>), dim3(P), dim3(threads), lds, st, a);
    else if constexpr (PASS == kWeights)
      hipLaunchKernelGGL((k_weights<T, C, MB>), dim3(P), dim3(threads), lds, st, a);
    else
      hipLaunchKernelGGL((k_slice_bwd<T, C, MB, PASS>), dim3(P), dim3(threads), lds, st, a);
    return hipGetLastError();
  }
}

template <int PASS, typename T, int C>
static hipError_t launch_c(int MB, const StreamArgs& a, int P, hipStream_t st) {
  switch (MB) {
    case 1: return launch_t<PASS, T, C, 1>(a, P, st);
    case 2: return launch_t<PASS, T, C, 2>(a, P, st);
    case 3: return launch_t<PASS, T, C, 3>(a, P, st);
    case 4: return launch_t<PASS, T, C, 4>(a, P, st);
    default: return hipErrorInvalidValue;
  }
}

template <int PASS>
static hipError_t launch_pass(int dtype, int C, int MB, const StreamArgs& a, int P,
                              hipStream_t st) {
  if (dtype == 1) {
    switch (C) {
      case 32: return launch_c<PASS, bf16, 32>(MB, a, P, st);
      case 64: return launch_c<PASS, bf16, 64>(MB, a, P, st);
      case 128: return launch_c<PASS, bf16, 128>(MB, a, P, st);
      case 256: return launch_c<PASS, bf16, 256>(MB, a, P, st);
      default: return hipErrorInvalidValue;
    }
  }
  switch (C) {
    case 32: return launch_c<PASS, float, 32>(MB, a, P, st);
    case 64: return launch_c<PASS, float, 64>(MB, a, P, st);
    case 128: return launch_c<PASS, float, 128>(MB, a, P, st);
    case 256: return launch_c<PASS, float, 256>(MB, a, P, st);
    default: return hipErrorInvalidValue;
  }
}

// Per-pass entry points (one translation unit each).
hipError_t launch_aggregate_pass(int dtype, int C, int MB, const StreamArgs& a, int P, hipStream_t st);
hipError_t launch_deslice_pass(int dtype, int C, int MB, const StreamArgs& a, int P, hipStream_t st);
hipError_t launch_deslice_bwd_pass(int dtype, int C, int MB, const StreamArgs& a, int P, hipStream_t st);
hipError_t launch_weights_pass(int dtype, int C, int MB, const StreamArgs& a, int P, hipStream_t st);
hipError_t launch_slice_bwd_pass(int dtype, int C, int MB, const StreamArgs& a, int P, hipStream_t st);
hipError_t launch_weights_bwd_pass(int dtype, int C, int MB, const StreamArgs& a, int P, hipStream_t st);

}  // namespace pa
