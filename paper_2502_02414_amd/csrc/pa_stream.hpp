// Streaming passes over the N points of one Physics-Attention layer (gfx950).
//
// Every pass recomputes the slice weights of a 16-point tile on chip:
//   logits  l = x A + b  and  t = tau0 + b_t + x.a   (one MFMA contraction
//           over C against the table [A^T ; a], Eq. 3 and Eq. 4)
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
// for the transposed operand of the contractions over points); each
// contraction issues its LDS reads ahead of the MFMAs that consume them.
// Point outputs (y, dx) are staged in LDS and written back as whole rows, the
// same 1 KB-per-instruction pattern as the loads.  Sums over points are
// accumulated in registers, reduced across the block's waves in LDS in wave
// order and written as one fp32 record per block; a separate kernel adds the
// P records in block order.
#pragma once

#include <type_traits>

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
  const float* tb_dev;   // nullable: a device scalar added to tb
  float tau_min;
  int flags;
  // per-head batch (see StreamLaunch)
  int heads;
  int64_t hs_x, hs_g, hs_dy, hs_out, hs_img, hs_part, hs_tb;
  int cr;                // channels of the point rows (<= C, a multiple of 16)
};

enum Flags { kHasG = 1, kStatesTerm = 2, kDesliceTerm = 4 };

// Tiles of loads in flight per wave (register stages) in each streaming pass:
// two for the bf16 deslice with up to 32 slices, whose registers allow it;
// the aggregating passes stream 32-point tiles there (one stage holds as
// many points as two).  Rows of 64 bytes (a head's channel block of the
// per-head slicing, 32 bf16 channels) carry so few bytes per tile that the
// passes on 16-point tiles keep two stages (measured at 8 heads x 1M points,
// on top of the 8 waves of narrow rows, Geo::max_waves); the forward
// aggregate's 32-point stage already holds as many points (a second stage
// cost it 40 us per step there).
template <typename T, int C> constexpr bool narrow_rows() { return C * (int)sizeof(T) <= 64; }
template <typename T, int C, int MB, bool BWD> constexpr int agg_depth() {
  return narrow_rows<T, C>() && BWD ? 2 : 1;
}
template <typename T, int C, int MB> constexpr int des_depth() {
  return narrow_rows<T, C>() || (sizeof(T) == 2 && MB <= 2) ? 2 : 1;
}
template <typename T, int C, int MB> constexpr int bwd_depth() {
  return narrow_rows<T, C>() ? 2 : 1;
}
// Cache reuse between the passes of a layer step: the aggregate's loads of
// x keep their lines in the last-level cache, and the deslice (which reads
// the same x next) walks its tile ranges backwards, so it starts on the lines
// the aggregate read last (measured at N = 1M: deslice -41 us, aggregate
// +9 us; keeping G as well gained nothing).  The other passes stream
// non-temporally in the forward direction (keeping their loads too cost more
// than their successors gained).
constexpr bool kRevDeslice = true, kRevSliceBwd = false;
template <int PASS> constexpr bool keep_loads() { return PASS == kAggregate; }

// A per-head batch runs head blockIdx.y: its tensors at the batch's byte
// strides, its b_t the device scalar at tb_dev's stride (one head: nothing
// changes).  Only pointers move: an array among the by-value arguments would
// send them all to scratch.
template <typename P>
__device__ __forceinline__ P head_ptr(P p, int64_t stride) {
  using B = typename std::conditional<std::is_const<typename std::remove_pointer<P>::type>::value,
                                      const char*, char*>::type;
  return p ? reinterpret_cast<P>(reinterpret_cast<B>(p) + (int64_t)blockIdx.y * stride) : p;
}
__device__ __forceinline__ void head_offsets(StreamArgs& a) {
  if (gridDim.y == 1) return;
  a.x = head_ptr(a.x, a.hs_x);
  a.G = head_ptr(a.G, a.hs_g);
  a.dY = head_ptr(a.dY, a.hs_dy);
  a.out = head_ptr(a.out, a.hs_out);
  a.img = head_ptr(a.img, a.hs_img);
  a.partials = head_ptr(a.partials, a.hs_part);
  a.tb_dev = head_ptr(a.tb_dev, a.hs_tb);
}

// The temperature constant: tau0 + b_t, plus the device scalar when one is
// given (a folded Project step's bias term, computed on the GPU).
__device__ __forceinline__ void add_tb_dev(StreamArgs& a) {
  if (a.tb_dev) a.tb += (double)a.tb_dev[0];
}

// Point-side tensors are streamed once per pass: their 16-byte stores are
// non-temporal (no dirty data is left in the caches, so a pass does not pay
// for the previous pass's write-backs), and so are the loads of a pass
// unless it is marked as feeding the next pass through the last-level cache
// (NT = false: the lines it reads last stay cached for a next pass that
// walks the points in the opposite direction).
typedef unsigned int nt_u32x4 __attribute__((ext_vector_type(4)));
template <bool NT = true>
__device__ __forceinline__ uint4 ld_global16(const void* p) {
  if constexpr (NT)
    return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const nt_u32x4*>(p)));
  else
    return *reinterpret_cast<const uint4*>(p);
}
__device__ __forceinline__ void st_global16(void* p, const uint4& v) {
  __builtin_nontemporal_store(__builtin_bit_cast(nt_u32x4, v), reinterpret_cast<nt_u32x4*>(p));
}

// Orders a wave's LDS accesses across lanes: its LDS writes have completed
// (lgkmcnt) before any later LDS access, and the compiler moves no memory
// access across it.  (A wavefront-scope fence would also wait for every
// outstanding global load, i.e. for the tiles being prefetched.)
__device__ __forceinline__ void wave_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_wave_barrier();
}

// Block-wide LDS barrier: this wave's LDS accesses have completed (lgkmcnt)
// when it reaches the barrier, and no memory access moves across it.  Not
// __syncthreads(): its workgroup fence would also wait for every
// outstanding global load, i.e. for the tiles being prefetched.
__device__ __forceinline__ void block_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Software pipeline over N unrolled steps: the LDS reads of step i + D - 1
// are issued before the MFMAs of step i (the scheduling barrier keeps the
// compiler from sinking them back next to their use).
template <int N, int D, typename F, typename Load, typename Use>
__device__ __forceinline__ void pipelined(Load load, Use use) {
  F buf[D];
#pragma unroll
  for (int i = 0; i < D - 1; ++i)
    if (i < N) load(i, buf[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) {
    if (i + D - 1 < N) load(i + D - 1, buf[(i + D - 1) % D]);
    __builtin_amdgcn_sched_barrier(0);
    use(i, buf[i % D]);
  }
}

// ---------------------------------------------------------------------------
// LDS addressing.  Tables and point tiles have rows padded by 32 bytes
// (lds_off() in pa_device.hpp).  Every fragment read below is a per-lane
// base, computed once per kernel, plus a compile-time offset.
// ---------------------------------------------------------------------------
// K32 row fragment of lane (r, g): elements [col + 8g, col + 8g + 8) of row
// row0 + lr, at offset row0 * RB + col * sz.
template <typename T> struct RowBase { int lo, hi; };
template <typename T>
__device__ __forceinline__ RowBase<T> row_base(int lr, int RB) {
  const int g = lane_id() >> 4;
  constexpr int SZ = (int)sizeof(T);
  return {lr * RB + 8 * g * SZ, lr * RB + 8 * g * SZ + 16};
}
template <typename T>
__device__ __forceinline__ void ld_row(K32<T>& f, const char* a, const RowBase<T>& o, int off) {
  if constexpr (sizeof(T) == 2) {
    f.v = *reinterpret_cast<const bf16x8*>(a + o.lo + off);
  } else {
    f.lo = *reinterpret_cast<const f32x4*>(a + o.lo + off);
    f.hi = *reinterpret_cast<const f32x4*>(a + o.hi + off);
  }
}

// Transposed K16 fragment: lane (r, g) element i = arr[row0 + 4g + i][col0 + r]
// at offset row0 * RB + col0 * sz.  bf16 uses ds_read_b64_tr_b16: within
// each 16-lane group, lane 4a+e receives element e of the 8-byte chunks
// addressed by lanes a, a+4, a+8, a+12, so lane k addresses row 4g + k/4,
// columns 4 (k%4) .. +3.  fp32 reads four elements.
template <typename T>
__device__ __forceinline__ int tr_base(int RB) {
  const int r = lane_id() & 15, g = lane_id() >> 4;
  if constexpr (sizeof(T) == 2) {
    return (4 * g + (r >> 2)) * RB + 8 * (r & 3);
  } else {
    return 4 * g * RB + 4 * r;
  }
}
template <typename T>
__device__ __forceinline__ void ld_tr(K16<T>& f, const char* a, int base, int off, int RB) {
  if constexpr (sizeof(T) == 2) {
    typedef __bf16 v4 __attribute__((__vector_size__(4 * sizeof(__bf16))));
    v4 v = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (__attribute__((address_space(3))) v4*)(a + base + off));
    f.v = __builtin_bit_cast(bf16x4, v);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) f.v[i] = *reinterpret_cast<const float*>(a + base + off + i * RB);
  }
}

// SP-layout output fragment (lane (r, g): channels [c0 + 4g, +4) of point r)
// into a tile, at offset c0 * sz.
template <typename T>
__device__ __forceinline__ int stage_base(int RB) {
  const int r = lane_id() & 15, g = lane_id() >> 4;
  return r * RB + 4 * g * (int)sizeof(T);
}
template <typename T>
__device__ __forceinline__ void stage4(char* tile, int base, int off, const f32x4& d) {
  if constexpr (sizeof(T) == 2) {
    bf16x4 o;
    o[0] = (bf16)d[0]; o[1] = (bf16)d[1]; o[2] = (bf16)d[2]; o[3] = (bf16)d[3];
    *reinterpret_cast<bf16x4*>(tile + base + off) = o;
  } else {
    *reinterpret_cast<f32x4*>(tile + base + off) = d;
  }
}

// ---------------------------------------------------------------------------
// Point tiles: HBM -> registers -> padded LDS rows, and staged outputs back.
// A tile holds ROWS rows of C channels; lane l holds 16-byte chunks
// q = l + 64k (row q / RCH, chunk q % RCH).  Rows >= N re-read row N - 1
// (finite data; their points are masked).  The tensor's rows hold cr <= C
// channels (cr a multiple of 16, so rows are whole 16-byte chunks): the
// chunks past a row's end re-read its last chunk (finite data), and the
// tables hold zeros for those channels, so they contribute nothing; outputs
// are written for the cr channels only.  EX (cr == C, chosen per launch):
// the row length is the compile-time C, and the per-chunk addresses fold.
// ---------------------------------------------------------------------------
template <typename T, int C, int ROWS = 16>
struct TileRegs {
  static constexpr int RCH = C * (int)sizeof(T) / 16;  // chunks per row
  static constexpr int NCH = ROWS * RCH / 64;          // chunks per lane
  uint4 c[NCH];
};

// Last valid row of the tile at p0 (at most ROWS - 1).
template <int ROWS>
__device__ __forceinline__ int last_row(int64_t p0, int64_t N) {
  return N - 1 - p0 < ROWS - 1 ? (int)(N - 1 - p0) : ROWS - 1;
}

template <typename T, int C, int ROWS = 16, bool NT = true, bool EX = true>
__device__ __forceinline__ void load_tile(TileRegs<T, C, ROWS>& R, const T* base, int64_t p0,
                                          int64_t N, int cr) {
  // no predicated loads, so the compiler can track these loads exactly
  constexpr int RCH = TileRegs<T, C, ROWS>::RCH;
  const int lane = lane_id();
  const int lim = last_row<ROWS>(p0, N);
  const int w = EX ? C : cr;                            // channels of a row
  const int rb = w * (int)sizeof(T), lc = rb / 16 - 1;  // row bytes, its last chunk
  const char* src = reinterpret_cast<const char*>(base + p0 * w);
#pragma unroll
  for (int k = 0; k < TileRegs<T, C, ROWS>::NCH; ++k) {
    const int q = lane + 64 * k;
    const int row = q / RCH, cc = q - row * RCH;
    const int rr = row < lim ? row : lim;
    const int c = EX ? cc : (cc < lc ? cc : lc);
    R.c[k] = ld_global16<NT>(src + (uint32_t)(rr * rb + 16 * c));
  }
}

template <typename T, int C, int ROWS = 16>
__device__ __forceinline__ void store_tile(char* tile, const TileRegs<T, C, ROWS>& R) {
  constexpr int RCH = TileRegs<T, C, ROWS>::RCH;
  constexpr int ROW = C * (int)sizeof(T) + 32;
  const int lane = lane_id();
#pragma unroll
  for (int k = 0; k < TileRegs<T, C, ROWS>::NCH; ++k) {
    const int q = lane + 64 * k;
    const int row = q / RCH, cc = q - row * RCH;
    *reinterpret_cast<uint4*>(tile + lds_off(row, 16 * cc, ROW)) = R.c[k];
  }
}

// Staged output tile (padded LDS rows) -> rows [p0, p0 + nvalid) of dst,
// their cr channels.
template <typename T, int C, int ROWS = 16, bool EX = true>
__device__ __forceinline__ void write_tile(T* dst, int64_t p0, const char* tile, int nvalid,
                                           int cr) {
  constexpr int RCH = TileRegs<T, C, ROWS>::RCH;
  constexpr int NCH = TileRegs<T, C, ROWS>::NCH;
  constexpr int ROW = C * (int)sizeof(T) + 32;
  const int lane = lane_id();
  const int w = EX ? C : cr;
  const int rb = w * (int)sizeof(T);
  char* d = reinterpret_cast<char*>(dst + p0 * w);
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const int q = lane + 64 * k;
    const int row = q / RCH, cc = q - row * RCH;
    const uint4 v = *reinterpret_cast<const uint4*>(tile + lds_off(row, 16 * cc, ROW));
    // (whole rows: chunk q of the tile sits at byte 16 q of the run)
    const uint32_t off = EX ? (uint32_t)(16 * lane + 1024 * k) : (uint32_t)(row * rb + 16 * cc);
    if (row < nvalid && (EX || 16 * cc < rb)) st_global16(d + off, v);
  }
}

// The Gumbel rows of a tile: ROWS*M elements, contiguous in G.  GCH 16-byte
// chunks per lane cover the largest tile (M = 16*MB).  In LDS they keep the
// same layout, element (row, j) at (row*M + j)*sz; reads of a padded slice
// j >= M land on finite data (the next row, or the tile's zeroed tail) and
// are masked by the -inf bias.
template <typename T, int MB, int ROWS = 16>
struct GRegs {
  static constexpr int BYTES = ROWS * 16 * MB * (int)sizeof(T);
  static constexpr int GCH = (BYTES / 16 + 63) / 64;
  uint4 c[GCH];
};

template <typename T, int MB, int ROWS = 16, bool NT = true>
__device__ __forceinline__ void load_g(GRegs<T, MB, ROWS>& gr, const T* G, const void* safe,
                                       int64_t p0, int64_t N, int M, bool hasG) {
  // A full tile's ROWS*M elements are whole 16-byte chunks (lanes past the
  // last one re-read it).  Without noise, or for the tail tile, every lane
  // reads the 16 bytes at `safe` instead, and the tile body rewrites the rows
  // (g_fixup): no predicated loads, no partial chunks read past the end of G.
  const int lane = lane_id();
  const int nchunk = ROWS * M * (int)sizeof(T) / 16;
  const bool full = hasG && p0 + ROWS <= N;
  const char* src = full ? reinterpret_cast<const char*>(G + p0 * M)
                         : reinterpret_cast<const char*>(safe);
#pragma unroll
  for (int k = 0; k < GRegs<T, MB, ROWS>::GCH; ++k) {
    const int q = lane + 64 * k < nchunk ? lane + 64 * k : nchunk - 1;
    gr.c[k] = ld_global16<NT>(src + (full ? (uint32_t)(16 * q) : 0u));
  }
}

// Gumbel rows of a tile that load_g did not read (no noise: zeros; the tail
// tile: its valid elements, element by element), written into the G tile.
template <typename T, int MB, int ROWS = 16>
__device__ __forceinline__ void g_fixup(char* gt, const T* G, int64_t p0, int64_t N, int M,
                                        bool hasG) {
  const int64_t nel = hasG ? (N - p0 < ROWS ? N - p0 : ROWS) * M : 0;
  T* d = reinterpret_cast<T*>(gt);
  for (int e = lane_id(); e < ROWS * M; e += 64) d[e] = e < nel ? G[p0 * M + e] : from_f<T>(0.f);
}

template <typename T, int MB, int ROWS = 16>
__device__ __forceinline__ void store_g(char* gt, const GRegs<T, MB, ROWS>& gr, int M, bool hasG) {
  // the tile is the rows' ROWS*M contiguous elements, copied chunk by chunk
  const int lane = lane_id();
  const int nchunk = ROWS * M * (int)sizeof(T) / 16;
#pragma unroll
  for (int k = 0; k < GRegs<T, MB, ROWS>::GCH; ++k) {
    const int q = lane + 64 * k;
    if (q < nchunk) *reinterpret_cast<uint4*>(gt + 16 * q) = gr.c[k];
  }
}

// One tile's rows in registers: x, dY (unused registers are dropped by the
// compiler in the passes that do not read dY), and the Gumbel rows.
template <typename T, int C, int MB>
struct TileStage {
  TileRegs<T, C> x, y;
  GRegs<T, MB> g;
};

// Streams tiles [t0, t1) with DEPTH register stages: at the top of tile t
// its stage is written to the wave's LDS tiles and immediately reloaded
// with tile t + DEPTH, so DEPTH tiles of loads are in flight while body(t)
// computes.  The pipelined tiles are full ones (t < tfull).  The main loop runs whole rounds
// of DEPTH tiles with every stage reloaded on every tile -- past the end with
// the current tile again (an L2 hit) -- so all loads are unconditional and
// every path into the loop head has issued the stages in the same order:
// the compiler's wait before a stage's store then covers that stage only.
// The last (fewer than DEPTH) tiles, already loaded, follow the loop; a
// partial last tile is left to tail(t).  load(stage, tile) / store(stage);
// init() is the block's set-up (tables into LDS), run by every wave first
// (its loads then do not queue behind the tiles').
template <int DEPTH, typename Stage, bool REV = false, typename Load, typename Store,
          typename Body, typename Tail, typename Init>
__device__ __forceinline__ void stream_tiles(int64_t t0, int64_t t1, int64_t tfull, Load load,
                                             Store store, Body body, Tail tail, Init init) {
  const int64_t te = t1 < tfull ? t1 : tfull;
  // REV walks the range from its end: tile(i) for i = t0 .. te - 1
  auto tile = [&](int64_t i) { return REV ? t0 + te - 1 - i : i; };
  Stage st[DEPTH];
  init();  // the block's set-up (every wave)
  if (t0 < te) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) load(st[d], tile(t0 + d < te ? t0 + d : te - 1));
  }
  if (REV && t0 <= te && te < t1) tail(te);  // this wave owns the partial last tile
  if (t0 < te) {
    int64_t t = t0;
    for (; t + DEPTH <= te; t += DEPTH) {
#pragma unroll
      for (int d = 0; d < DEPTH; ++d) {
        const int64_t tt = t + d;
        wave_sync();
        store(st[d]);
        wave_sync();
        load(st[d], tile(tt + DEPTH < te ? tt + DEPTH : tt));
        body(tile(tt));
      }
    }
#pragma unroll
    for (int d = 0; d + 1 < DEPTH; ++d) {
      if (t + d < te) {
        wave_sync();
        store(st[d]);
        wave_sync();
        body(tile(t + d));
      }
    }
  }
  if (!REV && t0 <= te && te < t1) tail(te);  // this wave owns the partial last tile
}

// ---------------------------------------------------------------------------
// Logits and temperature: one contraction over C against the logits table.
//   PS layout (SP = false): D[point][slice]; lane (r,g) holds point 4g+i,
//                           slice 16nb+r.
//   SP layout (SP = true):  D[slice][point]; lane (r,g) holds slice
//                           16nb+4g+i, point r.
// bf16: block nb = MB is the temperature block (every lane reads the single
// table row a), so every lane receives x.a for its point(s).  The point
// fragments xa are returned for reuse (the dw contraction of the backward).
// ---------------------------------------------------------------------------
template <typename T, int C, int MB>
struct LogitsBases {
  RowBase<T> x, t, a;
};
template <typename T, int C, int MB, bool SP>
__device__ __forceinline__ LogitsBases<T, C, MB> logits_bases() {
  using G_ = Geo<sizeof(T), C, MB>;
  using V = typename LAcc<T, SP>::v;
  const int r = lane_id() & 15;
  return {row_base<T>(r, G_::XT_ROW), row_base<T>(SP ? a_row<V>(r) : r, G_::TROW),
          row_base<T>(0, G_::TROW)};
}

// init (nullable): starting values of the slice blocks' accumulators (the
// biases, so that the contraction adds them); the temperature block starts
// at zero.
template <typename T, int C, int MB, bool SP, bool KEEP_X = true>
__device__ __forceinline__ void logits(typename LAcc<T, SP>::v (&acc)[MB + 1],
                                       K32<T> (&xa)[C / 32], const char* xt, const char* tabL,
                                       const LogitsBases<T, C, MB>& lb,
                                       const typename LAcc<T, SP>::v* init = nullptr) {
  using G_ = Geo<sizeof(T), C, MB>;
  using V = typename LAcc<T, SP>::v;
  constexpr int NT = sizeof(T) == 2 ? MB + 1 : MB;
  constexpr int SZ = (int)sizeof(T);
#pragma unroll
  for (int nb = 0; nb <= MB; ++nb) acc[nb] = (init && nb < MB) ? init[nb] : zero_acc<V>();
  // KEEP_X: all point fragments are read up front and returned in xa (for
  // reuse by the caller); otherwise each is read with its step's table
  // fragments and dropped after use (fewer live registers).
  if constexpr (KEEP_X) {
#pragma unroll
    for (int s = 0; s < C / 32; ++s) ld_row<T>(xa[s], xt, lb.x, 32 * s * SZ);
  }
  struct F { K32<T> t[NT]; K32<T> x; };
  pipelined<C / 32, 2, F>(
      [&](int s, F& f) {
        if constexpr (!KEEP_X) ld_row<T>(f.x, xt, lb.x, 32 * s * SZ);
#pragma unroll
        for (int nb = 0; nb < NT; ++nb) {
          if (nb < MB)
            ld_row<T>(f.t[nb], tabL, lb.t, 16 * nb * G_::TROW + 32 * s * SZ);
          else
            ld_row<T>(f.t[nb], tabL, lb.a, G_::M16 * G_::TROW + 32 * s * SZ);
        }
      },
      [&](int s, F& f) {
        const K32<T>& x = KEEP_X ? xa[s] : f.x;
#pragma unroll
        for (int nb = 0; nb < NT; ++nb)
          acc[nb] = SP ? mma_acc(f.t[nb], x, acc[nb]) : mma_acc(x, f.t[nb], acc[nb]);
      });
}

// Logits (SP layout, bf16) of H 16-point halves in one pass over the table:
// each table fragment feeds every half.  xfrag(h, s, f) gives the point
// fragment of half h at step s.  Block MB is the temperature block.
template <typename T, int C, int MB, int H, typename XFrag>
__device__ __forceinline__ void logits_h(f32x4 (&acc)[H][MB + 1], const char* tabL,
                                         const LogitsBases<T, C, MB>& lb, XFrag xfrag) {
  using G_ = Geo<sizeof(T), C, MB>;
  constexpr int SZ = (int)sizeof(T);
#pragma unroll
  for (int h = 0; h < H; ++h)
#pragma unroll
    for (int nb = 0; nb <= MB; ++nb) acc[h][nb] = zero4();
  struct F { K32<T> t[MB + 1]; K32<T> x[H]; };
  pipelined<C / 32, 2, F>(
      [&](int s, F& f) {
#pragma unroll
        for (int h = 0; h < H; ++h) xfrag(h, s, f.x[h]);
#pragma unroll
        for (int nb = 0; nb <= MB; ++nb) {
          if (nb < MB)
            ld_row<T>(f.t[nb], tabL, lb.t, 16 * nb * G_::TROW + 32 * s * SZ);
          else
            ld_row<T>(f.t[nb], tabL, lb.a, G_::M16 * G_::TROW + 32 * s * SZ);
        }
      },
      [&](int s, F& f) {
#pragma unroll
        for (int h = 0; h < H; ++h)
#pragma unroll
          for (int nb = 0; nb <= MB; ++nb) acc[h][nb] = mma_acc(f.t[nb], f.x[h], acc[h][nb]);
      });
}

// Unclamped temperature t = tau0 + b_t + x.a of the lane's own point (row r
// of the tile).  bf16 storage: the MFMA temperature block (fp32 accumulate).
// fp32 storage: the products x_c a_c are exact in fp64 and are summed in
// fp64, because t can sit just above tau_min after cancellation (tau0 vs
// x.a) and the backward scales with 1/tau^2; an fp32 sum would lose about
// 1e-5 of tau there.
template <typename T, int C, int MB, typename V>
__device__ __forceinline__ float temperature_own(const V (&acc)[MB + 1], const K32<T> (&xa)[C / 32],
                                                 const char* tabL, const RowBase<T>& ab,
                                                 double tb) {
  using G_ = Geo<sizeof(T), C, MB>;
  if constexpr (sizeof(T) == 2) {
    return (float)acc[MB][0] + (float)tb;
  } else {
    double s = 0.0;
#pragma unroll
    for (int q = 0; q < C / 32; ++q) {
      K32<float> av;
      ld_row<float>(av, tabL, ab, G_::M16 * G_::TROW + 32 * q * 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s = fma((double)xa[q].lo[e], (double)av.lo[e], s);
        s = fma((double)xa[q].hi[e], (double)av.hi[e], s);
      }
    }
    s = s + __shfl_xor(s, 16);
    s = s + __shfl_xor(s, 32);
    return (float)(tb + s);
  }
}

// PS layout: temperatures of points 4g+i (i = 0..3).
template <typename T, int C, int MB, typename V>
__device__ __forceinline__ void temperature_ps(const V (&acc)[MB + 1], const K32<T> (&xa)[C / 32],
                                               const char* tabL, const RowBase<T>& ab, double tb,
                                               float (&t)[4]) {
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int i = 0; i < 4; ++i) t[i] = (float)acc[MB][i] + (float)tb;
  } else {
    const float own = temperature_own<T, C, MB, V>(acc, xa, tabL, ab, tb);
    const int g = lane_id() >> 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) t[i] = __shfl(own, 4 * g + i);
  }
}

// Softmax over slices, PS layout.  u = l + b + g (the noisy logit), m its
// row maximum; the base-2 exponent zs = (u - m) log2(e) / tau is formed
// after the shift, so its error is relative to u - m (not to u / tau, which
// is large when tau is clamped); w = 2^zs / sum.  Padded slices (j >= M)
// have bias -inf in the table header and Gumbel 0 (the G tile starts zeroed
// and only its first M columns are ever written), so they get w = 0; points
// beyond N get w = 0.  The Gumbel values are read transposed from the G tile
// (rows 4g+i, column 16nb+r).
template <typename T, int MB, typename V>
__device__ __forceinline__ void softmax_ps(const V (&acc)[MB + 1], const char* gt, int M,
                                           const float (&bias)[MB], const float (&t)[4],
                                           float tau_min, int nvalid, float (&w)[MB][4],
                                           float (&tau)[4]) {
  using R = decltype(acc[0][0] + 0.f);
  const int g = lane_id() >> 4;
  const int r = lane_id() & 15;
  R u[MB][4];
#pragma unroll
  for (int nb = 0; nb < MB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float gv = to_f<T>(reinterpret_cast<const T*>(gt)[(4 * g + i) * M + 16 * nb + r]);
      u[nb][i] = (R)acc[nb][i] + (R)bias[nb] + (R)gv;
    }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    tau[i] = fmaxf(t[i], tau_min);
    const R k = (R)(kLog2e * fast_rcp(tau[i]));
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
    const float inv = (4 * g + i) < nvalid ? fast_rcp(s) : 0.f;
#pragma unroll
    for (int nb = 0; nb < MB; ++nb) w[nb][i] = e[nb] * inv;
  }
}

// Softmax over slices, SP layout (the lane's point is r).  Also returns the
// shifted base-2 exponents zs (the natural logit is zs ln 2 + const) for
// the temperature gradient.  The Gumbel values are four consecutive
// elements of row r of the G tile.  With bf16 storage the exponent is one
// fma, u k - m k (its rounding error, relative to u k, stays far below the
// bf16 tolerance); fp32 storage keeps the shift before the scale.
template <typename T, int MB, typename V>
__device__ __forceinline__ void softmax_sp(const V (&acc)[MB + 1], const char* gt, int M,
                                           const float (&bias)[MB][4], float t, float tau_min,
                                           int nvalid, float (&w)[MB][4], float (&zs)[MB][4],
                                           float& tau) {
  using R = decltype(acc[0][0] + 0.f);
  constexpr int SZ = (int)sizeof(T);
  const int r = lane_id() & 15, g = lane_id() >> 4;
  tau = fmaxf(t, tau_min);
  const R k = (R)(kLog2e * fast_rcp(tau));
  R u[MB][4];
  float m = -INFINITY;
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) {
    float gv[4];
    const int e = r * M + 16 * nb + 4 * g;  // element index in the G tile
    if (M % 4 == 0) {                        // 4 aligned elements
      if constexpr (SZ == 2) {
        const bf16x4 q = *reinterpret_cast<const bf16x4*>(gt + e * SZ);
#pragma unroll
        for (int i = 0; i < 4; ++i) gv[i] = (float)q[i];
      } else {
        const f32x4 q = *reinterpret_cast<const f32x4*>(gt + e * SZ);
#pragma unroll
        for (int i = 0; i < 4; ++i) gv[i] = q[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) gv[i] = to_f<T>(reinterpret_cast<const T*>(gt)[e + i]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      u[nb][i] = (R)acc[nb][i] + (R)bias[nb][i] + (R)gv[i];
      m = fmaxf(m, (float)u[nb][i]);
    }
  }
  m = groups_max(m);
  float s = 0.f;
  float e[MB][4];
  const float mk = (float)((R)m * k);
#pragma unroll
  for (int nb = 0; nb < MB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if constexpr (SZ == 2)
        zs[nb][i] = fmaf((float)u[nb][i], (float)k, -mk);
      else
        zs[nb][i] = (float)((u[nb][i] - (R)m) * k);
      e[nb][i] = fast_exp2(zs[nb][i]);
      s += e[nb][i];
    }
  s = groups_sum(s);
  const float inv = r < nvalid ? fast_rcp(s) : 0.f;
#pragma unroll
  for (int nb = 0; nb < MB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) w[nb][i] = e[nb][i] * inv;
}

// Stored weights of a tile's points -- a [16][M] tile laid out like the
// Gumbel rows (W has G's shape and dtype) -- in the SP layout softmax_sp
// returns: lane (r, g) gets slices 16nb + 4g + i of point r.  Slices >= M
// and points >= nvalid are 0 (selected, so whatever the padding holds).
template <typename T, int MB>
__device__ __forceinline__ void w_tile(const char* wt, int M, int nvalid, float (&w)[MB][4]) {
  constexpr int SZ = (int)sizeof(T);
  const int r = lane_id() & 15, g = lane_id() >> 4;
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) {
    const int j0 = 16 * nb + 4 * g, e = r * M + j0;
    float v[4];
    if (M % 4 == 0) {  // 4 aligned elements
      if constexpr (SZ == 2) {
        const bf16x4 q = *reinterpret_cast<const bf16x4*>(wt + e * SZ);
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = (float)q[i];
      } else {
        const f32x4 q = *reinterpret_cast<const f32x4*>(wt + e * SZ);
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = q[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = to_f<T>(reinterpret_cast<const T*>(wt)[e + i]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) w[nb][i] = (r < nvalid && j0 + i < M) ? v[i] : 0.f;
  }
}

// The weights of a tile's first nvalid points, staged in LDS as rows of
// stride `rowb` bytes (slices contiguous), written to rows [p0, p0 + nvalid)
// of W [N,M]: 16-byte stores when a row is a whole number of 16-byte chunks
// (the rows are then one contiguous run), else element by element.  These
// stores go through the caches, unlike the other streamed outputs: the
// deslice reads W next, walking backwards onto the lines written last
// (measured at N = 1M: aggregate -8 us, deslice -16 us against non-temporal
// stores).  Each lane issues a fixed number of (masked) stores: the vector
// memory counter also counts stores, and with a data-dependent number of
// them the compiler can only wait for the prefetched tile by waiting for
// everything.
template <typename T, int ROWS, int M16>
__device__ __forceinline__ void write_w_rows(T* W, int64_t p0, int nvalid, const char* wl, int M,
                                             int rowb) {
  constexpr int SZ = (int)sizeof(T);
  const int lane = lane_id();
  char* d = reinterpret_cast<char*>(W + p0 * M);
  if ((M * SZ) % 16 == 0) {
    constexpr int K = (ROWS * M16 * SZ / 16 + 63) / 64;
    const int cpr = M * SZ / 16, n = nvalid * cpr;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int q = lane + 64 * k;
      const int row = q / cpr, c = q - row * cpr;
      if (q < n)
        *reinterpret_cast<uint4*>(d + (int64_t)16 * q) =
            *reinterpret_cast<const uint4*>(wl + row * rowb + 16 * c);
    }
  } else {
    constexpr int K = (ROWS * M16 + 63) / 64;
    const int n = nvalid * M;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int e = lane + 64 * k;
      const int row = e / M, j = e - row * M;
      if (e < n) reinterpret_cast<T*>(d)[e] = *reinterpret_cast<const T*>(wl + row * rowb + j * SZ);
    }
  }
}

// Zero a wave-private LDS region (16-byte multiple).
__device__ __forceinline__ void zero_lds(char* p, int bytes) {
  for (int q = lane_id(); q < bytes / 16; q += 64) reinterpret_cast<uint4*>(p)[q] = uint4{0, 0, 0, 0};
}

// Copy the table image (BYTES, a multiple of 16) from global memory into LDS
// with the block's THREADS threads: each thread issues the loads of all its
// 16-byte chunks before it stores any (a copy loop that stores each chunk
// before loading the next waits one memory round trip per chunk: 10 to 14 of
// them for the larger images, at the start of every block).  Chunks past the
// end are the last chunk again, loaded and stored again (the same bytes to
// the same place), so no lane-dependent branch separates the loads.
template <int U, int END, int THREADS, int NQ>
__device__ __forceinline__ void copy_chunks(uint4* dst, const uint4* src, int t) {
  if constexpr (U < END) {
    const int q = t + U * THREADS;
    const int qq = q < NQ ? q : NQ - 1;
    const uint4 v = src[qq];
    copy_chunks<U + 1, END, THREADS, NQ>(dst, src, t);  // later chunks' loads first
    dst[qq] = v;
  }
}
// (batches of at most 16 chunks in registers per thread)
template <int B0, int PER, int THREADS, int NQ>
__device__ __forceinline__ void copy_batches(uint4* dst, const uint4* src, int t) {
  if constexpr (B0 < PER) {
    constexpr int END = B0 + 16 < PER ? B0 + 16 : PER;
    copy_chunks<B0, END, THREADS, NQ>(dst, src, t);
    copy_batches<END, PER, THREADS, NQ>(dst, src, t);
  }
}
template <int BYTES, int THREADS>
__device__ __forceinline__ void copy_image(char* lds, const void* img) {
  static_assert(BYTES % 16 == 0, "image bytes must be a multiple of 16");
  constexpr int NQ = BYTES / 16;
  constexpr int PER = (NQ + THREADS - 1) / THREADS;  // chunks per thread
  copy_batches<0, PER, THREADS, NQ>(reinterpret_cast<uint4*>(lds),
                                    reinterpret_cast<const uint4*>(img), (int)threadIdx.x);
}

// (wave: the wave's index in its block, uniform, so the range is scalar)
__device__ __forceinline__ void tile_range(int64_t N, int waves, int wave, int64_t& t0,
                                           int64_t& t1, int rows = 16) {
  const int64_t tiles = (N + rows - 1) / rows;
  const int64_t tw = (int64_t)gridDim.x * waves;
  const int64_t gw = (int64_t)blockIdx.x * waves + wave;
  t0 = tiles * gw / tw;
  t1 = tiles * (gw + 1) / tw;
}

// Sum of per-wave register partials over the block's waves, pairwise in a
// fixed order (((w0 + w1) + (w2 + w3)) + ...), through LDS slots (the
// tables and tiles are dead by then; WAVES/2 slots of NV f32x4 per lane at
// lds); wave 0 ends with the block total.  visit(f) calls f(f32x4&) on every
// partial vector, always in the same order.
template <int WAVES, int NV, typename Visit>
__device__ __forceinline__ void block_tree_reduce(char* lds, Visit visit) {
  const int wave = threadIdx.x >> 6, lane = lane_id();
  f32x4* slots = reinterpret_cast<f32x4*>(lds);
#pragma unroll
  for (int span = 1; span < WAVES; span *= 2) {
    __syncthreads();  // the LDS is free (main loop, or the previous round, done)
    f32x4* slot = slots + (wave / (2 * span)) * NV * 64;
    if ((wave & (2 * span - 1)) == span) {
      int k = 0;
      visit([&](f32x4& v) { slot[64 * k++ + lane] = v; });
    }
    __syncthreads();
    if ((wave & (2 * span - 1)) == 0) {
      int k = 0;
      visit([&](f32x4& v) { v += slot[64 * k++ + lane]; });
    }
  }
}

// ---------------------------------------------------------------------------
// kAggregate and kDesliceBwd: W^T x (with den = W^T 1) or W^T dY.  The
// weights come out of the softmax in the SP layout (lane: one point, 4
// slices per block); they are staged in LDS and read back transposed, which
// gives the contraction over points its A operand (lane: one slice, 4
// points).  den is the same contraction against a B operand of ones, so it
// uses exactly the rounded weights of num.  With 32-row tiles the two
// 16-point halves share the logits' table reads and their contractions over
// points pair into K32 MFMAs.
// ---------------------------------------------------------------------------
template <typename T, int C, int MB, int ROWS, bool BWD>
struct AggStage {
  TileRegs<T, C, ROWS> x;  // x rows
  TileRegs<T, C, ROWS> y;  // dY rows (BWD)
  GRegs<T, MB, ROWS> g;
};

// WV (stored weights): the forward also writes the weights it contracts
// (kAggregateW); the backward reads them from W (given as a.G) instead of
// recomputing them from x and G (kDesliceBwdW: no table, no x tile).
constexpr int agg_pass(bool bwd, bool wv) {
  return bwd ? (wv ? kDesliceBwdW : kDesliceBwd) : (wv ? kAggregateW : kAggregate);
}

template <typename T, int C, int MB, bool BWD, bool WV = false, bool EX = true>
__global__ void __launch_bounds__((64 * Geo<sizeof(T), C, MB>::waves(agg_pass(BWD, WV))))
k_aggregate(StreamArgs a) {
  using G_ = Geo<sizeof(T), C, MB>;
  constexpr int PASS = agg_pass(BWD, WV);
  constexpr bool WIN = BWD && WV, WOUT = !BWD && WV;
  constexpr int WAVES = G_::waves(PASS);
  constexpr int ROWS = G_::rows(PASS), H = ROWS / 16;
  constexpr int SZ = (int)sizeof(T);
  using V = typename LAcc<T, true>::v;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  head_offsets(a);
  add_tb_dev(a);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane_id() & 15, g = lane_id() >> 4;
  const bool hasG = WIN || (a.flags & kHasG);  // WIN: the Gumbel rows' buffer holds W

  const char* tabL = smem + G_::OFF_L;
  char* wreg = smem + G_::img_bytes(PASS) + wave * G_::wave_bytes(PASS);
  // x tile (logits), contracted tile (x, or dY), Gumbel rows (or stored
  // weights), transposed weights
  char* const xt = wreg;
  char* const yt = BWD ? wreg + H * G_::XT : wreg;
  char* const gbuf = wreg + (BWD ? 2 : 1) * H * G_::XT;
  char* const wbuf = gbuf + H * G_::GT;
  const auto lb = logits_bases<T, C, MB, true>();
  const int xtr = tr_base<T>(G_::XT_ROW);
  const int wtr = tr_base<T>(G_::GROW);
  const int wsb = r * G_::GROW + 4 * g * SZ;  // SP weights of point r, slices 16nb + 4g ..

  float bias[MB][4];
  auto init = [&]() {
    if constexpr (!WIN) {
      copy_image<G_::img_bytes(PASS), 64 * WAVES>(smem, a.img);
      __syncthreads();
    }
    zero_lds(gbuf, 2 * H * G_::GT);
#pragma unroll
    for (int nb = 0; nb < MB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        bias[nb][i] = WIN ? 0.f : reinterpret_cast<const float*>(smem)[16 * nb + 4 * g + i];
  };

  f32x4 acc[MB][G_::CB], dacc[MB];
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) {
    dacc[nb] = zero4();
#pragma unroll
    for (int cb = 0; cb < G_::CB; ++cb) acc[nb][cb] = zero4();
  }
  K16<T> ones;
  set_k16(ones, 1.f, 1.f, 1.f, 1.f);

  const T* X = reinterpret_cast<const T*>(a.x);
  const T* Y = reinterpret_cast<const T*>(a.dY);
  const T* Gp = reinterpret_cast<const T*>(a.G);
  int64_t t0, t1;
  tile_range(a.N, WAVES, wave, t0, t1, ROWS);
  using Stage = AggStage<T, C, MB, ROWS, BWD>;

  auto tile_body = [&](int64_t t) {
    const int64_t p0 = t * ROWS;
    int nv[H];
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const int64_t rem = a.N - p0 - 16 * h;
      nv[h] = rem < 0 ? 0 : rem > 16 ? 16 : (int)rem;
    }
    float w[H][MB][4];
    if constexpr (WIN) {
#pragma unroll
      for (int h = 0; h < H; ++h) w_tile<T, MB>(gbuf + h * 16 * a.M * SZ, a.M, nv[h], w[h]);
    } else {
      V lg[H][MB + 1];
      float tt[H];
      if constexpr (H == 1) {
        K32<T> xa[G_::XF];
        logits<T, C, MB, true, (SZ == 4)>(lg[0], xa, xt, tabL, lb);
        tt[0] = temperature_own<T, C, MB>(lg[0], xa, tabL, lb.a, a.tb);
      } else {
        logits_h<T, C, MB, H>(lg, tabL, lb, [&](int h, int s, K32<T>& f) {
          ld_row<T>(f, xt, lb.x, h * 16 * G_::XT_ROW + 32 * s * SZ);
        });
#pragma unroll
        for (int h = 0; h < H; ++h) tt[h] = (float)lg[h][MB][0] + (float)a.tb;
      }
      float zs[MB][4], tau;
#pragma unroll
      for (int h = 0; h < H; ++h)
        softmax_sp<T, MB>(lg[h], gbuf + h * 16 * a.M * SZ, a.M, bias, tt[h], a.tau_min, nv[h],
                          w[h], zs, tau);
    }

    // SP -> PS through the weights buffer
    wave_sync();
#pragma unroll
    for (int h = 0; h < H; ++h)
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) {
        f32x4 v{w[h][nb][0], w[h][nb][1], w[h][nb][2], w[h][nb][3]};
        stage4<T>(wbuf, wsb + h * 16 * G_::GROW, 16 * nb * SZ, v);
      }
    wave_sync();
    // the rows just staged are the tile's weights as the contraction rounds
    // them (point rows, slices contiguous)
    if constexpr (WOUT) {
      int nvt = 0;
#pragma unroll
      for (int h = 0; h < H; ++h) nvt += nv[h];
      write_w_rows<T, ROWS, G_::M16>(reinterpret_cast<T*>(a.out), p0, nvt, wbuf, a.M, G_::GROW);
    }
    K16<T> wt[H][MB];
#pragma unroll
    for (int h = 0; h < H; ++h)
#pragma unroll
      for (int nb = 0; nb < MB; ++nb)
        ld_tr<T>(wt[h][nb], wbuf, wtr, h * 16 * G_::GROW + 16 * nb * SZ, G_::GROW);
    if constexpr (!BWD) {
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) {
        if constexpr (H == 2)
          dacc[nb] = mma16x2(wt[0][nb], ones, wt[1][nb], ones, dacc[nb]);
        else
          dacc[nb] = mma16(wt[0][nb], ones, dacc[nb]);
      }
    }
    struct F { K16<T> xb[H]; };
    pipelined<G_::CB, 4, F>(
        [&](int cb, F& f) {
#pragma unroll
          for (int h = 0; h < H; ++h)
            ld_tr<T>(f.xb[h], yt, xtr, h * 16 * G_::XT_ROW + 16 * cb * SZ, G_::XT_ROW);
        },
        [&](int cb, F& f) {
#pragma unroll
          for (int nb = 0; nb < MB; ++nb) {
            if constexpr (H == 2)
              acc[nb][cb] = mma16x2(wt[0][nb], f.xb[0], wt[1][nb], f.xb[1], acc[nb][cb]);
            else
              acc[nb][cb] = mma16(wt[0][nb], f.xb[0], acc[nb][cb]);
          }
        });
  };

  auto load = [&](Stage& st, int64_t tile) {
    const int64_t p0 = tile * ROWS;
    constexpr bool NT = !keep_loads<PASS>();
    if constexpr (!WIN) load_tile<T, C, ROWS, NT, EX>(st.x, X, p0, a.N, a.cr);
    if constexpr (BWD) load_tile<T, C, ROWS, NT, EX>(st.y, Y, p0, a.N, a.cr);
    // G (or W): streamed either way; `safe` is any readable 16 bytes
    const void* safe = WIN ? a.img : static_cast<const void*>(X);
    load_g<T, MB, ROWS, true>(st.g, Gp, safe, p0, a.N, a.M, hasG);
  };
  auto store = [&](const Stage& st) {
    if constexpr (!WIN) store_tile<T, C, ROWS>(xt, st.x);
    if constexpr (BWD) store_tile<T, C, ROWS>(yt, st.y);
    if (hasG) store_g<T, MB, ROWS>(gbuf, st.g, a.M, hasG);
  };
  auto tail = [&](int64_t t) {
    Stage st;
    load(st, t);
    wave_sync();
    store(st);
    g_fixup<T, MB, ROWS>(gbuf, Gp, t * ROWS, a.N, a.M, hasG);
    wave_sync();
    tile_body(t);
  };
  stream_tiles<agg_depth<T, C, MB, BWD>(), Stage>(t0, t1, a.N / ROWS, load, store, tile_body, tail,
                                             init);

  // block total in wave 0, written as this block's record: num [M][C]
  // (or dS' [M][C]), then den [M]
  block_tree_reduce<WAVES, MB * G_::CB + (BWD ? 0 : MB)>(smem, [&](auto f) {
#pragma unroll
    for (int nb = 0; nb < MB; ++nb)
#pragma unroll
      for (int cb = 0; cb < G_::CB; ++cb) f(acc[nb][cb]);
    if constexpr (!BWD)
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) f(dacc[nb]);
  });
  if (wave == 0) {
    float* rec = a.partials + (int64_t)blockIdx.x * a.rec;
    const int cw = EX ? C : a.cr;  // the record's channels
#pragma unroll
    for (int nb = 0; nb < MB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = 16 * nb + 4 * g + i;
        if (j < a.M) {
#pragma unroll
          for (int cb = 0; cb < G_::CB; ++cb)
            if (16 * cb < cw) rec[j * cw + 16 * cb + r] = acc[nb][cb][i];
          if (!BWD && r == 0) rec[a.M * cw + j] = dacc[nb][i];
        }
      }
  }
}

// ---------------------------------------------------------------------------
// kDeslice (SP layout): y = W S'.  The y tile is staged in the x tile, which
// the logits are done with, and written back as whole rows.
// ---------------------------------------------------------------------------
// WIN (kDesliceW): the weights are read from W (given as a.G, in the Gumbel
// rows' buffer) instead of recomputed; only the deslice table is in LDS.
template <typename T, int C, int MB, bool WIN = false, bool EX = true>
__global__ void __launch_bounds__((64 * Geo<sizeof(T), C, MB>::waves(WIN ? kDesliceW : kDeslice)))
k_deslice(StreamArgs a) {
  using G_ = Geo<sizeof(T), C, MB>;
  constexpr int PASS = WIN ? kDesliceW : kDeslice;
  constexpr int WAVES = G_::waves(PASS);
  constexpr int SZ = (int)sizeof(T);
  extern __shared__ __attribute__((aligned(16))) char smem[];
  head_offsets(a);
  add_tb_dev(a);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane_id() & 15, g = lane_id() >> 4;
  const bool hasG = WIN || (a.flags & kHasG);

  const char* tabL = smem + G_::OFF_L;
  const char* tabS = smem + (WIN ? 0 : G_::OFF_2);
  char* xt = smem + G_::img_bytes(PASS) + wave * G_::wave_bytes(PASS);
  char* gt = xt + G_::XT;
  const auto lb = logits_bases<T, C, MB, true>();
  const int sb = r * G_::SROW + 4 * g * SZ;  // S'^T row 16cb + r, slices 16nb + 4g ..
  const int stb = stage_base<T>(G_::XT_ROW);

  float bias[MB][4];
  auto init = [&]() {
    if constexpr (WIN)  // the deslice table part of the image only
      copy_image<G_::SZ_S, 64 * WAVES>(smem, reinterpret_cast<const char*>(a.img) + G_::OFF_2);
    else
      copy_image<G_::img_bytes(kDeslice), 64 * WAVES>(smem, a.img);
    __syncthreads();
    zero_lds(gt, G_::GT);
#pragma unroll
    for (int nb = 0; nb < MB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        bias[nb][i] = WIN ? 0.f : reinterpret_cast<const float*>(smem)[16 * nb + 4 * g + i];
  };

  const T* X = reinterpret_cast<const T*>(a.x);
  const T* Gp = reinterpret_cast<const T*>(a.G);
  T* Y = reinterpret_cast<T*>(a.out);
  int64_t t0, t1;
  tile_range(a.N, WAVES, wave, t0, t1);

  using Stage = TileStage<T, C, MB>;
  auto load = [&](Stage& st, int64_t tile) {
    constexpr bool NT = !keep_loads<PASS>();
    if constexpr (WIN) {
      load_g<T, MB, 16, NT>(st.g, Gp, a.img, tile * 16, a.N, a.M, hasG);
    } else {
      load_tile<T, C, 16, NT, EX>(st.x, X, tile * 16, a.N, a.cr);
      load_g<T, MB, 16, NT>(st.g, Gp, X, tile * 16, a.N, a.M, hasG);
    }
  };
  auto store = [&](const Stage& st) {
    if constexpr (!WIN) store_tile<T, C>(xt, st.x);
    if (hasG) store_g<T, MB>(gt, st.g, a.M, hasG);
  };
  auto body = [&](int64_t t) {
    const int64_t p0 = t * 16;
    const int nvalid = (int)(a.N - p0 < 16 ? a.N - p0 : 16);

    float w[MB][4];
    if constexpr (WIN) {
      w_tile<T, MB>(gt, a.M, nvalid, w);
    } else {
      typename LAcc<T, true>::v lg[MB + 1];
      K32<T> xa[G_::XF];
      logits<T, C, MB, true>(lg, xa, xt, tabL, lb);
      float zs[MB][4], tau;
      const float tt = temperature_own<T, C, MB>(lg, xa, tabL, lb.a, a.tb);
      softmax_sp<T, MB>(lg, gt, a.M, bias, tt, a.tau_min, nvalid, w, zs, tau);
    }

    K16<T> wb[MB];
#pragma unroll
    for (int nb = 0; nb < MB; ++nb) set_k16(wb[nb], w[nb][0], w[nb][1], w[nb][2], w[nb][3]);
    wave_sync();  // the logits reads of the x tile are done: it becomes the y tile
    struct F { K16<T> s[MB]; };
    pipelined<G_::CB, 4, F>(
        [&](int cb, F& f) {
#pragma unroll
          for (int nb = 0; nb < MB; ++nb) ld_k16(f.s[nb], tabS + sb + 16 * cb * G_::SROW + 16 * nb * SZ);
        },
        [&](int cb, F& f) {
          f32x4 d = zero4();
#pragma unroll
          for (int nb = 0; nb + 1 < MB; nb += 2)
            d = mma16x2(f.s[nb], wb[nb], f.s[nb + 1], wb[nb + 1], d);
          if constexpr (MB % 2 == 1) {
            // the odd product stays a K32 MFMA (zero second half): one MFMA
            // shape per accumulator chain (a 16x16x16 MFMA taking the
            // accumulator of a preceding 16x16x32 one gave wrong sums)
            if constexpr (SZ == 2) {
              K16<T> z;
              set_k16(z, 0.f, 0.f, 0.f, 0.f);
              d = mma16x2(f.s[MB - 1], wb[MB - 1], z, z, d);
            } else {
              d = mma16(f.s[MB - 1], wb[MB - 1], d);
            }
          }
          stage4<T>(xt, stb, 16 * cb * SZ, d);
        });
    wave_sync();
    write_tile<T, C, 16, EX>(Y, p0, xt, nvalid, a.cr);
  };
  auto tail = [&](int64_t t) {
    Stage st;
    load(st, t);
    wave_sync();
    store(st);
    g_fixup<T, MB>(gt, Gp, t * 16, a.N, a.M, hasG);
    wave_sync();
    body(t);
  };
  stream_tiles<des_depth<T, C, MB>(), Stage, kRevDeslice>(t0, t1, a.N / 16, load, store, body, tail,
                                                     init);
}

// ---------------------------------------------------------------------------
// kWeights (PS layout): W [N,M] fp32 and tau [N] written out.
// ---------------------------------------------------------------------------
template <typename T, int C, int MB, bool EX = true>
__global__ void __launch_bounds__((64 * Geo<sizeof(T), C, MB>::waves(kWeights))) k_weights(StreamArgs a) {
  using G_ = Geo<sizeof(T), C, MB>;
  constexpr int WAVES = G_::waves(kWeights);
  extern __shared__ __attribute__((aligned(16))) char smem[];
  head_offsets(a);
  add_tb_dev(a);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane_id() & 15, g = lane_id() >> 4;
  const bool hasG = a.flags & kHasG;

  copy_image<G_::img_bytes(kWeights), 64 * WAVES>(smem, a.img);
  __syncthreads();
  const char* tabL = smem + G_::OFF_L;
  char* xt = smem + G_::img_bytes(kWeights) + wave * G_::wave_bytes(kWeights);
  char* gt = xt + G_::XT;
  zero_lds(gt, G_::GT);
  const auto lb = logits_bases<T, C, MB, false>();
  float bias[MB];
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) bias[nb] = reinterpret_cast<const float*>(smem)[16 * nb + r];

  const T* X = reinterpret_cast<const T*>(a.x);
  const T* Gp = reinterpret_cast<const T*>(a.G);
  float* W = reinterpret_cast<float*>(a.out);
  int64_t t0, t1;
  tile_range(a.N, WAVES, wave, t0, t1);
  TileRegs<T, C> xr;
  GRegs<T, MB> gr;
  for (int64_t t = t0; t < t1; ++t) {
    const int64_t p0 = t * 16;
    load_tile<T, C, 16, true, EX>(xr, X, p0, a.N, a.cr);
    load_g<T, MB>(gr, Gp, X, p0, a.N, a.M, hasG);
    const int nvalid = (int)(a.N - p0 < 16 ? a.N - p0 : 16);
    wave_sync();
    store_tile<T, C>(xt, xr);
    store_g<T, MB>(gt, gr, a.M, hasG);
    wave_sync();
    if (!hasG || p0 + 16 > a.N) {  // Gumbel rows load_g did not read
      g_fixup<T, MB>(gt, Gp, p0, a.N, a.M, hasG);
      wave_sync();
    }
    typename LAcc<T, false>::v lg[MB + 1];
    K32<T> xa[G_::XF];
    logits<T, C, MB, false>(lg, xa, xt, tabL, lb);
    float w[MB][4], tau[4], tt[4];
    temperature_ps<T, C, MB>(lg, xa, tabL, lb.a, a.tb, tt);
    softmax_ps<T, MB>(lg, gt, a.M, bias, tt, a.tau_min, nvalid, w, tau);
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
//   dx   = W dnum + A dl + a dt
//   dA  += x^T dl,  db += 1^T dl,  da += x^T dt,  db_t += 1^T dt
// The backward table rows hold dnum_j - cN and s'_j - cS (a shift common to
// all slices, which the softmax backward does not see); the header's dden is
// centred here by its den-weighted mean cD.  Without the states term the
// dnum rows, cN and dden are zero in the table image; without the deslice
// term the dY contraction is skipped.  The dx tile is staged in the dY tile
// (dw is done with it) and written back as whole rows.
// ---------------------------------------------------------------------------
template <typename T, int C, int MB, int PASS, bool EX = true>
__global__ void __launch_bounds__((64 * Geo<sizeof(T), C, MB>::waves(PASS))) k_slice_bwd(StreamArgs a) {
  using G_ = Geo<sizeof(T), C, MB>;
  using V = typename LAcc<T, true>::v;
  constexpr int WAVES = G_::waves(PASS);
  constexpr int M16 = G_::M16;
  constexpr int SZ = (int)sizeof(T);
  constexpr int SROWF = M16 + 1;  // dl transpose row stride (floats)
  extern __shared__ __attribute__((aligned(16))) char smem[];
  head_offsets(a);
  add_tb_dev(a);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane_id() & 15, g = lane_id() >> 4;
  const bool hasG = a.flags & kHasG;
  const bool deslice = (PASS == kSliceBwd) && (a.flags & kDesliceTerm);

  const float* hdr = reinterpret_cast<const float*>(smem);
  const float* dden_tab = hdr + M16;
  const float* cN = hdr + 2 * M16;
  const float* af = hdr + 3 * M16 + 2 * C;  // a in fp32
  const char* tabL = smem + G_::OFF_L;
  const char* tabW = smem + G_::OFF_2;
  char* wreg = smem + G_::img_bytes(PASS) + wave * G_::wave_bytes(PASS);
  char* xt = wreg;
  char* yt = wreg + G_::XT;  // dY tile, then the dx staging tile
  char* gt = wreg + 2 * G_::XT;
  float* scr = reinterpret_cast<float*>(gt + G_::GT);  // [16][M16+1]
  float* scr_dt = scr + 16 * SROWF;                     // [16]
  const auto lb = logits_bases<T, C, MB, true>();
  const RowBase<T> yb = row_base<T>(r, G_::XT_ROW);
  const RowBase<T> wrb = row_base<T>(a_row<V>(r), G_::WROW);
  const int xtr = tr_base<T>(G_::XT_ROW);
  const int ltr = tr_base<T>(G_::TROW);
  const int wtr = tr_base<T>(G_::WROW);
  const int stb = stage_base<T>(G_::XT_ROW);

  float bias[MB][4], dden[MB][4];
  auto init = [&]() {
    copy_image<G_::img_bytes(PASS), 64 * WAVES>(smem, a.img);
    __syncthreads();
    zero_lds(gt, G_::GT);
    // dden_j centred by its den-weighted mean (a shift common to all slices)
    float cD = 0.f;
    const float* sw = hdr + 2 * M16 + 2 * C;
    for (int j = 0; j < a.M; ++j) cD += sw[j] * dden_tab[j];
#pragma unroll
    for (int nb = 0; nb < MB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = 16 * nb + 4 * g + i;
        bias[nb][i] = hdr[j];
        dden[nb][i] = j < a.M ? dden_tab[j] - cD : 0.f;
      }
  };

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
  tile_range(a.N, WAVES, wave, t0, t1);

  using Stage = TileStage<T, C, MB>;
  auto load = [&](Stage& st, int64_t tile) {
    // dY is loaded unconditionally (x stands in without the deslice term),
    // so that the loads are never predicated
    constexpr bool NT = !keep_loads<PASS>();
    load_tile<T, C, 16, NT, EX>(st.x, X, tile * 16, a.N, a.cr);
    load_tile<T, C, 16, NT, EX>(st.y, deslice ? Y : X, tile * 16, a.N, a.cr);
    load_g<T, MB, 16, NT>(st.g, Gp, X, tile * 16, a.N, a.M, hasG);
  };
  auto store = [&](const Stage& st) {
    store_tile<T, C>(xt, st.x);
    if (deslice) store_tile<T, C>(yt, st.y);
    if (hasG) store_g<T, MB>(gt, st.g, a.M, hasG);
  };
  auto body = [&](int64_t t) {
    const int64_t p0 = t * 16;
    const int nvalid = (int)(a.N - p0 < 16 ? a.N - p0 : 16);
    const bool pv = r < nvalid;

    V lg[MB + 1];
    K32<T> xa[G_::XF];
    float w[MB][4], zs[MB][4], tau, tt;
    // narrow rows (a pass bound by instruction issue): the logit contraction
    // starts at the biases and the dw contraction below at dden (no
    // separate adds per slice); the softmax then adds -0, which the
    // compiler drops.  (On wide rows, bound by memory, the separate adds
    // measured slightly faster.)
    constexpr bool NARROW = narrow_rows<T, C>() && SZ == 2;
    if constexpr (NARROW) {
      V bi[MB];
      float nob[MB][4];
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) {
        bi[nb] = V{bias[nb][0], bias[nb][1], bias[nb][2], bias[nb][3]};
#pragma unroll
        for (int i = 0; i < 4; ++i) nob[nb][i] = -0.f;
      }
      logits<T, C, MB, true>(lg, xa, xt, tabL, lb, bi);
      tt = temperature_own<T, C, MB>(lg, xa, tabL, lb.a, a.tb);
      softmax_sp<T, MB>(lg, gt, a.M, nob, tt, a.tau_min, nvalid, w, zs, tau);
    } else {
      logits<T, C, MB, true>(lg, xa, xt, tabL, lb);
      tt = temperature_own<T, C, MB>(lg, xa, tabL, lb.a, a.tb);
      softmax_sp<T, MB>(lg, gt, a.M, bias, tt, a.tau_min, nvalid, w, zs, tau);
    }

    // dw in the SP layout
    float dw[MB][4];
    if constexpr (PASS == kSliceBwd) {
      V acc[MB];
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) {
        if constexpr (NARROW)
          acc[nb] = V{dden[nb][0], dden[nb][1], dden[nb][2], dden[nb][3]};
        else
          acc[nb] = zero_acc<V>();
      }
      // states term: x . (dnum_j - cN)  (zero rows without the states term)
      struct FS { K32<T> tw[MB]; };
      pipelined<G_::XF, 2, FS>(
          [&](int s, FS& f) {
#pragma unroll
            for (int nb = 0; nb < MB; ++nb)
              ld_row<T>(f.tw[nb], tabW, wrb, 16 * nb * G_::WROW + 32 * s * SZ);
          },
          [&](int s, FS& f) {
#pragma unroll
            for (int nb = 0; nb < MB; ++nb) acc[nb] = mma_acc(f.tw[nb], xa[s], acc[nb]);
          });
      if (deslice) {
        // deslice term: dY . (s'_j - cS)
        struct FD { K32<T> ya; K32<T> tw[MB]; };
        pipelined<G_::XF, 2, FD>(
            [&](int s, FD& f) {
              ld_row<T>(f.ya, yt, yb, 32 * s * SZ);
#pragma unroll
              for (int nb = 0; nb < MB; ++nb)
                ld_row<T>(f.tw[nb], tabW, wrb, 16 * nb * G_::WROW + (C + 32 * s) * SZ);
            },
            [&](int s, FD& f) {
#pragma unroll
              for (int nb = 0; nb < MB; ++nb) acc[nb] = mma_acc(f.tw[nb], f.ya, acc[nb]);
            });
      }
#pragma unroll
      for (int nb = 0; nb < MB; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          dw[nb][i] = NARROW ? (float)acc[nb][i] : (float)(acc[nb][i] + dden[nb][i]);
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
    const float rtau = fast_rcp(tau);
    float dl[MB][4];
    float zdz = 0.f;
#pragma unroll
    for (int nb = 0; nb < MB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float dz = w[nb][i] * ((dw[nb][i] - wdw) - res);
        dl[nb][i] = dz * rtau;
        // a padded slice has the exponent -inf and dz exactly 0 (w = 0):
        // narrow rows clamp the exponent to a finite value (one
        // median-of-three, not a compare and select), which keeps their
        // product 0
        if constexpr (NARROW)
          zdz = fmaf(dz, __builtin_amdgcn_fmed3f(zs[nb][i], -__FLT_MAX__, __FLT_MAX__), zdz);
        else if (w[nb][i] != 0.f)
          zdz += dz * zs[nb][i];
      }
    zdz = groups_sum(zdz);
    float dtau = -kLn2 * zdz * rtau;
    if (PASS == kWeightsBwd && a.dtau != nullptr && pv) dtau += a.dtau[p0 + r];
    const float dt = (pv && tt > a.tau_min) ? dtau : 0.f;

    // dx = [W | dl] [dnum - cN ; A^T] + a dt + cN   (SP: D[channel][point])
    K16<T> wb[MB], lbk[MB];
#pragma unroll
    for (int nb = 0; nb < MB; ++nb) {
      set_k16(wb[nb], w[nb][0], w[nb][1], w[nb][2], w[nb][3]);
      set_k16(lbk[nb], dl[nb][0], dl[nb][1], dl[nb][2], dl[nb][3]);
    }
    wave_sync();  // the dw reads of the dY tile are done: it becomes the dx tile
    struct FX { K16<T> ta[MB], tn[MB]; f32x4 av, cn; };
    pipelined<G_::CB, 2, FX>(
        [&](int cb, FX& f) {
#pragma unroll
          for (int nb = 0; nb < MB; ++nb) {
            // A^T rows of the logits table and (dnum_j - cN) rows of the
            // backward table, read transposed: [channel][slice]
            ld_tr<T>(f.ta[nb], tabL, ltr, 16 * nb * G_::TROW + 16 * cb * SZ, G_::TROW);
            ld_tr<T>(f.tn[nb], tabW, wtr, 16 * nb * G_::WROW + 16 * cb * SZ, G_::WROW);
          }
          f.av = *reinterpret_cast<const f32x4*>(af + 16 * cb + 4 * g);
          f.cn = *reinterpret_cast<const f32x4*>(cN + 16 * cb + 4 * g);
        },
        [&](int cb, FX& f) {
          // the 2 MB products [A^T | dnum - cN] x [dl ; w], two per MFMA
          auto fa = [&](int q) -> const K16<T>& { return q < MB ? f.ta[q] : f.tn[q - MB]; };
          auto fb = [&](int q) -> const K16<T>& { return q < MB ? lbk[q] : wb[q - MB]; };
          // + a dt, + cN (the table rows hold dnum_j - cN, and sum_j w_j =
          // 1): on narrow rows, whose pass is bound by instruction issue, as
          // the products' starting value (one fma per element); on wider
          // rows added after them (as a starting value the accumulators
          // would move into AGPRs first)
          f32x4 d;
#pragma unroll
          for (int i = 0; i < 4; ++i) d[i] = NARROW ? fmaf(f.av[i], dt, f.cn[i]) : 0.f;
#pragma unroll
          for (int q = 0; q < 2 * MB; q += 2) d = mma16x2(fa(q), fb(q), fa(q + 1), fb(q + 1), d);
          if constexpr (!NARROW) {
#pragma unroll
            for (int i = 0; i < 4; ++i) d[i] += f.av[i] * dt + f.cn[i];
          }
          stage4<T>(yt, stb, 16 * cb * SZ, d);
        });

    // parameter gradients: transpose dl (and dt) to the PS layout
#pragma unroll
    for (int nb = 0; nb < MB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) scr[r * SROWF + 16 * nb + 4 * g + i] = dl[nb][i];
    if (g == 0) scr_dt[r] = dt;
    wave_sync();
    write_tile<T, C, 16, EX>(DX, p0, yt, nvalid, a.cr);
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
    const bf16x2 dt01{(bf16)dtp[0], (bf16)dtp[1]}, dt23{(bf16)dtp[2], (bf16)dtp[3]};
    struct FA { K16<T> xa; };
    pipelined<G_::CB, 8, FA>(
        [&](int cb, FA& f) { ld_tr<T>(f.xa, xt, xtr, 16 * cb * SZ, G_::XT_ROW); },
        [&](int cb, FA& f) {
          if constexpr (SZ == 2) {
            da[cb] = __builtin_amdgcn_fdot2_f32_bf16(
                bf16x2{f.xa.v[2], f.xa.v[3]}, dt23,
                __builtin_amdgcn_fdot2_f32_bf16(bf16x2{f.xa.v[0], f.xa.v[1]}, dt01, da[cb], false),
                false);
          } else {
            da[cb] += (k16_elem(f.xa, 0) * dtp[0] + k16_elem(f.xa, 1) * dtp[1]) +
                      (k16_elem(f.xa, 2) * dtp[2] + k16_elem(f.xa, 3) * dtp[3]);
          }
#pragma unroll
          for (int nb = 0; nb < MB; ++nb) dA[cb][nb] = mma16(f.xa, lp[nb], dA[cb][nb]);
        });
  };
  auto tail = [&](int64_t t) {
    Stage st;
    load(st, t);
    wave_sync();
    store(st);
    g_fixup<T, MB>(gt, Gp, t * 16, a.N, a.M, hasG);
    wave_sync();
    body(t);
  };
  stream_tiles<bwd_depth<T, C, MB>(), Stage, kRevSliceBwd>(t0, t1, a.N / 16, load, store, body, tail,
                                                       init);

  // lane partials -> wave totals
#pragma unroll
  for (int nb = 0; nb < MB; ++nb) db[nb] = groups_sum(db[nb]);
#pragma unroll
  for (int cb = 0; cb < G_::CB; ++cb) da[cb] = groups_sum(da[cb]);
  dbt = row16_sum(dbt);  // only g == 0 lanes carry values; sum their row

  // block total in wave 0, written as this block's record: dA [C][M],
  // db [M], da [C], db_t
  constexpr int NDA = (G_::CB + 3) / 4, NSC = (MB + 1 + 3) / 4;
  f32x4 dav[NDA], scv[NSC];
#pragma unroll
  for (int k = 0; k < 4 * NDA; ++k) dav[k / 4][k % 4] = k < G_::CB ? da[k] : 0.f;
#pragma unroll
  for (int k = 0; k < 4 * NSC; ++k) scv[k / 4][k % 4] = k < MB ? db[k] : k == MB ? dbt : 0.f;
  block_tree_reduce<WAVES, G_::CB * MB + NDA + NSC>(smem, [&](auto f) {
#pragma unroll
    for (int cb = 0; cb < G_::CB; ++cb)
#pragma unroll
      for (int nb = 0; nb < MB; ++nb) f(dA[cb][nb]);
#pragma unroll
    for (int k = 0; k < NDA; ++k) f(dav[k]);
#pragma unroll
    for (int k = 0; k < NSC; ++k) f(scv[k]);
  });
  if (wave == 0) {
    float* rec = a.partials + (int64_t)blockIdx.x * a.rec;
    const int M = a.M;
    const int cw = EX ? C : a.cr;  // the record's channels
#pragma unroll
    for (int nb = 0; nb < MB; ++nb) {
      const int j = 16 * nb + r;
      if (j < M) {
#pragma unroll
        for (int cb = 0; cb < G_::CB; ++cb) {
          if (16 * cb < cw) {
#pragma unroll
            for (int i = 0; i < 4; ++i) rec[(16 * cb + 4 * g + i) * M + j] = dA[cb][nb][i];
          }
        }
        if (g == 0) rec[cw * M + j] = scv[nb / 4][nb % 4];
      }
    }
    if (g == 0) {
#pragma unroll
      for (int cb = 0; cb < G_::CB; ++cb)
        if (16 * cb < cw) rec[cw * M + M + 16 * cb + r] = dav[cb / 4][cb % 4];
      if (r == 0) rec[cw * M + M + cw] = scv[MB / 4][MB % 4];
    }
  }
}

// ---------------------------------------------------------------------------
// Launch of one pass, dispatched over dtype, C and slice blocks.  Each pass
// is instantiated in its own translation unit (pa_stream_<pass>.hip).
// ---------------------------------------------------------------------------
// EX: rows of exactly C channels (the addresses of the tiles' chunks fold);
// otherwise rows of a.cr < C channels.
template <int PASS, typename T, int C, int MB, bool EX>
static void launch_k(const StreamArgs& a, dim3 grid, int threads, size_t lds, hipStream_t st) {
  if constexpr (PASS == kAggregate)
    hipLaunchKernelGGL((k_aggregate<T, C, MB, false, false, EX>), grid, dim3(threads), lds, st, a);
  else if constexpr (PASS == kAggregateW)
    hipLaunchKernelGGL((k_aggregate<T, C, MB, false, true, EX>), grid, dim3(threads), lds, st, a);
  else if constexpr (PASS == kDesliceBwd)
    hipLaunchKernelGGL((k_aggregate<T, C, MB, true, false, EX>), grid, dim3(threads), lds, st, a);
  else if constexpr (PASS == kDesliceBwdW)
    hipLaunchKernelGGL((k_aggregate<T, C, MB, true, true, EX>), grid, dim3(threads), lds, st, a);
  else if constexpr (PASS == kDeslice)
    hipLaunchKernelGGL((k_deslice<T, C, MB, false, EX>), grid, dim3(threads), lds, st, a);
  else if constexpr (PASS == kDesliceW)
    hipLaunchKernelGGL((k_deslice<T, C, MB, true, EX>), grid, dim3(threads), lds, st, a);
  else if constexpr (PASS == kWeights)
    hipLaunchKernelGGL((k_weights<T, C, MB, EX>), grid, dim3(threads), lds, st, a);
  else
    hipLaunchKernelGGL((k_slice_bwd<T, C, MB, PASS, EX>), grid, dim3(threads), lds, st, a);
}

template <int PASS, typename T, int C, int MB>
static hipError_t launch_t(const StreamArgs& a, int P, hipStream_t st) {
  using G_ = Geo<sizeof(T), C, MB>;
  if constexpr (!G_::fits(PASS)) {
    return hipErrorInvalidConfiguration;
  } else {
    const int threads = 64 * G_::waves(PASS);
    const size_t lds = (size_t)G_::lds_bytes(PASS);
    const dim3 grid(P, a.heads);
    if (a.cr == C)
      launch_k<PASS, T, C, MB, true>(a, grid, threads, lds, st);
    else
      launch_k<PASS, T, C, MB, false>(a, grid, threads, lds, st);
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
hipError_t launch_aggregate_w_pass(int dtype, int C, int MB, const StreamArgs& a, int P, hipStream_t st);
hipError_t launch_deslice_w_pass(int dtype, int C, int MB, const StreamArgs& a, int P, hipStream_t st);
hipError_t launch_deslice_bwd_w_pass(int dtype, int C, int MB, const StreamArgs& a, int P, hipStream_t st);

}  // namespace pa
