// Device building blocks for the gfx950 (CDNA4) Physics-Attention kernels.
//
// Wave64 MFMA conventions used throughout (16x16 output tiles):
//   lane l = r + 16 g  (r = l % 16, g = l / 16)
//   A operand: lane holds row r, a run of K elements indexed by g
//   B operand: lane holds column r, the same run of K elements
//   D (f32x4): lane holds D[4 g + i][r], i = 0..3
// "K32" fragments hold 8 elements per lane (one v_mfma_f32_16x16x32_bf16, or
// eight v_mfma_f32_16x16x4_f32 steps); "K16" fragments hold 4 elements per
// lane (one v_mfma_f32_16x16x16_bf16, or four 16x16x4 f32 steps).  Only the
// pairing of A and B elements matters for a contraction, and it is the same
// (lane group, element) on both sides, so the order in which the hardware
// walks K inside a fragment never enters the result beyond fp32 rounding.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pa {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef double f64x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// Byte offset of (row, byte column) in an LDS array whose rows are padded by
// 32 bytes (row stride RB): consecutive rows start 32 bytes apart modulo the
// bank width, which makes the 16-byte row reads of 16 rows and the
// transposed 8-byte reads of 4 rows x 32 bytes conflict-free (measured on
// gfx950; an XOR swizzle of the 16-byte chunks does worse for the row reads).
__device__ __forceinline__ int lds_off(int row, int bcol, int RB) { return row * RB + bcol; }

// ---------------------------------------------------------------------------
// Scalar conversions
// ---------------------------------------------------------------------------
template <typename T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<bf16>(bf16 v) { return (float)v; }

template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float v) { return (bf16)v; }  // RNE

// Value as the MFMA will see it (bf16 rounding for bf16 operands).
template <typename T> __device__ __forceinline__ float as_operand(float v) {
  return to_f<T>(from_f<T>(v));
}

// ---------------------------------------------------------------------------
// MFMA fragments
// ---------------------------------------------------------------------------
template <typename T> struct K32;
template <> struct K32<bf16> { bf16x8 v; };
template <> struct K32<float> { f32x4 lo, hi; };

template <typename T> struct K16;
template <> struct K16<bf16> { bf16x4 v; };
template <> struct K16<float> { f32x4 v; };

// 8 consecutive elements from LDS (16 B for bf16, 32 B for fp32).
__device__ __forceinline__ void ld_k32(K32<bf16>& f, const char* p) {
  f.v = *reinterpret_cast<const bf16x8*>(p);
}
__device__ __forceinline__ void ld_k32(K32<float>& f, const char* p) {
  f.lo = *reinterpret_cast<const f32x4*>(p);
  f.hi = *reinterpret_cast<const f32x4*>(p + 16);
}
// 4 consecutive elements from LDS (8 B for bf16, 16 B for fp32).
__device__ __forceinline__ void ld_k16(K16<bf16>& f, const char* p) {
  f.v = *reinterpret_cast<const bf16x4*>(p);
}
__device__ __forceinline__ void ld_k16(K16<float>& f, const char* p) {
  f.v = *reinterpret_cast<const f32x4*>(p);
}

__device__ __forceinline__ f32x4 mma32(const K32<bf16>& a, const K32<bf16>& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma32(const K32<float>& a, const K32<float>& b, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo[0], b.lo[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo[1], b.lo[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo[2], b.lo[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo[3], b.lo[3], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi[0], b.hi[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi[1], b.hi[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi[2], b.hi[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi[3], b.hi[3], c, 0, 0, 0);
  return c;
}
__device__ __forceinline__ f32x4 mma16(const K16<bf16>& a, const K16<bf16>& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a.v, b.v, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma16(const K16<float>& a, const K16<float>& b, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[0], b.v[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[1], b.v[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[2], b.v[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[3], b.v[3], c, 0, 0, 0);
  return c;
}

// Two K16 products as one: the concatenated fragments pair the same
// elements (lane group g: a0 with b0, a1 with b1), so one K32 MFMA gives the
// sum of both products (bf16); fp32 runs the two products.
__device__ __forceinline__ f32x4 mma16x2(const K16<bf16>& a0, const K16<bf16>& b0,
                                         const K16<bf16>& a1, const K16<bf16>& b1, f32x4 c) {
  const bf16x8 a = __builtin_shufflevector(a0.v, a1.v, 0, 1, 2, 3, 4, 5, 6, 7);
  const bf16x8 b = __builtin_shufflevector(b0.v, b1.v, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma16x2(const K16<float>& a0, const K16<float>& b0,
                                         const K16<float>& a1, const K16<float>& b1, f32x4 c) {
  return mma16(a1, b1, mma16(a0, b0, c));
}

// K16 fragment from four floats (rounded to the operand type).
__device__ __forceinline__ void set_k16(K16<bf16>& f, float a, float b, float c, float d) {
  f.v[0] = (bf16)a; f.v[1] = (bf16)b; f.v[2] = (bf16)c; f.v[3] = (bf16)d;
}
__device__ __forceinline__ void set_k16(K16<float>& f, float a, float b, float c, float d) {
  f.v[0] = a; f.v[1] = b; f.v[2] = c; f.v[3] = d;
}
__device__ __forceinline__ float k16_elem(const K16<bf16>& f, int i) { return (float)f.v[i]; }
__device__ __forceinline__ float k16_elem(const K16<float>& f, int i) { return f.v[i]; }

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// Accumulator of a contraction over channels (logits, dw).  fp32 for bf16
// storage.  For fp32 storage the SP-layout passes (deslice, backward) use
// v_mfma_f64_16x16x4_f64 (exact products, fp64 sums): the temperature
// amplifies logit errors by up to 1/tau_min there, and the backward needs
// the logits and dw to better than fp32 accumulation.
template <typename T, bool SP> struct LAcc { typedef f32x4 v; typedef float s; };
template <> struct LAcc<float, true> { typedef f64x4 v; typedef double s; };

template <typename V> __device__ __forceinline__ V zero_acc();
template <> __device__ __forceinline__ f32x4 zero_acc<f32x4>() { return zero4(); }
template <> __device__ __forceinline__ f64x4 zero_acc<f64x4>() { return f64x4{0.0, 0.0, 0.0, 0.0}; }

template <typename T>
__device__ __forceinline__ f32x4 mma_acc(const K32<T>& a, const K32<T>& b, f32x4 c) {
  return mma32(a, b, c);
}
__device__ __forceinline__ f64x4 mma_acc(const K32<float>& a, const K32<float>& b, f64x4 c) {
#pragma unroll
  for (int e = 0; e < 4; ++e)
    c = __builtin_amdgcn_mfma_f64_16x16x4f64((double)a.lo[e], (double)b.lo[e], c, 0, 0, 0);
#pragma unroll
  for (int e = 0; e < 4; ++e)
    c = __builtin_amdgcn_mfma_f64_16x16x4f64((double)a.hi[e], (double)b.hi[e], c, 0, 0, 0);
  return c;
}

// The fp64 MFMA places D row 4i+g (not 4g+i) in element i of lane group g.
// An A operand whose lane r supplies row sigma(r) = 4 (r % 4) + r / 4 makes
// element i of group g hold row 4g+i again, the layout used everywhere else.
template <typename V> __device__ __forceinline__ int a_row(int r) { return r; }
template <> __device__ __forceinline__ int a_row<f64x4>(int r) { return 4 * (r & 3) + (r >> 2); }

// ---------------------------------------------------------------------------
// Cross-lane reductions
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
// DPP controls: quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror,
// row_mirror.  Each step pairs lanes whose partial results cover disjoint
// lane sets, so after four steps every lane of a 16-lane row holds the
// reduction of the whole row (bitwise equal on all 16 lanes).
constexpr int kQuadSwap1 = 0xB1, kQuadSwap2 = 0x4E, kHalfMirror = 0x141, kMirror = 0x140;

__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp<kQuadSwap1>(v));
  v = fmaxf(v, dpp<kQuadSwap2>(v));
  v = fmaxf(v, dpp<kHalfMirror>(v));
  v = fmaxf(v, dpp<kMirror>(v));
  return v;
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp<kQuadSwap1>(v);
  v += dpp<kQuadSwap2>(v);
  v += dpp<kHalfMirror>(v);
  v += dpp<kMirror>(v);
  return v;
}
// Reduction over the four lane groups (lanes l, l^16, l^32, l^48) with the
// gfx950 lane-swap instructions (VALU, no LDS round trip).  With both
// operands equal to v, v_permlane16_swap leaves in each lane the values of
// rows (2k, 2k+1) as the two operands (lower row first), and
// v_permlane32_swap does the same for the two halves, so every lane forms
// (v0 + v1) + (v2 + v3) in the same order: the result is bitwise equal on
// the four lanes.  s_nop 1 covers the VALU-write to lane-swap-read hazard.
__device__ __forceinline__ void lane_swap16(float& a, float& b) {
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ void lane_swap32(float& a, float& b) {
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ float groups_max(float v) {
  float a = v, b = v;
  lane_swap16(a, b);
  float c = fmaxf(a, b), d = c;
  lane_swap32(c, d);
  return fmaxf(c, d);
}
__device__ __forceinline__ float groups_sum(float v) {
  float a = v, b = v;
  lane_swap16(a, b);
  float c = a + b, d = c;
  lane_swap32(c, d);
  return c + d;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

}  // namespace pa
