// Compile-time geometry shared by the host launchers and the gfx950 kernels:
// the byte layout of the per-block LDS "table image" (built once per call by
// the prep kernel into the workspace, then copied by every block into LDS),
// the per-wave LDS regions, and the partial-sum record sizes.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace pa {

// The stored-weights passes follow Algorithm 1's dataflow, where the weights
// are computed once and the deslice reuses them: kAggregateW is kAggregate
// that also writes W [N,M] (storage dtype); kDesliceW and kDesliceBwdW read
// that W in place of recomputing it from x and G.
enum Pass { kAggregate = 0, kDeslice = 1, kDesliceBwd = 2, kWeights = 3, kSliceBwd = 4,
            kWeightsBwd = 5, kAggregateW = 6, kDesliceW = 7, kDesliceBwdW = 8 };
constexpr int kNumPasses = 9;
constexpr bool agg_fwd(int pass) { return pass == kAggregate || pass == kAggregateW; }
constexpr bool agg_bwd(int pass) { return pass == kDesliceBwd || pass == kDesliceBwdW; }

constexpr int kLdsBytes = 160 * 1024;  // LDS per CU on gfx950
constexpr int kPartialsMax = 256;      // blocks (point chunks) per streaming pass

// LDS rows of the tables and point tiles are padded by 32 bytes (lds_off()
// in pa_device.hpp): row reads of 16 bytes per lane (MFMA operands) over 16
// rows and the transposed reads of 8 bytes per lane (ds_read_b64_tr_b16)
// then hit distinct banks.
template <int SZ, int C, int MB>
struct Geo {
  static constexpr int M16 = 16 * MB;            // slices padded to 16
  static constexpr int XF = C / 32;              // K32 fragments per point row
  static constexpr int CB = C / 16;              // 16-channel blocks
  // table image (bytes); every region starts on a 16-byte boundary
  static constexpr int TROW = C * SZ + 32;       // logits table row: A[:,j] or a
  static constexpr int SROW = M16 * SZ + 16;     // deslice table row: s'[:,c]
  static constexpr int WROW = 2 * C * SZ + 32;   // dw table row: (dnum_j | s'_j)
  // header (fp32): bias[M16], dden[M16], cN[C], cS[C], sw[M16], a[C]: cN and
  // cS are the den-weighted means over slices of dnum_j and s'_j that the
  // backward table rows are centred by; sw_j = den_j / sum den are those
  // weights; a is the temperature projection in fp32
  static constexpr int HDR = (3 * M16 + 3 * C) * 4;
  static constexpr int OFF_L = HDR;
  static constexpr int SZ_L = (M16 + 1) * TROW;  // rows: A[:, j] (j < M16), then a
  static constexpr int OFF_2 = OFF_L + SZ_L;     // second table (S or W)
  static constexpr int SZ_S = C * SROW;
  static constexpr int SZ_W = M16 * WROW;
  // per-wave regions: point tiles (x, dY), the Gumbel rows, backward scratch
  static constexpr int XT_ROW = C * SZ + 32;
  static constexpr int XT = 16 * XT_ROW;
  static constexpr int GROW = M16 * SZ + 16;     // Gumbel tile row (M used)
  static constexpr int GT = 16 * GROW;
  static constexpr int SCR = 16 * (M16 + 1) * 4 + 64;  // dl transpose + dt

  // points per streamed tile: the forward aggregate with bf16 storage and up
  // to 32 slices takes two 16-point halves at once (more independent work
  // per wave; its contraction over points pairs into K32 MFMAs); the
  // backward aggregate, with two streamed tensors, measured faster with
  // 16-point tiles (fewer loads in flight per wave)
  static constexpr int rows(int pass) {
    return agg_fwd(pass) && SZ == 2 && MB <= 2 ? 32 : 16;
  }
  // LDS image of a pass: the stored-weights deslice holds only the deslice
  // table (at offset 0), its backward no table at all
  static constexpr int img_bytes(int pass) {
    return pass == kDeslice ? OFF_2 + SZ_S
         : pass == kDesliceW ? SZ_S
         : pass == kDesliceBwdW ? 0
         : (pass == kSliceBwd || pass == kWeightsBwd) ? OFF_2 + SZ_W
         : OFF_2;
  }
  // per wave: x tile, (dY tile or output staging), Gumbel rows, scratch
  // (the aggregating passes: the transposed weights); 32-row tiles hold x,
  // Gumbel and weight rows for 32 points
  static constexpr int wave_bytes(int pass) {
    return (pass == kSliceBwd || pass == kWeightsBwd) ? 2 * XT + GT + SCR
         : agg_fwd(pass) && rows(pass) == 32 ? 2 * XT + 4 * GT
         : agg_bwd(pass) ? 2 * XT + 2 * GT
         : agg_fwd(pass) ? XT + 2 * GT
         : XT + GT;
  }
  // f32x4 per lane of a wave's partial sums (the cross-wave reduction)
  static constexpr int red_vecs(int pass) {
    return agg_fwd(pass) ? MB * CB + MB
         : agg_bwd(pass) ? MB * CB
         : (pass == kSliceBwd || pass == kWeightsBwd) ? CB * MB + (CB + 3) / 4 + (MB + 4) / 4
         : 0;
  }
  // LDS of the cross-wave reduction: waves/2 slots of red_vecs x 64 lanes
  static constexpr int red_bytes(int pass, int waves) {
    return (waves / 2 > 0 ? waves / 2 : 1) * red_vecs(pass) * 64 * 16;
  }
  // the light passes run 8 waves per block with bf16 storage (two waves per
  // SIMD hide each other's latency); the accumulating passes, and fp32
  // storage (whose tiles take twice the registers), run 4; rows of 64 bytes
  // (a head's block of 32 bf16 channels) run 8 in every pass: their tiles
  // are small in registers and in bytes, so more waves keep more loads in
  // flight (measured at 8 heads x 1M points: the per-head step -24 %; 16
  // waves spill the backward's registers)
  static constexpr int max_waves(int pass) {
    return C * SZ <= 64 ? 8
         : (pass == kDeslice || pass == kDesliceW || pass == kWeights) && SZ == 2 ? 8 : 4;
  }
  static constexpr int waves(int pass) {
    return (max_waves(pass) >= 8 && img_bytes(pass) + 8 * wave_bytes(pass) <= kLdsBytes) ? 8
         : (img_bytes(pass) + 4 * wave_bytes(pass) <= kLdsBytes) ? 4
         : (img_bytes(pass) + 2 * wave_bytes(pass) <= kLdsBytes) ? 2 : 1;
  }
  static constexpr int lds_bytes(int pass) {
    return (img_bytes(pass) + waves(pass) * wave_bytes(pass)) > red_bytes(pass, waves(pass))
               ? img_bytes(pass) + waves(pass) * wave_bytes(pass)
               : red_bytes(pass, waves(pass));
  }
  static constexpr bool fits(int pass) {
    return img_bytes(pass) + wave_bytes(pass) <= kLdsBytes &&
           red_bytes(pass, waves(pass)) <= kLdsBytes;
  }
};

// Number of point chunks (blocks) of a streaming pass: a function of N only,
// so every reduction sums the same partials in the same order everywhere.
inline int num_chunks(int64_t N, int waves) {
  int64_t tiles = (N + 15) / 16;
  int64_t p = (tiles + waves - 1) / waves;
  return (int)(p < kPartialsMax ? (p > 0 ? p : 1) : kPartialsMax);
}

// Floats in the record a pass writes per block (valid slices only).
inline int64_t record_floats(int pass, int C, int M) {
  switch (pass) {
    case kAggregate:
    case kAggregateW: return (int64_t)M * C + M;
    case kDesliceBwd:
    case kDesliceBwdW: return (int64_t)M * C;
    case kSliceBwd:
    case kWeightsBwd: return (int64_t)C * M + M + C + 1;
    default: return 0;
  }
}

}  // namespace pa
