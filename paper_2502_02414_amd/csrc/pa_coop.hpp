// kSliceBwd for many slices and wide rows (bf16, C = 256, M > 32): groups
// of four waves work together on one 16-point tile at a time (gfx950).
//
// The per-wave kernel of pa_stream.hpp gives every wave its own tiles and
// the whole chain rule of a point: at C = 256 with up to 64 slices its
// tables (104 KB of LDS) leave room for two such waves per CU, and its dA
// accumulator (C M floats per wave) does not fit in the register file.
// Here the work of a tile is split over a group of four waves, each phase
// split the way its data falls:
//   A. contractions over channels, by slice block: wave w forms the logits
//      and dw of slices 16w .. 16w + 15 for the tile's 16 points (MFMA over
//      x and dY against its rows of the tables), and the temperature's
//      partial sum over channels 64w .. 64w + 63; all of them go to the
//      tile's exchange rows in LDS (one fp32 row per point);
//   B. the softmax over the slices and its backward, by point: wave w takes
//      points 4w .. 4w + 3, one 16-lane row per point with four slices per
//      lane, so every sum over slices is a reduction within a row of lanes
//      (no further exchange between waves); w and dl (bf16) and dt are
//      written back into the point's exchange row;
//   C. by channel block and slice block again: dx of channels
//      64w .. 64w + 63 (MFMA over all slices against [A^T | dnum - cN]),
//      staged and written back; dA of slice block w += x^T dl; da of its
//      channels += x^T dt.
// Two barriers per tile separate the phases (and two more the stores of
// the next tile's rows).  A block holds NG groups (two: one wave of each per
// SIMD) that share the tables and take alternate tiles of the block's
// range.  The barriers are the block's, so the second group runs one barrier
// interval behind the first: while one group is in its MFMA and LDS heavy
// phase A, the other is in its VALU-bound phase B (measured at N = 2.5M,
// M = 64: -4 % against both groups in the same phase).  Every sum is formed
// in a fixed order: the groups' and waves' partial sums are added in group
// and wave order at the end, so the result is deterministic.
#pragma once

#include "pa_stream.hpp"

namespace pa {

template <typename T, int C, int MB, int NG = 1>
struct CoopGeo {
  using G_ = Geo<sizeof(T), C, MB>;
  static constexpr int WAVES = 4 * NG;  // NG groups of four waves
  static constexpr int SZ = (int)sizeof(T);
  static constexpr int M16 = G_::M16;
  static constexpr int IMG = G_::img_bytes(kSliceBwd);
  // Exchange row of a point: logits and dw of every slice (fp32), then the
  // four waves' temperature partial sums; after the softmax the row's first
  // 4 M16 bytes hold w and dl (bf16) and dt sits where dw began.  The row
  // stride (16 bytes over a multiple of 256) keeps the 16-byte writes of 16
  // points and the 8-byte reads of w and dl across 16 points conflict-free.
  static constexpr int EXROW = 2 * M16 * 4 + 16;
  static constexpr int E_DW = M16 * 4;
  static constexpr int E_T = 2 * M16 * 4;
  static constexpr int E_W = 0;
  static constexpr int E_L = M16 * SZ;
  static constexpr int E_DT = E_DW;
  // per tile: x, dY (then the dx staging), Gumbel rows, exchange rows
  static constexpr int OFF_X = 0;
  static constexpr int OFF_Y = OFF_X + G_::XT;
  static constexpr int OFF_G = OFF_Y + G_::XT;
  static constexpr int OFF_E = OFF_G + G_::GT;
  static constexpr int TILE = OFF_E + 16 * EXROW;
  static constexpr int LDS = IMG + NG * TILE;
  // at the end, over the tables and tiles (no longer read): the second
  // group's per-lane partial sums, then every wave's db and db_t totals
  static constexpr int PART = 80;  // floats per lane: dA 64, da 4
  static constexpr int OFF_RED = 4 * 64 * PART * 4;
  static constexpr int RED_BYTES = (WAVES * M16 + WAVES) * 4;
  // a quarter of a tile's rows per wave: 16-byte chunks per lane
  static constexpr int QCH = 4 * C * SZ / 16 / 64;
  static constexpr bool fits = LDS <= kLdsBytes && QCH >= 1 && 4 * C * SZ == QCH * 16 * 64 &&
                               OFF_RED + RED_BYTES <= LDS && C / 32 % 4 == 0;
};

// Two groups of four waves (two waves per SIMD, one of each group: one
// group's compute overlaps the other's waits) when both tiles fit in LDS
// beside the tables.
template <typename T, int C, int MB>
constexpr int coop_groups() {
  return CoopGeo<T, C, MB, 2>::fits ? 2 : 1;
}

// Whether kSliceBwd runs the block-cooperative kernel at this shape.
template <typename T, int C, int MB>
constexpr bool coop_slice_bwd() {
  return sizeof(T) == 2 && C == 256 && MB >= 3 && CoopGeo<T, C, MB, 1>::fits;
}

template <typename T, int C, int MB>
struct CoopStage {
  uint4 x[CoopGeo<T, C, MB>::QCH], y[CoopGeo<T, C, MB>::QCH];
  uint4 g;
};

// Register prefetch (tiles in flight per group): two with one group (one
// wave per SIMD), one with two groups (whose registers then fit two waves
// per SIMD).
template <int NG>
constexpr int coop_depth() {
  return NG == 1 ? 2 : 1;
}

template <typename T, int C, int MB, int NG>
__global__ void __launch_bounds__(256 * NG) __attribute__((amdgpu_waves_per_eu(NG)))
k_slice_bwd_coop(StreamArgs a) {
  using G_ = Geo<sizeof(T), C, MB>;
  using CG = CoopGeo<T, C, MB, NG>;
  using Stage = CoopStage<T, C, MB>;
  constexpr int M16 = G_::M16, SZ = CG::SZ, CB = G_::CB, XF = G_::XF;
  constexpr int RCH = C * SZ / 16;  // 16-byte chunks per row
  constexpr int XQ = XF / 4;        // K32 steps of a wave's temperature partial
  constexpr int DEPTH = coop_depth<NG>();
  constexpr int EXROW = CG::EXROW;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  head_offsets(a);
  add_tb_dev(a);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) & 3;  // in its group
  const int grp = __builtin_amdgcn_readfirstlane(threadIdx.x >> 8);
  const int lane = lane_id(), r = lane & 15, g = lane >> 4;
  const bool hasG = a.flags & kHasG;
  const bool deslice = a.flags & kDesliceTerm;
  const bool own = wave < MB;  // the wave owns slice block `wave`
  const int nb = own ? wave : 0;
  // phase B: lane (r, g) takes point 4 wave + g, slices 4r .. 4r + 3
  // (lanes with 4r >= M16 hold no slice)
  const bool sact = 4 * r < M16;

  const float* hdr = reinterpret_cast<const float*>(smem);
  const float* dden_tab = hdr + M16;
  const float* cN = hdr + 2 * M16;
  const float* af = hdr + 3 * M16 + 2 * C;
  const char* tabL = smem + G_::OFF_L;
  const char* tabW = smem + G_::OFF_2;
  char* const tl = smem + CG::IMG + grp * CG::TILE;  // the group's tile
  char* const ex = tl + CG::OFF_E;

  const auto lb = logits_bases<T, C, MB, true>();
  const RowBase<T> yb = row_base<T>(r, G_::XT_ROW);
  const RowBase<T> wrb = row_base<T>(r, G_::WROW);
  const int xtr = tr_base<T>(G_::XT_ROW);
  const int ltr = tr_base<T>(G_::TROW);
  const int wtr = tr_base<T>(G_::WROW);
  const int etr = tr_base<T>(EXROW);
  const int stb = stage_base<T>(G_::XT_ROW);

  // block set-up: the table image, zeroed Gumbel tiles, the bias and
  // centred dden of the lane's softmax slices
  copy_image<CG::IMG, 256 * NG>(smem, a.img);
  for (int q = threadIdx.x & 255; q < G_::GT / 16; q += 256)
    reinterpret_cast<uint4*>(tl + CG::OFF_G)[q] = uint4{0, 0, 0, 0};
  __syncthreads();  // (before any prefetch: a full fence costs nothing here)
  float bias[4], dden[4];
  {
    float cD = 0.f;
    const float* sw = hdr + 2 * M16 + 2 * C;
    for (int j = 0; j < a.M; ++j) cD += sw[j] * dden_tab[j];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = 4 * r + i;
      bias[i] = sact ? hdr[j] : -INFINITY;  // -inf for the padded slices j >= M
      dden[i] = j < a.M ? dden_tab[j] - cD : 0.f;
    }
  }

  f32x4 dA[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) dA[cb] = zero4();
  float da[4] = {0.f, 0.f, 0.f, 0.f};  // channel blocks 4 wave + k, lane r
  float db[4] = {0.f, 0.f, 0.f, 0.f};  // slices 4r + i, points 4 wave + g
  float dbt = 0.f;                     // lanes r == 0: points 4 wave + g

  const T* X = reinterpret_cast<const T*>(a.x);
  const T* Y = reinterpret_cast<const T*>(a.dY);
  const T* Gp = reinterpret_cast<const T*>(a.G);
  T* DX = reinterpret_cast<T*>(a.out);
  // the block's tiles [t0, t1), group grp taking tiles t0 + NG rd + grp; a
  // round's tile past t1 is the last tile again, with no contribution
  const int64_t T_ = (a.N + 15) / 16;
  const int64_t t0 = T_ * blockIdx.x / gridDim.x, t1 = T_ * (blockIdx.x + 1) / gridDim.x;
  const int64_t nr = (t1 - t0 + NG - 1) / NG;  // rounds
  auto tile_at = [&](int64_t rd) { return t0 + NG * rd + grp; };
  auto tile_of = [&](int64_t rd) {
    const int64_t t = tile_at(rd);
    return t < t1 ? t : t1 - 1;
  };
  const int gchunks = 16 * a.M * SZ / 16;  // the Gumbel rows of a full tile

  // this wave's quarter of a tile's rows (rows 4 wave .. 4 wave + 3; Gumbel
  // chunks wave + 4 lane): every load unconditional, rows past N re-read
  // row N - 1
  auto load = [&](Stage& st, int64_t rd) {
    const int64_t p0 = tile_of(rd) * 16;
    const int lim = last_row<16>(p0, a.N);
    const char* xs = reinterpret_cast<const char*>(X + p0 * C);
    const char* ys = reinterpret_cast<const char*>((deslice ? Y : X) + p0 * C);
#pragma unroll
    for (int k = 0; k < CG::QCH; ++k) {
      const int q = 64 * CG::QCH * wave + lane + 64 * k;
      const int row = q / RCH, cc = q - row * RCH;
      const int rr = row < lim ? row : lim;
      const uint32_t off = (uint32_t)(rr * C * SZ + 16 * cc);
      st.x[k] = ld_global16<true>(xs + off);
      st.y[k] = ld_global16<true>(ys + off);
    }
    const bool full = hasG && p0 + 16 <= a.N;
    const int qg = wave + 4 * lane < gchunks ? wave + 4 * lane : gchunks - 1;
    st.g = ld_global16<true>(full ? reinterpret_cast<const char*>(Gp + p0 * a.M) + 16 * qg
                                  : reinterpret_cast<const char*>(X));
  };
  auto store = [&](const Stage& st, int64_t rd) {
#pragma unroll
    for (int k = 0; k < CG::QCH; ++k) {
      const int q = 64 * CG::QCH * wave + lane + 64 * k;
      const int row = q / RCH, cc = q - row * RCH;
      *reinterpret_cast<uint4*>(tl + CG::OFF_X + lds_off(row, 16 * cc, G_::XT_ROW)) = st.x[k];
      if (deslice)
        *reinterpret_cast<uint4*>(tl + CG::OFF_Y + lds_off(row, 16 * cc, G_::XT_ROW)) = st.y[k];
    }
    const int64_t p0 = tile_of(rd) * 16;
    if (hasG && p0 + 16 <= a.N) {
      // lanes past the last chunk loaded that chunk again and store it
      // again (the same bytes): no lane-dependent branch around the memory
      // instructions, so the compiler's waits stay exact
      const int qg = wave + 4 * lane < gchunks ? wave + 4 * lane : gchunks - 1;
      *reinterpret_cast<uint4*>(tl + CG::OFF_G + 16 * qg) = st.g;
    } else if (hasG && wave == 0) {
      // the tail tile's valid rows, element by element (without noise the
      // tile keeps the zeros of the set-up)
      g_fixup<T, MB>(tl + CG::OFF_G, Gp, p0, a.N, a.M, hasG);
    }
  };

  auto body = [&](int64_t rd) {
    const bool live = tile_at(rd) < t1;  // uniform over the group
    const int64_t p0 = tile_of(rd) * 16;
    const int nvalid = (int)(a.N - p0 < 16 ? a.N - p0 : 16);
    const char* xt = tl + CG::OFF_X;

    // A. logits and dw of slices 16 nb + 4g + i (point r), the temperature's
    // partial sum over channel steps [XQ wave, XQ wave + XQ)
    f32x4 lacc = zero4(), wacc = zero4(), tacc = zero4();
    if (own) {
      // x . A (logits) and x . (dnum - cN) (dw) share the x fragments
      struct FL { K32<T> t, tw, ta, x; };
      pipelined<XF, 2, FL>(
          [&](int s, FL& f) {
            ld_row<T>(f.t, tabL, lb.t, 16 * nb * G_::TROW + 32 * s * SZ);
            ld_row<T>(f.tw, tabW, wrb, 16 * nb * G_::WROW + 32 * s * SZ);
            ld_row<T>(f.x, xt, lb.x, 32 * s * SZ);
            if (s / XQ == wave) ld_row<T>(f.ta, tabL, lb.a, M16 * G_::TROW + 32 * s * SZ);
          },
          [&](int s, FL& f) {
            lacc = mma32(f.t, f.x, lacc);
            wacc = mma32(f.tw, f.x, wacc);
            if (s / XQ == wave) tacc = mma32(f.ta, f.x, tacc);
          });
      if (deslice) {
        struct FD { K32<T> tw, y; };
        pipelined<XF, 2, FD>(
            [&](int s, FD& f) {
              ld_row<T>(f.tw, tabW, wrb, 16 * nb * G_::WROW + (C + 32 * s) * SZ);
              ld_row<T>(f.y, tl + CG::OFF_Y, yb, 32 * s * SZ);
            },
            [&](int s, FD& f) { wacc = mma32(f.tw, f.y, wacc); });
      }
      char* er = ex + r * EXROW + (16 * nb + 4 * g) * 4;
      *reinterpret_cast<f32x4*>(er) = lacc;
      *reinterpret_cast<f32x4*>(er + CG::E_DW) = wacc;
    } else {
#pragma unroll
      for (int s2 = 0; s2 < XQ; ++s2) {
        const int s = XQ * wave + s2;
        K32<T> ta, x;
        ld_row<T>(ta, tabL, lb.a, M16 * G_::TROW + 32 * s * SZ);
        ld_row<T>(x, xt, lb.x, 32 * s * SZ);
        tacc = mma32(ta, x, tacc);
      }
    }
    if (g == 0) *reinterpret_cast<float*>(ex + r * EXROW + CG::E_T + 4 * wave) = tacc[0];
    block_sync();

    // B. softmax and its backward of point pt = 4 wave + g over its row of
    // 16 lanes (slices 4r + i)
    {
      const int pt = 4 * wave + g;
      char* er = ex + pt * EXROW;
      const int qo = sact ? 16 * r : 0;
      const f32x4 lg = *reinterpret_cast<const f32x4*>(er + qo);
      const f32x4 dwv = *reinterpret_cast<const f32x4*>(er + CG::E_DW + qo);
      const f32x4 tp = *reinterpret_cast<const f32x4*>(er + CG::E_T);
      const char* gt = tl + CG::OFF_G;
      const int e = pt * a.M + (sact ? 4 * r : 0);  // element of the G tile
      float gv[4];
      if (a.M % 4 == 0) {
        const bf16x4 q4 = *reinterpret_cast<const bf16x4*>(gt + e * SZ);
#pragma unroll
        for (int i = 0; i < 4; ++i) gv[i] = (float)q4[i];
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) gv[i] = to_f<T>(reinterpret_cast<const T*>(gt)[e + i]);
      }
      const float tt = ((tp[0] + tp[1]) + (tp[2] + tp[3])) + (float)a.tb;
      const float tau = fmaxf(tt, a.tau_min);
      const float k2 = kLog2e * fast_rcp(tau);
      float u[4], m = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        u[i] = lg[i] + bias[i] + gv[i];
        m = fmaxf(m, u[i]);
      }
      m = row16_max(m);
      const float mk = m * k2;
      float zs[4], e4[4], ssum = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        zs[i] = fmaf(u[i], k2, -mk);
        e4[i] = fast_exp2(zs[i]);
        ssum += e4[i];
      }
      ssum = row16_sum(ssum);
      const bool pv = live && pt < nvalid;
      const float sc = pv ? fast_rcp(ssum) : 0.f;
      float w[4], dw[4], p1 = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        w[i] = e4[i] * sc;
        dw[i] = dwv[i] + dden[i];
        p1 += w[i] * dw[i];
      }
      // softmax backward: <w, dw>, compensated by the residual pass; the
      // temperature's <dz, zs> = <w (dw - wdw), zs> - res <w, zs> (the shift
      // of zs common to all slices drops out, as sum_j dz_j = 0)
      const float wdw = row16_sum(p1);
      float res = 0.f, q1 = 0.f, q2 = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float d = w[i] * (dw[i] - wdw);
        res += d;
        // a padded slice: exponent -inf, w = d = 0; the exponent clamped to
        // a finite value keeps the products 0
        const float zc = __builtin_amdgcn_fmed3f(zs[i], -__FLT_MAX__, __FLT_MAX__);
        q1 = fmaf(d, zc, q1);
        q2 = fmaf(w[i], zc, q2);
      }
      res = row16_sum(res);
      q1 = row16_sum(q1);
      q2 = row16_sum(q2);
      const float rtau = fast_rcp(tau);
      const float dtau = -kLn2 * (q1 - res * q2) * rtau;
      const float dt = (pv && tt > a.tau_min) ? dtau : 0.f;
      bf16x4 wq, lq;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float dl = w[i] * ((dw[i] - wdw) - res) * rtau;
        wq[i] = (bf16)w[i];
        lq[i] = (bf16)dl;
        db[i] += dl;
      }
      // the row's logits and dw are read (by this wave only): w, dl and dt
      // take their place
      if (sact) {
        *reinterpret_cast<bf16x4*>(er + CG::E_W + 8 * r) = wq;
        *reinterpret_cast<bf16x4*>(er + CG::E_L + 8 * r) = lq;
      }
      if (r == 0) {
        *reinterpret_cast<float*>(er + CG::E_DT) = dt;
        dbt += dt;
      }
    }
    block_sync();

    // C. dx of the wave's channel blocks: [A^T | dnum - cN] x [dl ; w] + a dt + cN
    const float dtr = *reinterpret_cast<const float*>(ex + r * EXROW + CG::E_DT);
    K16<T> wb[MB], lbk[MB];
#pragma unroll
    for (int q = 0; q < MB; ++q) {
      ld_k16(wb[q], ex + r * EXROW + CG::E_W + (16 * q + 4 * g) * SZ);
      ld_k16(lbk[q], ex + r * EXROW + CG::E_L + (16 * q + 4 * g) * SZ);
    }
    struct FX { K16<T> ta[MB], tn[MB]; f32x4 av, cn; };
    pipelined<4, 2, FX>(
        [&](int k, FX& f) {
          const int cb = 4 * wave + k;
#pragma unroll
          for (int q = 0; q < MB; ++q) {
            ld_tr<T>(f.ta[q], tabL, ltr, 16 * q * G_::TROW + 16 * cb * SZ, G_::TROW);
            ld_tr<T>(f.tn[q], tabW, wtr, 16 * q * G_::WROW + 16 * cb * SZ, G_::WROW);
          }
          f.av = *reinterpret_cast<const f32x4*>(af + 16 * cb + 4 * g);
          f.cn = *reinterpret_cast<const f32x4*>(cN + 16 * cb + 4 * g);
        },
        [&](int k, FX& f) {
          f32x4 d = zero4();
#pragma unroll
          for (int q = 0; q < MB; ++q) d = mma16x2(f.ta[q], lbk[q], f.tn[q], wb[q], d);
#pragma unroll
          for (int i = 0; i < 4; ++i) d[i] += f.av[i] * dtr + f.cn[i];
          stage4<T>(tl + CG::OFF_Y, stb, 16 * (4 * wave + k) * SZ, d);
        });
    wave_sync();
    if (live) {  // uniform over the group
      // the wave's 64 channels of the tile's rows: 8 chunks per row (rows
      // past the tile's last point write that point's chunk again: the same
      // bytes, and every lane stores unconditionally)
      char* dst = reinterpret_cast<char*>(DX + p0 * C);
      const char* yt = tl + CG::OFF_Y;
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int q = lane + 64 * k;  // < 128
        const int row = (q >> 3) < nvalid ? (q >> 3) : nvalid - 1;
        const int cc = 8 * wave + (q & 7);
        const uint4 v = *reinterpret_cast<const uint4*>(yt + lds_off(row, 16 * cc, G_::XT_ROW));
        st_global16(dst + (uint32_t)(row * C * SZ + 16 * cc), v);
      }
    }

    // da (the wave's channel blocks) += x^T dt, dA (its slices) += x^T dl
    {
      float dtp[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        dtp[i] = *reinterpret_cast<const float*>(ex + (4 * g + i) * EXROW + CG::E_DT);
      const bf16x2 dt01{(bf16)dtp[0], (bf16)dtp[1]}, dt23{(bf16)dtp[2], (bf16)dtp[3]};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        K16<T> xa;
        ld_tr<T>(xa, xt, xtr, 16 * (4 * wave + k) * SZ, G_::XT_ROW);
        da[k] = __builtin_amdgcn_fdot2_f32_bf16(
            bf16x2{xa.v[2], xa.v[3]}, dt23,
            __builtin_amdgcn_fdot2_f32_bf16(bf16x2{xa.v[0], xa.v[1]}, dt01, da[k], false), false);
      }
    }
    if (own) {
      K16<T> lp;
      ld_tr<T>(lp, ex + CG::E_L, etr, 16 * nb * SZ, EXROW);
      struct FA { K16<T> xa; };
      pipelined<CB, 4, FA>(
          [&](int cb, FA& f) { ld_tr<T>(f.xa, xt, xtr, 16 * cb * SZ, G_::XT_ROW); },
          [&](int cb, FA& f) { dA[cb] = mma16(f.xa, lp, dA[cb]); });
    }
  };

  // the block's rounds, DEPTH of them in flight in registers; the shared
  // tiles are rewritten only after every wave is done with the previous
  // round.  The main loop runs whole groups of DEPTH rounds with every stage
  // reloaded on every round (past the end with the last round again, L2
  // hits), so that every path into the loop head has issued the same memory
  // instructions in the same order and the compiler's waits cover exactly
  // the stage being stored; the last (fewer than DEPTH) rounds, already
  // loaded, follow.
  Stage st[DEPTH];
  if (nr > 0) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) load(st[d], d < nr ? d : nr - 1);
  }
  // the second group runs one barrier interval behind the first (one extra
  // barrier before its first round; the first group takes one after its
  // last, so both pass the same number)
  if (NG == 2 && grp == 1) block_sync();
  int64_t rd = 0;
  for (; rd + DEPTH <= nr; rd += DEPTH) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      block_sync();
      store(st[d], rd + d);
      const int64_t nx = rd + d + DEPTH;
      load(st[d], nx < nr ? nx : nr - 1);
      block_sync();
      body(rd + d);
    }
  }
#pragma unroll
  for (int d = 0; d < DEPTH - 1; ++d) {
    if (rd + d < nr) {  // uniform over the block (every group runs nr rounds)
      block_sync();
      store(st[d], rd + d);
      block_sync();
      body(rd + d);
    }
  }

  if (NG == 2 && grp == 0) block_sync();
  // lane partials -> wave totals of db (over the wave's four points) and
  // db_t; then, over the tables and tiles (no longer read), every wave's
  // totals and the second group's per-lane dA and da partials, added to the
  // first's in group and wave order
#pragma unroll
  for (int i = 0; i < 4; ++i) db[i] = groups_sum(db[i]);
  dbt = groups_sum(dbt);
  float* red = reinterpret_cast<float*>(smem + CG::OFF_RED);  // [WAVES][M16], then [WAVES]
  const int gw = 4 * grp + wave;
  block_sync();
  if (g == 0 && sact)
    *reinterpret_cast<f32x4*>(red + gw * M16 + 4 * r) = f32x4{db[0], db[1], db[2], db[3]};
  if (lane == 0) red[CG::WAVES * M16 + gw] = dbt;
  if constexpr (NG == 2) {
    static_assert(CG::OFF_RED >= 4 * 64 * CG::PART * 4, "group partials must fit below the totals");
    float* part = reinterpret_cast<float*>(smem) + (wave * 64 + lane) * CG::PART;
    if (grp == 1) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) *reinterpret_cast<f32x4*>(part + 4 * cb) = dA[cb];
#pragma unroll
      for (int i = 0; i < 4; ++i) part[4 * CB + i] = da[i];
    }
    block_sync();
    if (grp == 1) return;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) dA[cb] += *reinterpret_cast<const f32x4*>(part + 4 * cb);
#pragma unroll
    for (int i = 0; i < 4; ++i) da[i] += part[4 * CB + i];
  } else {
    block_sync();
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) da[k] = groups_sum(da[k]);
  // the block's record: dA [C][M], db [M], da [C], db_t, each part written
  // by the wave that owns it
  float* rec = a.partials + (int64_t)blockIdx.x * a.rec;
  const int M = a.M;
  if (own) {
    const int j = 16 * nb + r;
    if (j < M) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int i = 0; i < 4; ++i) rec[(16 * cb + 4 * g + i) * M + j] = dA[cb][i];
    }
  }
  if (g == 0) {
#pragma unroll
    for (int k = 0; k < 4; ++k) rec[C * M + M + 16 * (4 * wave + k) + r] = da[k];
  }
  if (wave == 0) {
    for (int j = lane; j < M; j += 64) {
      float s = 0.f;
      for (int v = 0; v < CG::WAVES; ++v) s += red[v * M16 + j];
      rec[C * M + j] = s;
    }
    if (lane == 0) {
      float s = 0.f;
      for (int v = 0; v < CG::WAVES; ++v) s += red[CG::WAVES * M16 + v];
      rec[C * M + M + C] = s;
    }
  }
}

}  // namespace pa
