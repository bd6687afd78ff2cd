// kSliceBwd for many slices and wide rows (bf16, C = 256, M > 32): groups
// of four waves work together on one 16-point tile at a time (gfx950).
//
// The per-wave kernel of pa_stream.hpp gives every wave its own tiles and
// the whole chain rule of a point: at C = 256 with up to 64 slices its
// tables (104 KB of LDS) leave room for two such waves per CU, and its dA
// accumulator (C M floats per wave) does not fit in the register file.
// Here the work of a tile is split over a group of four waves: wave w owns
// slice block w (slices 16w .. 16w + 15) for the logits, the softmax, dw
// and the dA accumulator (C x 16 floats), and channel blocks 4w .. 4w + 3
// for dx and da.  A block holds NG groups (two: one wave of each per SIMD)
// that share the tables and each take their own tiles (TT per round).  Per
// round, in each group:
//   1. the tiles' x, dY and Gumbel rows (each wave loads a quarter, a round
//      or more ahead in registers) are stored into the group's tiles;
//   2. logits of the wave's slices and the temperature (MFMA over C); a
//      softmax over all slices from per-wave partial (max, sum) pairs
//      exchanged in LDS;
//   3. dw of the wave's slices (MFMA over [x | dY] against the backward
//      table), then <w, dw>, its compensation and the temperature terms
//      from exchanged per-wave partial sums;
//   4. w and dl of every slice published in LDS; dx of the wave's channel
//      blocks (MFMA over [dl | w] against [A^T | dnum - cN]) staged and
//      written back;
//   5. dA (its slice block) += x^T dl and da (its channel blocks) += x^T dt.
// Every cross-wave sum is formed in the same fixed order in every wave, and
// the groups' partial sums are added in group order at the end, so the
// result is deterministic; each block's record is written by the waves of
// the first group that own its parts.
#pragma once

#include "pa_stream.hpp"

namespace pa {

template <typename T, int C, int MB, int TT, int NG = 1>
struct CoopGeo {
  using G_ = Geo<sizeof(T), C, MB>;
  static constexpr int WAVES = 4 * NG;  // NG groups of four waves
  static constexpr int SZ = (int)sizeof(T);
  static constexpr int IMG = G_::img_bytes(kSliceBwd);
  static constexpr int SROW = G_::M16 * SZ + 16;  // published w / dl rows (per point)
  // per tile: x, dY (then the dx staging), Gumbel rows, published w and dl
  static constexpr int OFF_X = 0;
  static constexpr int OFF_Y = OFF_X + G_::XT;
  static constexpr int OFF_G = OFF_Y + G_::XT;
  static constexpr int OFF_W = OFF_G + G_::GT;
  static constexpr int OFF_L = OFF_W + 16 * SROW;
  static constexpr int TILE = OFF_L + 16 * SROW;
  // per tile and wave: (max, sum), <w, dw>, (res, P1, P2, -) for 16 points
  static constexpr int OFF_EX = IMG + NG * TT * TILE;
  static constexpr int EX = 4 * 16 * (8 + 4 + 16);
  static constexpr int LDS = OFF_EX + NG * TT * EX;
  // the second group's per-lane partial sums at the end (over the tables
  // and tiles, no longer read then)
  static constexpr int PART = 80;  // floats per lane: dA 64, db 4, da 4, db_t 1
  // a quarter of a tile's rows per wave: 16-byte chunks per lane
  static constexpr int QCH = 4 * C * SZ / 16 / 64;
  static constexpr bool fits = LDS <= kLdsBytes && QCH >= 1 && 4 * C * SZ == QCH * 16 * 64;
};

// Tiles per round and groups: two groups of four waves, each on its own
// tile (two waves per SIMD, one per group: one group's compute overlaps the
// other's waits), when both tiles fit in LDS beside the tables.
template <typename T, int C, int MB>
constexpr int coop_groups() {
  return CoopGeo<T, C, MB, 1, 2>::fits ? 2 : 1;
}
template <typename T, int C, int MB>
constexpr int coop_tiles() {
  return 1;
}

// Whether kSliceBwd runs the block-cooperative kernel at this shape.
template <typename T, int C, int MB>
constexpr bool coop_slice_bwd() {
  return sizeof(T) == 2 && C == 256 && MB >= 3 && CoopGeo<T, C, MB, 1>::fits;
}

template <typename T, int C, int MB, int TT>
struct CoopStage {
  uint4 x[TT][CoopGeo<T, C, MB, TT>::QCH], y[TT][CoopGeo<T, C, MB, TT>::QCH];
  uint4 g[TT];
};

// Register prefetch (rounds in flight) of the cooperative kernel: two with
// one group (one wave per SIMD), one with two groups (whose registers then
// fit two waves per SIMD).
template <int NG>
constexpr int coop_depth() {
  return NG == 1 ? 2 : 1;
}

template <typename T, int C, int MB, int TT, int NG>
__global__ void __launch_bounds__(256 * NG) __attribute__((amdgpu_waves_per_eu(NG)))
k_slice_bwd_coop(StreamArgs a) {
  using G_ = Geo<sizeof(T), C, MB>;
  using CG = CoopGeo<T, C, MB, TT, NG>;
  using Stage = CoopStage<T, C, MB, TT>;
  constexpr int M16 = G_::M16, SZ = CG::SZ, CB = G_::CB, XF = G_::XF;
  constexpr int RCH = C * SZ / 16;  // 16-byte chunks per row
  constexpr int DEPTH = coop_depth<NG>();
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

  const float* hdr = reinterpret_cast<const float*>(smem);
  const float* dden_tab = hdr + M16;
  const float* cN = hdr + 2 * M16;
  const float* af = hdr + 3 * M16 + 2 * C;
  const char* tabL = smem + G_::OFF_L;
  const char* tabW = smem + G_::OFF_2;
  // the group's tiles and exchange slots
  auto tile_lds = [&](int tt) { return smem + CG::IMG + (grp * TT + tt) * CG::TILE; };
  auto ex_at = [&](int tt) { return smem + CG::OFF_EX + (grp * TT + tt) * CG::EX; };
  auto ex_ms = [&](int tt) { return reinterpret_cast<float2*>(ex_at(tt)); };
  auto ex_s1 = [&](int tt) { return reinterpret_cast<float*>(ex_at(tt) + 4 * 16 * 8); };
  auto ex_s3 = [&](int tt) { return reinterpret_cast<f32x4*>(ex_at(tt) + 4 * 16 * 12); };

  const auto lb = logits_bases<T, C, MB, true>();
  const RowBase<T> yb = row_base<T>(r, G_::XT_ROW);
  const RowBase<T> wrb = row_base<T>(r, G_::WROW);
  const int xtr = tr_base<T>(G_::XT_ROW);
  const int ltr = tr_base<T>(G_::TROW);
  const int wtr = tr_base<T>(G_::WROW);
  const int str = tr_base<T>(CG::SROW);
  const int stb = stage_base<T>(G_::XT_ROW);

  // block set-up: the table image, zeroed Gumbel tiles, the wave's bias and
  // centred dden for its slices
  copy_image(smem, a.img, CG::IMG);
#pragma unroll
  for (int tt = 0; tt < TT; ++tt)
    for (int q = threadIdx.x & 255; q < G_::GT / 16; q += 256)
      reinterpret_cast<uint4*>(tile_lds(tt) + CG::OFF_G)[q] = uint4{0, 0, 0, 0};
  __syncthreads();  // (before any prefetch: a full fence costs nothing here)
  float bias[4], dden[4];
  {
    float cD = 0.f;
    const float* sw = hdr + 2 * M16 + 2 * C;
    for (int j = 0; j < a.M; ++j) cD += sw[j] * dden_tab[j];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = 16 * nb + 4 * g + i;
      bias[i] = hdr[j];
      dden[i] = j < a.M ? dden_tab[j] - cD : 0.f;
    }
  }

  f32x4 dA[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) dA[cb] = zero4();
  float da[4] = {0.f, 0.f, 0.f, 0.f};  // channel blocks 4 wave + k, lane r
  float db[4] = {0.f, 0.f, 0.f, 0.f};  // slices 16 nb + 4g + i, this lane's points
  float dbt = 0.f;

  const T* X = reinterpret_cast<const T*>(a.x);
  const T* Y = reinterpret_cast<const T*>(a.dY);
  const T* Gp = reinterpret_cast<const T*>(a.G);
  T* DX = reinterpret_cast<T*>(a.out);
  // the block's tiles [t0, t1) in rounds of NG TT (group grp: TT tiles from
  // the round's grp-th); a round's tile past t1 is the last tile again, with
  // no contribution (live = false)
  const int64_t T_ = (a.N + 15) / 16;
  const int64_t t0 = T_ * blockIdx.x / gridDim.x, t1 = T_ * (blockIdx.x + 1) / gridDim.x;
  const int64_t nr = (t1 - t0 + NG * TT - 1) / (NG * TT);  // rounds
  auto tile_at = [&](int64_t rd, int tt) { return t0 + (NG * rd + grp) * TT + tt; };
  auto tile_of = [&](int64_t rd, int tt) {
    const int64_t t = tile_at(rd, tt);
    return t < t1 ? t : t1 - 1;
  };
  const int gchunks = 16 * a.M * SZ / 16;  // the Gumbel rows of a full tile

  // this wave's quarter of a round's tiles (rows 4 wave .. 4 wave + 3;
  // Gumbel chunks wave + 4 lane): every load unconditional, rows past N
  // re-read row N - 1
  auto load = [&](Stage& st, int64_t rd) {
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      const int64_t p0 = tile_of(rd, tt) * 16;
      const int lim = last_row<16>(p0, a.N);
      const char* xs = reinterpret_cast<const char*>(X + p0 * C);
      const char* ys = reinterpret_cast<const char*>((deslice ? Y : X) + p0 * C);
#pragma unroll
      for (int k = 0; k < CG::QCH; ++k) {
        const int q = 64 * CG::QCH * wave + lane + 64 * k;
        const int row = q / RCH, cc = q - row * RCH;
        const int rr = row < lim ? row : lim;
        const uint32_t off = (uint32_t)(rr * C * SZ + 16 * cc);
        st.x[tt][k] = ld_global16<true>(xs + off);
        st.y[tt][k] = ld_global16<true>(ys + off);
      }
      const bool full = hasG && p0 + 16 <= a.N;
      const int qg = wave + 4 * lane < gchunks ? wave + 4 * lane : gchunks - 1;
      st.g[tt] = ld_global16<true>(full ? reinterpret_cast<const char*>(Gp + p0 * a.M) + 16 * qg
                                        : reinterpret_cast<const char*>(X));
    }
  };
  auto store = [&](const Stage& st, int64_t rd) {
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      char* tl = tile_lds(tt);
#pragma unroll
      for (int k = 0; k < CG::QCH; ++k) {
        const int q = 64 * CG::QCH * wave + lane + 64 * k;
        const int row = q / RCH, cc = q - row * RCH;
        *reinterpret_cast<uint4*>(tl + CG::OFF_X + lds_off(row, 16 * cc, G_::XT_ROW)) =
            st.x[tt][k];
        if (deslice)
          *reinterpret_cast<uint4*>(tl + CG::OFF_Y + lds_off(row, 16 * cc, G_::XT_ROW)) =
              st.y[tt][k];
      }
      const int64_t p0 = tile_of(rd, tt) * 16;
      if (hasG && p0 + 16 <= a.N) {
        // lanes past the last chunk loaded that chunk again and store it
        // again (the same bytes): no lane-dependent branch around the memory
        // instructions, so the compiler's waits stay exact
        const int qg = wave + 4 * lane < gchunks ? wave + 4 * lane : gchunks - 1;
        *reinterpret_cast<uint4*>(tl + CG::OFF_G + 16 * qg) = st.g[tt];
      } else if (hasG && wave == 0) {
        // the tail tile's valid rows, element by element (without noise
        // the tile keeps the zeros of the set-up)
        g_fixup<T, MB>(tl + CG::OFF_G, Gp, p0, a.N, a.M, hasG);
      }
    }
  };

  auto body = [&](int64_t rd) {
    int64_t p0[TT];
    int nvalid[TT];
    bool live[TT], pv[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      live[tt] = tile_at(rd, tt) < t1;  // uniform over the group
      p0[tt] = tile_of(rd, tt) * 16;
      nvalid[tt] = (int)(a.N - p0[tt] < 16 ? a.N - p0[tt] : 16);
      pv[tt] = live[tt] && r < nvalid[tt];
    }

    // 2. logits of slices 16 nb + 4g + i (point r) and the temperature
    f32x4 lacc[TT], tacc[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) lacc[tt] = tacc[tt] = zero4();
    struct FL { K32<T> t, ta, x[TT]; };
    pipelined<XF, 2, FL>(
        [&](int s, FL& f) {
          ld_row<T>(f.t, tabL, lb.t, 16 * nb * G_::TROW + 32 * s * SZ);
          ld_row<T>(f.ta, tabL, lb.a, M16 * G_::TROW + 32 * s * SZ);
#pragma unroll
          for (int tt = 0; tt < TT; ++tt)
            ld_row<T>(f.x[tt], tile_lds(tt) + CG::OFF_X, lb.x, 32 * s * SZ);
        },
        [&](int s, FL& f) {
#pragma unroll
          for (int tt = 0; tt < TT; ++tt) {
            lacc[tt] = mma32(f.t, f.x[tt], lacc[tt]);
            tacc[tt] = mma32(f.ta, f.x[tt], tacc[tt]);
          }
        });
    float tt_[TT], tau[TT], k2[TT], w[TT][4], zs[TT][4], e4[TT][4], mloc[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      tt_[tt] = tacc[tt][0] + (float)a.tb;
      tau[tt] = fmaxf(tt_[tt], a.tau_min);
      k2[tt] = kLog2e * fast_rcp(tau[tt]);
      const char* gt = tile_lds(tt) + CG::OFF_G;
      const int e = r * a.M + 16 * nb + 4 * g;  // element of the G tile
      float gv[4];
      if (a.M % 4 == 0) {
        const bf16x4 q4 = *reinterpret_cast<const bf16x4*>(gt + e * SZ);
#pragma unroll
        for (int i = 0; i < 4; ++i) gv[i] = (float)q4[i];
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) gv[i] = to_f<T>(reinterpret_cast<const T*>(gt)[e + i]);
      }
      float u[4], m = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        u[i] = own ? lacc[tt][i] + bias[i] + gv[i] : -INFINITY;
        m = fmaxf(m, u[i]);
      }
      mloc[tt] = groups_max(m);
      float sloc = 0.f;
      const float mk = mloc[tt] * k2[tt];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        zs[tt][i] = own ? fmaf(u[i], k2[tt], -mk) : -INFINITY;
        e4[tt][i] = own ? fast_exp2(zs[tt][i]) : 0.f;
        sloc += e4[tt][i];
      }
      sloc = groups_sum(sloc);
      if (g == 0) ex_ms(tt)[16 * wave + r] = float2{own ? mloc[tt] : -INFINITY, sloc};
    }
    block_sync();
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      const float2* ms = ex_ms(tt);
      float m = -INFINITY;
#pragma unroll
      for (int v = 0; v < 4; ++v) m = fmaxf(m, ms[16 * v + r].x);
      float ssum = 0.f;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float2 p = ms[16 * v + r];
        ssum += p.y == 0.f ? 0.f : p.y * fast_exp2((p.x - m) * k2[tt]);
      }
      const float shift = own ? (mloc[tt] - m) * k2[tt] : 0.f;  // this wave's exponent offset
      const float scale = pv[tt] ? fast_exp2(shift) * fast_rcp(ssum) : 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        w[tt][i] = e4[tt][i] * scale;
        zs[tt][i] += shift;
      }
    }

    // 3. dw of the wave's slices: x . (dnum_j - cN) + dY . (s'_j - cS) + dden_j
    f32x4 wacc[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) wacc[tt] = zero4();
    {
      struct FS { K32<T> tw, x[TT]; };
      pipelined<XF, 2, FS>(
          [&](int s, FS& f) {
            ld_row<T>(f.tw, tabW, wrb, 16 * nb * G_::WROW + 32 * s * SZ);
#pragma unroll
            for (int tt = 0; tt < TT; ++tt)
              ld_row<T>(f.x[tt], tile_lds(tt) + CG::OFF_X, lb.x, 32 * s * SZ);
          },
          [&](int s, FS& f) {
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) wacc[tt] = mma32(f.tw, f.x[tt], wacc[tt]);
          });
      if (deslice) {
        struct FD { K32<T> tw, y[TT]; };
        pipelined<XF, 2, FD>(
            [&](int s, FD& f) {
              ld_row<T>(f.tw, tabW, wrb, 16 * nb * G_::WROW + (C + 32 * s) * SZ);
#pragma unroll
              for (int tt = 0; tt < TT; ++tt)
                ld_row<T>(f.y[tt], tile_lds(tt) + CG::OFF_Y, yb, 32 * s * SZ);
            },
            [&](int s, FD& f) {
#pragma unroll
              for (int tt = 0; tt < TT; ++tt) wacc[tt] = mma32(f.tw, f.y[tt], wacc[tt]);
            });
      }
    }
    float dw[TT][4];
    // softmax backward: <w, dw> from the waves' partial sums, compensated by
    // the residual pass; the temperature's <dz, zs> from two more partial
    // sums, <w (dw - wdw), zs> - res <w, zs> (the shift of zs common to all
    // slices drops out, as sum_j dz_j = 0)
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      float p1 = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        dw[tt][i] = own ? wacc[tt][i] + dden[i] : 0.f;
        p1 += w[tt][i] * dw[tt][i];
      }
      p1 = groups_sum(p1);
      if (g == 0) ex_s1(tt)[16 * wave + r] = p1;
    }
    block_sync();
    float wdw[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      const float* s1 = ex_s1(tt);
      wdw[tt] = (s1[r] + s1[16 + r]) + (s1[32 + r] + s1[48 + r]);
      float res = 0.f, q1 = 0.f, q2 = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float d = w[tt][i] * (dw[tt][i] - wdw[tt]);
        res += d;
        if (w[tt][i] != 0.f) {
          q1 += d * zs[tt][i];
          q2 += w[tt][i] * zs[tt][i];
        }
      }
      res = groups_sum(res);
      q1 = groups_sum(q1);
      q2 = groups_sum(q2);
      if (g == 0) ex_s3(tt)[16 * wave + r] = f32x4{res, q1, q2, 0.f};
    }
    block_sync();
    float dt[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      const f32x4* s3 = ex_s3(tt);
      f32x4 tot = zero4();
#pragma unroll
      for (int v = 0; v < 4; ++v) tot += s3[16 * v + r];
      const float rtau = fast_rcp(tau[tt]);
      const float zdz = tot[1] - tot[0] * tot[2];
      const float dtau = -kLn2 * zdz * rtau;
      dt[tt] = (pv[tt] && tt_[tt] > a.tau_min) ? dtau : 0.f;
      // 4. publish w and dl of the wave's slices ([point][slice] rows)
      if (own) {
        bf16x4 wq, lq;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float dl = w[tt][i] * ((dw[tt][i] - wdw[tt]) - tot[0]) * rtau;
          wq[i] = (bf16)w[tt][i];
          lq[i] = (bf16)dl;
          db[i] += dl;
        }
        char* tl = tile_lds(tt);
        *reinterpret_cast<bf16x4*>(tl + CG::OFF_W + r * CG::SROW + (16 * nb + 4 * g) * SZ) = wq;
        *reinterpret_cast<bf16x4*>(tl + CG::OFF_L + r * CG::SROW + (16 * nb + 4 * g) * SZ) = lq;
      }
      if (wave == 0 && g == 0) dbt += dt[tt];
    }
    block_sync();

    // dx of the wave's channel blocks: [A^T | dnum - cN] x [dl ; w] + a dt + cN
    K16<T> wb[TT][MB], lbk[TT][MB];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
      for (int q = 0; q < MB; ++q) {
        const char* tl = tile_lds(tt);
        ld_k16(wb[tt][q], tl + CG::OFF_W + r * CG::SROW + (16 * q + 4 * g) * SZ);
        ld_k16(lbk[tt][q], tl + CG::OFF_L + r * CG::SROW + (16 * q + 4 * g) * SZ);
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
#pragma unroll
          for (int tt = 0; tt < TT; ++tt) {
            f32x4 d = zero4();
#pragma unroll
            for (int q = 0; q < MB; ++q) d = mma16x2(f.ta[q], lbk[tt][q], f.tn[q], wb[tt][q], d);
#pragma unroll
            for (int i = 0; i < 4; ++i) d[i] += f.av[i] * dt[tt] + f.cn[i];
            stage4<T>(tile_lds(tt) + CG::OFF_Y, stb, 16 * (4 * wave + k) * SZ, d);
          }
        });
    wave_sync();
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      if (live[tt]) {  // uniform over the group
        // the wave's 64 channels of the tile's rows: 8 chunks per row (rows
        // past the tile's last point write that point's chunk again: the
        // same bytes, and every lane stores unconditionally)
        char* dst = reinterpret_cast<char*>(DX + p0[tt] * C);
        const char* yt = tile_lds(tt) + CG::OFF_Y;
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const int q = lane + 64 * k;  // < 128
          const int row = (q >> 3) < nvalid[tt] ? (q >> 3) : nvalid[tt] - 1;
          const int cc = 8 * wave + (q & 7);
          const uint4 v = *reinterpret_cast<const uint4*>(yt + lds_off(row, 16 * cc, G_::XT_ROW));
          st_global16(dst + (uint32_t)(row * C * SZ + 16 * cc), v);
        }
      }
    }

    // 5. dA (the wave's slices) += x^T dl, da (its channel blocks) += x^T dt
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      float dtp[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) dtp[i] = __shfl(dt[tt], 4 * g + i);
      const bf16x2 dt01{(bf16)dtp[0], (bf16)dtp[1]}, dt23{(bf16)dtp[2], (bf16)dtp[3]};
      const char* xt = tile_lds(tt) + CG::OFF_X;
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
      K16<T> lp[TT];
#pragma unroll
      for (int tt = 0; tt < TT; ++tt)
        ld_tr<T>(lp[tt], tile_lds(tt) + CG::OFF_L, str, 16 * nb * SZ, CG::SROW);
      struct FA { K16<T> xa[TT]; };
      pipelined<CB, 4, FA>(
          [&](int cb, FA& f) {
#pragma unroll
            for (int tt = 0; tt < TT; ++tt)
              ld_tr<T>(f.xa[tt], tile_lds(tt) + CG::OFF_X, xtr, 16 * cb * SZ, G_::XT_ROW);
          },
          [&](int cb, FA& f) {
            if constexpr (TT == 2) {
              // the two tiles' K16 products as one K32 product (32 points)
              dA[cb] = mma16x2(f.xa[0], lp[0], f.xa[1], lp[1], dA[cb]);
            } else {
#pragma unroll
              for (int tt = 0; tt < TT; ++tt) dA[cb] = mma16(f.xa[tt], lp[tt], dA[cb]);
            }
          });
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

  // two groups: the second group's per-lane partials through LDS (over the
  // tables and tiles, no longer read), added to the first's in that order
  if constexpr (NG == 2) {
    static_assert(4 * 64 * CG::PART * 4 <= CG::LDS, "group partials must fit in LDS");
    float* part = reinterpret_cast<float*>(smem) + (wave * 64 + lane) * CG::PART;
    block_sync();
    if (grp == 1) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) *reinterpret_cast<f32x4*>(part + 4 * cb) = dA[cb];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        part[4 * CB + i] = db[i];
        part[4 * CB + 4 + i] = da[i];
      }
      part[4 * CB + 8] = dbt;
    }
    block_sync();
    if (grp == 1) return;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) dA[cb] += *reinterpret_cast<const f32x4*>(part + 4 * cb);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      db[i] += part[4 * CB + i];
      da[i] += part[4 * CB + 4 + i];
    }
    dbt += part[4 * CB + 8];
  }
  // lane partials -> wave totals, then the block's record: dA [C][M],
  // db [M], da [C], db_t, each part written by the wave that owns it
#pragma unroll
  for (int i = 0; i < 4; ++i) db[i] = row16_sum(db[i]);
#pragma unroll
  for (int k = 0; k < 4; ++k) da[k] = groups_sum(da[k]);
  dbt = row16_sum(dbt);
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
    if (r == 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int jj = 16 * nb + 4 * g + i;
        if (jj < M) rec[C * M + jj] = db[i];
      }
    }
  }
  if (g == 0) {
#pragma unroll
    for (int k = 0; k < 4; ++k) rec[C * M + M + 16 * (4 * wave + k) + r] = da[k];
  }
  if (wave == 0 && lane == 0) rec[C * M + M + C] = dbt;
}

}  // namespace pa
