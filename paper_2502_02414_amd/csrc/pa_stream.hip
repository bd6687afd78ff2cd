// Dispatch of the streaming passes (kernels in pa_stream.hpp, instantiated
// per pass in pa_stream_<pass>.hip).
#include "pa_coop.hpp"

namespace pa {

template <int SZ>
static int waves_of(int pass, int C, int MB, int cr) {
  // the block-cooperative slice backward (groups of four waves per block;
  // rows of exactly 256 channels)
  const bool coop = pass == kSliceBwd && SZ == 2 && C == 256 && cr == 256;
  if (coop && MB == 4 && coop_slice_bwd<bf16, 256, 4>())
    return CoopGeo<bf16, 256, 4, coop_groups<bf16, 256, 4>()>::WAVES;
  if (coop && MB == 3 && coop_slice_bwd<bf16, 256, 3>())
    return CoopGeo<bf16, 256, 3, coop_groups<bf16, 256, 3>()>::WAVES;
#define PA_W(CC, BB) \
  if (C == CC && MB == BB) return Geo<SZ, CC, BB>::fits(pass) ? Geo<SZ, CC, BB>::waves(pass) : 0;
  PA_W(32, 1) PA_W(32, 2) PA_W(32, 3) PA_W(32, 4)
  PA_W(64, 1) PA_W(64, 2) PA_W(64, 3) PA_W(64, 4)
  PA_W(128, 1) PA_W(128, 2) PA_W(128, 3) PA_W(128, 4)
  PA_W(256, 1) PA_W(256, 2) PA_W(256, 3) PA_W(256, 4)
#undef PA_W
  return 0;
}

int stream_waves(int pass, int dtype, int C, int MB, int cr) {
  if (cr < 16 || cr > C || cr % 16) return 0;
  return dtype == 1 ? waves_of<2>(pass, C, MB, cr) : waves_of<4>(pass, C, MB, cr);
}

hipError_t launch_stream(int pass, int dtype, int C, int MB, const StreamLaunch& L,
                         hipStream_t st) {
  // every pointer a pass dereferences must be there (a NULL is an error here,
  // never a device fault)
  // (the stored-weights passes read W, given as G, in place of x and G)
  const bool win = pass == kDesliceW || pass == kDesliceBwdW;
  if ((win ? !L.G : !L.x) || !L.img || L.N < 1 || L.M < 1 || L.M > 16 * MB || L.P < 1 ||
      L.cr < 16 || L.cr > C || L.cr % 16)
    return hipErrorInvalidValue;
  const bool reduces = agg_fwd(pass) || agg_bwd(pass) || pass == kSliceBwd || pass == kWeightsBwd;
  if (reduces && !L.partials) return hipErrorInvalidValue;
  if ((pass == kDeslice || pass == kDesliceW || pass == kWeights || pass == kSliceBwd ||
       pass == kWeightsBwd || pass == kAggregateW) && !L.out)
    return hipErrorInvalidValue;
  if (agg_bwd(pass) && !L.dY) return hipErrorInvalidValue;
  if (pass == kSliceBwd && L.deslice && !L.dY) return hipErrorInvalidValue;
  if (pass == kWeightsBwd && !L.dW) return hipErrorInvalidValue;
  StreamArgs a;
  a.x = L.x; a.G = L.G; a.dY = L.dY; a.img = L.img; a.out = L.out; a.tau_out = L.tau_out;
  a.dW = L.dW; a.dtau = L.dtau; a.partials = L.partials; a.N = L.N; a.M = L.M; a.cr = L.cr;
  a.rec = L.rec;
  a.tb = L.tb; a.tb_dev = L.tb_dev; a.tau_min = L.tau_min;
  a.flags = (L.G ? kHasG : 0) | (L.states ? kStatesTerm : 0) | (L.deslice ? kDesliceTerm : 0);
  if (L.heads < 1 || L.heads > kMaxHeads) return hipErrorInvalidValue;
  a.heads = L.heads;
  a.hs_x = L.hs_x; a.hs_g = L.hs_g; a.hs_dy = L.hs_dy; a.hs_out = L.hs_out;
  a.hs_img = L.hs_img; a.hs_part = L.hs_part; a.hs_tb = L.hs_tb;
  switch (pass) {
    case kAggregate: return launch_aggregate_pass(dtype, C, MB, a, L.P, st);
    case kDeslice: return launch_deslice_pass(dtype, C, MB, a, L.P, st);
    case kDesliceBwd: return launch_deslice_bwd_pass(dtype, C, MB, a, L.P, st);
    case kWeights: return launch_weights_pass(dtype, C, MB, a, L.P, st);
    case kSliceBwd: return launch_slice_bwd_pass(dtype, C, MB, a, L.P, st);
    case kWeightsBwd: return launch_weights_bwd_pass(dtype, C, MB, a, L.P, st);
    case kAggregateW: return launch_aggregate_w_pass(dtype, C, MB, a, L.P, st);
    case kDesliceW: return launch_deslice_w_pass(dtype, C, MB, a, L.P, st);
    case kDesliceBwdW: return launch_deslice_bwd_w_pass(dtype, C, MB, a, L.P, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace pa
