// Instantiation of the kSliceBwd streaming pass (see pa_stream.hpp): the
// per-wave kernel, or the block-cooperative one (pa_coop.hpp) for bf16 rows
// of 256 channels with more than 32 slices.
#include "pa_coop.hpp"

namespace pa {

template <int MB>
static hipError_t launch_coop(const StreamArgs& a, int P, hipStream_t st) {
  constexpr int NG = coop_groups<bf16, 256, MB>();
  using CG = CoopGeo<bf16, 256, MB, NG>;
  hipLaunchKernelGGL((k_slice_bwd_coop<bf16, 256, MB, NG>), dim3(P, a.heads),
                     dim3(64 * CG::WAVES), CG::LDS, st, a);
  return hipGetLastError();
}

hipError_t launch_slice_bwd_pass(int dtype, int C, int MB, const StreamArgs& a, int P, hipStream_t st) {
  const bool coop = dtype == 1 && C == 256 && a.cr == 256;  // rows of exactly 256 channels
  if (coop && MB == 4 && coop_slice_bwd<bf16, 256, 4>()) return launch_coop<4>(a, P, st);
  if (coop && MB == 3 && coop_slice_bwd<bf16, 256, 3>()) return launch_coop<3>(a, P, st);
  return launch_pass<kSliceBwd>(dtype, C, MB, a, P, st);
}
}  // namespace pa
