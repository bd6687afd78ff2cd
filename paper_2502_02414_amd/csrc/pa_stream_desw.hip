// Instantiation of the kDesliceW streaming pass (see pa_stream.hpp).
#include "pa_stream.hpp"

namespace pa {
hipError_t launch_deslice_w_pass(int dtype, int C, int MB, const StreamArgs& a, int P, hipStream_t st) {
  return launch_pass<kDesliceW>(dtype, C, MB, a, P, st);
}
}  // namespace pa
