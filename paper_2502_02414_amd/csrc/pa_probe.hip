// Stream probe (diagnostics, gfx950): the memory traffic of one streaming
// pass with none of its arithmetic.  k_probe moves the point tensors the
// per-wave kernel of a pass reads and writes exactly as that kernel does --
// its work split (P blocks of the pass's waves, a contiguous tile range per
// wave), tile height, register prefetch depth and walk direction, its 16-byte
// loads with the same cache hints into the same LDS tiles, and its output
// rows written back from an LDS tile -- and computes nothing (the written
// rows are the x tile's).  Its duration is what the pass's access pattern
// takes on its own, the rate the pass would reach if its arithmetic were
// free: the achievable bandwidth its roofline fraction is read against.
#include "pa_stream.hpp"

namespace pa {
namespace {

// The passes the probe mirrors: what each reads and writes, per point.
template <int PASS> constexpr bool probe_reads_dy() { return PASS == kDesliceBwd || PASS == kSliceBwd; }
template <int PASS> constexpr bool probe_writes() { return PASS == kDeslice || PASS == kSliceBwd; }
template <typename T, int C, int MB, int PASS> constexpr int probe_depth() {
  return PASS == kAggregate ? agg_depth<T, C, MB, false>()
       : PASS == kDesliceBwd ? agg_depth<T, C, MB, true>()
       : PASS == kDeslice ? des_depth<T, C, MB>()
       : bwd_depth<T, C, MB>();
}
template <int PASS> constexpr bool probe_rev() {
  return PASS == kDeslice ? kRevDeslice : PASS == kSliceBwd ? kRevSliceBwd : false;
}

template <typename T, int C, int MB, int ROWS>
struct ProbeStage {
  TileRegs<T, C, ROWS> x, y;
  GRegs<T, MB, ROWS> g;
};

template <typename T, int C, int MB, int PASS, bool EX>
__global__ void __launch_bounds__((64 * Geo<sizeof(T), C, MB>::waves(PASS))) k_probe(StreamArgs a) {
  using G_ = Geo<sizeof(T), C, MB>;
  constexpr int WAVES = G_::waves(PASS);
  constexpr int ROWS = G_::rows(PASS), H = ROWS / 16;
  constexpr bool NT = !keep_loads<PASS>();
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool hasG = a.flags & kHasG;
  char* const xt = smem + wave * G_::wave_bytes(PASS);
  char* const yt = probe_reads_dy<PASS>() ? xt + H * G_::XT : xt;
  char* const gt = xt + (probe_reads_dy<PASS>() ? 2 : 1) * H * G_::XT;
  const T* X = reinterpret_cast<const T*>(a.x);
  const T* Y = reinterpret_cast<const T*>(a.dY);
  const T* Gp = reinterpret_cast<const T*>(a.G);
  T* OUT = reinterpret_cast<T*>(a.out);
  int64_t t0, t1;
  tile_range(a.N, WAVES, wave, t0, t1, ROWS);

  using Stage = ProbeStage<T, C, MB, ROWS>;
  auto load = [&](Stage& st, int64_t tile) {
    const int64_t p0 = tile * ROWS;
    load_tile<T, C, ROWS, NT, EX>(st.x, X, p0, a.N, a.cr);
    if constexpr (probe_reads_dy<PASS>()) load_tile<T, C, ROWS, true, EX>(st.y, Y, p0, a.N, a.cr);
    load_g<T, MB, ROWS, true>(st.g, Gp, X, p0, a.N, a.M, hasG);
  };
  auto store = [&](const Stage& st) {
    store_tile<T, C, ROWS>(xt, st.x);
    if constexpr (probe_reads_dy<PASS>()) store_tile<T, C, ROWS>(yt, st.y);
    if (hasG) store_g<T, MB, ROWS>(gt, st.g, a.M, hasG);
  };
  auto body = [&](int64_t t) {
    if constexpr (probe_writes<PASS>()) {
      const int64_t p0 = t * ROWS;
      const int nvalid = (int)(a.N - p0 < ROWS ? a.N - p0 : ROWS);
      wave_sync();
      write_tile<T, C, ROWS, EX>(OUT, p0, xt, nvalid, a.cr);
    }
  };
  auto tail = [&](int64_t t) {
    Stage st;
    load(st, t);
    wave_sync();
    store(st);
    wave_sync();
    body(t);
  };
  stream_tiles<probe_depth<T, C, MB, PASS>(), Stage, probe_rev<PASS>()>(
      t0, t1, a.N / ROWS, load, store, body, tail, [] {});
}

template <typename T, int C, int MB, int PASS>
hipError_t launch_probe_t(const StreamArgs& a, int P, hipStream_t st) {
  using G_ = Geo<sizeof(T), C, MB>;
  if constexpr (!G_::fits(PASS)) {
    return hipErrorInvalidConfiguration;
  } else {
    const size_t lds = (size_t)G_::waves(PASS) * G_::wave_bytes(PASS);
    if (a.cr == C)
      hipLaunchKernelGGL((k_probe<T, C, MB, PASS, true>), dim3(P), dim3(64 * G_::waves(PASS)), lds,
                         st, a);
    else
      hipLaunchKernelGGL((k_probe<T, C, MB, PASS, false>), dim3(P), dim3(64 * G_::waves(PASS)), lds,
                         st, a);
    return hipGetLastError();
  }
}

template <typename T, int C, int PASS>
hipError_t launch_probe_c(int MB, const StreamArgs& a, int P, hipStream_t st) {
  switch (MB) {
    case 1: return launch_probe_t<T, C, 1, PASS>(a, P, st);
    case 2: return launch_probe_t<T, C, 2, PASS>(a, P, st);
    case 3: return launch_probe_t<T, C, 3, PASS>(a, P, st);
    case 4: return launch_probe_t<T, C, 4, PASS>(a, P, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename T, int PASS>
hipError_t launch_probe_p(int C, int MB, const StreamArgs& a, int P, hipStream_t st) {
  switch (C) {
    case 32: return launch_probe_c<T, 32, PASS>(MB, a, P, st);
    case 64: return launch_probe_c<T, 64, PASS>(MB, a, P, st);
    case 128: return launch_probe_c<T, 128, PASS>(MB, a, P, st);
    case 256: return launch_probe_c<T, 256, PASS>(MB, a, P, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t launch_probe_d(int pass, int C, int MB, const StreamArgs& a, int P, hipStream_t st) {
  switch (pass) {
    case kAggregate: return launch_probe_p<T, kAggregate>(C, MB, a, P, st);
    case kDeslice: return launch_probe_p<T, kDeslice>(C, MB, a, P, st);
    case kDesliceBwd: return launch_probe_p<T, kDesliceBwd>(C, MB, a, P, st);
    case kSliceBwd: return launch_probe_p<T, kSliceBwd>(C, MB, a, P, st);
    default: return hipErrorInvalidValue;
  }
}

template <int SZ>
int probe_waves_of(int pass, int C, int MB) {
#define PA_PW(CC, BB) \
  if (C == CC && MB == BB) return Geo<SZ, CC, BB>::fits(pass) ? Geo<SZ, CC, BB>::waves(pass) : 0;
  PA_PW(32, 1) PA_PW(32, 2) PA_PW(32, 3) PA_PW(32, 4)
  PA_PW(64, 1) PA_PW(64, 2) PA_PW(64, 3) PA_PW(64, 4)
  PA_PW(128, 1) PA_PW(128, 2) PA_PW(128, 3) PA_PW(128, 4)
  PA_PW(256, 1) PA_PW(256, 2) PA_PW(256, 3) PA_PW(256, 4)
#undef PA_PW
  return 0;
}

}  // namespace

int probe_waves(int pass, int dtype, int C, int MB) {
  if (pass != kAggregate && pass != kDeslice && pass != kDesliceBwd && pass != kSliceBwd) return 0;
  return dtype == 1 ? probe_waves_of<2>(pass, C, MB) : probe_waves_of<4>(pass, C, MB);
}

hipError_t launch_probe(int pass, int dtype, int C, int MB, const StreamLaunch& L, hipStream_t st) {
  if (!L.x || L.N < 1 || L.M < 1 || L.M > 16 * MB || L.P < 1 || L.cr < 16 || L.cr > C ||
      L.cr % 16)
    return hipErrorInvalidValue;
  if ((pass == kDesliceBwd || pass == kSliceBwd) && !L.dY) return hipErrorInvalidValue;
  if ((pass == kDeslice || pass == kSliceBwd) && !L.out) return hipErrorInvalidValue;
  StreamArgs a{};
  a.x = L.x; a.G = L.G; a.dY = L.dY; a.out = L.out; a.N = L.N; a.M = L.M; a.cr = L.cr;
  a.flags = L.G ? kHasG : 0;
  a.heads = 1;
  return dtype == 1 ? launch_probe_d<bf16>(pass, C, MB, a, L.P, st)
                    : launch_probe_d<float>(pass, C, MB, a, L.P, st);
}

}  // namespace pa
