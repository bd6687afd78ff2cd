// C ABI of the Physics-Attention hot path (see include/pa.h): host-side
// validation, workspace carving and the launch sequence of every call.  No
// arithmetic of the layer happens here; it all runs in the HIP kernels.
#include "pa.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>

#include "pa_internal.h"
#include "pa_layout.h"

namespace {

thread_local std::string g_err;

pa_status fail(pa_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
pa_status fail(pa_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

pa_status hip_fail(hipError_t e, const char* what) {
  return fail(PA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define PA_HIP(call, what)                      \
  do {                                          \
    hipError_t e_ = (call);                     \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

constexpr size_t kAlign = 256;
size_t up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

int mblocks(int M) { return (M + 15) / 16; }

// The width the streaming kernels are built for that holds C channels: rows
// of C channels run on the kernels of the next width up, with the tables'
// extra channels zero.
int cpad(int C) { return C <= 32 ? 32 : C <= 64 ? 64 : C <= 128 ? 128 : 256; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Workspace carve-up (offsets in bytes).
struct Layout {
  size_t img, parts, attn, total;
  int P;          // point chunks (the largest over the streaming passes)
};

Layout layout_of(const pa_dims& d) {
  Layout L{};
  const int MB = mblocks(d.M);
  size_t img = 0;
  for (int pass = 0; pass < pa::kNumPasses; ++pass) {
    size_t b = pa::image_bytes(pass, d.dtype, cpad(d.C), MB);
    if (b > img) img = b;
  }
  // chunks: every pass uses at most kPartialsMax blocks
  const int64_t rec = (int64_t)d.C * d.M + d.M + d.C + 1;  // the largest record
  const int P = pa::kPartialsMax;
  const size_t mc = (size_t)d.M * d.C;
  // token scratch: eight [M,C] matrices in double (fp32 storage) or float,
  // and the attention matrices of the heads
  const size_t attn = (16 * mc + (size_t)d.H * d.M * d.M) * sizeof(float);
  L.img = 0;
  L.parts = up(img);
  L.attn = L.parts + up((size_t)P * rec * sizeof(float));
  L.total = L.attn + up(attn);
  L.P = P;
  return L;
}

pa_status check_dims(const pa_dims* d) {
  if (!d) return fail(PA_ERR_INVALID, "dims is NULL");
  if (d->N < 1) return fail(PA_ERR_INVALID, "N must be >= 1 (got %lld)", (long long)d->N);
  if (d->M < 1 || d->M > 64) return fail(PA_ERR_INVALID, "M must be in [1, 64] (got %d)", d->M);
  if (d->C < 1) return fail(PA_ERR_INVALID, "C must be >= 1 (got %d)", d->C);
  if (d->H < 1 || d->C % d->H != 0)
    return fail(PA_ERR_INVALID, "H must be >= 1 and divide C (C=%d, H=%d)", d->C, d->H);
  if (!(d->tau_min > 0.f) || !std::isfinite(d->tau_min))
    return fail(PA_ERR_INVALID, "tau_min must be finite and > 0");
  if (!(d->eps > 0.f) || !std::isfinite(d->eps))
    return fail(PA_ERR_INVALID, "eps must be finite and > 0");
  if (!std::isfinite(d->tau0)) return fail(PA_ERR_INVALID, "tau0 must be finite");
  if (d->dtype != PA_F32 && d->dtype != PA_BF16)
    return fail(PA_ERR_INVALID, "dtype must be PA_F32 or PA_BF16 (got %d)", d->dtype);
  if (d->C % 16 != 0 || d->C > 256)
    return fail(PA_ERR_UNSUPPORTED, "C must be a multiple of 16 in [16, 256] (got %d)", d->C);
  return PA_OK;
}

pa_status check_pass(const pa_dims& d, int pass) {
  if (pa::stream_waves(pass, d.dtype, cpad(d.C), mblocks(d.M), d.C) <= 0)
    return fail(PA_ERR_UNSUPPORTED,
                "shape C=%d M=%d dtype=%d does not fit the on-chip tables of this pass", d.C,
                d.M, d.dtype);
  return PA_OK;
}

pa_status check_ptr(const void* p, const char* name, bool required) {
  if (!p) return required ? fail(PA_ERR_INVALID, "%s is NULL", name) : PA_OK;
  if (!aligned16(p)) return fail(PA_ERR_INVALID, "%s is not 16-byte aligned", name);
  return PA_OK;
}

pa_status check_ws(const pa_dims& d, const void* ws, size_t ws_bytes) {
  const Layout L = layout_of(d);
  if (!ws) return fail(PA_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", L.total);
  if (ws_bytes < L.total)
    return fail(PA_ERR_WORKSPACE, "workspace too small: %zu < %zu bytes", ws_bytes, L.total);
  if (((uintptr_t)ws & (kAlign - 1)) != 0)
    return fail(PA_ERR_INVALID, "workspace is not %zu-byte aligned", kAlign);
  return PA_OK;
}

#define PA_TRY(x)                \
  do {                           \
    pa_status s_ = (x);          \
    if (s_ != PA_OK) return s_;  \
  } while (0)

char* wsb(void* ws) { return reinterpret_cast<char*>(ws); }

int chunks(const pa_dims& d, int pass) {
  return pa::num_chunks(d.N, pa::stream_waves(pass, d.dtype, cpad(d.C), mblocks(d.M), d.C));
}

pa::PrepArgs prep_of(const pa_dims& d, int pass, const pa_slice_params* sp, void* ws) {
  pa::PrepArgs p;
  p.pass = pass;
  p.dtype = d.dtype;
  p.C = cpad(d.C);
  p.cr = d.C;
  p.M = d.M;
  p.MB = mblocks(d.M);
  p.eps = d.eps;
  if (sp) {  // (the stored-weights deslice builds no logits table)
    p.A = sp->A;
    p.b = sp->b;
    p.a = sp->a;
  }
  p.img = wsb(ws) + layout_of(d).img;
  return p;
}

pa::StreamLaunch stream_of(const pa_dims& d, int pass, const void* x, const void* G,
                           const pa_slice_params* sp, void* ws) {
  pa::StreamLaunch L;
  const Layout lay = layout_of(d);
  L.x = x;
  L.G = G;
  L.img = wsb(ws) + lay.img;
  L.partials = reinterpret_cast<float*>(wsb(ws) + lay.parts);
  L.N = d.N;
  L.M = d.M;
  L.cr = d.C;
  L.rec = (int)pa::record_floats(pass, d.C, d.M);
  L.P = chunks(d, pass);
  L.tb = (double)d.tau0 + (sp ? (double)sp->b_t : 0.0);
  L.tb_dev = sp ? sp->b_t_dev : nullptr;
  L.tau_min = d.tau_min;
  return L;
}

pa_status check_slice(const pa_dims* dims, const void* x, const void* G,
                      const pa_slice_params* sp) {
  PA_TRY(check_dims(dims));
  if (!sp) return fail(PA_ERR_INVALID, "slice params are NULL");
  PA_TRY(check_ptr(x, "x", true));
  PA_TRY(check_ptr(G, "G", false));
  PA_TRY(check_ptr(sp->A, "A", true));
  PA_TRY(check_ptr(sp->b, "b", false));
  PA_TRY(check_ptr(sp->a, "a", false));
  if (!std::isfinite(sp->b_t)) return fail(PA_ERR_INVALID, "b_t must be finite");
  return PA_OK;
}

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

}  // namespace

void pa::set_last_error(const char* msg) { g_err = msg; }

namespace {

// pa_time_kernel's hook: the pass whose streaming kernel is bracketed by the
// caller's events on this thread (-1: disarmed).
struct KernelTimer {
  int pass = -1;
  hipEvent_t start = nullptr, stop = nullptr;
};
thread_local KernelTimer g_timer;

// Launches the streaming kernel of a pass, between the armed events when it
// is the timed pass.
hipError_t run_stream(int pass, const pa_dims& d, const pa::StreamLaunch& L, hipStream_t st) {
  const bool timed = g_timer.pass == pass;
  if (timed) {
    hipError_t e = hipEventRecord(g_timer.start, st);
    if (e != hipSuccess) return e;
  }
  hipError_t e = pa::launch_stream(pass, d.dtype, cpad(d.C), mblocks(d.M), L, st);
  if (e == hipSuccess && timed) e = hipEventRecord(g_timer.stop, st);
  return e;
}

}  // namespace

extern "C" {

int pa_version(void) { return PA_VERSION; }

const char* pa_last_error(void) { return g_err.c_str(); }

pa_status pa_time_kernel(const char* call, void* start, void* stop) {
  if (!call) {
    g_timer = KernelTimer{};
    return PA_OK;
  }
  static const struct { const char* name; int pass; } kCalls[] = {
      {"pa_slice_weights", pa::kWeights},
      {"pa_slice_aggregate", pa::kAggregate},
      {"pa_deslice", pa::kDeslice},
      {"pa_deslice_backward", pa::kDesliceBwd},
      {"pa_slice_aggregate_backward", pa::kSliceBwd},
      {"pa_slice_weights_backward", pa::kWeightsBwd},
      {"pa_slice_aggregate_w", pa::kAggregateW},
      {"pa_deslice_w", pa::kDesliceW},
      {"pa_deslice_backward_w", pa::kDesliceBwdW},
  };
  int pass = -1;
  for (const auto& c : kCalls)
    if (std::strcmp(call, c.name) == 0) pass = c.pass;
  if (pass < 0) return fail(PA_ERR_INVALID, "pa_time_kernel: no streaming kernel in '%s'", call);
  if (!start || !stop) return fail(PA_ERR_INVALID, "pa_time_kernel: start and stop are required");
  g_timer.pass = pass;
  g_timer.start = static_cast<hipEvent_t>(start);
  g_timer.stop = static_cast<hipEvent_t>(stop);
  return PA_OK;
}

pa_status pa_stream_probe(const pa_dims* dims, const char* call, const void* x, const void* dY,
                          const void* G, void* out, void* stream) {
  PA_TRY(check_dims(dims));
  static const struct { const char* name; int pass; } kProbed[] = {
      {"pa_slice_aggregate", pa::kAggregate},
      {"pa_deslice", pa::kDeslice},
      {"pa_deslice_backward", pa::kDesliceBwd},
      {"pa_slice_aggregate_backward", pa::kSliceBwd},
  };
  int pass = -1;
  if (call)
    for (const auto& c : kProbed)
      if (std::strcmp(call, c.name) == 0) pass = c.pass;
  if (pass < 0)
    return fail(PA_ERR_INVALID, "pa_stream_probe: no probed streaming pass in '%s'",
                call ? call : "(null)");
  PA_TRY(check_ptr(x, "x", true));
  PA_TRY(check_ptr(G, "G", false));
  PA_TRY(check_ptr(dY, "dY", pass == pa::kDesliceBwd || pass == pa::kSliceBwd));
  PA_TRY(check_ptr(out, "out", pass == pa::kDeslice || pass == pa::kSliceBwd));
  const pa_dims& d = *dims;
  const int waves = pa::probe_waves(pass, d.dtype, cpad(d.C), mblocks(d.M));
  if (waves <= 0)
    return fail(PA_ERR_UNSUPPORTED, "pa_stream_probe: shape C=%d M=%d dtype=%d not served", d.C,
                d.M, d.dtype);
  pa::StreamLaunch L;
  L.x = x;
  L.G = G;
  L.dY = dY;
  L.out = out;
  L.N = d.N;
  L.M = d.M;
  L.cr = d.C;
  L.P = pa::num_chunks(d.N, waves);
  PA_HIP(pa::launch_probe(pass, d.dtype, cpad(d.C), mblocks(d.M), L, as_stream(stream)),
         "stream probe");
  return PA_OK;
}

pa_status pa_workspace_size(const pa_dims* dims, size_t* bytes) {
  PA_TRY(check_dims(dims));
  if (!bytes) return fail(PA_ERR_INVALID, "bytes is NULL");
  *bytes = layout_of(*dims).total;
  return PA_OK;
}

pa_status pa_slice_weights(const pa_dims* dims, const void* x, const void* G,
                           const pa_slice_params* sp, float* W, float* tau, void* ws,
                           size_t ws_bytes, void* stream) {
  PA_TRY(check_slice(dims, x, G, sp));
  PA_TRY(check_ptr(W, "W", true));
  PA_TRY(check_ptr(tau, "tau", false));
  PA_TRY(check_pass(*dims, pa::kWeights));
  PA_TRY(check_ws(*dims, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  PA_HIP(pa::launch_prep(prep_of(*dims, pa::kWeights, sp, ws), st), "prep");
  pa::StreamLaunch L = stream_of(*dims, pa::kWeights, x, G, sp, ws);
  L.out = W;
  L.tau_out = tau;
  PA_HIP(run_stream(pa::kWeights, *dims, L, st),
         "slice weights");
  return PA_OK;
}

}  // extern "C"

namespace {
pa_status check_aggregate(int pass, const pa_dims* dims, const void* x, const void* G,
                          const pa_slice_params* sp, float* num, float* den, float* S,
                          void* W) {
  PA_TRY(check_slice(dims, x, G, sp));
  PA_TRY(check_ptr(num, "num", true));
  PA_TRY(check_ptr(den, "den", true));
  PA_TRY(check_ptr(S, "S", true));
  PA_TRY(check_ptr(W, "W", pass == pa::kAggregateW));
  return check_pass(*dims, pass);
}

// The launches of pa_slice_aggregate(_w) on a validated workspace: the
// table image at its start, the block records at the layout's offset.
pa_status slice_aggregate_launch(int pass, const pa_dims* dims, const void* x, const void* G,
                                 const pa_slice_params* sp, float* num, float* den, float* S,
                                 void* W, void* ws, hipStream_t st) {
  PA_HIP(pa::launch_prep(prep_of(*dims, pass, sp, ws), st), "prep");
  pa::StreamLaunch L = stream_of(*dims, pass, x, G, sp, ws);
  L.out = W;
  PA_HIP(run_stream(pass, *dims, L, st), "slice aggregate");
  pa::Segments seg{};
  seg.dst[0] = num; seg.len[0] = (int64_t)dims->M * dims->C;
  seg.dst[1] = den; seg.len[1] = dims->M;
  seg.n = 2;
  seg.S = S;
  seg.nS = (int64_t)dims->M * dims->C;
  seg.den_col = seg.nS;
  seg.C = dims->C;
  seg.eps = dims->eps;
  PA_HIP(pa::launch_reduce(L.partials, L.P, L.rec, seg, st), "reduce");
  return PA_OK;
}

// pa_slice_aggregate and pa_slice_aggregate_w (which also writes W).
pa_status slice_aggregate(int pass, const pa_dims* dims, const void* x, const void* G,
                          const pa_slice_params* sp, float* num, float* den, float* S, void* W,
                          void* ws, size_t ws_bytes, void* stream) {
  PA_TRY(check_aggregate(pass, dims, x, G, sp, num, den, S, W));
  PA_TRY(check_ws(*dims, ws, ws_bytes));
  return slice_aggregate_launch(pass, dims, x, G, sp, num, den, S, W, ws, as_stream(stream));
}
}  // namespace

extern "C" {

pa_status pa_slice_aggregate(const pa_dims* dims, const void* x, const void* G,
                             const pa_slice_params* sp, float* num, float* den, float* S,
                             void* ws, size_t ws_bytes, void* stream) {
  return slice_aggregate(pa::kAggregate, dims, x, G, sp, num, den, S, nullptr, ws, ws_bytes,
                         stream);
}

pa_status pa_slice_aggregate_w(const pa_dims* dims, const void* x, const void* G,
                               const pa_slice_params* sp, float* num, float* den, float* S,
                               void* W, void* ws, size_t ws_bytes, void* stream) {
  return slice_aggregate(pa::kAggregateW, dims, x, G, sp, num, den, S, W, ws, ws_bytes, stream);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// pa_slice_aggregate_noalloc: the aggregate's table image and block records
// in a static device array instead of a caller's workspace.  Each device
// holds its own copy of the array for the life of the process; host code
// uses only the address hipGetSymbolAddress returns for it on that device
// (the array's name is a host-side stand-in, not a device address).
// ---------------------------------------------------------------------------
namespace {
constexpr size_t kNoallocScratchBytes = (size_t)17 << 20;  // 17 MiB
constexpr int kNoallocMaxDevices = 64;
std::mutex g_noalloc_mu;
void* g_noalloc_scratch[kNoallocMaxDevices] = {};
}  // namespace

static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

namespace {
// Device address of `scratch` on the current device, looked up on the first
// call on that device (with it current) and kept.
pa_status noalloc_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kNoallocMaxDevices)
    return fail(PA_ERR_UNSUPPORTED, "pa_slice_aggregate_noalloc: device %d beyond %d", dev,
                kNoallocMaxDevices);
  std::lock_guard<std::mutex> lock(g_noalloc_mu);
  if (!g_noalloc_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(PA_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_noalloc_scratch[dev] = p;
  }
  *out = g_noalloc_scratch[dev];
  return PA_OK;
}

// Scratch bytes the aggregate needs: the workspace layout up to the end of
// the aggregate's own block records (its table image sits at offset 0).
size_t noalloc_bytes(const pa_dims& d) {
  return layout_of(d).parts +
         (size_t)chunks(d, pa::kAggregate) * pa::record_floats(pa::kAggregate, d.C, d.M) *
             sizeof(float);
}
}  // namespace

extern "C" {

pa_status pa_slice_aggregate_noalloc(const pa_dims* dims, const void* x, const void* G,
                                     const pa_slice_params* sp, float* num, float* den,
                                     float* S, void* stream) {
  PA_TRY(check_aggregate(pa::kAggregate, dims, x, G, sp, num, den, S, nullptr));
  const size_t need = noalloc_bytes(*dims);
  if (need > kNoallocScratchBytes)
    return fail(PA_ERR_UNSUPPORTED,
                "pa_slice_aggregate_noalloc: this shape needs %zu bytes of scratch, more than "
                "the %zu the library holds",
                need, kNoallocScratchBytes);
  void* base = nullptr;
  PA_TRY(noalloc_scratch(&base));
  return slice_aggregate_launch(pa::kAggregate, dims, x, G, sp, num, den, S, nullptr, base,
                                as_stream(stream));
}

pa_status pa_deslice_w(const pa_dims* dims, const void* W, const float* Sp, void* y, void* ws,
                       size_t ws_bytes, void* stream) {
  PA_TRY(check_dims(dims));
  PA_TRY(check_ptr(W, "W", true));
  PA_TRY(check_ptr(Sp, "Sp", true));
  PA_TRY(check_ptr(y, "y", true));
  PA_TRY(check_pass(*dims, pa::kDesliceW));
  PA_TRY(check_ws(*dims, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  pa::PrepArgs p = prep_of(*dims, pa::kDesliceW, nullptr, ws);
  p.Sp = Sp;
  PA_HIP(pa::launch_prep(p, st), "prep");
  pa::StreamLaunch L = stream_of(*dims, pa::kDesliceW, nullptr, W, nullptr, ws);
  L.out = y;
  PA_HIP(run_stream(pa::kDesliceW, *dims, L, st), "deslice (stored weights)");
  return PA_OK;
}

pa_status pa_deslice_backward_w(const pa_dims* dims, const void* W, const void* dY, float* dSp,
                                void* ws, size_t ws_bytes, void* stream) {
  PA_TRY(check_dims(dims));
  PA_TRY(check_ptr(W, "W", true));
  PA_TRY(check_ptr(dY, "dY", true));
  PA_TRY(check_ptr(dSp, "dSp", true));
  PA_TRY(check_pass(*dims, pa::kDesliceBwdW));
  PA_TRY(check_ws(*dims, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  pa::StreamLaunch L = stream_of(*dims, pa::kDesliceBwdW, nullptr, W, nullptr, ws);
  L.dY = dY;
  PA_HIP(run_stream(pa::kDesliceBwdW, *dims, L, st), "deslice backward (stored weights)");
  pa::Segments seg{};
  seg.dst[0] = dSp; seg.len[0] = (int64_t)dims->M * dims->C;
  seg.n = 1;
  PA_HIP(pa::launch_reduce(L.partials, L.P, L.rec, seg, st), "reduce");
  return PA_OK;
}

static pa_status check_attn(const pa_dims* dims, const float* S, const pa_attn_params* ap) {
  PA_TRY(check_dims(dims));
  if (!ap) return fail(PA_ERR_INVALID, "attention params are NULL");
  PA_TRY(check_ptr(S, "S", true));
  PA_TRY(check_ptr(ap->Wq, "Wq", true));
  PA_TRY(check_ptr(ap->Wk, "Wk", true));
  PA_TRY(check_ptr(ap->Wv, "Wv", true));
  PA_TRY(check_ptr(ap->bq, "bq", false));
  PA_TRY(check_ptr(ap->bk, "bk", false));
  PA_TRY(check_ptr(ap->bv, "bv", false));
  PA_TRY(check_ptr(ap->Wo, "Wo", false));
  PA_TRY(check_ptr(ap->bo, "bo", false));
  if (ap->bo && !ap->Wo) return fail(PA_ERR_INVALID, "bo given without Wo");
  return PA_OK;
}

namespace {
struct AttnWs {
  float *Q, *K, *V, *O, *dO, *dQ, *dK, *dV, *P;
};
AttnWs attn_ws(const pa_dims& d, void* ws) {
  const size_t mc = (size_t)d.M * d.C;
  float* base = reinterpret_cast<float*>(wsb(ws) + layout_of(d).attn);
  AttnWs a;
  a.Q = base; a.K = base + mc; a.V = base + 2 * mc; a.O = base + 3 * mc;
  a.dO = base + 4 * mc; a.dQ = base + 5 * mc; a.dK = base + 6 * mc; a.dV = base + 7 * mc;
  a.P = base + 8 * mc;
  return a;
}

// General path (heads too large for the fused kernel): Q, K, V, P, O in the
// workspace, O -> Sp when Sp is wanted and there is no output projection.
pa_status attn_forward_general(const pa_dims& d, const float* S, const pa_attn_params* ap,
                               float* Sp, const AttnWs& w, hipStream_t st) {
  const int M = d.M, C = d.C;
  pa::Proj q{};
  q.n = 3; q.M = M; q.Cin = C; q.Cout = C;
  q.in[0] = q.in[1] = q.in[2] = S;
  q.W[0] = ap->Wq; q.W[1] = ap->Wk; q.W[2] = ap->Wv;
  q.b[0] = ap->bq; q.b[1] = ap->bk; q.b[2] = ap->bv;
  q.out[0] = w.Q; q.out[1] = w.K; q.out[2] = w.V;
  PA_HIP(pa::launch_proj(q, st), "QKV projection");
  float* O = (ap->Wo || !Sp) ? w.O : Sp;
  PA_HIP(pa::launch_attn_core(w.Q, w.K, w.V, w.P, O, M, C, d.H, st), "attention core");
  return PA_OK;
}

// Double-precision token forward (fp32 storage): S' feeds the slice
// backward through the differences of nearly equal tokens, where an fp32
// evaluation error of ~1e-7 moves dA by ~1e-5; so Q, K, V, the attention
// and S' are formed in double and S' is rounded once.  The backward's dS
// is ten times less sensitive and keeps the fp32 kernels.  Its matrices
// (as doubles) share the token scratch region.
struct AttnWs64 {
  double *Q, *K, *V, *O, *dO, *dQ, *dK, *dV;
};
AttnWs64 attn_ws64(const pa_dims& d, void* ws) {
  const size_t mc = (size_t)d.M * d.C;
  double* base = reinterpret_cast<double*>(wsb(ws) + layout_of(d).attn);
  return {base, base + mc, base + 2 * mc, base + 3 * mc,
          base + 4 * mc, base + 5 * mc, base + 6 * mc, base + 7 * mc};
}

// (this block has C linkage: no overloads)
pa::Opnd64 opf(const float* p, int64_t rs, int64_t cs) { return {p, rs, cs, 0}; }
pa::Opnd64 opd(const double* p, int64_t rs, int64_t cs) { return {p, rs, cs, 1}; }

// out [rows, cols] = sum_t A_t B_t (+ bias): one product of a batch.
pa::MM64& mm64_add(pa::MM64Batch& b, int rows, int cols, void* out, bool out_dbl,
                   const float* bias = nullptr) {
  pa::MM64& q = b.p[b.n++];
  q = pa::MM64{};
  q.rows = rows; q.cols = cols; q.ld = cols;
  q.out = out; q.out_dbl = out_dbl ? 1 : 0; q.bias = bias;
  return q;
}
void mm64_term(pa::MM64& q, pa::Opnd64 A, pa::Opnd64 B, int K) {
  q.A[q.nt] = A; q.B[q.nt] = B; q.K[q.nt] = K;
  ++q.nt;
}

// Q, K, V = S W + b in double.
pa_status attn64_project(const pa_dims& d, const float* S, const pa_attn_params* ap,
                         const AttnWs64& w, hipStream_t st) {
  const int M = d.M, C = d.C;
  const float* W[3] = {ap->Wq, ap->Wk, ap->Wv};
  const float* bias[3] = {ap->bq, ap->bk, ap->bv};
  double* out[3] = {w.Q, w.K, w.V};
  pa::MM64Batch b{};
  for (int p = 0; p < 3; ++p)
    mm64_term(mm64_add(b, M, C, out[p], true, bias[p]), opf(S, C, 1), opf(W[p], C, 1), C);
  PA_HIP(pa::launch_mm64(b, st), "QKV projection (double)");
  return PA_OK;
}

pa_status attn64_forward(const pa_dims& d, const float* S, const pa_attn_params* ap, float* Sp,
                         void* ws, hipStream_t st) {
  const int M = d.M, C = d.C;
  const AttnWs64 w = attn_ws64(d, ws);
  PA_TRY(attn64_project(d, S, ap, w, st));
  if (!ap->Wo) {
    PA_HIP(pa::launch_core64(w.Q, w.K, w.V, Sp, false, M, C, d.H, st), "attention core (double)");
    return PA_OK;
  }
  PA_HIP(pa::launch_core64(w.Q, w.K, w.V, w.O, true, M, C, d.H, st), "attention core (double)");
  pa::MM64Batch b{};
  mm64_term(mm64_add(b, M, C, Sp, false, ap->bo), opd(w.O, C, 1), opf(ap->Wo, C, 1), C);
  PA_HIP(pa::launch_mm64(b, st), "output projection (double)");
  return PA_OK;
}

pa::HeadArgs head_args(const pa_dims& d, const float* S, const pa_attn_params* ap) {
  pa::HeadArgs h{};
  h.S = S;
  h.W[0] = ap->Wq; h.W[1] = ap->Wk; h.W[2] = ap->Wv;
  h.b[0] = ap->bq; h.b[1] = ap->bk; h.b[2] = ap->bv;
  h.geo.M = d.M; h.geo.C = d.C; h.geo.H = d.H;
  return h;
}
}  // namespace

pa_status pa_token_attention(const pa_dims* dims, const float* S, const pa_attn_params* ap,
                             float* Sp, void* ws, size_t ws_bytes, void* stream) {
  PA_TRY(check_attn(dims, S, ap));
  PA_TRY(check_ptr(Sp, "Sp", true));
  PA_TRY(check_ws(*dims, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  const pa_dims& d = *dims;
  if (d.dtype == PA_F32) return attn64_forward(d, S, ap, Sp, ws, st);
  const AttnWs w = attn_ws(d, ws);
  // the heads' output: straight to Sp without an output projection
  float* O = ap->Wo ? w.O : Sp;
  if (pa::head_fits(d.M, d.C, d.H)) {
    pa::HeadArgs h = head_args(d, S, ap);
    h.O = O;
    PA_HIP(pa::launch_head(h, false, st), "attention heads");
  } else {
    PA_TRY(attn_forward_general(d, S, ap, Sp, w, st));
  }
  if (ap->Wo) {
    pa::Proj o{};
    o.n = 1; o.M = d.M; o.Cin = d.C; o.Cout = d.C;
    o.in[0] = w.O; o.W[0] = ap->Wo; o.b[0] = ap->bo; o.out[0] = Sp;
    PA_HIP(pa::launch_proj(o, st), "output projection");
  }
  return PA_OK;
}

pa_status pa_token_attention_backward(const pa_dims* dims, const float* S,
                                      const pa_attn_params* ap, const float* dSp, float* dS,
                                      const pa_attn_grads* ag, void* ws, size_t ws_bytes,
                                      void* stream) {
  PA_TRY(check_attn(dims, S, ap));
  PA_TRY(check_ptr(dSp, "dSp", true));
  PA_TRY(check_ptr(dS, "dS", true));
  if (ag) {
    const float* gs[] = {ag->dWq, ag->dbq, ag->dWk, ag->dbk, ag->dWv, ag->dbv, ag->dWo, ag->dbo};
    for (const float* p : gs) PA_TRY(check_ptr(p, "attention gradient", false));
  }
  PA_TRY(check_ws(*dims, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  const pa_dims& d = *dims;
  const int M = d.M, C = d.C;
  const AttnWs w = attn_ws(d, ws);
  const float* dO = dSp;
  if (ap->Wo) {
    pa::Proj q{};  // dO = dSp Wo^T
    q.n = 1; q.M = M; q.Cin = C; q.Cout = C; q.transW = 1;
    q.in[0] = dSp; q.W[0] = ap->Wo; q.out[0] = w.dO;
    PA_HIP(pa::launch_proj(q, st), "dO");
    dO = w.dO;
  }
  const bool wantWo = ag && ap->Wo && (ag->dWo || ag->dbo);
  if (pa::head_fits(M, C, d.H)) {
    pa::HeadArgs h = head_args(d, S, ap);  // recomputes the forward per head
    h.dO = dO;
    h.O = wantWo ? w.O : nullptr;
    h.dX[0] = w.dQ; h.dX[1] = w.dK; h.dX[2] = w.dV;
    PA_HIP(pa::launch_head(h, true, st), "attention heads backward");
  } else {
    PA_TRY(attn_forward_general(d, S, ap, nullptr, w, st));  // Q, K, V, P, O
    PA_HIP(pa::launch_attn_core_bwd(w.Q, w.K, w.V, w.P, dO, w.dQ, w.dK, w.dV, M, C, d.H, st),
           "attention core backward");
  }
  // dS = dQ Wq^T + dK Wk^T + dV Wv^T; dW = S^T dX, db = 1^T dX; dWo = O^T dSp
  pa::GradArgs g{};
  g.M = M; g.C = C;
  g.nS = 3; g.dS = dS;
  g.X[0] = w.dQ; g.X[1] = w.dK; g.X[2] = w.dV;
  g.W[0] = ap->Wq; g.W[1] = ap->Wk; g.W[2] = ap->Wv;
  if (ag) {
    float* dW4[4] = {ag->dWq, ag->dWk, ag->dWv, ag->dWo};
    float* db4[4] = {ag->dbq, ag->dbk, ag->dbv, ag->dbo};
    const float* B4[4] = {w.dQ, w.dK, w.dV, dSp};
    const float* A4[4] = {S, S, S, w.O};
    for (int t = 0; t < 4; ++t) {
      if (!dW4[t] && !db4[t]) continue;
      if (t == 3 && !ap->Wo) continue;
      g.A[g.nO] = A4[t]; g.B[g.nO] = B4[t]; g.dW[g.nO] = dW4[t]; g.db[g.nO] = db4[t];
      ++g.nO;
    }
  }
  PA_HIP(pa::launch_token_grads(g, st), "token gradients");
  return PA_OK;
}

pa_status pa_deslice(const pa_dims* dims, const void* x, const void* G,
                     const pa_slice_params* sp, const float* Sp, void* y, void* ws,
                     size_t ws_bytes, void* stream) {
  PA_TRY(check_slice(dims, x, G, sp));
  PA_TRY(check_ptr(Sp, "Sp", true));
  PA_TRY(check_ptr(y, "y", true));
  PA_TRY(check_pass(*dims, pa::kDeslice));
  PA_TRY(check_ws(*dims, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  pa::PrepArgs p = prep_of(*dims, pa::kDeslice, sp, ws);
  p.Sp = Sp;
  PA_HIP(pa::launch_prep(p, st), "prep");
  pa::StreamLaunch L = stream_of(*dims, pa::kDeslice, x, G, sp, ws);
  L.out = y;
  PA_HIP(run_stream(pa::kDeslice, *dims, L, st),
         "deslice");
  return PA_OK;
}

pa_status pa_deslice_backward(const pa_dims* dims, const void* x, const void* G,
                              const pa_slice_params* sp, const void* dY, float* dSp, void* ws,
                              size_t ws_bytes, void* stream) {
  PA_TRY(check_slice(dims, x, G, sp));
  PA_TRY(check_ptr(dY, "dY", true));
  PA_TRY(check_ptr(dSp, "dSp", true));
  PA_TRY(check_pass(*dims, pa::kDesliceBwd));
  PA_TRY(check_ws(*dims, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  PA_HIP(pa::launch_prep(prep_of(*dims, pa::kDesliceBwd, sp, ws), st), "prep");
  pa::StreamLaunch L = stream_of(*dims, pa::kDesliceBwd, x, G, sp, ws);
  L.dY = dY;
  PA_HIP(run_stream(pa::kDesliceBwd, *dims, L, st),
         "deslice backward");
  pa::Segments seg{};
  seg.dst[0] = dSp; seg.len[0] = (int64_t)dims->M * dims->C;
  seg.n = 1;
  PA_HIP(pa::launch_reduce(L.partials, L.P, L.rec, seg, st), "reduce");
  return PA_OK;
}

namespace {
pa_status reduce_slice_grads(const pa_dims& d, const pa::StreamLaunch& L,
                             const pa_slice_grads* gr, hipStream_t st) {
  if (!gr) return PA_OK;
  pa::Segments seg{};
  seg.dst[0] = gr->dA; seg.len[0] = (int64_t)d.C * d.M;
  seg.dst[1] = gr->db; seg.len[1] = d.M;
  seg.dst[2] = gr->da; seg.len[2] = d.C;
  seg.dst[3] = gr->db_t; seg.dst2[3] = gr->dtau0; seg.len[3] = 1;  // d tau0 = d b_t
  seg.n = 4;
  PA_HIP(pa::launch_reduce(L.partials, L.P, L.rec, seg, st), "reduce");
  return PA_OK;
}

pa_status check_grads(const pa_slice_grads* gr) {
  if (!gr) return PA_OK;
  PA_TRY(check_ptr(gr->dA, "dA", false));
  PA_TRY(check_ptr(gr->db, "db", false));
  PA_TRY(check_ptr(gr->da, "da", false));
  if (gr->db_t && ((uintptr_t)gr->db_t & 3u)) return fail(PA_ERR_INVALID, "db_t misaligned");
  if (gr->dtau0 && ((uintptr_t)gr->dtau0 & 3u)) return fail(PA_ERR_INVALID, "dtau0 misaligned");
  return PA_OK;
}
}  // namespace

pa_status pa_slice_aggregate_backward(const pa_dims* dims, const void* x, const void* G,
                                      const pa_slice_params* sp, const float* num,
                                      const float* den, const float* dS, const float* Sp,
                                      const void* dY, void* dx, const pa_slice_grads* gr,
                                      void* ws, size_t ws_bytes, void* stream) {
  PA_TRY(check_slice(dims, x, G, sp));
  PA_TRY(check_ptr(dS, "dS", false));
  PA_TRY(check_ptr(Sp, "Sp", false));
  PA_TRY(check_ptr(dY, "dY", false));
  PA_TRY(check_ptr(dx, "dx", true));
  if ((Sp == nullptr) != (dY == nullptr))
    return fail(PA_ERR_INVALID, "Sp and dY must both be given or both be NULL");
  if (dS) {
    PA_TRY(check_ptr(num, "num", true));
    PA_TRY(check_ptr(den, "den", true));
  }
  PA_TRY(check_grads(gr));
  PA_TRY(check_pass(*dims, pa::kSliceBwd));
  PA_TRY(check_ws(*dims, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  pa::PrepArgs p = prep_of(*dims, pa::kSliceBwd, sp, ws);
  p.num = num;
  p.den = den;
  p.dS = dS;
  p.Sp = Sp;
  PA_HIP(pa::launch_prep(p, st), "prep");
  pa::StreamLaunch L = stream_of(*dims, pa::kSliceBwd, x, G, sp, ws);
  L.dY = dY;
  L.out = dx;
  L.states = dS != nullptr;
  L.deslice = Sp != nullptr;
  PA_HIP(run_stream(pa::kSliceBwd, *dims, L, st),
         "slice backward");
  return reduce_slice_grads(*dims, L, gr, st);
}

// ---------------------------------------------------------------------------
// Per-head batches: `heads` independent layers of one head each (dims: one
// head), x, G, y, dY, dx, the states and the gradients stacked head after
// head; head h's table image and partial records in its own copy of the
// one-head workspace.  Every launch covers all heads (blockIdx.y = head).
// ---------------------------------------------------------------------------
namespace {
struct HeadsCall {
  int heads = 1;
  int64_t sx = 0, sg = 0, sMD = 0, sM = 0, sA = 0, sb = 0, sa = 0;  // byte strides
  int64_t wtot = 0;                                                // workspace per head
};

pa_status check_heads(const pa_dims* dims, int heads, const void* x, const void* G,
                      const pa_heads_params* hp, HeadsCall& hc) {
  PA_TRY(check_dims(dims));
  const pa_dims& d = *dims;
  if (heads < 1 || heads > pa::kMaxHeads)
    return fail(PA_ERR_INVALID, "heads must be in [1, %d] (got %d)", pa::kMaxHeads, heads);
  if (d.M % 8) return fail(PA_ERR_INVALID, "per-head calls need M a multiple of 8 (got %d)", d.M);
  if (!hp) return fail(PA_ERR_INVALID, "per-head slice params are NULL");
  PA_TRY(check_ptr(x, "x", true));
  PA_TRY(check_ptr(G, "G", false));
  PA_TRY(check_ptr(hp->A, "A", true));
  PA_TRY(check_ptr(hp->b, "b", false));
  PA_TRY(check_ptr(hp->a, "a", false));
  if (hp->b_t && ((uintptr_t)hp->b_t & 3u)) return fail(PA_ERR_INVALID, "b_t misaligned");
  const int64_t sz = d.dtype == PA_BF16 ? 2 : 4;
  hc.heads = heads;
  hc.sx = d.N * d.C * sz;
  hc.sg = d.N * d.M * sz;
  hc.sMD = (int64_t)d.M * d.C * 4;
  hc.sM = (int64_t)d.M * 4;
  hc.sA = hp->shared ? 0 : (int64_t)d.C * d.M * sz;
  hc.sb = hp->shared ? 0 : (int64_t)d.M * 4;
  hc.sa = hp->shared ? 0 : (int64_t)d.C * sz;
  hc.wtot = (int64_t)layout_of(d).total;
  return PA_OK;
}

pa_status check_heads_ws(const pa_dims& d, int heads, const void* ws, size_t ws_bytes) {
  const size_t need = layout_of(d).total * (size_t)heads;
  if (!ws) return fail(PA_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", need);
  if (ws_bytes < need)
    return fail(PA_ERR_WORKSPACE, "workspace too small: %zu < %zu bytes", ws_bytes, need);
  if (((uintptr_t)ws & (kAlign - 1)) != 0)
    return fail(PA_ERR_INVALID, "workspace is not %zu-byte aligned", kAlign);
  return PA_OK;
}

pa::PrepArgs heads_prep(const pa_dims& d, int pass, const pa_heads_params* hp,
                        const HeadsCall& hc, void* ws) {
  pa::PrepArgs p = prep_of(d, pass, nullptr, ws);
  p.A = hp->A;
  p.b = hp->b;
  p.a = hp->a;
  p.heads = hc.heads;
  p.hs_A = hc.sA; p.hs_b = hc.sb; p.hs_a = hc.sa;
  p.hs_Sp = p.hs_num = p.hs_dS = hc.sMD;
  p.hs_den = hc.sM;
  p.hs_img = hc.wtot;
  return p;
}

pa::StreamLaunch heads_stream(const pa_dims& d, int pass, const void* x, const void* G,
                              const pa_heads_params* hp, const HeadsCall& hc, void* ws) {
  pa::StreamLaunch L = stream_of(d, pass, x, G, nullptr, ws);
  L.heads = hc.heads;
  L.hs_x = L.hs_dy = L.hs_out = hc.sx;
  L.hs_g = hc.sg;
  L.hs_img = L.hs_part = hc.wtot;
  // tau0 + b_t in double, b_t the head's device scalar (as b_t_dev adds it)
  L.tb = (double)d.tau0;
  L.tb_dev = hp->b_t;
  L.hs_tb = hp->shared ? 0 : 4;
  return L;
}

pa::Segments heads_segments(const HeadsCall& hc) {
  pa::Segments seg{};
  seg.heads = hc.heads;
  seg.hs_parts = hc.wtot;
  return seg;
}
}  // namespace

pa_status pa_heads_workspace_size(const pa_dims* dims, int heads, size_t* bytes) {
  PA_TRY(check_dims(dims));
  if (heads < 1 || heads > pa::kMaxHeads)
    return fail(PA_ERR_INVALID, "heads must be in [1, %d] (got %d)", pa::kMaxHeads, heads);
  if (!bytes) return fail(PA_ERR_INVALID, "bytes is NULL");
  *bytes = layout_of(*dims).total * (size_t)heads;
  return PA_OK;
}

pa_status pa_heads_slice_aggregate(const pa_dims* dims, int heads, const void* x, const void* G,
                                   const pa_heads_params* hp, float* num, float* den, float* S,
                                   void* ws, size_t ws_bytes, void* stream) {
  HeadsCall hc;
  PA_TRY(check_heads(dims, heads, x, G, hp, hc));
  PA_TRY(check_ptr(num, "num", true));
  PA_TRY(check_ptr(den, "den", true));
  PA_TRY(check_ptr(S, "S", true));
  PA_TRY(check_pass(*dims, pa::kAggregate));
  PA_TRY(check_heads_ws(*dims, heads, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  const pa_dims& d = *dims;
  PA_HIP(pa::launch_prep(heads_prep(d, pa::kAggregate, hp, hc, ws), st), "prep");
  pa::StreamLaunch L = heads_stream(d, pa::kAggregate, x, G, hp, hc, ws);
  PA_HIP(run_stream(pa::kAggregate, d, L, st), "per-head slice aggregate");
  pa::Segments seg = heads_segments(hc);
  seg.dst[0] = num; seg.len[0] = (int64_t)d.M * d.C; seg.hs_dst[0] = hc.sMD;
  seg.dst[1] = den; seg.len[1] = d.M; seg.hs_dst[1] = hc.sM;
  seg.n = 2;
  seg.S = S; seg.hs_S = hc.sMD;
  seg.nS = (int64_t)d.M * d.C;
  seg.den_col = seg.nS;
  seg.C = d.C;
  seg.eps = d.eps;
  PA_HIP(pa::launch_reduce(L.partials, L.P, L.rec, seg, st), "reduce");
  return PA_OK;
}

pa_status pa_heads_deslice(const pa_dims* dims, int heads, const void* x, const void* G,
                           const pa_heads_params* hp, const float* Sp, void* y, void* ws,
                           size_t ws_bytes, void* stream) {
  HeadsCall hc;
  PA_TRY(check_heads(dims, heads, x, G, hp, hc));
  PA_TRY(check_ptr(Sp, "Sp", true));
  PA_TRY(check_ptr(y, "y", true));
  PA_TRY(check_pass(*dims, pa::kDeslice));
  PA_TRY(check_heads_ws(*dims, heads, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  const pa_dims& d = *dims;
  pa::PrepArgs p = heads_prep(d, pa::kDeslice, hp, hc, ws);
  p.Sp = Sp;
  PA_HIP(pa::launch_prep(p, st), "prep");
  pa::StreamLaunch L = heads_stream(d, pa::kDeslice, x, G, hp, hc, ws);
  L.out = y;
  PA_HIP(run_stream(pa::kDeslice, d, L, st), "per-head deslice");
  return PA_OK;
}

pa_status pa_heads_deslice_backward(const pa_dims* dims, int heads, const void* x, const void* G,
                                    const pa_heads_params* hp, const void* dY, float* dSp,
                                    void* ws, size_t ws_bytes, void* stream) {
  HeadsCall hc;
  PA_TRY(check_heads(dims, heads, x, G, hp, hc));
  PA_TRY(check_ptr(dY, "dY", true));
  PA_TRY(check_ptr(dSp, "dSp", true));
  PA_TRY(check_pass(*dims, pa::kDesliceBwd));
  PA_TRY(check_heads_ws(*dims, heads, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  const pa_dims& d = *dims;
  PA_HIP(pa::launch_prep(heads_prep(d, pa::kDesliceBwd, hp, hc, ws), st), "prep");
  pa::StreamLaunch L = heads_stream(d, pa::kDesliceBwd, x, G, hp, hc, ws);
  L.dY = dY;
  PA_HIP(run_stream(pa::kDesliceBwd, d, L, st), "per-head deslice backward");
  pa::Segments seg = heads_segments(hc);
  seg.dst[0] = dSp; seg.len[0] = (int64_t)d.M * d.C; seg.hs_dst[0] = hc.sMD;
  seg.n = 1;
  PA_HIP(pa::launch_reduce(L.partials, L.P, L.rec, seg, st), "reduce");
  return PA_OK;
}

pa_status pa_heads_slice_aggregate_backward(const pa_dims* dims, int heads, const void* x,
                                            const void* G, const pa_heads_params* hp,
                                            const float* num, const float* den, const float* dS,
                                            const float* Sp, const void* dY, void* dx,
                                            const pa_slice_grads* gr, void* ws, size_t ws_bytes,
                                            void* stream) {
  HeadsCall hc;
  PA_TRY(check_heads(dims, heads, x, G, hp, hc));
  PA_TRY(check_ptr(dS, "dS", false));
  PA_TRY(check_ptr(Sp, "Sp", false));
  PA_TRY(check_ptr(dY, "dY", false));
  PA_TRY(check_ptr(dx, "dx", true));
  if ((Sp == nullptr) != (dY == nullptr))
    return fail(PA_ERR_INVALID, "Sp and dY must both be given or both be NULL");
  if (dS) {
    PA_TRY(check_ptr(num, "num", true));
    PA_TRY(check_ptr(den, "den", true));
  }
  PA_TRY(check_grads(gr));
  PA_TRY(check_pass(*dims, pa::kSliceBwd));
  PA_TRY(check_heads_ws(*dims, heads, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  const pa_dims& d = *dims;
  pa::PrepArgs p = heads_prep(d, pa::kSliceBwd, hp, hc, ws);
  p.num = num;
  p.den = den;
  p.dS = dS;
  p.Sp = Sp;
  PA_HIP(pa::launch_prep(p, st), "prep");
  pa::StreamLaunch L = heads_stream(d, pa::kSliceBwd, x, G, hp, hc, ws);
  L.dY = dY;
  L.out = dx;
  L.states = dS != nullptr;
  L.deslice = Sp != nullptr;
  PA_HIP(run_stream(pa::kSliceBwd, d, L, st), "per-head slice backward");
  if (!gr) return PA_OK;
  pa::Segments seg = heads_segments(hc);
  seg.dst[0] = gr->dA; seg.len[0] = (int64_t)d.C * d.M; seg.hs_dst[0] = (int64_t)d.C * d.M * 4;
  seg.dst[1] = gr->db; seg.len[1] = d.M; seg.hs_dst[1] = (int64_t)d.M * 4;
  seg.dst[2] = gr->da; seg.len[2] = d.C; seg.hs_dst[2] = (int64_t)d.C * 4;
  seg.dst[3] = gr->db_t; seg.dst2[3] = gr->dtau0; seg.len[3] = 1;  // d tau0 = d b_t
  seg.hs_dst[3] = seg.hs_dst2[3] = 4;
  seg.n = 4;
  PA_HIP(pa::launch_reduce(L.partials, L.P, L.rec, seg, st), "reduce");
  return PA_OK;
}

pa_status pa_slice_weights_backward(const pa_dims* dims, const void* x, const void* G,
                                    const pa_slice_params* sp, const float* dW,
                                    const float* dtau, void* dx, const pa_slice_grads* gr,
                                    void* ws, size_t ws_bytes, void* stream) {
  PA_TRY(check_slice(dims, x, G, sp));
  PA_TRY(check_ptr(dW, "dW", true));
  PA_TRY(check_ptr(dtau, "dtau", false));
  PA_TRY(check_ptr(dx, "dx", true));
  PA_TRY(check_grads(gr));
  PA_TRY(check_pass(*dims, pa::kWeightsBwd));
  PA_TRY(check_ws(*dims, ws, ws_bytes));
  hipStream_t st = as_stream(stream);
  PA_HIP(pa::launch_prep(prep_of(*dims, pa::kWeightsBwd, sp, ws), st), "prep");
  pa::StreamLaunch L = stream_of(*dims, pa::kWeightsBwd, x, G, sp, ws);
  L.dW = dW;
  L.dtau = dtau;
  L.out = dx;
  PA_HIP(run_stream(pa::kWeightsBwd, *dims, L, st),
         "slice weights backward");
  return reduce_slice_grads(*dims, L, gr, st);
}

}  // extern "C"
