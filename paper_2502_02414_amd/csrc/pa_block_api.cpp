// C ABI of the block-stack primitives (see include/pa.h): host-side
// validation and launches.  The arithmetic runs in pa_block.hip's kernels
// and, for the plain GEMMs, in hipBLASLt.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "pa.h"
#include "pa_internal.h"

namespace {

pa_status err(pa_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
pa_status err(pa_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  pa::set_last_error(buf);
  return s;
}

#define PB_HIP(call, what)                                                      \
  do {                                                                          \
    hipError_t e_ = (call);                                                     \
    if (e_ != hipSuccess) return err(PA_ERR_HIP, "%s: %s", what, hipGetErrorString(e_)); \
  } while (0)
#define PB_TRY(x)                \
  do {                           \
    pa_status s_ = (x);          \
    if (s_ != PA_OK) return s_;  \
  } while (0)

bool a16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

pa_status need(const void* p, const char* name) {
  if (!p) return err(PA_ERR_INVALID, "%s is NULL", name);
  if (!a16(p)) return err(PA_ERR_INVALID, "%s is not 16-byte aligned", name);
  return PA_OK;
}
pa_status opt(const void* p, const char* name) { return p ? need(p, name) : PA_OK; }
pa_status dtype_ok(int dt) {
  return (dt == PA_F32 || dt == PA_BF16) ? PA_OK : err(PA_ERR_INVALID, "dtype must be PA_F32 or PA_BF16");
}

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }


// Partial records -> dst segments, added in block order.
pa_status reduce_to(const float* parts, int P, int64_t rec, float* d0, int64_t l0, float* d1,
                    int64_t l1, hipStream_t st) {
  pa::Segments seg{};
  seg.dst[0] = d0; seg.len[0] = l0;
  seg.n = 1;
  if (d1) {
    seg.dst[1] = d1; seg.len[1] = l1;
    seg.n = 2;
  } else if (l1 > 0) {  // a skipped segment still occupies its place in the record
    seg.dst[1] = nullptr; seg.len[1] = l1;
    seg.n = 2;
  }
  PB_HIP(pa::launch_reduce(parts, P, rec, seg, st), "reduce");
  return PA_OK;
}

}  // namespace

extern "C" {

static pa_status gemm_call(const char* who, bool tune, int transA, int transB, int64_t m,
                           int64_t n, int64_t k, float alpha, const void* A, pa_dtype a_dtype,
                           const void* B, pa_dtype b_dtype, float beta, const void* C, void* D,
                           pa_dtype d_dtype, const float* bias, void* ws, size_t ws_bytes,
                           void* stream) {
  if (m < 1 || n < 1 || k < 1) return err(PA_ERR_INVALID, "%s: m, n, k must be >= 1", who);
  PB_TRY(dtype_ok(a_dtype));
  PB_TRY(dtype_ok(b_dtype));
  PB_TRY(dtype_ok(d_dtype));
  PB_TRY(need(A, "A"));
  PB_TRY(need(B, "B"));
  PB_TRY(opt(C, "C"));
  PB_TRY(need(D, "D"));
  PB_TRY(opt(bias, "bias"));
  if (ws_bytes && !ws) return err(PA_ERR_WORKSPACE, "%s: workspace is NULL", who);
  pa::Gemm g;
  g.transA = transA != 0;
  g.transB = transB != 0;
  g.m = m; g.n = n; g.k = k;
  g.alpha = alpha; g.beta = beta;
  g.A = A; g.B = B; g.Cin = C; g.D = D;
  g.ta = a_dtype; g.tb = b_dtype; g.td = d_dtype;
  g.bias = bias;
  g.ws = ws; g.ws_bytes = ws_bytes;
  const int s = pa::gemm(g, as_stream(stream), tune);
  if (s != 0)
    return err(s == 7 /* HIPBLAS_STATUS_NOT_SUPPORTED */ ? PA_ERR_UNSUPPORTED : PA_ERR_HIP,
               "%s: hipBLASLt status %d (m=%lld n=%lld k=%lld types %d,%d->%d)", who, s,
               (long long)m, (long long)n, (long long)k, a_dtype, b_dtype, d_dtype);
  return PA_OK;
}

pa_status pa_gemm(int transA, int transB, int64_t m, int64_t n, int64_t k, float alpha,
                  const void* A, pa_dtype a_dtype, const void* B, pa_dtype b_dtype, float beta,
                  const void* C, void* D, pa_dtype d_dtype, const float* bias, void* ws,
                  size_t ws_bytes, void* stream) {
  return gemm_call("pa_gemm", false, transA, transB, m, n, k, alpha, A, a_dtype, B, b_dtype, beta,
                   C, D, d_dtype, bias, ws, ws_bytes, stream);
}

pa_status pa_gemm_prepare(int transA, int transB, int64_t m, int64_t n, int64_t k, float alpha,
                          const void* A, pa_dtype a_dtype, const void* B, pa_dtype b_dtype,
                          float beta, const void* C, void* D, pa_dtype d_dtype,
                          const float* bias, void* ws, size_t ws_bytes, void* stream) {
  return gemm_call("pa_gemm_prepare", true, transA, transB, m, n, k, alpha, A, a_dtype, B, b_dtype,
                   beta, C, D, d_dtype, bias, ws, ws_bytes, stream);
}

pa_status pa_layernorm(int64_t N, int C, float eps, pa_dtype dtype, const void* x, const void* r,
                       void* xs, const float* g, const float* b, void* y, float* mean,
                       float* rstd, void* stream) {
  PB_TRY(dtype_ok(dtype));
  if (N < 1 || C < 16 || C > 1024 || (C & (C - 1)))
    return err(PA_ERR_INVALID, "pa_layernorm: N >= 1 and C a power of two in [16, 1024]");
  if (!(eps > 0.f)) return err(PA_ERR_INVALID, "pa_layernorm: eps must be > 0");
  PB_TRY(need(x, "x"));
  PB_TRY(opt(r, "r"));
  PB_TRY(opt(xs, "xs"));
  PB_TRY(need(y, "y"));
  PB_TRY(need(mean, "mean"));
  PB_TRY(need(rstd, "rstd"));
  if (xs && !r) return err(PA_ERR_INVALID, "pa_layernorm: xs needs r");
  if ((dtype == PA_F32 && C > 256) || (dtype == PA_BF16 && C > 512))
    return err(PA_ERR_UNSUPPORTED, "pa_layernorm: a row must fit one wave (16 bytes per lane)");
  pa::LayerNormArgs a;
  a.N = N; a.C = C; a.eps = eps;
  a.x = x; a.r = r; a.xs = xs; a.g = g; a.b = b; a.y = y; a.mean = mean; a.rstd = rstd;
  PB_HIP(pa::launch_layernorm(a, dtype, false, as_stream(stream)), "layernorm");
  return PA_OK;
}

pa_status pa_layernorm_backward(int64_t N, int C, pa_dtype dtype, const void* x, const float* g,
                                const float* mean, const float* rstd, const void* dy,
                                const void* dres, void* dx, float* dg, float* db, void* ws,
                                size_t ws_bytes, void* stream) {
  PB_TRY(dtype_ok(dtype));
  if (N < 1 || C < 16 || C > 1024 || (C & (C - 1)))
    return err(PA_ERR_INVALID, "pa_layernorm_backward: N >= 1 and C a power of two in [16, 1024]");
  if ((dtype == PA_F32 && C > 256) || (dtype == PA_BF16 && C > 512))
    return err(PA_ERR_UNSUPPORTED, "pa_layernorm_backward: a row must fit one wave");
  PB_TRY(need(x, "x"));
  PB_TRY(need(mean, "mean"));
  PB_TRY(need(rstd, "rstd"));
  PB_TRY(need(dy, "dy"));
  PB_TRY(opt(dres, "dres"));
  PB_TRY(need(dx, "dx"));
  const bool sums = dg || db;
  const int P = pa::layernorm_blocks(N, C, dtype, true);
  const size_t need_ws = sums ? (size_t)P * 2 * C * sizeof(float) : 0;
  if (sums && (!ws || ws_bytes < need_ws))
    return err(PA_ERR_WORKSPACE, "pa_layernorm_backward: workspace needs %zu bytes", need_ws);
  pa::LayerNormArgs a;
  a.N = N; a.C = C;
  a.x = x; a.g = g; a.mean = const_cast<float*>(mean); a.rstd = const_cast<float*>(rstd);
  a.dy = dy; a.dres = dres; a.dx = dx;
  a.partials = sums ? reinterpret_cast<float*>(ws) : nullptr;
  a.blocks = P;
  hipStream_t st = as_stream(stream);
  PB_HIP(pa::launch_layernorm(a, dtype, true, st), "layernorm backward");
  if (sums) {
    // records [dg | db]; a NULL output's segment is skipped
    pa::Segments seg{};
    seg.dst[0] = dg; seg.len[0] = C;
    seg.dst[1] = db; seg.len[1] = C;
    seg.n = 2;
    PB_HIP(pa::launch_reduce(a.partials, (int)P, 2 * C, seg, st), "reduce");
  }
  return PA_OK;
}

pa_status pa_gelu(int64_t n, pa_dtype dtype, const void* x, void* y, void* stream) {
  PB_TRY(dtype_ok(dtype));
  const int E = dtype == PA_BF16 ? 8 : 4;
  if (n < 1 || n % E) return err(PA_ERR_INVALID, "pa_gelu: n must be a positive multiple of %d", E);
  PB_TRY(need(x, "x"));
  PB_TRY(need(y, "y"));
  PB_HIP(pa::launch_gelu(n, dtype, x, nullptr, y, as_stream(stream)), "gelu");
  return PA_OK;
}

pa_status pa_gelu_backward(int64_t n, pa_dtype dtype, const void* x, const void* dy, void* dx,
                           void* stream) {
  PB_TRY(dtype_ok(dtype));
  const int E = dtype == PA_BF16 ? 8 : 4;
  if (n < 1 || n % E)
    return err(PA_ERR_INVALID, "pa_gelu_backward: n must be a positive multiple of %d", E);
  PB_TRY(need(x, "x"));
  PB_TRY(need(dy, "dy"));
  PB_TRY(need(dx, "dx"));
  PB_HIP(pa::launch_gelu(n, dtype, x, dy, dx, as_stream(stream)), "gelu backward");
  return PA_OK;
}

static pa_status mlp_up(const char* who, int64_t N, int K, int F, const void* X,
                        const void* W1, const float* b1, const void* dY, const void* W2,
                        void* out, void* ws, size_t ws_bytes, void* stream) {
  if (N < 1) return err(PA_ERR_INVALID, "%s: N must be >= 1", who);
  if (!pa::mlp_up_served(K, F))
    return err(PA_ERR_UNSUPPORTED, "%s: K must be 64, 128 or 256 and F a multiple of 64", who);
  const void* ps[] = {X, W1, b1, out, ws};
  const char* names[] = {"X", "W1", "b1", "out", "ws"};
  for (int i = 0; i < 5; ++i) {
    PB_TRY(need(ps[i], names[i]));
    if (!a16(ps[i])) return err(PA_ERR_INVALID, "%s: %s must be 16-byte aligned", who, names[i]);
  }
  if (dY) {
    PB_TRY(need(W2, "W2"));
    if (!a16(dY) || !a16(W2)) return err(PA_ERR_INVALID, "%s: dY and W2 must be 16-byte aligned", who);
  }
  const size_t need_ws = (size_t)2 * F * K;
  if (ws_bytes < need_ws) return err(PA_ERR_WORKSPACE, "%s: workspace needs %zu bytes", who, need_ws);
  PB_HIP(pa::launch_mlp_up(N, K, F, X, W1, b1, dY, W2, out, ws, as_stream(stream)), who);
  return PA_OK;
}

pa_status pa_mlp_up(int64_t N, int K, int F, const void* X, const void* W1, const float* b1,
                    void* G, void* ws, size_t ws_bytes, void* stream) {
  return mlp_up("pa_mlp_up", N, K, F, X, W1, b1, nullptr, nullptr, G, ws, ws_bytes, stream);
}

pa_status pa_mlp_up_backward(int64_t N, int K, int F, const void* X, const void* W1,
                             const float* b1, const void* dY, const void* W2, void* dU,
                             void* ws, size_t ws_bytes, void* stream) {
  PB_TRY(need(dY, "dY"));
  return mlp_up("pa_mlp_up_backward", N, K, F, X, W1, b1, dY, W2, dU, ws, ws_bytes, stream);
}

pa_status pa_colsum(int64_t N, int C, pa_dtype dtype, const void* x, float* out, void* ws,
                    size_t ws_bytes, void* stream) {
  PB_TRY(dtype_ok(dtype));
  const int E = dtype == PA_BF16 ? 8 : 4;
  if (N < 1 || C < E || C % E || C / E > 256)
    return err(PA_ERR_INVALID, "pa_colsum: C must be a multiple of %d, at most %d", E, 256 * E);
  PB_TRY(need(x, "x"));
  PB_TRY(need(out, "out"));
  const int P = pa::colsum_blocks(N);
  const size_t need_ws = (size_t)P * C * sizeof(float);
  if (!ws || ws_bytes < need_ws)
    return err(PA_ERR_WORKSPACE, "pa_colsum: workspace needs %zu bytes", need_ws);
  hipStream_t st = as_stream(stream);
  float* parts = reinterpret_cast<float*>(ws);
  PB_HIP(pa::launch_colsum(N, C, dtype, x, parts, P, st), "colsum");
  PB_TRY(reduce_to(parts, P, C, out, C, nullptr, 0, st));
  return PA_OK;
}

pa_status pa_project_fold(const pa_dims* dims, const float* Wp, const float* bp, const float* A,
                          const float* b, const float* a, void* A_out, float* b_out,
                          void* a_out, float* b_t_out, void* stream) {
  if (!dims) return err(PA_ERR_INVALID, "dims is NULL");
  PB_TRY(dtype_ok(dims->dtype));
  if (dims->C < 1 || dims->M < 1 || dims->M > 64) return err(PA_ERR_INVALID, "bad C or M");
  PB_TRY(need(Wp, "Wp"));
  PB_TRY(need(bp, "bp"));
  PB_TRY(need(A, "A"));
  PB_TRY(opt(b, "b"));
  PB_TRY(opt(a, "a"));
  PB_TRY(need(A_out, "A_out"));
  PB_TRY(need(b_out, "b_out"));
  PB_TRY(need(a_out, "a_out"));
  PB_TRY(need(b_t_out, "b_t_out"));
  pa::FoldArgs f;
  f.C = dims->C; f.M = dims->M;
  f.Wp = Wp; f.bp = bp; f.A = A; f.b = b; f.a = a;
  f.A_out = A_out; f.a_out = a_out; f.b_out = b_out; f.bt_out = b_t_out;
  PB_HIP(pa::launch_fold(f, dims->dtype, as_stream(stream)), "project fold");
  return PA_OK;
}

pa_status pa_project_states(const pa_dims* dims, const float* S, const float* Wp, const float* bp,
                            float* S_proj, void* stream) {
  if (!dims) return err(PA_ERR_INVALID, "dims is NULL");
  if (dims->C < 1 || dims->M < 1 || dims->M > 64) return err(PA_ERR_INVALID, "bad C or M");
  PB_TRY(need(S, "S"));
  PB_TRY(need(Wp, "Wp"));
  PB_TRY(need(bp, "bp"));
  PB_TRY(need(S_proj, "S_proj"));
  PB_HIP(pa::launch_project_states(dims->M, dims->C, S, Wp, bp, S_proj, as_stream(stream)),
         "project states");
  return PA_OK;
}

pa_status pa_project_backward(const pa_dims* dims, const float* Wp, const float* bp,
                              const float* A, const float* a, const float* S,
                              const float* dS_proj, const pa_slice_grads* folded, float* dWp,
                              float* dbp, float* dS, const pa_slice_grads* gr, void* stream) {
  if (!dims) return err(PA_ERR_INVALID, "dims is NULL");
  if (dims->C < 1 || dims->M < 1 || dims->M > 64) return err(PA_ERR_INVALID, "bad C or M");
  if (!folded || !gr) return err(PA_ERR_INVALID, "folded and gr are required");
  PB_TRY(need(Wp, "Wp"));
  PB_TRY(need(bp, "bp"));
  PB_TRY(need(A, "A"));
  PB_TRY(opt(a, "a"));
  PB_TRY(need(S, "S"));
  PB_TRY(need(dS_proj, "dS_proj"));
  PB_TRY(need(folded->dA, "folded dA"));
  PB_TRY(need(folded->db, "folded db"));
  PB_TRY(need(folded->da, "folded da"));
  PB_TRY(need(folded->db_t, "folded db_t"));
  PB_TRY(need(dWp, "dWp"));
  PB_TRY(need(dbp, "dbp"));
  PB_TRY(opt(dS, "dS"));
  PB_TRY(need(gr->dA, "dA"));
  pa::FoldGradArgs f;
  f.C = dims->C; f.M = dims->M;
  f.Wp = Wp; f.bp = bp; f.A = A; f.a = a; f.S = S; f.dSp = dS_proj;
  f.dAf = folded->dA; f.dbf = folded->db; f.daf = folded->da; f.dbtf = folded->db_t;
  f.dWp = dWp; f.dbp = dbp; f.dA = gr->dA; f.db = gr->db; f.da = gr->da; f.dbt = gr->db_t;
  f.dS = dS;
  PB_HIP(pa::launch_fold_grads(f, as_stream(stream)), "project backward");
  return PA_OK;
}

pa_status pa_heads_relayout(int64_t R, int H, int D, pa_dtype dtype, int to_heads,
                            const void* src, void* dst, void* stream) {
  PB_TRY(dtype_ok(dtype));
  const int E = dtype == PA_BF16 ? 8 : 4;
  if (R < 1 || H < 1 || D < E || D % E)
    return err(PA_ERR_INVALID, "pa_heads_relayout: R, H >= 1 and D a positive multiple of %d", E);
  PB_TRY(need(src, "src"));
  PB_TRY(need(dst, "dst"));
  const int64_t bytes = R * H * D * (dtype == PA_BF16 ? 2 : 4);
  const uintptr_t s0 = (uintptr_t)src, d0 = (uintptr_t)dst;
  if (s0 < d0 + (uintptr_t)bytes && d0 < s0 + (uintptr_t)bytes)
    return err(PA_ERR_INVALID, "pa_heads_relayout: src and dst overlap");
  PB_HIP(pa::launch_heads_relayout(R, H, D, dtype, to_heads ? 1 : 0, src, dst,
                                   as_stream(stream)), "heads relayout");
  return PA_OK;
}

static pa_status heads_small(const char* what, int H, int64_t L, int blockdiag,
                             const float* src, float* dst) {
  if (H < 1 || L < 1 || (blockdiag && (int64_t)H * L > 4096))
    return err(PA_ERR_INVALID, "%s: H, L >= 1 (H L <= 4096 for a block-diagonal matrix)", what);
  if (!src || !dst) return err(PA_ERR_INVALID, "%s: src and dst are required", what);
  if (((uintptr_t)src & 3u) || ((uintptr_t)dst & 3u))
    return err(PA_ERR_INVALID, "%s: src and dst must be 4-byte aligned", what);
  return PA_OK;
}

pa_status pa_heads_expand(int H, int64_t L, int blockdiag, const float* src, float* dst,
                          void* stream) {
  PB_TRY(heads_small("pa_heads_expand", H, L, blockdiag, src, dst));
  PB_HIP(pa::launch_heads_expand(H, L, blockdiag ? 1 : 0, src, dst, as_stream(stream)),
         "heads expand");
  return PA_OK;
}

pa_status pa_heads_sum(int H, int64_t L, int blockdiag, const float* src, float* dst,
                       void* stream) {
  PB_TRY(heads_small("pa_heads_sum", H, L, blockdiag, src, dst));
  PB_HIP(pa::launch_heads_sum(H, L, blockdiag ? 1 : 0, src, dst, as_stream(stream)),
         "heads sum");
  return PA_OK;
}

pa_status pa_heads_sum_batch(int H, int n, const pa_heads_sum_item* items, void* stream) {
  if (n < 1 || n > pa::kHeadSumMax)
    return err(PA_ERR_INVALID, "pa_heads_sum_batch: n must be in [1, %d] (got %d)",
               pa::kHeadSumMax, n);
  if (!items) return err(PA_ERR_INVALID, "pa_heads_sum_batch: items is NULL");
  pa::HeadSumBatch b{};
  b.n = n;
  for (int i = 0; i < n; ++i) {
    PB_TRY(heads_small("pa_heads_sum_batch", H, items[i].L, items[i].blockdiag, items[i].src,
                       items[i].dst));
    b.it[i] = {items[i].src, items[i].dst, items[i].L, items[i].blockdiag ? 1 : 0};
  }
  PB_HIP(pa::launch_heads_sum_batch(H, b, as_stream(stream)), "heads sum batch");
  return PA_OK;
}

}  // extern "C"
