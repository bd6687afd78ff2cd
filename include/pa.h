/*
 * pa.h -- C ABI of the MI355X (gfx950) Physics-Attention hot path.
 *
 * One Transolver++ Physics-Attention layer ("Transolver++: An Accurate Neural
 * Solver for PDEs on Million-Scale Geometries", arXiv 2502.02414), forward and
 * backward, for N mesh points with C channels, M slices and H heads:
 *
 *   t_i   = tau0 + a.x_i + b_t,  tau_i = max(t_i, tau_min)      Eq. 3 (Ada-Temp)
 *   w_i   = softmax_j((x_i A + b + g_i) / tau_i)                Eq. 4 (Rep-Slice)
 *   num_j = sum_i w_ij x_i,  den_j = sum_i w_ij,
 *   s_j   = num_j / max(den_j, eps)                              Eq. 1, as the
 *           partial sums of Section 4.2 (Algorithm 1, states step)
 *   s'    = multi-head attention among the M states              Eq. 2
 *   y_i   = sum_j w_ij s'_j                                      deslice, Section 3
 *
 * The backward calls are the chain rule of the above (the paper gives none).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Every tensor argument is a DEVICE pointer owned by the caller, row-major
 *   and contiguous, 16-byte aligned.  Structs and scalars are host memory.
 * - `dims->dtype` (pa_dtype) is the storage type of the point-side tensors
 *   x [N,C], G [N,M], y [N,C], dY [N,C], dx [N,C] and of the slice
 *   projection A [C,M] and a [C].  Everything else -- b [M], tokens [M,C],
 *   num, den, attention parameters and every parameter gradient -- is fp32.
 *   Arithmetic accumulates in fp32 (MFMA with fp32 accumulation).
 * - Weights use the x*W ("in, out") layout: A is [C,M], W_q is [C,C].
 * - G is the Gumbel sample g = -log(-log U), passed in as data so runs are
 *   reproducible; NULL means no noise.  a = NULL means t_i = tau0 + b_t
 *   (Transolver's constant temperature when b_t = 0).  b = NULL means 0.
 * - Outputs are overwritten, never accumulated, and must not alias inputs.
 * - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *   stream).  The library never allocates, frees or synchronises device
 *   memory.  Calls that take a workspace need at least
 *   pa_workspace_size(dims) bytes of device memory; a workspace must not be
 *   shared by calls that may run concurrently.
 * - Results are deterministic: identical inputs give bitwise identical
 *   outputs (fixed point partition that depends on N only, fixed-order
 *   reductions, no floating-point atomics).
 * - Arguments are validated on the host before anything is launched:
 *   N >= 1; 1 <= M <= 64; H >= 1 and C % H == 0; tau_min > 0; eps > 0;
 *   required pointers non-NULL; workspace large enough.  Served channel
 *   counts: C a multiple of 16 in [16, 256] (other C >= 1 return
 *   PA_ERR_UNSUPPORTED; C = 256 with M > 48 in fp32 does not fit the slice
 *   backward's on-chip tables either).  Failures return PA_ERR_INVALID,
 *   PA_ERR_UNSUPPORTED or
 *   PA_ERR_WORKSPACE and set the thread-local message of pa_last_error().
 *   A failed HIP launch returns PA_ERR_HIP with HIP's message.  Non-finite
 *   input values propagate; there are no device-side checks.
 */
#ifndef PA_H
#define PA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PA_VERSION 8

typedef enum { PA_F32 = 0, PA_BF16 = 1 } pa_dtype;

typedef enum {
  PA_OK = 0,
  PA_ERR_INVALID = -1,     /* bad argument value or NULL pointer           */
  PA_ERR_UNSUPPORTED = -2, /* valid, but a shape the library does not serve */
  PA_ERR_WORKSPACE = -3,   /* workspace smaller than pa_workspace_size     */
  PA_ERR_HIP = -4          /* a HIP runtime call or launch failed          */
} pa_status;

/* Layer dimensions and scalars (host struct). */
typedef struct {
  int64_t N;      /* mesh points                                  */
  int32_t C;      /* channels                                     */
  int32_t H;      /* heads of the token attention (D = C / H)     */
  int32_t M;      /* slices (physical states)                     */
  float tau0;     /* temperature constant of Eq. 3                */
  float tau_min;  /* temperature floor: tau = max(t, tau_min)     */
  float eps;      /* denominator floor: s = num / max(den, eps)   */
  int32_t dtype;  /* pa_dtype of the point-side tensors and A, a  */
} pa_dims;

/* Slice projection (Eq. 4 Linear) and Ada-Temp projection (Eq. 3 Linear). */
typedef struct {
  const void* A;  /* [C,M] dtype, required                        */
  const float* b; /* [M] fp32, nullable (0)                       */
  const void* a;  /* [C] dtype, nullable (0)                      */
  float b_t;      /* scalar bias of the Ada-Temp projection       */
  const float* b_t_dev; /* nullable: a device fp32 scalar added to b_t
                           (e.g. the bias term of a folded Project step,
                           pa_project_fold), read by the streaming kernels */
} pa_slice_params;

/* Token attention parameters (Eq. 2), all fp32 [C,C] / [C]. */
typedef struct {
  const float *Wq, *bq; /* W required, b nullable */
  const float *Wk, *bk;
  const float *Wv, *bv;
  const float *Wo, *bo; /* Wo NULL: no output projection (s' = heads) */
} pa_attn_params;

/* Gradients of the slice and Ada-Temp projections; fp32; each nullable. */
typedef struct {
  float* dA;    /* [C,M] */
  float* db;    /* [M]   */
  float* da;    /* [C]   */
  float* db_t;  /* [1]   */
  float* dtau0; /* [1], equal to db_t */
} pa_slice_grads;

/* Gradients of the token attention parameters; fp32; each nullable. */
typedef struct {
  float *dWq, *dbq;
  float *dWk, *dbk;
  float *dWv, *dbv;
  float *dWo, *dbo; /* only written when the forward had Wo */
} pa_attn_grads;

/* Library version (PA_VERSION). */
int pa_version(void);

/* Thread-local message of the last failed call on this thread ("" if none). */
const char* pa_last_error(void);

/* Bytes of device workspace that every call below needs at these dims. */
pa_status pa_workspace_size(const pa_dims* dims, size_t* bytes);

/* Eq. 3 + Eq. 4 written out: W [N,M] fp32 (rows sum to 1) and, if tau is
 * not NULL, the clamped temperature tau [N] fp32.  For tests and
 * diagnostics; the fused calls below never write W. */
pa_status pa_slice_weights(const pa_dims* dims, const void* x, const void* G,
                           const pa_slice_params* sp, float* W, float* tau,
                           void* ws, size_t ws_bytes, void* stream);

/* Eq. 3 + Eq. 4 + Eq. 1 fused in one streaming pass over x and G (the
 * weights stay on chip), reduced over fixed point chunks in a fixed order
 * (the partial-sum form of Section 4.2): num [M,C], den [M], S [M,C], all
 * fp32. */
pa_status pa_slice_aggregate(const pa_dims* dims, const void* x, const void* G,
                             const pa_slice_params* sp, float* num, float* den,
                             float* S, void* ws, size_t ws_bytes, void* stream);

/* Eq. 2: Q,K,V = S W_q + b_q, ...; per head h (channels [hD, hD+D)),
 * softmax(Q_h K_h^T / sqrt(D)) V_h; heads concatenated; then, if Wo is
 * given, Sp = O W_o + b_o.  S, Sp [M,C] fp32. */
pa_status pa_token_attention(const pa_dims* dims, const float* S,
                             const pa_attn_params* ap, float* Sp, void* ws,
                             size_t ws_bytes, void* stream);

/* Deslice (Section 3) with the weights recomputed from x and G exactly as
 * in pa_slice_aggregate: y [N,C] (dtype) = W Sp. */
pa_status pa_deslice(const pa_dims* dims, const void* x, const void* G,
                     const pa_slice_params* sp, const float* Sp, void* y,
                     void* ws, size_t ws_bytes, void* stream);

/* Backward of the deslice, token half: dSp [M,C] fp32 = W^T dY, with the
 * weights recomputed.  (The weight half, dY Sp^T, is folded into
 * pa_slice_aggregate_backward.) */
pa_status pa_deslice_backward(const pa_dims* dims, const void* x,
                              const void* G, const pa_slice_params* sp,
                              const void* dY, float* dSp, void* ws,
                              size_t ws_bytes, void* stream);

/* Backward of Eq. 2 (recomputes the forward from S): dS [M,C] fp32 and the
 * parameter gradients requested in *ag (ag may be NULL). */
pa_status pa_token_attention_backward(const pa_dims* dims, const float* S,
                                      const pa_attn_params* ap,
                                      const float* dSp, float* dS,
                                      const pa_attn_grads* ag, void* ws,
                                      size_t ws_bytes, void* stream);

/* Backward of the slice side of the layer, in one streaming pass with the
 * weights recomputed.  With dw_ij = <dY_i, Sp_j> + <x_i, dnum_j> + dden_j
 * (dnum_j = dS_j / max(den_j, eps); dden_j = -<dS_j, S_j>/den_j when
 * den_j >= eps, else 0), it writes
 *   dx_i = sum_j w_ij dnum_j + A dl_i + a dt_i        (dx [N,C] dtype)
 * and the projection gradients in *gr (gr may be NULL), where dl, dt are
 * the chain rule of Eq. 4 and Eq. 3.  num, den are pa_slice_aggregate's
 * outputs.  dS may be NULL (no states term); Sp and dY must both be NULL
 * (no deslice term) or both be given. */
pa_status pa_slice_aggregate_backward(const pa_dims* dims, const void* x,
                                      const void* G, const pa_slice_params* sp,
                                      const float* num, const float* den,
                                      const float* dS, const float* Sp,
                                      const void* dY, void* dx,
                                      const pa_slice_grads* gr, void* ws,
                                      size_t ws_bytes, void* stream);

/* Backward of pa_slice_weights: from dW [N,M] fp32 and optional dtau [N]
 * fp32 (the gradient of the clamped temperature), dx [N,C] dtype =
 * A dl + a dt and the projection gradients in *gr (nullable). */
pa_status pa_slice_weights_backward(const pa_dims* dims, const void* x,
                                    const void* G, const pa_slice_params* sp,
                                    const float* dW, const float* dtau,
                                    void* dx, const pa_slice_grads* gr,
                                    void* ws, size_t ws_bytes, void* stream);

/* Stored-weights variant of the forward and of the deslice backward.
 * Algorithm 1 computes the weights once and reuses them in the deslice;
 * the calls above recompute them from x and G in every pass instead.
 * These three calls store them once: W [N,M] in dtype (row-major, exactly
 * the weights the aggregate contracted, i.e. rounded to dtype), written by
 * pa_slice_aggregate_w, then read by pa_deslice_w and pa_deslice_backward_w
 * in place of x and G (64 B per point at M = 32 in bf16 instead of 576).
 * pa_slice_aggregate_backward needs x anyway and recomputes them as before.
 * W is caller-owned device memory, 16-byte aligned, and must not alias any
 * other argument.  Results equal those of the recomputing calls up to the
 * fp32 accumulation order.
 *
 * pa_slice_aggregate_w: pa_slice_aggregate, plus W written. */
pa_status pa_slice_aggregate_w(const pa_dims* dims, const void* x, const void* G,
                               const pa_slice_params* sp, float* num, float* den,
                               float* S, void* W, void* ws, size_t ws_bytes,
                               void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * computation as pa_slice_aggregate, bit for bit, with no workspace
 * argument.  Its table image and per-block partial records live in a
 * static device array of the library (17 MiB on each device it runs on,
 * held until the process ends); the call allocates and frees nothing.
 * Shapes whose scratch would exceed the array return PA_ERR_UNSUPPORTED
 * (every shape the layer calls serve fits).  The first call on a device
 * looks up the array's address there (hipGetSymbolAddress, with that device
 * current; the stream must belong to the current device) and keeps it.
 * Every call on one device uses that device's one array: calls that overlap
 * on a device (other streams, other threads) race and must be ordered by
 * the caller.  Nothing in the array has to start at zero: every call
 * rewrites what it reads. */
pa_status pa_slice_aggregate_noalloc(const pa_dims* dims, const void* x, const void* G,
                                     const pa_slice_params* sp, float* num, float* den,
                                     float* S, void* stream);

/* pa_deslice_w: y = W Sp (the deslice of Section 3) from a stored W [N,M]
 * dtype; y [N,C] dtype.  dims->tau0, tau_min and eps are not used. */
pa_status pa_deslice_w(const pa_dims* dims, const void* W, const float* Sp, void* y,
                       void* ws, size_t ws_bytes, void* stream);

/* pa_deslice_backward_w: dSp [M,C] fp32 = W^T dY from a stored W [N,M]
 * dtype and dY [N,C] dtype. */
pa_status pa_deslice_backward_w(const pa_dims* dims, const void* W, const void* dY,
                                float* dSp, void* ws, size_t ws_bytes, void* stream);

/* Diagnostics: time the streaming kernel of one entry point with the
 * caller's HIP events (hipEvent_t passed as void*), without a profiler.
 * While armed, every later call on this thread of the entry point named
 * `call` (pa_slice_weights, pa_slice_aggregate, pa_deslice,
 * pa_deslice_backward, pa_slice_aggregate_backward,
 * pa_slice_weights_backward, pa_slice_aggregate_w, pa_deslice_w or
 * pa_deslice_backward_w) records `start` on its stream right before
 * its streaming kernel and `stop` right after it, so hipEventElapsedTime
 * gives that kernel's duration alone (without the table set-up and the
 * partial-sum reduction around it).  The events stay owned by the caller
 * and must outlive the calls they time; re-arming replaces the pair.
 * call = NULL disarms.  An unknown name or a NULL event returns
 * PA_ERR_INVALID and leaves the hook as it was.  Host-only: it launches
 * nothing. */
pa_status pa_time_kernel(const char* call, void* start, void* stop);

/* Diagnostics: the memory traffic of one streaming pass with none of its
 * arithmetic, the rate its access pattern reaches on its own (what the
 * pass would reach if its arithmetic were free; the achievable bandwidth
 * its roofline fraction is read against).  For call = pa_slice_aggregate,
 * pa_deslice, pa_deslice_backward or pa_slice_aggregate_backward, it runs
 * one kernel that moves the point tensors that call's per-wave streaming
 * kernel reads and writes at these dims exactly as that kernel does: the
 * same blocks and waves, tile ranges, tile height, register prefetch depth,
 * walk direction and cache hints of its 16-byte loads, the rows staged in
 * LDS, and its output rows written back from an LDS tile.  Nothing is
 * computed: out [N,C] dtype (pa_deslice, pa_slice_aggregate_backward;
 * otherwise unused, may be NULL) receives the rows of x.  x [N,C] dtype,
 * dY [N,C] dtype (pa_deslice_backward, pa_slice_aggregate_backward; may be
 * NULL otherwise), G [N,M] dtype or NULL (no noise); no workspace.  Shapes
 * whose call runs a block-cooperative kernel (bf16, C = 256, M > 32) are
 * probed with the per-wave kernel's split.  An unknown call returns
 * PA_ERR_INVALID. */
pa_status pa_stream_probe(const pa_dims* dims, const char* call, const void* x,
                          const void* dY, const void* G, void* out, void* stream);

/* ---------------------------------------------------------------------
 * Block-stack primitives.  A Transolver++ block is the Transformer block
 * with Physics-Attention in place of attention (Section 3; the block
 * diagram of Figure 2a), read here as pre-norm with residual adds:
 *   x1 = x + PA(LN1(x)),  x2 = x1 + GELU(LN2(x1) W1 + b1) W2 + b2,
 * where PA starts with Algorithm 1's Project step x_proj = h Wp + bp.  The
 * stack runner (paper_2502_02414_amd/stack.py) composes these calls with
 * the layer's calls above.  Same conventions as above (device pointers,
 * 16-byte aligned, asynchronous on `stream`, host validation first);
 * parameters are fp32 unless said otherwise; "dtype" tensors are bf16 or
 * fp32.  Sums over rows are per-block partial sums added in block order
 * (bitwise deterministic), except inside hipBLASLt.
 * --------------------------------------------------------------------- */

/* Row-major D[m,n] = alpha op(A) op(B) + beta C (+ bias[n] added to every
 * row), op(X) = X^T when trans; A is [m,k] ([k,m] when transA), B [k,n]
 * ([n,k] when transB); C [m,n] in D's dtype (nullable: C = D, in place;
 * a residual add when it is another tensor and beta = 1).  The plain GEMMs of the MLP and the linear layers,
 * on hipBLASLt (fp32 accumulation).  The first call on a device creates
 * one hipBLASLt handle there (kept until the process ends); ws/ws_bytes is
 * hipBLASLt's workspace (may be 0).  pa_gemm itself never synchronises: a
 * problem (shape, dtypes, transposes, bias) that pa_gemm_prepare has not
 * tuned runs hipBLASLt's first heuristic candidate.  A long reduction into a small fp32 output (transA, K >= 2^17, D at most
 * 8 MB, beta = 0, no bias: the weight gradients) is split over K into up to
 * 64 partial products kept at the end of ws (at most half of it) and added
 * in order, deterministically.  A combination of dtypes hipBLASLt does
 * not serve returns PA_ERR_UNSUPPORTED. */
pa_status pa_gemm(int transA, int transB, int64_t m, int64_t n, int64_t k, float alpha,
                  const void* A, pa_dtype a_dtype, const void* B, pa_dtype b_dtype,
                  float beta, const void* C, void* D, pa_dtype d_dtype, const float* bias,
                  void* ws, size_t ws_bytes, void* stream);

/* pa_gemm, and the tuning of its problem (same arguments, same result):
 * up to 8 of hipBLASLt's candidate algorithms are timed on `stream` (the
 * stream is synchronised) and the fastest is kept for every later pa_gemm
 * of that problem on this device, unless D is also the accumulated input
 * (beta != 0, C = D: the first candidate is kept).  It also creates the
 * device's hipBLASLt handle: calling it once per problem before a timed or
 * captured loop leaves pa_gemm with no allocation and no synchronisation. */
pa_status pa_gemm_prepare(int transA, int transB, int64_t m, int64_t n, int64_t k, float alpha,
                          const void* A, pa_dtype a_dtype, const void* B, pa_dtype b_dtype,
                          float beta, const void* C, void* D, pa_dtype d_dtype,
                          const float* bias, void* ws, size_t ws_bytes, void* stream);

/* LayerNorm over the C channels of each of N rows (biased variance):
 * s = x (+ r when r is given, rounded to dtype and written to xs when xs is
 * given: the residual add that precedes a block's LayerNorm), y = (s -
 * mean) / sqrt(var + eps) * g + b (g, b [C] nullable: 1, 0); mean, rstd [N]
 * are saved for the backward.  C a power of two, 16 <= C <= 256 (fp32) or
 * 512 (bf16). */
pa_status pa_layernorm(int64_t N, int C, float eps, pa_dtype dtype, const void* x,
                       const void* r, void* xs, const float* g, const float* b, void* y,
                       float* mean, float* rstd, void* stream);

/* Chain rule of pa_layernorm (x = the normalised input s): dx = the
 * LayerNorm backward of dy, plus dres when given (the residual branch's
 * gradient); dg, db [C] (nullable) need at most 1024 * 2C floats of
 * workspace (one partial record per block). */
pa_status pa_layernorm_backward(int64_t N, int C, pa_dtype dtype, const void* x,
                                const float* g, const float* mean, const float* rstd,
                                const void* dy, const void* dres, void* dx, float* dg,
                                float* db, void* ws, size_t ws_bytes, void* stream);

/* GELU in its exact form y = x Phi(x) = x (1 + erf(x / sqrt 2)) / 2 over n
 * elements (n a multiple of 16 bytes' worth), and its chain rule
 * dx = dy GELU'(x), GELU'(x) = Phi(x) + x phi(x). */
pa_status pa_gelu(int64_t n, pa_dtype dtype, const void* x, void* y, void* stream);
pa_status pa_gelu_backward(int64_t n, pa_dtype dtype, const void* x, const void* dy, void* dx,
                           void* stream);

/* The first product of the block's feed-forward layer (Figure 2a) with
 * its activation, as one kernel (bf16 storage, fp32 accumulation):
 * G [N,F] = GELU(X W1 + b1), X [N,K] and W1 [K,F] bf16, b1 [F] fp32,
 * K in {64, 128, 256}, F a positive multiple of 64, all pointers 16-byte
 * aligned.  GELU(u) = u Phi(u) is applied to the fp32 accumulator (Phi
 * from an erf approximation with absolute error below 1.5e-7) and rounded
 * to bf16 once; the pre-activation u is not written.  ws: at least 2 F K
 * bytes (W1 transposed), caller-owned, clobbered.  bf16 only: with fp32
 * storage the stack uses pa_gemm and pa_gelu.  Unserved K or F return
 * PA_ERR_UNSUPPORTED. */
pa_status pa_mlp_up(int64_t N, int K, int F, const void* X, const void* W1, const float* b1,
                    void* G, void* ws, size_t ws_bytes, void* stream);
/* Its chain rule with the pre-activation recomputed from X:
 * dU [N,F] = (dY W2^T) GELU'(X W1 + b1), dY [N,K] and W2 [F,K] bf16 (the
 * second product's input gradient and weight), the rest as pa_mlp_up. */
pa_status pa_mlp_up_backward(int64_t N, int K, int F, const void* X, const void* W1,
                             const float* b1, const void* dY, const void* W2, void* dU,
                             void* ws, size_t ws_bytes, void* stream);

/* out[c] = sum over the N rows of x [N,C] (the bias gradient of a linear
 * layer; C a multiple of 16 bytes' worth, at most 256 x 16 bytes);
 * workspace min(N, 1024) * C floats. */
pa_status pa_colsum(int64_t N, int C, pa_dtype dtype, const void* x, float* out, void* ws,
                    size_t ws_bytes, void* stream);

/* Algorithm 1's Project step x_proj = h Wp + bp (Wp [C,C], bp [C]) folded
 * into the slice parameters (A [C,M], b [M] nullable, a [C] nullable, all
 * fp32): A_out = Wp A (dtype), b_out = b + bp A, a_out = Wp a (dtype),
 * b_t_out[0] = bp.a (fp32 device scalar, for pa_slice_params.b_t_dev).  The
 * logits and temperature of x_proj are then those of h under the folded
 * parameters, so the layer's streaming calls run on h. */
pa_status pa_project_fold(const pa_dims* dims, const float* Wp, const float* bp,
                          const float* A, const float* b, const float* a, void* A_out,
                          float* b_out, void* a_out, float* b_t_out, void* stream);

/* The states of x_proj from those of h: S_proj [M,C] = S Wp + bp (each
 * point's weights sum to 1; exact for every slice with den >= eps). */
pa_status pa_project_states(const pa_dims* dims, const float* S, const float* Wp,
                            const float* bp, float* S_proj, void* stream);

/* Chain rule of pa_project_fold and pa_project_states: from the gradients
 * of the folded parameters (*folded: dA, db, da, db_t, as
 * pa_slice_aggregate_backward returns them for the folded call) and of the
 * projected states dS_proj [M,C]: dWp [C,C], dbp [C], dS [M,C] (nullable;
 * dS_proj Wp^T, the states gradient that pa_slice_aggregate_backward
 * takes, which a caller forms before that call, e.g. with pa_gemm) and the
 * gradients of the unfolded parameters in *gr (dA required; db, da, db_t
 * nullable). */
pa_status pa_project_backward(const pa_dims* dims, const float* Wp, const float* bp,
                              const float* A, const float* a, const float* S,
                              const float* dS_proj, const pa_slice_grads* folded, float* dWp,
                              float* dbp, float* dS, const pa_slice_grads* gr, void* stream);

/* ---------------------------------------------------------------------
 * Per-head slicing: the heads of Eq. 2 carried into the slicing of Eq. 1.
 * The C channels split into H contiguous blocks of D = C/H.  Head h slices
 * its own block x_h [N,D] with its own slice parameters and Gumbel noise
 * [N,M] (Eq. 3, Eq. 4), forms its own M states [M,D] (Eq. 1) and deslices
 * them into the channels of its block; the token attention is one head of
 * width D with projections shared by the heads (Eq. 2's Linear acting on
 * the last axis of the [H,M,D] states).  On the GPU each head runs the
 * layer's streaming calls above on x_h stored head-major ([H,N,D], dims
 * with C = D, H = 1), and the token attention of all heads is one
 * pa_token_attention call (dims with C = H D and H heads) on the heads'
 * states side by side, [M, H D], with the shared D x D projections on the
 * block diagonal.  The runner (paper_2502_02414_amd/heads.py) composes
 * these calls.  Same conventions as above.
 * --------------------------------------------------------------------- */

/* Moves R rows of H blocks of D elements between the point-major layout
 * [R,H,D] (= [R, H D]) and the head-major layout [H,R,D]: to_heads = 1
 * reads src as [R,H,D] and writes dst as [H,R,D], 0 the reverse.  D a
 * multiple of 16 bytes' worth; src and dst 16-byte aligned and disjoint
 * (PA_ERR_INVALID otherwise).  A plain copy, bit-exact. */
pa_status pa_heads_relayout(int64_t R, int H, int D, pa_dtype dtype, int to_heads,
                            const void* src, void* dst, void* stream);

/* One fp32 parameter shared by the heads, laid out for all H of them:
 * blockdiag = 1 takes a D x D matrix (L = D) and writes the [H D, H D]
 * matrix with it in every diagonal block and zeros elsewhere (the token
 * projection of the H-head call); blockdiag = 0 takes L floats and writes
 * them H times, [H,L] (a bias).  H L at most 4096 for a matrix; src, dst
 * 4-byte aligned. */
pa_status pa_heads_expand(int H, int64_t L, int blockdiag, const float* src, float* dst,
                          void* stream);

/* The gradient of a parameter shared by the heads, from the H-head
 * gradient: blockdiag = 1 sums the H diagonal D x D blocks of an [H D, H D]
 * matrix (L = D; the off-diagonal blocks belong to no parameter);
 * blockdiag = 0 sums src [H,L] over its first axis (per-head gradients of
 * a vector or, with L = 1, a scalar).  Added in head order in double
 * precision, rounded once to fp32. */
pa_status pa_heads_sum(int H, int64_t L, int blockdiag, const float* src, float* dst,
                       void* stream);

/* Up to 8 pa_heads_sum in one launch (a layer's shared-parameter gradients
 * at once): item i sums items[i].src into items[i].dst with its own L and
 * blockdiag, each exactly as pa_heads_sum does it (same order, same bits).
 * n in [1, 8]; items is a host array, read before the call returns; every
 * item is validated as pa_heads_sum validates its arguments. */
typedef struct {
  const float* src;
  float* dst;
  int64_t L;
  int blockdiag;
} pa_heads_sum_item;
pa_status pa_heads_sum_batch(int H, int n, const pa_heads_sum_item* items, void* stream);

/* ---------------------------------------------------------------------
 * Per-head slicing in one launch per kernel.  The calls below run the
 * layer's aggregate, deslice, deslice backward and slice backward for all
 * `heads` heads of a per-head sliced layer together (1 <= heads <= 16):
 * `dims` describes ONE head (C = D channels, H = 1, M slices per head; M a
 * multiple of 8), and every per-head tensor is stacked head after head:
 * x, y, dY, dx [heads][N][D] (dtype), G [heads][N][M] (dtype, nullable),
 * num, S, Sp, dSp, dS [heads][M][D] and den [heads][M] (fp32), the slice
 * gradients dA [heads][D][M], db [heads][M], da [heads][D], db_t and
 * dtau0 [heads] (fp32, *gr pointing at head 0's).  Each head's results are
 * bit for bit those of the one-head call on its own tensors (same kernels,
 * same ordered sums).  The workspace holds one one-head workspace per head
 * (pa_heads_workspace_size).  Errors as in the one-head calls.
 * --------------------------------------------------------------------- */

/* The heads' slice parameters, stacked: A [heads][D][M] and a [heads][D]
 * (dtype; a nullable), b [heads][M] and b_t [heads] (fp32 device arrays,
 * nullable: 0; b_t is added to tau0 in double on the GPU, as
 * pa_slice_params.b_t_dev, and not validated on the host).  With shared = 1
 * one set serves every head: A [D][M], a [D], b [M], b_t [1]. */
typedef struct {
  const void* A;
  const float* b;
  const void* a;
  const float* b_t;
  int shared;
} pa_heads_params;

pa_status pa_heads_workspace_size(const pa_dims* dims, int heads, size_t* bytes);

/* Eq. 1 per head (as pa_slice_aggregate). */
pa_status pa_heads_slice_aggregate(const pa_dims* dims, int heads, const void* x, const void* G,
                                   const pa_heads_params* hp, float* num, float* den, float* S,
                                   void* ws, size_t ws_bytes, void* stream);
/* The deslice per head (as pa_deslice). */
pa_status pa_heads_deslice(const pa_dims* dims, int heads, const void* x, const void* G,
                           const pa_heads_params* hp, const float* Sp, void* y, void* ws,
                           size_t ws_bytes, void* stream);
/* Chain rule of the deslice per head (as pa_deslice_backward). */
pa_status pa_heads_deslice_backward(const pa_dims* dims, int heads, const void* x, const void* G,
                                    const pa_heads_params* hp, const void* dY, float* dSp,
                                    void* ws, size_t ws_bytes, void* stream);
/* Chain rule of Eq. 1, 3 and 4 per head (as pa_slice_aggregate_backward;
 * the gradients per head, a shared parameter's to be summed over the heads
 * with pa_heads_sum). */
pa_status pa_heads_slice_aggregate_backward(const pa_dims* dims, int heads, const void* x,
                                            const void* G, const pa_heads_params* hp,
                                            const float* num, const float* den, const float* dS,
                                            const float* Sp, const void* dY, void* dx,
                                            const pa_slice_grads* gr, void* ws, size_t ws_bytes,
                                            void* stream);

#ifdef __cplusplus
}
#endif
#endif /* PA_H */
