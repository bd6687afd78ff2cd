// Internal launch interface between the C-ABI layer (pa_api.cpp) and the
// kernels (pa_stream.hip, pa_small.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pa {

// Heads of one batched per-head call (pa_heads_*): head h = blockIdx.y of
// every launch, its tensors at fixed byte strides from head 0's.
constexpr int kMaxHeads = 16;

struct StreamLaunch {
  const void* x = nullptr;
  const void* G = nullptr;
  const void* dY = nullptr;
  const void* img = nullptr;
  void* out = nullptr;
  float* tau_out = nullptr;
  const float* dW = nullptr;
  const float* dtau = nullptr;
  float* partials = nullptr;
  int64_t N = 0;
  int M = 0;
  int cr = 0;   // channels of the point rows (<= the kernels' C, a multiple of 16)
  int rec = 0;
  int P = 1;
  double tb = 0.0;  // tau0 + b_t
  const float* tb_dev = nullptr;  // nullable device scalar added to tb
  float tau_min = 0.f;
  bool states = false;
  bool deslice = false;
  // per-head batch: heads (gridDim.y), byte strides of x, G, dY, out, the
  // table image, the partial records and tb_dev (each head's b_t)
  int heads = 1;
  int64_t hs_x = 0, hs_g = 0, hs_dy = 0, hs_out = 0, hs_img = 0, hs_part = 0, hs_tb = 0;
};

// Streaming passes (pass = pa::Pass).  dtype: 0 fp32, 1 bf16.
// C is the width the kernels are built for (32, 64, 128 or 256); rows of
// L.cr <= C channels are laid out in LDS as C channels, the others zero in
// the tables.
hipError_t launch_stream(int pass, int dtype, int C, int MB, const StreamLaunch& L,
                         hipStream_t st);
// Waves per block of a pass at this shape (0 = shape not served); cr the
// channels of the point rows.
int stream_waves(int pass, int dtype, int C, int MB, int cr);

// Stream probe (pa_probe.hip): the per-wave kernel of `pass` (kAggregate,
// kDeslice, kDesliceBwd or kSliceBwd) with its loads and stores and no
// arithmetic; probe_waves is its block's waves (0 = not served).
int probe_waves(int pass, int dtype, int C, int MB);
hipError_t launch_probe(int pass, int dtype, int C, int MB, const StreamLaunch& L,
                        hipStream_t st);

// Table image for a pass, written into `img` (device).
struct PrepArgs {
  int pass = 0;
  int dtype = 0;
  int C = 0, M = 0, MB = 0;  // C: the tables' (padded) width
  int cr = 0;                // channels of the parameters and states (<= C)
  float eps = 0.f;
  const void* A = nullptr;    // [cr,M] dtype
  const float* b = nullptr;   // [M]
  const void* a = nullptr;    // [cr] dtype
  const float* Sp = nullptr;  // [M,cr]  (kDeslice, kSliceBwd deslice term)
  const float* num = nullptr; // [M,cr]  (kSliceBwd states term)
  const float* den = nullptr; // [M]
  const float* dS = nullptr;  // [M,cr]
  void* img = nullptr;
  // per-head batch: heads (gridDim.y) and byte strides (0: shared by heads)
  int heads = 1;
  int64_t hs_A = 0, hs_b = 0, hs_a = 0, hs_Sp = 0, hs_num = 0, hs_den = 0, hs_dS = 0, hs_img = 0;
};
hipError_t launch_prep(const PrepArgs& p, hipStream_t st);
// Bytes of the table image of a pass.
size_t image_bytes(int pass, int dtype, int C, int MB);

// out[k] = sum_{p < P} partials[p * rec + k] (k < rec), in order p = 0..P-1,
// scattered into up to 6 destination segments (each written to dst[i] and,
// if given, also to dst2[i]).  With S set, the first nS columns are the
// numerators [M,C] of Eq. 1 and the states S = num / max(den, eps) are
// written too, den_j being column den_col + j reduced in the same order.
struct Segments {
  float* dst[6];
  float* dst2[6];
  int64_t len[6];
  int n;
  float* S;
  int64_t nS, den_col;
  int C;
  float eps;
  // per-head batch (heads < 2: one): byte strides of the partial records,
  // the destinations and S
  int heads;
  int64_t hs_parts, hs_dst[6], hs_dst2[6], hs_S;
};
hipError_t launch_reduce(const float* partials, int P, int64_t rec, const Segments& seg,
                         hipStream_t st);

// Token-side products (fp32, M <= 64 rows):
//   sum = 0: out_p [M,Cout] = in_p [M,Cin] op(W_p) + b_p   for p < n
//   sum = 1: out_0 [M,Cout] = sum_p in_p op(W_p) + b_0
//   op(W) = W ([Cin,Cout]) or, with transW, W^T (W given as [Cout,Cin]).
struct Proj {
  const float* in[3];
  const float* W[3];
  const float* b[3];
  float* out[3];
  int n, M, Cin, Cout, transW, sum;
};
hipError_t launch_proj(const Proj& q, hipStream_t st);
// Fused per-head token attention (one block per head, channels [hD, hD+D)):
//   forward:  O_h = softmax(Q_h K_h^T / sqrt(D)) V_h with [Q|K|V]_h = S W_h + b_h
//   backward: the same forward, then dQ_h, dK_h, dV_h from dO_h (and O_h if
//             O is given).
// M, C, H are set by the caller; launch_head fills the rest of the geometry
// and returns hipErrorInvalidConfiguration when a head does not fit on chip
// (head_fits tells beforehand).
struct HeadGeo {
  int M, C, H, D;
  int M16, D16, MT, NT, T;  // padded rows / head columns, projection tiles
  int KC, SR;               // K chunk, chunk row stride (floats)
  size_t lds;
};
struct HeadArgs {
  const float* S;     // [M,C]
  const float* W[3];  // Wq, Wk, Wv [C,C]
  const float* b[3];  // [C], nullable
  const float* dO;    // [M,C] (backward)
  float* O;           // [M,C] forward output; backward: nullable
  float* dX[3];       // dQ, dK, dV [M,C] (backward)
  HeadGeo geo;
};
bool head_fits(int M, int C, int H);
hipError_t launch_head(HeadArgs a, bool bwd, hipStream_t st);
// Parameter-side products of the token backward, one launch:
//   dS = sum_{p < nS} X_p W_p^T           (X_p [M,C], W_p [C,C]; dS [M,C])
//   dW_p = A_p^T B_p, db_p = 1^T B_p      (p < nO; A_p, B_p [M,C]; NULL
//                                          outputs skipped)
struct GradArgs {
  const float* X[3];
  const float* W[3];
  int nS;
  float* dS;
  const float* A[4];
  const float* B[4];
  float* dW[4];
  float* db[4];
  int nO;
  int M, C;
};
hipError_t launch_token_grads(const GradArgs& a, hipStream_t st);
// Per-head attention core: P_h = softmax(Q_h K_h^T * scale), O_h = P_h V_h.
hipError_t launch_attn_core(const float* Q, const float* K, const float* V, float* P, float* O,
                            int M, int C, int H, hipStream_t st);
// Per-head attention backward core: from dO, P, Q, K, V -> dQ, dK, dV.
hipError_t launch_attn_core_bwd(const float* Q, const float* K, const float* V,
                                const float* P, const float* dO, float* dQ, float* dK,
                                float* dV, int M, int C, int H, hipStream_t st);

// Token attention forward in double precision (pa_tokens64.hip; the
// fp32-storage path).
// Operand element (i, k) = p[i rs + k cs], fp32 or fp64; p == NULL: all ones.
struct Opnd64 {
  const void* p;
  int64_t rs, cs;
  int dbl;
};
// out[i, j] (row stride ld, fp32 or fp64) = sum_{t < nt} sum_{k < K_t}
// A_t(i, k) B_t(k, j) + bias[j] (bias nullable), i < rows, j < cols.
struct MM64 {
  Opnd64 A[3], B[3];
  int K[3];
  int nt;
  const float* bias;
  void* out;
  int out_dbl;
  int rows, cols;
  int64_t ld;
};
constexpr int kMM64Max = 3;
struct MM64Batch {
  MM64 p[kMM64Max];
  int n;
};
hipError_t launch_mm64(const MM64Batch& b, hipStream_t st);
// Per head h (channels [hD, hD + D)): O_h = softmax(Q_h K_h^T / sqrt(D)) V_h
// (O fp32 or fp64); Q, K, V: [M,C] fp64.
hipError_t launch_core64(const double* Q, const double* K, const double* V, void* O, bool O_dbl,
                         int M, int C, int H, hipStream_t st);

// Sets the thread-local message of pa_last_error() (pa_api.cpp).
void set_last_error(const char* msg);

// ---- Block stack (pa_block.hip, pa_gemm.cpp) ----
// LayerNorm over C channels: forward (s = x + r, optional; y = LN(s);
// mean/rstd saved) or backward (dx = LN'(dy) + dres; dg/db partial records
// of 2C floats per block, `blocks` = layernorm_blocks(...) of them).
struct LayerNormArgs {
  int64_t N = 0;
  int C = 0;
  float eps = 1e-5f;
  const void* x = nullptr;
  const void* r = nullptr;
  void* xs = nullptr;
  const float* g = nullptr;
  const float* b = nullptr;
  void* y = nullptr;
  float* mean = nullptr;
  float* rstd = nullptr;
  const void* dy = nullptr;
  const void* dres = nullptr;
  void* dx = nullptr;
  float* partials = nullptr;
  int blocks = 0;
};
hipError_t launch_layernorm(const LayerNormArgs& a, int dtype, bool bwd, hipStream_t st);
// Blocks (= partial records of the backward) of the LayerNorm launches, and
// of the column sums; at most kLnPartials records.
constexpr int kLnPartials = 1024;
int layernorm_blocks(int64_t N, int C, int dtype, bool bwd);
int colsum_blocks(int64_t N);
// out = GELU(x), or out = dy GELU'(x) when dy is given (n a multiple of 16 B).
hipError_t launch_gelu(int64_t n, int dtype, const void* x, const void* dy, void* out,
                       hipStream_t st);
// Per-block column sums of x [N,C] (P records of C floats).
hipError_t launch_colsum(int64_t N, int C, int dtype, const void* x, float* partials, int P,
                         hipStream_t st);
// The MLP's first product with its activation (pa_mlp.hip, bf16): forward
// (DY == NULL) out = GELU(X W1 + b1); backward out = (DY W2^T) GELU'(X W1 +
// b1).  X, DY [N, K]; W1 [K, F]; W2 [F, K]; b1 [F]; out [N, F]; W1T: F K
// bf16 of scratch for W1 transposed.
bool mlp_up_served(int K, int F);
hipError_t launch_mlp_up(int64_t N, int K, int F, const void* X, const void* W1, const float* b1,
                         const void* DY, const void* W2, void* out, void* W1T, hipStream_t st);
// Project folding (fp32 parameters; A_out, a_out in dtype).
struct FoldArgs {
  int C = 0, M = 0;
  const float *Wp = nullptr, *bp = nullptr, *A = nullptr, *b = nullptr, *a = nullptr;
  void* A_out = nullptr;
  void* a_out = nullptr;
  float* b_out = nullptr;
  float* bt_out = nullptr;
};
hipError_t launch_fold(const FoldArgs& f, int dtype, hipStream_t st);
hipError_t launch_project_states(int M, int C, const float* S, const float* Wp, const float* bp,
                                 float* Sp, hipStream_t st);
struct FoldGradArgs {
  int C = 0, M = 0;
  const float *Wp = nullptr, *bp = nullptr, *A = nullptr, *a = nullptr, *S = nullptr;
  const float *dSp = nullptr, *dAf = nullptr, *dbf = nullptr, *daf = nullptr, *dbtf = nullptr;
  float *dWp = nullptr, *dbp = nullptr, *dA = nullptr, *db = nullptr, *da = nullptr;
  float *dbt = nullptr, *dS = nullptr;
};
hipError_t launch_fold_grads(const FoldGradArgs& f, hipStream_t st);
// Per-head slicing layout: [R,H,D] <-> [H,R,D] (D elements a multiple of
// 16 bytes), a shared fp32 parameter expanded to every head (block-diagonal
// or tiled) and the sum over the heads.
hipError_t launch_heads_relayout(int64_t R, int H, int D, int dtype, int to_heads,
                                 const void* src, void* dst, hipStream_t st);
hipError_t launch_heads_expand(int H, int64_t L, int blockdiag, const float* src, float* dst,
                               hipStream_t st);
// Up to kHeadSumMax head sums in one launch (item blockIdx.y).
constexpr int kHeadSumMax = 8;
struct HeadSumItem {
  const float* src;
  float* dst;
  int64_t L;
  int blockdiag;
};
struct HeadSumBatch {
  HeadSumItem it[kHeadSumMax];
  int n;
};
hipError_t launch_heads_sum_batch(int H, const HeadSumBatch& b, hipStream_t st);
hipError_t launch_heads_sum(int H, int64_t L, int blockdiag, const float* src, float* dst,
                            hipStream_t st);
// Row-major D[m,n] = alpha op(A) op(B) + beta D (+ bias[n]) on hipBLASLt;
// dtypes 0 fp32, 1 bf16.  Returns 0 or a hipblasStatus_t.
struct Gemm {
  bool transA = false, transB = false;
  int64_t m = 0, n = 0, k = 0;
  float alpha = 1.f, beta = 0.f;
  const void* A = nullptr;
  const void* B = nullptr;
  const void* Cin = nullptr;  // beta's input (nullable: D itself), D's dtype and shape
  void* D = nullptr;
  int ta = 0, tb = 0, td = 0;
  const float* bias = nullptr;
  void* ws = nullptr;
  size_t ws_bytes = 0;
};
// tune: time hipBLASLt's candidates for this problem (synchronising st) and
// keep the fastest for later calls; otherwise a problem not tuned before
// takes the heuristic's first candidate (no synchronisation).
int gemm(const Gemm& g, hipStream_t st, bool tune = false);

}  // namespace pa
