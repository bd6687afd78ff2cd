/*
 * Physics-Attention oracle: plain, slow, double-precision CPU evaluation of
 * one Transolver++ Physics-Attention layer and its chain-rule backward.
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists so that the tests, the smoke
 * check and the CPU-baseline leg of the benchmark can check and time the HIP
 * path.  Nothing in the product path may include, link or call it, and it
 * includes, links and calls nothing from the product path.
 *
 * Paper: "Transolver++: An Accurate Neural Solver for PDEs on Million-Scale
 * Geometries" (arXiv 2502.02414).  Equation numbers below are the paper's:
 *   Eq. 1  slice weights and physical states (Section 3)
 *   Eq. 2  attention among the physical states (Section 3)
 *   Eq. 3  Ada-Temp, a per-point temperature (Section 4.1)
 *   Eq. 4  Rep-Slice, the Gumbel-softmax slice weights (Section 4.1)
 *   deslice: x'_i = sum_j w_ij s'_j (Section 3, text after Eq. 2)
 *   sharded states: numerator and denominator as sums of per-shard partial
 *   sums (Section 4.2, parallelism formulation; Algorithm 1)
 * The backward is not given in the paper; it is the chain rule of the above.
 *
 * Conventions: every array is row-major, contiguous, double precision and
 * owned by the caller.  x [N,C]; G [N,M] Gumbel samples (nullable = no noise);
 * A [C,M] and b [M] (nullable = 0) the slice projection; a [C] (nullable = 0)
 * and scalar b_t the Ada-Temp projection; tokens [M,C].  All weights use the
 * x*W ("in, out") layout.  Outputs are overwritten, never accumulated.
 *
 * Readings of points the paper leaves open (each one is listed in the design
 * notes with its reason):
 *   - the temperature is clamped from below: tau_i = max(t_i, tau_min),
 *     t_i = tau0 + a.x_i + b_t; the gradient through the clamp is 0;
 *   - the Gumbel noise is a full [N,M] sample, added to the logits;
 *   - the state denominator is floored: s_j = num_j / max(den_j, eps);
 *   - heads split only the token attention, by contiguous channel blocks of
 *     D = C/H channels, with scale 1/sqrt(D); W_o/b_o optional (NULL = none).
 *
 * Parity: every function here is pinned by the CPU tests (closed forms,
 * invariants, a hand-derived worked example, library routines and finite
 * differences).
 */
#ifndef PA_ORACLE_H
#define PA_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Points per shard in the sharded (partial-sum) evaluation of the states. */
int pao_shard_points(void);

/* Number of OpenMP threads the oracle uses (1 when built without OpenMP). */
int pao_num_threads(void);
void pao_set_num_threads(int n);

/* Eq. 3 + Eq. 4: W [N,M]; tau [N] (nullable) the clamped temperature;
 * t [N] (nullable) the unclamped tau0 + a.x + b_t. */
void pao_slice_weights(int64_t N, int C, int M, double tau0, double tau_min,
                       const double* x, const double* G, const double* A,
                       const double* b, const double* a, double b_t,
                       double* W, double* tau, double* t);

/* Eq. 1 (states), in the sharded form of Section 4.2:
 * num [M,C] = W^T x, den [M] = column sums of W, S = num / max(den, eps). */
void pao_aggregate(int64_t N, int C, int M, double eps, const double* x,
                   const double* W, double* num, double* den, double* S);

/* Eq. 2 with H heads: Q,K,V = S*Wq+bq, ...; per head softmax(QK^T/sqrt(D))V;
 * optional output projection Sp = O*Wo + bo.  W* [C,C]; b* [C] nullable;
 * Wo NULL means Sp = O. */
void pao_token_attention(int M, int C, int H, const double* S,
                         const double* Wq, const double* bq,
                         const double* Wk, const double* bk,
                         const double* Wv, const double* bv,
                         const double* Wo, const double* bo, double* Sp);

/* Deslice: y [N,C] = W Sp. */
void pao_deslice(int64_t N, int C, int M, const double* W, const double* Sp,
                 double* y);

/* Backward of the deslice: dSp [M,C] = W^T dY, dW [N,M] = dY Sp^T. */
void pao_deslice_backward(int64_t N, int C, int M, const double* W,
                          const double* Sp, const double* dY, double* dSp,
                          double* dW);

/* Backward of Eq. 2.  dS [M,C]; every parameter-gradient pointer is
 * nullable (not computed).  dWo/dbo are only meaningful when Wo != NULL. */
void pao_token_attention_backward(int M, int C, int H, const double* S,
                                  const double* Wq, const double* bq,
                                  const double* Wk, const double* bk,
                                  const double* Wv, const double* bv,
                                  const double* Wo, const double* bo,
                                  const double* dSp, double* dS,
                                  double* dWq, double* dbq, double* dWk,
                                  double* dbk, double* dWv, double* dbv,
                                  double* dWo, double* dbo);

/* Backward of Eq. 1 from dS [M,C]: dx [N,C] = W dnum (the direct path
 * through the numerator) and dW [N,M] = x dnum^T + dden. */
void pao_aggregate_backward(int64_t N, int C, int M, double eps,
                            const double* x, const double* W,
                            const double* num, const double* den,
                            const double* dS, double* dx, double* dW);

/* Backward of Eq. 3 + Eq. 4 from dW [N,M] and optional dtau [N] (the
 * gradient of the clamped temperature output):
 * dx [N,C] = A dl + a dt; dA [C,M], db [M], da [C], db_t [1], dtau0 [1]
 * (each nullable). */
void pao_slice_weights_backward(int64_t N, int C, int M, double tau0,
                                double tau_min, const double* x,
                                const double* G, const double* A,
                                const double* b, const double* a, double b_t,
                                const double* dW, const double* dtau,
                                double* dx, double* dA, double* db, double* da,
                                double* db_t, double* dtau0);

/* ---- Block stack (pa_oracle_block.c): the parts of a Transolver++ block
 * around the layer (pre-norm Transformer block with Physics-Attention in
 * place of attention, Section 3 and Figure 2a). */

/* LayerNorm per row over C channels, biased variance; g, b nullable (1, 0);
 * mean, rstd [N] nullable. */
void pao_layernorm(int64_t N, int C, double eps, const double* x, const double* g,
                   const double* b, double* y, double* mean, double* rstd);
/* Its chain rule: dx [N,C], dg [C], db [C] (each nullable). */
void pao_layernorm_backward(int64_t N, int C, double eps, const double* x, const double* g,
                            const double* dy, double* dx, double* dg, double* db);
/* GELU x Phi(x), Phi the standard normal CDF, and its chain rule. */
void pao_gelu(int64_t n, const double* x, double* y);
void pao_gelu_backward(int64_t n, const double* x, const double* dy, double* dx);
/* (The block's Linear layers, y = x W + b, are plain matrix products taken
 * from the host BLAS by the Python wrapper.) */

#ifdef __cplusplus
}
#endif
#endif
