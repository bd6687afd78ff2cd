/*
 * Physics-Attention oracle (see pa_oracle.h for the contract).
 *
 * TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the
 * CPU-baseline leg of the benchmark; never by the product path.
 *
 * Plain loops in double precision, in the order the paper states the layer.
 * The only restructuring is the one the paper itself gives: the states'
 * numerator and denominator (and, for the backward, every sum over points)
 * are formed as per-shard partial sums added in shard order (Section 4.2),
 * which makes the result independent of the thread count.  A library
 * primitive is never used; exp/log/sqrt come from libm.
 */
#include "pa_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define SHARD 1024 /* points per shard of the Section 4.2 partial sums */

int pao_shard_points(void) { return SHARD; }

int pao_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void pao_set_num_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

static int64_t n_shards(int64_t N) { return (N + SHARD - 1) / SHARD; }

/* ---------------------------------------------------------------------- */
/* Eq. 3 and Eq. 4 for one point.                                          */
/*   l_j   = b_j + sum_c x_c A_cj                 (Linear(x) of Eq. 4)     */
/*   t     = tau0 + b_t + sum_c x_c a_c           (Eq. 3)                  */
/*   tau   = max(t, tau_min)                      (clamp reading)          */
/*   z_j   = (l_j + g_j) / tau                    (Eq. 4, Gumbel added)    */
/*   w_j   = exp(z_j - max z) / sum_k exp(z_k - max z)  (softmax over M)   */
/* ---------------------------------------------------------------------- */
static void point_weights(int C, int M, double tau0, double tau_min,
                          const double* xi, const double* gi, const double* A,
                          const double* b, const double* a, double b_t,
                          double* z, double* w, double* tau_out,
                          double* t_out) {
  double t = tau0 + b_t;
  if (a)
    for (int c = 0; c < C; ++c) t += xi[c] * a[c];
  double tau = t > tau_min ? t : tau_min;
  for (int j = 0; j < M; ++j) {
    double l = b ? b[j] : 0.0;
    for (int c = 0; c < C; ++c) l += xi[c] * A[(int64_t)c * M + j];
    double g = gi ? gi[j] : 0.0;
    z[j] = (l + g) / tau;
  }
  double zmax = z[0];
  for (int j = 1; j < M; ++j)
    if (z[j] > zmax) zmax = z[j];
  double sum = 0.0;
  for (int j = 0; j < M; ++j) {
    w[j] = exp(z[j] - zmax);
    sum += w[j];
  }
  for (int j = 0; j < M; ++j) w[j] /= sum;
  if (tau_out) *tau_out = tau;
  if (t_out) *t_out = t;
}

void pao_slice_weights(int64_t N, int C, int M, double tau0, double tau_min,
                       const double* x, const double* G, const double* A,
                       const double* b, const double* a, double b_t,
                       double* W, double* tau, double* t) {
#pragma omp parallel
  {
    double* z = (double*)malloc(sizeof(double) * M);
#pragma omp for schedule(static)
    for (int64_t i = 0; i < N; ++i)
      point_weights(C, M, tau0, tau_min, x + i * C, G ? G + i * M : NULL, A, b,
                    a, b_t, z, W + i * M, tau ? tau + i : NULL,
                    t ? t + i : NULL);
    free(z);
  }
}

/* ---------------------------------------------------------------------- */
/* Eq. 1 physical states, sharded as in Section 4.2:                       */
/*   num_j = sum_shards sum_{i in shard} w_ij x_i                          */
/*   den_j = sum_shards sum_{i in shard} w_ij                              */
/*   s_j   = num_j / max(den_j, eps)                 (floor reading)       */
/* ---------------------------------------------------------------------- */
void pao_aggregate(int64_t N, int C, int M, double eps, const double* x,
                   const double* W, double* num, double* den, double* S) {
  int64_t P = n_shards(N);
  int64_t part = (int64_t)M * C + M;
  double* parts = (double*)calloc((size_t)(P > 0 ? P : 1) * part, sizeof(double));
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < P; ++p) {
    double* pn = parts + p * part;
    double* pd = pn + (int64_t)M * C;
    int64_t i1 = (p + 1) * SHARD < N ? (p + 1) * SHARD : N;
    for (int64_t i = p * SHARD; i < i1; ++i) {
      const double* xi = x + i * C;
      const double* wi = W + i * M;
      for (int j = 0; j < M; ++j) {
        pd[j] += wi[j];
        for (int c = 0; c < C; ++c) pn[(int64_t)j * C + c] += wi[j] * xi[c];
      }
    }
  }
  memset(num, 0, sizeof(double) * M * C);
  memset(den, 0, sizeof(double) * M);
  for (int64_t p = 0; p < P; ++p) {
    const double* pn = parts + p * part;
    const double* pd = pn + (int64_t)M * C;
    for (int64_t k = 0; k < (int64_t)M * C; ++k) num[k] += pn[k];
    for (int j = 0; j < M; ++j) den[j] += pd[j];
  }
  free(parts);
  for (int j = 0; j < M; ++j) {
    double d = den[j] >= eps ? den[j] : eps;
    for (int c = 0; c < C; ++c) S[(int64_t)j * C + c] = num[(int64_t)j * C + c] / d;
  }
}

/* ---------------------------------------------------------------------- */
/* Eq. 2: attention among the M physical states.                           */
/* ---------------------------------------------------------------------- */

/* out [R,Cout] = in [R,Cin] * Wt [Cin,Cout] + bias (nullable). */
static void affine(int R, int Cin, int Cout, const double* in, const double* Wt,
                   const double* bias, double* out) {
  for (int r = 0; r < R; ++r)
    for (int o = 0; o < Cout; ++o) {
      double s = bias ? bias[o] : 0.0;
      for (int k = 0; k < Cin; ++k) s += in[(int64_t)r * Cin + k] * Wt[(int64_t)k * Cout + o];
      out[(int64_t)r * Cout + o] = s;
    }
}

/* Forward of the attention core; fills Q,K,V,O [M,C] and P [H,M,M]. */
static void attention_core(int M, int C, int H, const double* S,
                           const double* Wq, const double* bq,
                           const double* Wk, const double* bk,
                           const double* Wv, const double* bv, double* Q,
                           double* K, double* V, double* P, double* O) {
  int D = C / H;
  double scale = 1.0 / sqrt((double)D);
  affine(M, C, C, S, Wq, bq, Q);
  affine(M, C, C, S, Wk, bk, K);
  affine(M, C, C, S, Wv, bv, V);
  for (int h = 0; h < H; ++h) {
    double* Ph = P + (int64_t)h * M * M;
    for (int r = 0; r < M; ++r) {
      double mx = -INFINITY;
      for (int c = 0; c < M; ++c) {
        double s = 0.0;
        for (int d = 0; d < D; ++d)
          s += Q[(int64_t)r * C + h * D + d] * K[(int64_t)c * C + h * D + d];
        s *= scale;
        Ph[r * M + c] = s;
        if (s > mx) mx = s;
      }
      double sum = 0.0;
      for (int c = 0; c < M; ++c) {
        Ph[r * M + c] = exp(Ph[r * M + c] - mx);
        sum += Ph[r * M + c];
      }
      for (int c = 0; c < M; ++c) Ph[r * M + c] /= sum;
      for (int d = 0; d < D; ++d) {
        double s = 0.0;
        for (int c = 0; c < M; ++c) s += Ph[r * M + c] * V[(int64_t)c * C + h * D + d];
        O[(int64_t)r * C + h * D + d] = s;
      }
    }
  }
}

void pao_token_attention(int M, int C, int H, const double* S,
                         const double* Wq, const double* bq,
                         const double* Wk, const double* bk,
                         const double* Wv, const double* bv,
                         const double* Wo, const double* bo, double* Sp) {
  size_t mc = (size_t)M * C;
  double* Q = (double*)malloc(sizeof(double) * mc);
  double* K = (double*)malloc(sizeof(double) * mc);
  double* V = (double*)malloc(sizeof(double) * mc);
  double* O = (double*)malloc(sizeof(double) * mc);
  double* P = (double*)malloc(sizeof(double) * (size_t)H * M * M);
  attention_core(M, C, H, S, Wq, bq, Wk, bk, Wv, bv, Q, K, V, P, O);
  if (Wo)
    affine(M, C, C, O, Wo, bo, Sp);
  else
    memcpy(Sp, O, sizeof(double) * mc);
  free(Q); free(K); free(V); free(O); free(P);
}

/* ---------------------------------------------------------------------- */
/* Deslice (Section 3): y_i = sum_j w_ij s'_j.                             */
/* ---------------------------------------------------------------------- */
void pao_deslice(int64_t N, int C, int M, const double* W, const double* Sp,
                 double* y) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < N; ++i)
    for (int c = 0; c < C; ++c) {
      double s = 0.0;
      for (int j = 0; j < M; ++j) s += W[i * M + j] * Sp[(int64_t)j * C + c];
      y[i * C + c] = s;
    }
}

/* ---------------------------------------------------------------------- */
/* Backward (chain rule; the paper gives no backward).                     */
/* ---------------------------------------------------------------------- */

/* y = W Sp:  dSp_jc = sum_i w_ij dY_ic (sharded),  dW_ij = <dY_i, s'_j>. */
void pao_deslice_backward(int64_t N, int C, int M, const double* W,
                          const double* Sp, const double* dY, double* dSp,
                          double* dW) {
  int64_t P = n_shards(N);
  int64_t part = (int64_t)M * C;
  double* parts = (double*)calloc((size_t)(P > 0 ? P : 1) * part, sizeof(double));
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < P; ++p) {
    double* pp = parts + p * part;
    int64_t i1 = (p + 1) * SHARD < N ? (p + 1) * SHARD : N;
    for (int64_t i = p * SHARD; i < i1; ++i)
      for (int j = 0; j < M; ++j) {
        double wij = W[i * M + j];
        double g = 0.0;
        for (int c = 0; c < C; ++c) {
          pp[(int64_t)j * C + c] += wij * dY[i * C + c];
          g += dY[i * C + c] * Sp[(int64_t)j * C + c];
        }
        if (dW) dW[i * M + j] = g;
      }
  }
  memset(dSp, 0, sizeof(double) * part);
  for (int64_t p = 0; p < P; ++p)
    for (int64_t k = 0; k < part; ++k) dSp[k] += parts[p * part + k];
  free(parts);
}

/* Eq. 2 backward.  With O the concatenated head outputs:
 *   Sp = O Wo + bo         -> dO = dSp Wo^T, dWo = O^T dSp, dbo = 1^T dSp
 *   O_h = P_h V_h          -> dV_h = P_h^T dO_h, dP_h = dO_h V_h^T
 *   P_h = softmax(Q_h K_h^T * scale)
 *                          -> dE = P_h o (dP_h - rowsum(dP_h o P_h))
 *                             dQ_h = scale dE K_h, dK_h = scale dE^T Q_h
 *   Q = S Wq + bq (same K, V) -> dS = dQ Wq^T + dK Wk^T + dV Wv^T,
 *                                dWq = S^T dQ, dbq = 1^T dQ (same K, V). */
void pao_token_attention_backward(int M, int C, int H, const double* S,
                                  const double* Wq, const double* bq,
                                  const double* Wk, const double* bk,
                                  const double* Wv, const double* bv,
                                  const double* Wo, const double* bo,
                                  const double* dSp, double* dS,
                                  double* dWq, double* dbq, double* dWk,
                                  double* dbk, double* dWv, double* dbv,
                                  double* dWo, double* dbo) {
  (void)bo;
  int D = C / H;
  double scale = 1.0 / sqrt((double)D);
  size_t mc = (size_t)M * C;
  double* Q = (double*)malloc(sizeof(double) * mc);
  double* K = (double*)malloc(sizeof(double) * mc);
  double* V = (double*)malloc(sizeof(double) * mc);
  double* O = (double*)malloc(sizeof(double) * mc);
  double* P = (double*)malloc(sizeof(double) * (size_t)H * M * M);
  double* dO = (double*)malloc(sizeof(double) * mc);
  double* dQ = (double*)calloc(mc, sizeof(double));
  double* dK = (double*)calloc(mc, sizeof(double));
  double* dV = (double*)calloc(mc, sizeof(double));
  double* dE = (double*)malloc(sizeof(double) * (size_t)M * M);
  attention_core(M, C, H, S, Wq, bq, Wk, bk, Wv, bv, Q, K, V, P, O);

  if (Wo) {
    for (int r = 0; r < M; ++r)
      for (int k = 0; k < C; ++k) {
        double s = 0.0;
        for (int o = 0; o < C; ++o) s += dSp[(int64_t)r * C + o] * Wo[(int64_t)k * C + o];
        dO[(int64_t)r * C + k] = s;
      }
    if (dWo)
      for (int k = 0; k < C; ++k)
        for (int o = 0; o < C; ++o) {
          double s = 0.0;
          for (int r = 0; r < M; ++r) s += O[(int64_t)r * C + k] * dSp[(int64_t)r * C + o];
          dWo[(int64_t)k * C + o] = s;
        }
    if (dbo)
      for (int o = 0; o < C; ++o) {
        double s = 0.0;
        for (int r = 0; r < M; ++r) s += dSp[(int64_t)r * C + o];
        dbo[o] = s;
      }
  } else {
    memcpy(dO, dSp, sizeof(double) * mc);
  }

  for (int h = 0; h < H; ++h) {
    const double* Ph = P + (int64_t)h * M * M;
    int off = h * D;
    /* dV_h = P_h^T dO_h */
    for (int c = 0; c < M; ++c)
      for (int d = 0; d < D; ++d) {
        double s = 0.0;
        for (int r = 0; r < M; ++r) s += Ph[r * M + c] * dO[(int64_t)r * C + off + d];
        dV[(int64_t)c * C + off + d] = s;
      }
    /* dP = dO_h V_h^T; dE = P o (dP - rowsum(dP o P)) */
    for (int r = 0; r < M; ++r) {
      double rs = 0.0;
      for (int c = 0; c < M; ++c) {
        double s = 0.0;
        for (int d = 0; d < D; ++d) s += dO[(int64_t)r * C + off + d] * V[(int64_t)c * C + off + d];
        dE[r * M + c] = s;
        rs += s * Ph[r * M + c];
      }
      for (int c = 0; c < M; ++c) dE[r * M + c] = Ph[r * M + c] * (dE[r * M + c] - rs);
    }
    /* dQ_h = scale dE K_h; dK_h = scale dE^T Q_h */
    for (int r = 0; r < M; ++r)
      for (int d = 0; d < D; ++d) {
        double sq = 0.0, sk = 0.0;
        for (int c = 0; c < M; ++c) {
          sq += dE[r * M + c] * K[(int64_t)c * C + off + d];
          sk += dE[c * M + r] * Q[(int64_t)c * C + off + d];
        }
        dQ[(int64_t)r * C + off + d] = scale * sq;
        dK[(int64_t)r * C + off + d] = scale * sk;
      }
  }

  for (int r = 0; r < M; ++r)
    for (int k = 0; k < C; ++k) {
      double s = 0.0;
      for (int o = 0; o < C; ++o)
        s += dQ[(int64_t)r * C + o] * Wq[(int64_t)k * C + o] +
             dK[(int64_t)r * C + o] * Wk[(int64_t)k * C + o] +
             dV[(int64_t)r * C + o] * Wv[(int64_t)k * C + o];
      dS[(int64_t)r * C + k] = s;
    }
  const double* dproj[3] = {dQ, dK, dV};
  double* dWs[3] = {dWq, dWk, dWv};
  double* dbs[3] = {dbq, dbk, dbv};
  for (int t = 0; t < 3; ++t) {
    if (dWs[t])
      for (int k = 0; k < C; ++k)
        for (int o = 0; o < C; ++o) {
          double s = 0.0;
          for (int r = 0; r < M; ++r) s += S[(int64_t)r * C + k] * dproj[t][(int64_t)r * C + o];
          dWs[t][(int64_t)k * C + o] = s;
        }
    if (dbs[t])
      for (int o = 0; o < C; ++o) {
        double s = 0.0;
        for (int r = 0; r < M; ++r) s += dproj[t][(int64_t)r * C + o];
        dbs[t][o] = s;
      }
  }
  free(Q); free(K); free(V); free(O); free(P);
  free(dO); free(dQ); free(dK); free(dV); free(dE);
}

/* Eq. 1 backward.  s_j = num_j / d_j with d_j = max(den_j, eps):
 *   den_j >= eps: dnum_j = ds_j / den_j, dden_j = -<ds_j, s_j> / den_j
 *   den_j <  eps: dnum_j = ds_j / eps,   dden_j = 0
 * then num_j = sum_i w_ij x_i, den_j = sum_i w_ij give
 *   dx_i = sum_j w_ij dnum_j,  dW_ij = <x_i, dnum_j> + dden_j. */
void pao_aggregate_backward(int64_t N, int C, int M, double eps,
                            const double* x, const double* W,
                            const double* num, const double* den,
                            const double* dS, double* dx, double* dW) {
  double* dnum = (double*)malloc(sizeof(double) * M * C);
  double* dden = (double*)malloc(sizeof(double) * M);
  for (int j = 0; j < M; ++j) {
    if (den[j] >= eps) {
      double dot = 0.0;
      for (int c = 0; c < C; ++c) {
        double s = num[(int64_t)j * C + c] / den[j];
        dot += dS[(int64_t)j * C + c] * s;
        dnum[(int64_t)j * C + c] = dS[(int64_t)j * C + c] / den[j];
      }
      dden[j] = -dot / den[j];
    } else {
      for (int c = 0; c < C; ++c) dnum[(int64_t)j * C + c] = dS[(int64_t)j * C + c] / eps;
      dden[j] = 0.0;
    }
  }
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < N; ++i) {
    for (int c = 0; c < C; ++c) {
      double s = 0.0;
      for (int j = 0; j < M; ++j) s += W[i * M + j] * dnum[(int64_t)j * C + c];
      if (dx) dx[i * C + c] = s;
    }
    if (dW)
      for (int j = 0; j < M; ++j) {
        double s = dden[j];
        for (int c = 0; c < C; ++c) s += x[i * C + c] * dnum[(int64_t)j * C + c];
        dW[i * M + j] = s;
      }
  }
  free(dnum);
  free(dden);
}

/* Eq. 3 + Eq. 4 backward, per point (z, w, tau, t recomputed as forward):
 *   dz_j  = w_j (dW_j - sum_k w_k dW_k)          softmax
 *   dl_j  = dz_j / tau                           z = (l + g)/tau
 *   dtau  = dtau_in - sum_j dz_j z_j / tau
 *   dt    = dtau if t > tau_min else 0           clamp
 *   dx    = A dl + a dt
 * and over points (sharded): dA = sum_i x_i dl_i^T, db = sum_i dl_i,
 *   da = sum_i dt_i x_i, db_t = dtau0 = sum_i dt_i. */
void pao_slice_weights_backward(int64_t N, int C, int M, double tau0,
                                double tau_min, const double* x,
                                const double* G, const double* A,
                                const double* b, const double* a, double b_t,
                                const double* dW, const double* dtau,
                                double* dx, double* dA, double* db, double* da,
                                double* db_t, double* dtau0) {
  int64_t P = n_shards(N);
  int64_t part = (int64_t)C * M + M + C + 1;
  double* parts = (double*)calloc((size_t)(P > 0 ? P : 1) * part, sizeof(double));
#pragma omp parallel
  {
    double* z = (double*)malloc(sizeof(double) * M);
    double* w = (double*)malloc(sizeof(double) * M);
    double* dl = (double*)malloc(sizeof(double) * M);
#pragma omp for schedule(static)
    for (int64_t p = 0; p < P; ++p) {
      double* pA = parts + p * part;
      double* pb = pA + (int64_t)C * M;
      double* pa = pb + M;
      double* pbt = pa + C;
      int64_t i1 = (p + 1) * SHARD < N ? (p + 1) * SHARD : N;
      for (int64_t i = p * SHARD; i < i1; ++i) {
        const double* xi = x + i * C;
        double tau, t;
        point_weights(C, M, tau0, tau_min, xi, G ? G + i * M : NULL, A, b, a,
                      b_t, z, w, &tau, &t);
        const double* dwi = dW + i * M;
        double wdw = 0.0;
        for (int j = 0; j < M; ++j) wdw += w[j] * dwi[j];
        double dtau_i = dtau ? dtau[i] : 0.0;
        for (int j = 0; j < M; ++j) {
          double dz = w[j] * (dwi[j] - wdw);
          dl[j] = dz / tau;
          dtau_i -= dz * z[j] / tau;
        }
        double dt = t > tau_min ? dtau_i : 0.0;
        for (int c = 0; c < C; ++c) {
          double s = a ? a[c] * dt : 0.0;
          for (int j = 0; j < M; ++j) s += A[(int64_t)c * M + j] * dl[j];
          if (dx) dx[i * C + c] = s;
          for (int j = 0; j < M; ++j) pA[(int64_t)c * M + j] += xi[c] * dl[j];
          pa[c] += dt * xi[c];
        }
        for (int j = 0; j < M; ++j) pb[j] += dl[j];
        pbt[0] += dt;
      }
    }
    free(z);
    free(w);
    free(dl);
  }
  double* acc = (double*)calloc((size_t)part, sizeof(double));
  for (int64_t p = 0; p < P; ++p)
    for (int64_t k = 0; k < part; ++k) acc[k] += parts[p * part + k];
  if (dA) memcpy(dA, acc, sizeof(double) * C * M);
  if (db) memcpy(db, acc + (int64_t)C * M, sizeof(double) * M);
  if (da) memcpy(da, acc + (int64_t)C * M + M, sizeof(double) * C);
  if (db_t) *db_t = acc[part - 1];
  if (dtau0) *dtau0 = acc[part - 1];
  free(acc);
  free(parts);
}
