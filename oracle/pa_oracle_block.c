/*
 * Block-stack oracle: the parts of a Transolver++ block around the
 * Physics-Attention layer, in double precision (see pa_oracle.h).
 *
 * TEST INFRASTRUCTURE ONLY: used by the tests and the smoke check; never by
 * the product path.
 *
 * The block is the Transformer block with Physics-Attention in place of
 * attention (Section 3; the block diagram of Figure 2a), read as pre-norm
 * with residual adds:  x <- x + PA(LN(x));  x <- x + MLP(LN(x)),
 * MLP(h) = GELU(h W1 + b1) W2 + b2.  The composition lives in oracle/
 * __init__.py; this file holds the pieces, each written out from its
 * definition.  Sums over points are formed per shard of SHARD points and
 * added in shard order (as the states are), so results do not depend on the
 * thread count.
 */
#include "pa_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define SHARD 1024

/* LayerNorm over the C channels of each row (biased variance):
 *   y = (x - mean) / sqrt(var + eps) * g + b. */
void pao_layernorm(int64_t N, int C, double eps, const double* x, const double* g,
                   const double* b, double* y, double* mean, double* rstd) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < N; ++i) {
    const double* xi = x + i * C;
    double m = 0.0;
    for (int c = 0; c < C; ++c) m += xi[c];
    m /= C;
    double v = 0.0;
    for (int c = 0; c < C; ++c) v += (xi[c] - m) * (xi[c] - m);
    v /= C;
    const double r = 1.0 / sqrt(v + eps);
    for (int c = 0; c < C; ++c) y[i * C + c] = (xi[c] - m) * r * (g ? g[c] : 1.0) + (b ? b[c] : 0.0);
    if (mean) mean[i] = m;
    if (rstd) rstd[i] = r;
  }
}

/* Chain rule of pao_layernorm, with xhat = (x - mean) rstd and
 * gh = dy * g:  dx = rstd (gh - mean_c(gh) - xhat mean_c(gh xhat));
 * dg = sum_i dy xhat; db = sum_i dy (each output nullable). */
void pao_layernorm_backward(int64_t N, int C, double eps, const double* x, const double* g,
                            const double* dy, double* dx, double* dg, double* db) {
  const int64_t S = (N + SHARD - 1) / SHARD;
  double* pg = calloc((size_t)S * C, sizeof(double));
  double* pb = calloc((size_t)S * C, sizeof(double));
#pragma omp parallel for schedule(static)
  for (int64_t s = 0; s < S; ++s) {
    double* xh = malloc((size_t)C * sizeof(double));
    double* gh = malloc((size_t)C * sizeof(double));
    const int64_t i1 = (s + 1) * SHARD < N ? (s + 1) * SHARD : N;
    for (int64_t i = s * SHARD; i < i1; ++i) {
      const double* xi = x + i * C;
      const double* dyi = dy + i * C;
      double m = 0.0;
      for (int c = 0; c < C; ++c) m += xi[c];
      m /= C;
      double v = 0.0;
      for (int c = 0; c < C; ++c) v += (xi[c] - m) * (xi[c] - m);
      v /= C;
      const double r = 1.0 / sqrt(v + eps);
      double mg = 0.0, mgx = 0.0;
      for (int c = 0; c < C; ++c) {
        xh[c] = (xi[c] - m) * r;
        gh[c] = dyi[c] * (g ? g[c] : 1.0);
        mg += gh[c];
        mgx += gh[c] * xh[c];
        pg[s * C + c] += dyi[c] * xh[c];
        pb[s * C + c] += dyi[c];
      }
      mg /= C;
      mgx /= C;
      if (dx)
        for (int c = 0; c < C; ++c) dx[i * C + c] = r * (gh[c] - mg - xh[c] * mgx);
    }
    free(xh);
    free(gh);
  }
  for (int c = 0; c < C; ++c) {
    double a = 0.0, bb = 0.0;
    for (int64_t s = 0; s < S; ++s) {
      a += pg[s * C + c];
      bb += pb[s * C + c];
    }
    if (dg) dg[c] = a;
    if (db) db[c] = bb;
  }
  free(pg);
  free(pb);
}

/* GELU (the feedforward layer's activation; the paper names the layer but
 * not its activation, read as the Transformer's GELU in its defining form):
 *   y = x Phi(x),  Phi(x) = (1 + erf(x / sqrt 2)) / 2  (standard normal CDF). */
#define GELU_R2 0.7071067811865476      /* 1 / sqrt(2) */
#define GELU_IS2PI 0.3989422804014327   /* 1 / sqrt(2 pi) */
void pao_gelu(int64_t n, const double* x, double* y) {
#pragma omp parallel for schedule(static)
  for (int64_t k = 0; k < n; ++k) y[k] = 0.5 * x[k] * (1.0 + erf(x[k] * GELU_R2));
}

/* dx = dy (Phi(x) + x phi(x)),  phi(x) = exp(-x^2 / 2) / sqrt(2 pi). */
void pao_gelu_backward(int64_t n, const double* x, const double* dy, double* dx) {
#pragma omp parallel for schedule(static)
  for (int64_t k = 0; k < n; ++k) {
    const double Phi = 0.5 * (1.0 + erf(x[k] * GELU_R2));
    const double phi = GELU_IS2PI * exp(-0.5 * x[k] * x[k]);
    dx[k] = dy[k] * (Phi + x[k] * phi);
  }
}

