/*
 * Plain fp64 loops of the LoRA-adapted linear layer -- TEST INFRASTRUCTURE.
 *
 * The same definition as oracle/lora_oracle.py (Eq. 1 of JORA, Section 3,
 * "Model Transfer API": output = W0 x + b0 + B A x, row-major over m tokens,
 * b0 = 0, LoRA scale s = alpha / r; and its chain rule for the trainable A and
 * B with W0 frozen), written as loops over the index definitions with float64
 * accumulators:
 *
 *     U[i][t]  = sum_l X[i][l] A[t][l]
 *     Y[i][j]  = sum_l X[i][l] W[j][l] + s sum_t U[i][t] B[j][t]
 *     dU[i][t] = s sum_j dY[i][j] B[j][t]
 *     dX[i][l] = sum_j dY[i][j] W[j][l] + sum_t dU[i][t] A[t][l]
 *     dB[j][t] = s sum_i dY[i][j] U[i][t]
 *     dA[t][l] = sum_i dU[i][t] X[i][l]
 *
 * Inputs are float64 (the caller decodes bfloat16 exactly); every sum runs in
 * index order.  The only parallelism is over output rows (OpenMP), which
 * leaves each sum's order unchanged.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg load this; the HIP library shares nothing with
 * it.
 */
#include <stdint.h>
#include <stdlib.h>

#define AT(p, row, ld, col) ((p)[(int64_t)(row) * (ld) + (col)])

/* U [m][r] and Y [m][n] from X [m][k], W [n][k], A [r][k], B [n][r]. */
void lora_loops_forward(const double* X, const double* W, const double* A, const double* B, int64_t m,
                        int64_t n, int64_t k, int64_t r, double alpha, double* U, double* Y, int threads) {
  const double s = alpha / (double)r;
#pragma omp parallel for num_threads(threads) schedule(static)
  for (int64_t i = 0; i < m; ++i) {
    for (int64_t t = 0; t < r; ++t) {
      double u = 0.0;
      for (int64_t l = 0; l < k; ++l) u += AT(X, i, k, l) * AT(A, t, k, l);
      AT(U, i, r, t) = u;
    }
    for (int64_t j = 0; j < n; ++j) {
      double y = 0.0;
      for (int64_t l = 0; l < k; ++l) y += AT(X, i, k, l) * AT(W, j, k, l);
      double lo = 0.0;
      for (int64_t t = 0; t < r; ++t) lo += AT(U, i, r, t) * AT(B, j, r, t);
      AT(Y, i, n, j) = y + s * lo;
    }
  }
}

/* dU [m][r], dX [m][k], dA [r][k], dB [n][r] from dY [m][n] and the forward's
 * inputs (U is recomputed from X and A). */
void lora_loops_backward(const double* dY, const double* X, const double* W, const double* A, const double* B,
                         int64_t m, int64_t n, int64_t k, int64_t r, double alpha, double* dU, double* dX,
                         double* dA, double* dB, int threads) {
  const double s = alpha / (double)r;
  double* U = (double*)malloc(sizeof(double) * (size_t)(m * r));
  if (!U) abort();
#pragma omp parallel for num_threads(threads) schedule(static)
  for (int64_t i = 0; i < m; ++i) {
    for (int64_t t = 0; t < r; ++t) {
      double u = 0.0;
      for (int64_t l = 0; l < k; ++l) u += AT(X, i, k, l) * AT(A, t, k, l);
      AT(U, i, r, t) = u;
      double du = 0.0;
      for (int64_t j = 0; j < n; ++j) du += AT(dY, i, n, j) * AT(B, j, r, t);
      AT(dU, i, r, t) = s * du;
    }
    /* dX row i: the sum over j for every l at once (j outer, so each
     * dX[i][l] still adds its terms in j order), then the rank-r term */
    double* dxi = &AT(dX, i, k, 0);
    for (int64_t l = 0; l < k; ++l) dxi[l] = 0.0;
    for (int64_t j = 0; j < n; ++j) {
      const double g = AT(dY, i, n, j);
      for (int64_t l = 0; l < k; ++l) dxi[l] += g * AT(W, j, k, l);
    }
    for (int64_t l = 0; l < k; ++l) {
      double lo = 0.0;
      for (int64_t t = 0; t < r; ++t) lo += AT(dU, i, r, t) * AT(A, t, k, l);
      dxi[l] += lo;
    }
  }
#pragma omp parallel for num_threads(threads) schedule(static)
  for (int64_t j = 0; j < n; ++j) {
    for (int64_t t = 0; t < r; ++t) AT(dB, j, r, t) = 0.0;
    for (int64_t i = 0; i < m; ++i) {
      const double g = AT(dY, i, n, j);
      for (int64_t t = 0; t < r; ++t) AT(dB, j, r, t) += g * AT(U, i, r, t);
    }
    for (int64_t t = 0; t < r; ++t) AT(dB, j, r, t) *= s;
  }
#pragma omp parallel for num_threads(threads) schedule(static)
  for (int64_t l = 0; l < k; ++l) {
    for (int64_t t = 0; t < r; ++t) {
      double a = 0.0;
      for (int64_t i = 0; i < m; ++i) a += AT(dU, i, r, t) * AT(X, i, k, l);
      AT(dA, t, k, l) = a;
    }
  }
  free(U);
}
