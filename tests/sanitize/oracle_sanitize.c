/*
 * Memory- and UB-checking driver for the oracle's fp64 loops (oracle/lora_loops.c),
 * built with -fsanitize=address,undefined by tests/test_sanitizers.py.  Every
 * array is allocated at its exact size, so an index past a row or matrix end
 * is reported by the address sanitizer.  Besides running clean it checks two
 * exact facts: results do not depend on the thread count, and B = 0 gives
 * dU = dA = 0 and Y = X W^T.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void lora_loops_forward(const double* X, const double* W, const double* A, const double* B, int64_t m,
                        int64_t n, int64_t k, int64_t r, double alpha, double* U, double* Y, int threads);
void lora_loops_backward(const double* dY, const double* X, const double* W, const double* A, const double* B,
                         int64_t m, int64_t n, int64_t k, int64_t r, double alpha, double* dU, double* dX,
                         double* dA, double* dB, int threads);

static uint64_t state = 0x9E3779B97F4A7C15ull;
static double draw(void) {   /* xorshift64*, uniform in [-1, 1) */
  state ^= state >> 12;
  state ^= state << 25;
  state ^= state >> 27;
  return (double)((state * 0x2545F4914F6CDD1Dull) >> 11) / 4503599627370496.0 - 1.0;
}
static double* mat(int64_t rows, int64_t cols, int fill) {
  double* p = (double*)malloc(sizeof(double) * (size_t)(rows * cols));
  if (!p) abort();
  for (int64_t i = 0; i < rows * cols; ++i) p[i] = fill ? draw() : 0.0;
  return p;
}
static int same(const double* a, const double* b, int64_t count) {
  return memcmp(a, b, sizeof(double) * (size_t)count) == 0;
}

static int run(int64_t m, int64_t n, int64_t k, int64_t r, double alpha) {
  int bad = 0;
  double *X = mat(m, k, 1), *W = mat(n, k, 1), *A = mat(r, k, 1), *B = mat(n, r, 1), *dY = mat(m, n, 1);
  double *U1 = mat(m, r, 0), *Y1 = mat(m, n, 0), *U3 = mat(m, r, 0), *Y3 = mat(m, n, 0);
  double *dU1 = mat(m, r, 0), *dX1 = mat(m, k, 0), *dA1 = mat(r, k, 0), *dB1 = mat(n, r, 0);
  double *dU3 = mat(m, r, 0), *dX3 = mat(m, k, 0), *dA3 = mat(r, k, 0), *dB3 = mat(n, r, 0);
  lora_loops_forward(X, W, A, B, m, n, k, r, alpha, U1, Y1, 1);
  lora_loops_forward(X, W, A, B, m, n, k, r, alpha, U3, Y3, 3);
  lora_loops_backward(dY, X, W, A, B, m, n, k, r, alpha, dU1, dX1, dA1, dB1, 1);
  lora_loops_backward(dY, X, W, A, B, m, n, k, r, alpha, dU3, dX3, dA3, dB3, 3);
  if (!same(U1, U3, m * r) || !same(Y1, Y3, m * n) || !same(dU1, dU3, m * r) || !same(dX1, dX3, m * k) ||
      !same(dA1, dA3, r * k) || !same(dB1, dB3, n * r)) {
    fprintf(stderr, "thread count changed a result at m=%lld n=%lld k=%lld r=%lld\n", (long long)m,
            (long long)n, (long long)k, (long long)r);
    bad = 1;
  }
  for (int64_t i = 0; i < m * n; ++i)
    if (!isfinite(Y1[i])) bad = 1;
  /* B = 0: the adapter path vanishes */
  double* B0 = mat(n, r, 0);
  lora_loops_forward(X, W, A, B0, m, n, k, r, alpha, U1, Y1, 2);
  lora_loops_backward(dY, X, W, A, B0, m, n, k, r, alpha, dU1, dX1, dA1, dB1, 2);
  for (int64_t i = 0; i < m; ++i)
    for (int64_t j = 0; j < n; ++j) {
      double y = 0.0;
      for (int64_t l = 0; l < k; ++l) y += X[i * k + l] * W[j * k + l];
      if (Y1[i * n + j] != y) bad = 1;
    }
  for (int64_t i = 0; i < m * r; ++i)
    if (dU1[i] != 0.0) bad = 1;
  for (int64_t i = 0; i < r * k; ++i)
    if (dA1[i] != 0.0) bad = 1;
  if (bad) fprintf(stderr, "check failed at m=%lld n=%lld k=%lld r=%lld\n", (long long)m, (long long)n,
                   (long long)k, (long long)r);
  free(X); free(W); free(A); free(B); free(dY); free(B0);
  free(U1); free(Y1); free(U3); free(Y3);
  free(dU1); free(dX1); free(dA1); free(dB1); free(dU3); free(dX3); free(dA3); free(dB3);
  return bad;
}

int main(void) {
  const int64_t shapes[][4] = {{1, 8, 8, 1}, {3, 8, 16, 2}, {17, 24, 40, 5}, {33, 16, 8, 16}, {64, 72, 56, 64}};
  int bad = 0;
  for (size_t s = 0; s < sizeof(shapes) / sizeof(shapes[0]); ++s)
    bad |= run(shapes[s][0], shapes[s][1], shapes[s][2], shapes[s][3], 2.0 * (double)shapes[s][3]);
  printf(bad ? "oracle sanitizer driver: FAILED\n" : "oracle sanitizer driver: ok\n");
  return bad;
}
