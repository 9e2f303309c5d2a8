/* Exercise of the CPU oracle (oracle/oracle.h) for the sanitizer build:
 * every entry point over small nets of every activation pair, with buffers
 * allocated to their exact sizes, rounding on and off, one and two
 * threads, and the argument checks.  Also checks that the training step's
 * G equals the seeded backward's G for dY = 2 (Y32 - T) / (M out_dim), bit
 * for bit.  Exit status 0 when every check holds. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"

#define CHECK(c)                                                      \
  do {                                                                \
    if (!(c)) {                                                       \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      return 1;                                                       \
    }                                                                 \
  } while (0)

static double* vec(size_t n, unsigned seed) {
  double* v = (double*)malloc((n ? n : 1) * sizeof(double));
  for (size_t i = 0; i < n; ++i) v[i] = ((double)((seed * 2654435761u + (unsigned)i * 40503u) % 2001u) - 1000.0) / 1000.0;
  return v;
}

static int finite_all(const double* v, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!isfinite(v[i])) return 0;
  return 1;
}

static int one(int width, int depth, int in_dim, int out_dim, int act, int out_act, int64_t M,
               int round, int threads) {
  orc_net n = {width, depth, in_dim, out_dim, act, out_act, round, threads};
  const int64_t P = orc_param_count(&n);
  const size_t hid = (size_t)depth * M * width, nd = hid + (size_t)M * out_dim;
  double *W = vec(P, 1), *X = vec(M * in_dim, 2), *T = vec(M * out_dim, 3);
  double *Y = vec(M * out_dim, 0), *Y32 = vec(M * out_dim, 0), *A = vec(hid, 0);
  double *G = vec(P, 0), *G2 = vec(P, 0), *D = vec(nd, 0), *dX = vec(M * in_dim, 0);
  double* dY = vec(M * out_dim, 4);
  double loss = 0.0;
  CHECK(orc_forward(&n, W, X, M, Y, Y32, A) == 0);
  CHECK(finite_all(Y, M * out_dim) && finite_all(A, hid));
  CHECK(orc_backward(&n, W, X, M, dY, G, D) == 0);
  CHECK(orc_backward_dx(&n, W, X, M, dY, G2, NULL, dX) == 0);
  CHECK(memcmp(G, G2, P * sizeof(double)) == 0);
  CHECK(finite_all(G, P) && finite_all(D, nd) && finite_all(dX, M * in_dim));
  CHECK(orc_train_step(&n, W, X, T, M, Y, Y32, G, &loss, D) == 0);
  CHECK(isfinite(loss) && loss >= 0.0);
  /* the training step forms the output delta as (2 / (M out_dim)) (Y32 - T) */
  for (int64_t i = 0; i < M * out_dim; ++i) dY[i] = (2.0 / ((double)M * out_dim)) * (Y32[i] - T[i]);
  CHECK(orc_backward(&n, W, X, M, dY, G2, NULL) == 0);
  CHECK(memcmp(G, G2, P * sizeof(double)) == 0);
  free(W); free(X); free(T); free(Y); free(Y32); free(A); free(G); free(G2); free(D); free(dX); free(dY);
  return 0;
}

int main(void) {
  int cases = 0;
  for (int width = 1; width <= 9; width += 4)
    for (int depth = 0; depth <= 3; ++depth)
      for (int act = 0; act < 4; ++act)
        for (int out_act = 0; out_act < 4; ++out_act)
          for (int64_t M = 0; M <= 5; M += 5) {
            const int in_dim = 1 + (act + depth) % 3, out_dim = 1 + (out_act + width) % 3;
            if (one(width, depth, in_dim, out_dim, act, out_act, M, (act + out_act) & 1, 1 + (depth & 1))) {
              fprintf(stderr, "case w=%d d=%d act=%d out=%d M=%lld\n", width, depth, act, out_act, (long long)M);
              return 1;
            }
            ++cases;
          }
  /* argument checks */
  orc_net bad = {4, 1, 4, 4, 9, 0, 1, 1};
  double v[64] = {0};
  CHECK(orc_forward(&bad, v, v, 1, v, v, NULL) != 0);
  orc_net ok = {4, 1, 4, 4, 1, 0, 1, 1};
  CHECK(orc_forward(&ok, v, v, -1, v, v, NULL) != 0);
  CHECK(orc_forward(NULL, v, v, 1, v, v, NULL) != 0);
  CHECK(orc_layer_shape(&ok, 2, NULL, NULL, NULL) != 0);
  CHECK(orc_rne_bf16(1.0 + 1.0 / 256.0) == 1.0);
  printf("oracle ok: %d cases\n", cases);
  return 0;
}
