/* Host-only exercise of the C ABI (include/ffmlp.h) for the sanitizer
 * build: handles, shape and size queries and every argument check that
 * fails before a launch, over many shapes.  Never launches a kernel, so it
 * runs without a GPU.  Exit status 0 when every check holds. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "ffmlp.h"

#define CHECK(c)                                                      \
  do {                                                                \
    if (!(c)) {                                                       \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      return 1;                                                       \
    }                                                                 \
  } while (0)

static int one_net(int width, int depth, int in_dim, int out_dim, int act, int out_act) {
  mlp_t* h = NULL;
  CHECK(mlp_create(width, depth, in_dim, out_dim, act, &h) == MLP_OK && h != NULL);
  CHECK(mlp_set_output_activation(h, out_act) == MLP_OK);
  /* shapes: consecutive offsets summing to the parameter count */
  int64_t off_expect = 0;
  for (int l = 0; l <= depth; ++l) {
    int fi = 0, fo = 0;
    int64_t off = -1;
    CHECK(mlp_layer_shape(h, l, &fi, &fo, &off) == MLP_OK);
    CHECK(fi == (l == 0 ? in_dim : width) && fo == (l == depth ? out_dim : width));
    CHECK(off == off_expect);
    off_expect += (int64_t)fi * fo;
  }
  CHECK(mlp_layer_shape(h, depth + 1, NULL, NULL, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_layer_shape(h, -1, NULL, NULL, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(strlen(mlp_last_error()) > 0);
  CHECK(mlp_param_count(h) == off_expect);
  CHECK(mlp_packed_bytes(h) > 0 && mlp_packed_bytes(h) % 1024 == 0);
  /* workspace: 256-byte multiple, non-decreasing in M, none for inference */
  size_t prev = 0;
  const int64_t Ms[] = {0, 1, 15, 16, 17, 127, 128, 129, 1000, 4097, 1 << 20};
  for (size_t i = 0; i < sizeof Ms / sizeof Ms[0]; ++i) {
    const size_t b = mlp_workspace_bytes(h, Ms[i], MLP_MODE_TRAIN);
    CHECK(b % 256 == 0 && b >= prev);
    CHECK(mlp_workspace_bytes(h, Ms[i], MLP_MODE_INFER) == 0);
    prev = b;
  }
  CHECK(mlp_workspace_bytes(h, -1, MLP_MODE_TRAIN) == 0);
  /* argument checks that fail before anything is enqueued (the fake
   * pointers are never dereferenced) */
  void* f = (void*)(uintptr_t)0x1000;
  void* mis = (void*)(uintptr_t)0x1002;
  CHECK(mlp_forward(h, NULL, f, f, 10, NULL, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_forward(h, f, mis, f, 10, NULL, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_forward(h, f, f, f, -1, NULL, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_forward(h, f, f, f, 10, mis, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_forward(h, NULL, NULL, NULL, 0, NULL, NULL) == MLP_OK); /* empty batch */
  CHECK(mlp_backward(h, f, f, f, NULL, 10, f, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_backward_dx(h, f, f, f, f, mis, 10, f, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_train_step(h, f, f, NULL, NULL, f, NULL, 10, f, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_train_step(h, f, f, f, NULL, f, NULL, 10, mis, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_train_step_noalloc(h, f, f, f, NULL, f, NULL, (int64_t)1 << 30, NULL) == MLP_ERR_WORKSPACE);
  CHECK(mlp_pack_weights(h, NULL, f, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_pack_weights(h, f, mis, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_sgd_step(h, NULL, f, f, NULL, 0.1f, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_adam_step(h, f, f, f, f, f, NULL, 1e-3f, 0.9f, 0.999f, 1e-8f, 0, NULL) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_set_output_activation(h, 7) == MLP_ERR_UNSUPPORTED);
  mlp_destroy(h);
  return 0;
}

int main(void) {
  static const int widths[] = {16, 32, 64, 128};
  int n = 0;
  for (int wi = 0; wi < 4; ++wi) {
    const int w = widths[wi];
    const int depths[] = {0, 1, 2, 4, 17};
    for (int di = 0; di < 5; ++di) {
      const int ins[] = {1, w / 2 + 1, w};
      const int outs[] = {1, 3, w};
      for (int ii = 0; ii < 3; ++ii)
        for (int oi = 0; oi < 3; ++oi) {
          const int act = (wi + di + ii) % 4, out_act = (di + oi) % 4;
          if (one_net(w, depths[di], ins[ii], outs[oi], act, out_act)) {
            fprintf(stderr, "net w=%d d=%d in=%d out=%d\n", w, depths[di], ins[ii], outs[oi]);
            return 1;
          }
          ++n;
        }
    }
  }
  /* rejected shapes leave *out NULL */
  mlp_t* h = (mlp_t*)(uintptr_t)0x1;
  CHECK(mlp_create(48, 2, 8, 8, MLP_ACT_RELU, &h) == MLP_ERR_UNSUPPORTED && h == NULL);
  CHECK(mlp_create(64, 2, 8, 8, 9, &h) == MLP_ERR_UNSUPPORTED);
  CHECK(mlp_create(64, -1, 8, 8, MLP_ACT_RELU, &h) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_create(64, MLP_MAX_DEPTH + 1, 8, 8, MLP_ACT_RELU, &h) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_create(64, 2, 0, 8, MLP_ACT_RELU, &h) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_create(64, 2, 8, 65, MLP_ACT_RELU, &h) == MLP_ERR_INVALID_ARG);
  CHECK(mlp_create(64, 2, 8, 8, MLP_ACT_RELU, NULL) == MLP_ERR_INVALID_ARG);
  /* the deepest net */
  CHECK(mlp_create(16, MLP_MAX_DEPTH, 16, 16, MLP_ACT_SINE, &h) == MLP_OK);
  int fi = 0, fo = 0;
  int64_t off = 0;
  CHECK(mlp_layer_shape(h, MLP_MAX_DEPTH, &fi, &fo, &off) == MLP_OK && off == (int64_t)MLP_MAX_DEPTH * 256);
  CHECK(mlp_workspace_bytes(h, 4096, MLP_MODE_TRAIN) > 0);
  mlp_destroy(h);
  mlp_destroy(NULL);
  printf("abi ok: %d nets\n", n);
  return 0;
}
