/*
 * CPU oracle for fully-fused narrow MLPs (arXiv 2403.17607).
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the plain, slow, obviously
 * correct definition that the GPU library is checked against.  Only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg may load it;
 * the GPU product path never calls it.
 *
 * What it computes:
 *   - Inference, Algorithm 1 (section III-A): A_1 = X; C_l = A_l W_l;
 *     A_{l+1} = sigma(C_l); the last layer uses a separate output activation
 *     (the benchmarks of section IV use ReLU hidden layers with a linear
 *     output).  No bias terms: the algorithms have none.
 *   - Training, Algorithm 2 (section III-A): the forward pass with every A_l
 *     kept, the L2 loss with the mean over M*out_dim, the output delta
 *     D_{L+1} = sigma_b(A, 2 (Y - T) / (M out_dim)), backward propagation
 *     D_l = sigma_b(A_l, D_{l+1} W_l^T) down to l = 2 (no input gradient), and
 *     the weight gradients G_l = A_l^T D_{l+1}.  No optimizer step.
 *
 * Arithmetic is fp64.  With round_bf16 = 1 each value the GPU stores as
 * bf16 (activations A_l, deltas D_l, the output Y, the cos stash of sine
 * layers) is rounded once, from fp64 straight to bf16, round-to-nearest-even.
 * Products and sums are never rounded.  With round_bf16 = 0 nothing is
 * rounded (used for finite-difference checks).
 *
 * Weights are one concatenated array: layer l (0-based) is a row-major
 * fan_in(l) x fan_out(l) matrix used as C = A W (section III-A).
 * fan_in(0) = in_dim, fan_out(L-1) = out_dim, every other dim = width.
 * Any width >= 1 is accepted (no padding happens here).
 *
 * Parity status per function is recorded in oracle/__init__.py; every
 * function here is pinned by a CPU test.
 */
#ifndef FFMLP_ORACLE_H
#define FFMLP_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_LINEAR = 0, ORC_RELU = 1, ORC_SIGMOID = 2, ORC_SINE = 3 };

typedef struct {
  int width;      /* hidden width */
  int depth;      /* number of hidden layers; L = depth + 1 weight matrices */
  int in_dim;
  int out_dim;
  int act;        /* hidden activation */
  int out_act;    /* output activation */
  int round_bf16; /* 1: round at the GPU's rounding points; 0: pure fp64 */
  int threads;    /* OpenMP threads, <= 0 means the runtime default */
} orc_net;

/* Round an fp64 value to the nearest bf16 value, ties to even. */
double orc_rne_bf16(double x);

int64_t orc_param_count(const orc_net* n);

/* Shape and offset (in elements) of weight matrix l, 0 <= l < depth + 1. */
int orc_layer_shape(const orc_net* n, int l, int* fan_in, int* fan_out,
                    int64_t* offset);

/*
 * Forward pass, Algorithm 1.
 *   X  [M, in_dim]   inputs (values as given, normally bf16-exact)
 *   Y  [M, out_dim]  output, rounded to bf16 when round_bf16
 *   Y32 [M, out_dim] output before that rounding (may be NULL)
 *   A  [depth, M, width] hidden activations A_2..A_{L} (may be NULL)
 * Returns 0, or -1 on an invalid argument.
 */
int orc_forward(const orc_net* n, const double* W, const double* X,
                int64_t M, double* Y, double* Y32, double* A);

/*
 * Backward pass of Algorithm 2 seeded with a caller-given dY = dLoss/dY
 * (the loss is then whatever produced dY).  The forward pass is recomputed
 * from X.  Writes G (param_count values, same layout as W) and, when D is
 * not NULL, the deltas D_2..D_{L+1}: depth arrays [M, width] followed by
 * one [M, out_dim] array (layer-major).
 */
int orc_backward(const orc_net* n, const double* W, const double* X,
                 int64_t M, const double* dY, double* G, double* D);

/*
 * orc_backward plus the input gradient dX = dLoss/dX [M, in_dim], the
 * product of the first hidden layer's delta with the first weight
 * matrix's transpose, unrounded (dX may be NULL).
 */
int orc_backward_dx(const orc_net* n, const double* W, const double* X,
                    int64_t M, const double* dY, double* G, double* D,
                    double* dX);

/*
 * One training step of Algorithm 2 with the mean-squared-error loss:
 * Y and Y32 as in orc_forward (Y32 may be NULL), G and D as in
 * orc_backward, *loss = sum (Y32 - T)^2 / (M out_dim) (loss may be NULL).
 */
int orc_train_step(const orc_net* n, const double* W, const double* X,
                   const double* T, int64_t M, double* Y, double* Y32,
                   double* G, double* loss, double* D);

#ifdef __cplusplus
}
#endif

#endif
