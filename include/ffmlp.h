/*
 * ffmlp: fully-fused narrow MLPs on AMD Instinct MI355X (gfx950).
 *
 * C ABI of the library.  The operations are those of "Fully-fused
 * Multi-Layer Perceptrons on Intel Data Center GPUs" (arXiv 2403.17607),
 * section III-A:
 *   - inference, Algorithm 1: A_1 = X, C_i = A_i B_i, A_{i+1} = sigma(C_i);
 *   - the training step, Algorithm 2: the forward pass keeping every A_i,
 *     the L2 loss, the output delta, backward propagation of the deltas
 *     D_i = sigma_b(A_i, D_{i+1} B_i^T) down to i = 2 (no input gradient),
 *     and the weight gradients G_i = A_i^T D_{i+1}.  No optimizer step
 *     (the paper leaves it out of the algorithm).
 * Weights B_i are stored fan_in x fan_out and used as C = A B (section
 * III-A); there are no bias terms (the algorithms have none).
 *
 * Shapes.  An MLP has `depth` hidden layers of `width` neurons, i.e.
 * L = depth + 1 weight matrices: in_dim x width, (depth - 1) times
 * width x width, width x out_dim (for depth = 0: one in_dim x out_dim
 * matrix).  width is 16, 32, 64 or 128 (section I); 1 <= in_dim, out_dim
 * <= width; 0 <= depth <= MLP_MAX_DEPTH (the weight-gradient launch has one
 * grid row per matrix, and a grid dimension holds at most 65535).  Smaller input and output widths are reduced to the square case
 * by zero padding inside the library (section III-A).
 *
 * Precision.  All matrix products take bf16 operands and accumulate in fp32
 * (section III-B).  Every activation, delta and output stored is rounded
 * once to bf16, round-to-nearest-even; weight gradients are fp32.
 *
 * Memory.  Every pointer argument except `mlp_t*`, `fan_in`, `fan_out` and
 * `offset` of mlp_layer_shape is DEVICE memory on the current HIP device,
 * owned by the caller.  The library never allocates device memory, never
 * synchronizes the stream and keeps no device state: a handle holds host
 * metadata only and is immutable after mlp_set_output_activation, so one
 * handle may be used from several streams at once as long as each call has
 * its own workspace.  Calls that share a workspace on overlapping streams
 * race.  All work is enqueued on `stream` (a hipStream_t; NULL means the
 * default stream).
 *
 * Errors.  Every int-returning call returns MLP_OK (0) or a negative code.
 * Argument errors are detected on the host before anything is enqueued;
 * mlp_last_error() (thread-local) then describes the problem.  Faults of
 * enqueued kernels surface at the caller's next synchronization.
 */
#ifndef FFMLP_H
#define FFMLP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct mlp mlp_t;

/* Activations (the benchmarks of section IV use ReLU hidden layers with a
 * linear output; sigmoid and sine serve the application-shaped nets). */
enum {
  MLP_ACT_LINEAR = 0,
  MLP_ACT_RELU = 1,
  MLP_ACT_SIGMOID = 2, /* 1 / (1 + exp(-x)) */
  MLP_ACT_SINE = 3     /* sin(x) */
};

enum {
  MLP_OK = 0,
  MLP_ERR_INVALID_ARG = -1, /* null pointer, bad size, misaligned pointer */
  MLP_ERR_UNSUPPORTED = -2, /* width not in {16, 32, 64, 128}, bad activation */
  MLP_ERR_WORKSPACE = -3,   /* workspace smaller than mlp_workspace_bytes */
  MLP_ERR_HIP = -4          /* a HIP runtime call or launch failed */
};

enum { MLP_MODE_INFER = 0, MLP_MODE_TRAIN = 1 };

enum { MLP_MAX_DEPTH = 65534 };

/* Create a handle (host memory only).  `activation` applies to the hidden
 * layers; the output activation defaults to linear.  Returns
 * MLP_ERR_UNSUPPORTED for a width outside {16, 32, 64, 128} or an unknown
 * activation, MLP_ERR_INVALID_ARG for depth outside [0, MLP_MAX_DEPTH], in_dim or out_dim outside
 * [1, width], or out == NULL. */
int mlp_create(int width, int depth, int in_dim, int out_dim, int activation,
               mlp_t** out);

/* Set the activation of the output layer (default MLP_ACT_LINEAR). */
int mlp_set_output_activation(mlp_t* h, int activation);

/* Free the handle.  NULL is ignored. */
void mlp_destroy(mlp_t* h);

/* Number of weights, sum over layers of fan_in * fan_out (real dims). */
int64_t mlp_param_count(const mlp_t* h);

/* Real shape of weight matrix l (0-based, 0 <= l <= depth) and its offset,
 * in elements, inside the concatenated weight and gradient buffers.  Any of
 * the three output pointers may be NULL. */
int mlp_layer_shape(const mlp_t* h, int l, int* fan_in, int* fan_out,
                    int64_t* offset);

/* Bytes of the packed-weight buffer written by mlp_pack_weights. */
size_t mlp_packed_bytes(const mlp_t* h);

/* Rearrange the weights into the operand order of the matrix cores, zero
 * padded, in the two orientations the forward and backward passes use (the
 * counterpart of the packed format of section III-B).
 *   W       bf16 bit patterns, mlp_param_count(h) elements: the L matrices
 *           concatenated, each row-major [fan_in][fan_out].  2-byte aligned.
 *   packed  mlp_packed_bytes(h) bytes, 16-byte aligned, written in full.
 * Call it again after every weight update. */
int mlp_pack_weights(const mlp_t* h, const uint16_t* W, void* packed,
                     void* stream);

/* Workspace bytes for a batch of M rows.  MLP_MODE_INFER: 0 (inference
 * needs none).  MLP_MODE_TRAIN: the activation stash, the deltas and the
 * per-workgroup partial sums used by mlp_forward (with a stash),
 * mlp_backward and mlp_train_step.  Depends only on the handle and M. */
size_t mlp_workspace_bytes(const mlp_t* h, int64_t M, int mode);

/*
 * Forward pass, Algorithm 1.
 *   X      bf16 [M][in_dim], row-major, contiguous, 16-byte aligned.
 *   Y      bf16 [M][out_dim], row-major, contiguous, 8-byte aligned.
 *   stash  NULL for inference.  Otherwise a training workspace of at least
 *          mlp_workspace_bytes(h, M, MLP_MODE_TRAIN) bytes, 256-byte
 *          aligned: the forward pass of Algorithm 2 then also keeps every
 *          hidden activation there for a later mlp_backward.
 * M >= 0 rows (M = 0 enqueues nothing).
 */
int mlp_forward(const mlp_t* h, const void* packed, const uint16_t* X,
                uint16_t* Y, int64_t M, void* stash, void* stream);

/*
 * Backward pass of Algorithm 2 seeded with dY = dLoss/dY, after
 * mlp_forward(..., stash = ws) on the same X, M and packed weights.
 *   X   the forward's input (needed for G_1 = A_1^T D_2).
 *   dY  fp32 [M][out_dim], row-major, 16-byte aligned.
 *   G   fp32, mlp_param_count(h) elements, same layout as the weights;
 *       overwritten with the weight gradients.  No input gradient.
 *   ws  the workspace the forward pass stashed into.
 */
int mlp_backward(const mlp_t* h, const void* packed, const uint16_t* X,
                 const float* dY, float* G, int64_t M, void* ws,
                 void* stream);

/* mlp_backward plus the input gradient dX = dLoss/dX (an extension beyond
 * Algorithm 2 of section III-A, which stops at the first hidden layer: X
 * enters the first product linearly, so dX = D_1 W_1^T in 1-based layer
 * numbering, with no activation derivative).
 *   dX  fp32 [M][in_dim] row-major, 16-byte aligned, written in full (not
 *       rounded to bf16); the other arguments as for mlp_backward.
 * A caller chaining nets passes dX of one net as dY of the net before it.
 * Same error behaviour as mlp_backward; dX == NULL is mlp_backward. */
int mlp_backward_dx(const mlp_t* h, const void* packed, const uint16_t* X,
                    const float* dY, float* G, float* dX, int64_t M, void* ws,
                    void* stream);

/*
 * One training step, Algorithm 2: forward with stash, mean-squared-error
 * loss over the M * out_dim outputs, output delta 2 (Y - T) / (M out_dim)
 * times the output activation's derivative, backward propagation and the
 * weight gradients.  No optimizer step.
 *   T     fp32 targets [M][out_dim], row-major, 16-byte aligned.
 *   Y     optional bf16 output [M][out_dim] (NULL: not stored).
 *   G     fp32 gradients, mlp_param_count(h) elements (overwritten).
 *   loss  optional device float, set to sum (Y - T)^2 / (M out_dim)
 *         computed from the fp32 outputs before rounding.
 *   ws    mlp_workspace_bytes(h, M, MLP_MODE_TRAIN) bytes, 256-byte aligned.
 * Kernels: at widths 16, 32 and 64 with 2 to 5 weight matrices, one kernel
 * for the whole step (forward, loss, backward and weight gradients, the
 * hidden activations kept on chip: only X, T and Y touch memory).  Otherwise
 * the forward pass, then for nets of 2 to 5 weight matrices (at width 128
 * only ReLU nets with out_dim <= 16) one fused kernel that propagates the
 * deltas and accumulates the weight gradients without storing the deltas
 * (the fusion section V of the paper proposes), for other nets a backward
 * kernel and a weight-gradient kernel.  Then a fixed-order reduction, so G
 * and the loss are bitwise the same from run to run.  mlp_backward uses
 * the same rule for its backward kernels; mlp_backward_dx always the
 * unfused pair.
 */
int mlp_train_step(const mlp_t* h, const void* packed, const uint16_t* X,
                   const float* T, uint16_t* Y, float* G, float* loss,
                   int64_t M, void* ws, void* stream);

/* Bytes of the library's own static device scratch array (64 MiB), the
 * largest mlp_workspace_bytes(h, M, MLP_MODE_TRAIN) that
 * mlp_train_step_noalloc accepts. */
enum { MLP_SCRATCH_BYTES = 64 << 20 };

/*
 * mlp_train_step for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same computation, arguments and results as mlp_train_step, but the
 * workspace is a static array of MLP_SCRATCH_BYTES inside the library (one
 * per GPU, held until the process ends) instead of a caller buffer.  The
 * call allocates nothing (no hipMalloc, hipFree or allocating library
 * routine); on its first call on a device it looks up that device's array
 * once.  Nothing in the array has to start at zero: every byte a call reads
 * was written earlier in the same call.
 *   Returns MLP_ERR_WORKSPACE, before anything is enqueued, when
 *   mlp_workspace_bytes(h, M, MLP_MODE_TRAIN) > MLP_SCRATCH_BYTES (for
 *   example width 128, 4 hidden layers, out 16: up to 15 744 rows).
 * Every call on one GPU shares that GPU's array, so calls that overlap on
 * one GPU (several streams or host threads at once) race; calls that follow
 * each other in one stream do not.
 */
int mlp_train_step_noalloc(const mlp_t* h, const void* packed,
                           const uint16_t* X, const float* T, uint16_t* Y,
                           float* G, float* loss, int64_t M, void* stream);

/* Optimizer step on fp32 master weights (NEXT-4; the paper leaves the
 * optimizer out of its training step, section III-A).  One kernel updates
 * every parameter, then writes the bf16 weights the fused kernels read
 * (round to nearest even) and, when packed != NULL, re-packs them exactly as
 * mlp_pack_weights does.  All buffers hold mlp_param_count(h) values in the
 * weights' layout (the L matrices concatenated, each [fan_in][fan_out]).
 *   master  fp32, updated in place; 4-byte aligned.
 *   G       fp32 gradients (from mlp_train_step or mlp_backward).
 *   W       bf16 output; 2-byte aligned.
 *   packed  mlp_packed_bytes(h) bytes, 16-byte aligned, or NULL.
 * SGD: master -= lr G. */
int mlp_sgd_step(const mlp_t* h, float* master, const float* G, uint16_t* W,
                 void* packed, float lr, void* stream);

/* Adam (Kingma and Ba 2015, Algorithm 1), step t = 1, 2, ...:
 *   m = beta1 m + (1 - beta1) G;  v = beta2 v + (1 - beta2) G^2;
 *   master -= lr (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps).
 *   m, v  fp32 moment buffers, updated in place (start from zeros).
 * MLP_ERR_INVALID_ARG for t < 1, beta outside [0, 1), eps <= 0, a
 * non-finite lr, or null or misaligned pointers.  Other arguments as for
 * mlp_sgd_step. */
int mlp_adam_step(const mlp_t* h, float* master, float* m, float* v,
                  const float* G, uint16_t* W, void* packed, float lr,
                  float beta1, float beta2, float eps, int64_t t,
                  void* stream);

/* Description of the last error on this thread ("" if none). */
const char* mlp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif
