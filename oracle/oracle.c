/*
 * CPU oracle for fully-fused narrow MLPs (arXiv 2403.17607).
 * TEST INFRASTRUCTURE ONLY: see oracle.h.  Shares no code with the GPU
 * library.
 *
 * Rows are independent in the forward and backward passes (Algorithms 1 and
 * 2 act on the batch row by row except for the sums that form G), so every
 * row is pushed through the whole network on its own; G is summed over rows
 * in fp64, per thread, then the per-thread sums are added in thread order.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* bf16 keeps 8 significant bits (1 implicit + 7 stored), its smallest normal
 * is 2^-126 and its largest finite value is (2 - 2^-7) * 2^127. */
double orc_rne_bf16(double x) {
  if (!isfinite(x) || x == 0.0) return x;
  int e;
  (void)frexp(x, &e); /* |x| in [2^(e-1), 2^e) */
  int ulp_exp = e - 8;
  if (ulp_exp < -133) ulp_exp = -133; /* subnormal bf16 spacing */
  double q = ldexp(x, -ulp_exp);      /* exact power-of-two scaling */
  double r = nearbyint(q);            /* default mode: ties to even */
  double y = ldexp(r, ulp_exp);
  const double max_bf16 = ldexp(255.0, 120); /* (2 - 2^-7) * 2^127 */
  if (fabs(y) > max_bf16) return y > 0 ? INFINITY : -INFINITY;
  return y;
}

static double round_if(const orc_net* n, double v) {
  return n->round_bf16 ? orc_rne_bf16(v) : v;
}

static int n_layers(const orc_net* n) { return n->depth + 1; }

static int fan_in_of(const orc_net* n, int l) {
  return l == 0 ? n->in_dim : n->width;
}

static int fan_out_of(const orc_net* n, int l) {
  return l == n_layers(n) - 1 ? n->out_dim : n->width;
}

int64_t orc_param_count(const orc_net* n) {
  int64_t total = 0;
  for (int l = 0; l < n_layers(n); ++l)
    total += (int64_t)fan_in_of(n, l) * fan_out_of(n, l);
  return total;
}

int orc_layer_shape(const orc_net* n, int l, int* fan_in, int* fan_out,
                    int64_t* offset) {
  if (!n || l < 0 || l >= n_layers(n)) return -1;
  int64_t off = 0;
  for (int i = 0; i < l; ++i)
    off += (int64_t)fan_in_of(n, i) * fan_out_of(n, i);
  if (fan_in) *fan_in = fan_in_of(n, l);
  if (fan_out) *fan_out = fan_out_of(n, l);
  if (offset) *offset = off;
  return 0;
}

static int valid_act(int a) { return a >= ORC_LINEAR && a <= ORC_SINE; }

static int check_net(const orc_net* n, int64_t M) {
  if (!n || n->width < 1 || n->depth < 0 || n->in_dim < 1 || n->out_dim < 1)
    return -1;
  if (!valid_act(n->act) || !valid_act(n->out_act)) return -1;
  if (M < 0) return -1;
  return 0;
}

/* sigma: the activation functions themselves. */
static double act_fwd(int act, double c) {
  switch (act) {
    case ORC_RELU: return c > 0.0 ? c : 0.0;
    case ORC_SIGMOID: return 1.0 / (1.0 + exp(-c));
    case ORC_SINE: return sin(c);
    default: return c;
  }
}

/*
 * sigma_b for a hidden layer, Algorithm 2: the derivative is taken from the
 * stored activation a = A_l where the activation allows it (ReLU: a > 0;
 * sigmoid: a (1 - a)); for sine it is cos of the pre-activation c, stored
 * (and so rounded) like an activation.
 */
static double act_grad_hidden(const orc_net* n, double a, double c) {
  switch (n->act) {
    case ORC_RELU: return a > 0.0 ? 1.0 : 0.0;
    case ORC_SIGMOID: return a * (1.0 - a);
    case ORC_SINE: return round_if(n, cos(c));
    default: return 1.0;
  }
}

/* sigma_b at the output layer: taken from the unrounded output y32 and the
 * pre-activation c, which the GPU still holds in registers there. */
static double act_grad_out(int act, double y32, double c) {
  switch (act) {
    case ORC_RELU: return c > 0.0 ? 1.0 : 0.0;
    case ORC_SIGMOID: return y32 * (1.0 - y32);
    case ORC_SINE: return cos(c);
    default: return 1.0;
  }
}

/* Per-row working storage: the input to every layer and every
 * pre-activation. */
typedef struct {
  double* a; /* (L + 1) slots of max_dim: a[l] is the input of layer l */
  double* c; /* L slots of max_dim: c[l] = a[l] W_l */
  double* d; /* (L + 1) slots of max_dim: d[l + 1] = dLoss/dc[l] */
  double* y32;
} row_buf;

static int max_dim(const orc_net* n) {
  int m = n->width;
  if (n->in_dim > m) m = n->in_dim;
  if (n->out_dim > m) m = n->out_dim;
  return m;
}

static int row_buf_alloc(row_buf* b, const orc_net* n) {
  int L = n_layers(n), D = max_dim(n);
  b->a = (double*)calloc((size_t)(L + 1) * D, sizeof(double));
  b->c = (double*)calloc((size_t)L * D, sizeof(double));
  b->d = (double*)calloc((size_t)(L + 1) * D, sizeof(double));
  b->y32 = (double*)calloc((size_t)D, sizeof(double));
  return (b->a && b->c && b->d && b->y32) ? 0 : -1;
}

static void row_buf_free(row_buf* b) {
  free(b->a);
  free(b->c);
  free(b->d);
  free(b->y32);
}

/* Algorithm 1 for one row.  Leaves a[], c[] and y32 in the buffer. */
static void forward_row(const orc_net* n, const double* W, const double* x,
                        row_buf* b) {
  const int L = n_layers(n), D = max_dim(n);
  for (int k = 0; k < n->in_dim; ++k) b->a[k] = x[k];
  const double* Wl = W;
  for (int l = 0; l < L; ++l) {
    const int fi = fan_in_of(n, l), fo = fan_out_of(n, l);
    const double* a = b->a + (size_t)l * D;
    double* c = b->c + (size_t)l * D;
    for (int j = 0; j < fo; ++j) c[j] = 0.0;
    for (int k = 0; k < fi; ++k) {
      const double ak = a[k];
      const double* wrow = Wl + (size_t)k * fo;
      for (int j = 0; j < fo; ++j) c[j] += ak * wrow[j];
    }
    if (l < L - 1) {
      double* next = b->a + (size_t)(l + 1) * D;
      for (int j = 0; j < fo; ++j) next[j] = round_if(n, act_fwd(n->act, c[j]));
    } else {
      for (int j = 0; j < fo; ++j) b->y32[j] = act_fwd(n->out_act, c[j]);
    }
    Wl += (size_t)fi * fo;
  }
}

/*
 * Backward pass of Algorithm 2 for one row, given g = dLoss/dY for that row
 * and the forward state left by forward_row.  Leaves the deltas in b->d and
 * adds the row's contribution A_l^T D_{l+1} to G (fp64).
 */
static void backward_row(const orc_net* n, const double* W, const double* g,
                         row_buf* b, double* G, double* dx) {
  const int L = n_layers(n), D = max_dim(n);
  /* Output delta: D_{L+1} = sigma_b(Y, g). */
  {
    const double* c = b->c + (size_t)(L - 1) * D;
    double* d = b->d + (size_t)L * D;
    for (int j = 0; j < n->out_dim; ++j)
      d[j] = round_if(n, g[j] * act_grad_out(n->out_act, b->y32[j], c[j]));
  }
  /* Offsets of every weight matrix. */
  int64_t off = orc_param_count(n);
  for (int l = L - 1; l >= 0; --l) {
    const int fi = fan_in_of(n, l), fo = fan_out_of(n, l);
    off -= (int64_t)fi * fo;
    const double* Wl = W + off;
    const double* a = b->a + (size_t)l * D;
    const double* dn = b->d + (size_t)(l + 1) * D;
    /* G_l += A_l^T D_{l+1} (this row's outer product). */
    double* Gl = G + off;
    for (int k = 0; k < fi; ++k) {
      const double ak = a[k];
      double* grow = Gl + (size_t)k * fo;
      for (int j = 0; j < fo; ++j) grow[j] += ak * dn[j];
    }
    /* The input gradient (an extension beyond Algorithm 2, which stops at
     * the first hidden layer): X enters the first product linearly, so
     * dLoss/dX = D_1 W_1^T (1-based), with no activation derivative and no
     * rounding. */
    if (l == 0 && dx) {
      for (int k = 0; k < fi; ++k) {
        const double* wrow = Wl + (size_t)k * fo;
        double p = 0.0;
        for (int j = 0; j < fo; ++j) p += dn[j] * wrow[j];
        dx[k] = p;
      }
    }
    /* D_l = sigma_b(A_l, D_{l+1} W_l^T), only down to l = 2 (1-based):
     * the input layer gets no delta. */
    if (l >= 1) {
      double* d = b->d + (size_t)l * D;
      const double* cprev = b->c + (size_t)(l - 1) * D;
      for (int k = 0; k < fi; ++k) {
        const double* wrow = Wl + (size_t)k * fo;
        double p = 0.0;
        for (int j = 0; j < fo; ++j) p += dn[j] * wrow[j];
        d[k] = round_if(n, p * act_grad_hidden(n, a[k], cprev[k]));
      }
    }
  }
}

static void store_row_outputs(const orc_net* n, const row_buf* b, int64_t M,
                              int64_t r, double* Y, double* Y32, double* A) {
  const int L = n_layers(n), D = max_dim(n);
  for (int j = 0; j < n->out_dim; ++j) {
    if (Y) Y[r * n->out_dim + j] = round_if(n, b->y32[j]);
    if (Y32) Y32[r * n->out_dim + j] = b->y32[j];
  }
  if (A) {
    for (int l = 1; l < L; ++l) {
      double* dst = A + ((size_t)(l - 1) * M + r) * n->width;
      memcpy(dst, b->a + (size_t)l * D, sizeof(double) * n->width);
    }
  }
}

static void store_row_deltas(const orc_net* n, const row_buf* b, int64_t M,
                             int64_t r, double* Dout) {
  const int L = n_layers(n), D = max_dim(n);
  for (int l = 1; l < L; ++l) {
    double* dst = Dout + ((size_t)(l - 1) * M + r) * n->width;
    memcpy(dst, b->d + (size_t)l * D, sizeof(double) * n->width);
  }
  double* dst = Dout + (size_t)(L - 1) * M * n->width + (size_t)r * n->out_dim;
  memcpy(dst, b->d + (size_t)L * D, sizeof(double) * n->out_dim);
}

static int thread_count(const orc_net* n) {
#ifdef _OPENMP
  return n->threads > 0 ? n->threads : omp_get_max_threads();
#else
  (void)n;
  return 1;
#endif
}

int orc_forward(const orc_net* n, const double* W, const double* X,
                int64_t M, double* Y, double* Y32, double* A) {
  if (check_net(n, M) || !W || (M > 0 && (!X || !Y))) return -1;
  int failed = 0;
#pragma omp parallel num_threads(thread_count(n)) reduction(| : failed)
  {
    row_buf b;
    if (row_buf_alloc(&b, n)) {
      failed = 1;
    } else {
#pragma omp for schedule(static)
      for (int64_t r = 0; r < M; ++r) {
        forward_row(n, W, X + r * n->in_dim, &b);
        store_row_outputs(n, &b, M, r, Y, Y32, A);
      }
    }
    row_buf_free(&b);
  }
  return failed ? -1 : 0;
}

/* Shared driver of orc_backward and orc_train_step.  T == NULL means dY is
 * given; otherwise dY is NULL and g = 2 (Y32 - T) / (M out_dim). */
static int run_backward(const orc_net* n, const double* W, const double* X,
                        const double* T, const double* dY, int64_t M,
                        double* Y, double* Y32, double* G, double* loss,
                        double* Dout, double* dX) {
  const int64_t P = orc_param_count(n);
  const int nt = thread_count(n);
  double* partial = (double*)calloc((size_t)nt * P, sizeof(double));
  double* loss_part = (double*)calloc((size_t)nt, sizeof(double));
  if (!partial || !loss_part) {
    free(partial);
    free(loss_part);
    return -1;
  }
  const double scale = (T && M > 0) ? 2.0 / ((double)M * n->out_dim) : 0.0;
  int failed = 0;
#pragma omp parallel num_threads(nt) reduction(| : failed)
  {
    int tid = 0;
#ifdef _OPENMP
    tid = omp_get_thread_num();
#endif
    row_buf b;
    double* g = (double*)calloc((size_t)n->out_dim, sizeof(double));
    if (row_buf_alloc(&b, n) || !g) {
      failed = 1;
    } else {
      double* Gt = partial + (size_t)tid * P;
#pragma omp for schedule(static)
      for (int64_t r = 0; r < M; ++r) {
        forward_row(n, W, X + r * n->in_dim, &b);
        if (T) {
          const double* t = T + r * n->out_dim;
          for (int j = 0; j < n->out_dim; ++j) {
            const double diff = b.y32[j] - t[j];
            loss_part[tid] += diff * diff;
            g[j] = scale * diff;
          }
        } else {
          for (int j = 0; j < n->out_dim; ++j) g[j] = dY[r * n->out_dim + j];
        }
        backward_row(n, W, g, &b, Gt, dX ? dX + r * n->in_dim : NULL);
        store_row_outputs(n, &b, M, r, Y, Y32, NULL);
        if (Dout) store_row_deltas(n, &b, M, r, Dout);
      }
    }
    free(g);
    row_buf_free(&b);
  }
  if (!failed) {
    for (int64_t i = 0; i < P; ++i) G[i] = 0.0;
    double total_loss = 0.0;
    for (int t = 0; t < nt; ++t) {
      const double* Gt = partial + (size_t)t * P;
      for (int64_t i = 0; i < P; ++i) G[i] += Gt[i];
      total_loss += loss_part[t];
    }
    if (loss) *loss = M > 0 ? total_loss / ((double)M * n->out_dim) : 0.0;
  }
  free(partial);
  free(loss_part);
  return failed ? -1 : 0;
}

int orc_backward(const orc_net* n, const double* W, const double* X,
                 int64_t M, const double* dY, double* G, double* D) {
  return orc_backward_dx(n, W, X, M, dY, G, D, NULL);
}

int orc_backward_dx(const orc_net* n, const double* W, const double* X,
                    int64_t M, const double* dY, double* G, double* D,
                    double* dX) {
  if (check_net(n, M) || !W || !G || (M > 0 && (!X || !dY))) return -1;
  return run_backward(n, W, X, NULL, dY, M, NULL, NULL, G, NULL, D, dX);
}

int orc_train_step(const orc_net* n, const double* W, const double* X,
                   const double* T, int64_t M, double* Y, double* Y32,
                   double* G, double* loss, double* D) {
  if (check_net(n, M) || !W || !G || (M > 0 && (!X || !T))) return -1;
  return run_backward(n, W, X, T, NULL, M, Y, Y32, G, loss, D, NULL);
}
