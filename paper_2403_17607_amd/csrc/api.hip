// C ABI of the library (include/ffmlp.h): argument checks, workspace
// layout and the launch sequence of each entry point.  Host code only.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"
#include "ffmlp.h"

using namespace ffmlp;

struct mlp {
  int width, depth, in_dim, out_dim, act, out_act;
};

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(MLP_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int n_mats(const mlp* h) { return h->depth + 1; }
int fan_in_of(const mlp* h, int l) { return l == 0 ? h->in_dim : h->width; }
int fan_out_of(const mlp* h, int l) { return l == n_mats(h) - 1 ? h->out_dim : h->width; }
int kblocks(int n) { return (n + 31) / 32; }
int strips(int n) { return (n + 15) / 16; }

// Fragment counts of the packed buffer: forward layers 0 .. L-1, then
// backward layers 1 .. L-1, then backward layer 0 (input gradient only).
struct PackGeom {
  uint32_t fwd_frag[2], fwd_total;  // [0] = layer 0, [1] = hidden layers
  uint32_t bwd_hidden, bwd_total;   // backward layers 1 .. L-1
  uint32_t bwd0;                    // backward layer 0, after them
};

PackGeom pack_geom(const mlp* h) {
  const int W = h->width, L = n_mats(h);
  PackGeom g{};
  uint32_t total = 0;
  // Every packed layer has kblocks(W) k-blocks (zero-padded past a smaller
  // fan), so the kernels' contraction depth is a compile-time constant.
  for (int l = 0; l < L; ++l) {
    const uint32_t f = (uint32_t)strips(fan_out_of(h, l)) * kblocks(W);
    if (l == 0) g.fwd_frag[0] = f;
    if (l == 1) g.fwd_frag[1] = f;
    total += f;
  }
  g.fwd_total = total;
  g.fwd_frag[1] = (uint32_t)strips(W) * kblocks(W);
  uint32_t bt = 0;
  for (int l = 1; l < L; ++l) bt += (uint32_t)strips(fan_in_of(h, l)) * kblocks(W);
  g.bwd_hidden = (uint32_t)strips(W) * kblocks(W);
  g.bwd_total = bt;
  g.bwd0 = (uint32_t)strips(h->in_dim) * kblocks(W);
  return g;
}

// Workspace layout for a batch of M rows (byte offsets, 256-byte aligned).
struct WsLayout {
  int64_t M16;
  size_t stashA, stashS, reluMask, deltaH, deltaOut, cOut, partial, lossPart, total;
  int P, chunks_per_block;
};

WsLayout ws_layout(const mlp* h, int64_t M) {
  WsLayout w{};
  const int W = h->width, L = n_mats(h);
  const int OP = strips(h->out_dim) * 16;
  w.M16 = (M + 15) / 16 * 16;
  const size_t hid = (size_t)(L - 1) * w.M16 * W * 2;
  size_t o = 0;
  w.stashA = o; o = round_up(o + hid, 256);
  w.stashS = o; o = round_up(o + (h->act == MLP_ACT_SINE ? hid : 0), 256);
  // ReLU masks: one 32-bit word per lane of every 16-row block and layer
  w.reluMask = o; o = round_up(o + (h->act == MLP_ACT_RELU ? (size_t)(L - 1) * (w.M16 / 16) * 256 : 0), 256);
  w.deltaH = o; o = round_up(o + hid, 256);
  w.deltaOut = o; o = round_up(o + (size_t)w.M16 * OP * 2, 256);
  w.cOut = o; o = round_up(o + (h->out_act != MLP_ACT_LINEAR ? (size_t)w.M16 * OP * 4 : 0), 256);
  const int CH = wgrad_chunk(W);
  const int64_t nch = (M + CH - 1) / CH;
  int64_t P = (kWgradTargetBlocks + L - 1) / L;
  if (P > nch) P = nch;
  if (P < 1) P = 1;
  const int64_t cpb = nch > 0 ? (nch + P - 1) / P : 0;
  P = cpb > 0 ? (nch + cpb - 1) / cpb : 1;  // no empty workgroups
  w.P = (int)P;
  w.chunks_per_block = (int)cpb;
  // The fused backward writes one partial per workgroup, at most one per
  // row tile and at most kBwdgMaxBlocks.
  int64_t Pf = (M + kBwdgRows - 1) / kBwdgRows;
  if (Pf > kBwdgMaxBlocks) Pf = kBwdgMaxBlocks;
  const int64_t Pmax = P > Pf ? P : Pf;
  int64_t params = 0;
  for (int l = 0; l < L; ++l) params += (int64_t)fan_in_of(h, l) * fan_out_of(h, l);
  w.partial = o; o = round_up(o + (size_t)Pmax * params * 4, 256);
  w.lossPart = o; o = round_up(o + (size_t)kMaxLossParts * 4, 256);
  w.total = o;
  return w;
}

int64_t param_count(const mlp* h) {
  int64_t p = 0;
  for (int l = 0; l < n_mats(h); ++l) p += (int64_t)fan_in_of(h, l) * fan_out_of(h, l);
  return p;
}

bool valid_act(int a) { return a >= MLP_ACT_LINEAR && a <= MLP_ACT_SINE; }

int check_handle(const mlp* h) {
  if (!h) return fail(MLP_ERR_INVALID_ARG, "null handle");
  return MLP_OK;
}

FwdArgs fwd_args(const mlp* h, const void* packed, const uint16_t* X, int64_t M) {
  const PackGeom g = pack_geom(h);
  FwdArgs a{};
  a.packed = static_cast<const u32x4*>(packed);
  a.X = X;
  a.M = M;
  a.M16 = (M + 15) / 16 * 16;
  a.in_dim = h->in_dim;
  a.out_dim = h->out_dim;
  a.L = n_mats(h);
  a.out_act = h->out_act;
  a.scale = M > 0 ? (float)(2.0 / ((double)M * h->out_dim)) : 0.f;
  const int64_t rows = tile_rows(h->width);
  a.ntiles = (int)((M + rows - 1) / rows);
  a.lay0_frags = g.fwd_frag[0];
  a.layH_frags = g.fwd_frag[1];
  a.total_frags = g.fwd_total;
  return a;
}

BwdArgs bwd_args(const mlp* h, const void* packed, const WsLayout& w, uint8_t* ws, int64_t M) {
  const PackGeom g = pack_geom(h);
  BwdArgs b{};
  b.packed = reinterpret_cast<const u32x4*>(static_cast<const uint8_t*>(packed) + (size_t)g.fwd_total * 1024);
  b.stashA = reinterpret_cast<const uint16_t*>(ws + w.stashA);
  b.stashS = h->act == MLP_ACT_SINE ? reinterpret_cast<const uint16_t*>(ws + w.stashS) : nullptr;
  b.deltaH = reinterpret_cast<uint16_t*>(ws + w.deltaH);
  b.deltaOut = reinterpret_cast<uint16_t*>(ws + w.deltaOut);
  b.cOut = h->out_act != MLP_ACT_LINEAR ? reinterpret_cast<const float*>(ws + w.cOut) : nullptr;
  b.reluMask = h->act == MLP_ACT_RELU ? reinterpret_cast<const uint32_t*>(ws + w.reluMask) : nullptr;
  b.M = M;
  b.M16 = w.M16;
  b.in_dim = h->in_dim;
  b.out_dim = h->out_dim;
  b.L = n_mats(h);
  b.out_act = h->out_act;
  const int64_t rows = tile_rows(h->width);
  b.ntiles = (int)((M + rows - 1) / rows);
  b.layH_frags = g.bwd_hidden;
  b.total_frags = g.bwd_total;
  b.packed0 = reinterpret_cast<const u32x4*>(static_cast<const uint8_t*>(packed) +
                                             (size_t)(g.fwd_total + g.bwd_total) * 1024);
  b.dX = nullptr;
  return b;
}

// Fixed-order sum of P weight-gradient partials (and the loss partials).
int run_reduce(const mlp* h, const WsLayout& w, uint8_t* ws, int64_t M, int P, float* G,
               float* loss, int nloss, hipStream_t s) {
  ReduceArgs r{};
  r.partial = reinterpret_cast<const float*>(ws + w.partial);
  r.G = G;
  r.params = param_count(h);
  r.P = M > 0 ? P : 0;
  r.lossPart = reinterpret_cast<const float*>(ws + w.lossPart);
  r.nloss = M > 0 ? nloss : 0;
  r.loss = loss;
  r.loss_scale = M > 0 ? (float)(1.0 / ((double)M * h->out_dim)) : 0.f;
  hipError_t e = launch_reduce(r, s);
  if (e != hipSuccess) return hip_fail(e, "reduce kernel launch");
  return MLP_OK;
}

// The fused backward pass with the weight gradients, then the reduce.
// Returns 1 (nothing enqueued) when the fused kernel does not cover the net.
int run_fused_backward(const mlp* h, const void* packed, const uint16_t* X, const float* dY,
                       const WsLayout& w, uint8_t* ws, int64_t M, float* G, float* loss, int nloss,
                       int seeded, bool masks, hipStream_t s, bool stash_t = false) {
  if (M <= 0 || !backward_fused_supported(h->width, n_mats(h), h->act, h->in_dim, h->out_dim))
    return 1;
  const PackGeom g = pack_geom(h);
  BwdgArgs a{};
  a.packed = reinterpret_cast<const u32x4*>(static_cast<const uint8_t*>(packed) + (size_t)g.fwd_total * 1024);
  a.X = X;
  a.stashA = reinterpret_cast<const uint16_t*>(ws + w.stashA);
  a.reluMask = (h->act == MLP_ACT_RELU && masks) ? reinterpret_cast<const uint32_t*>(ws + w.reluMask)
                                                 : nullptr;
  a.stashS = h->act == MLP_ACT_SINE ? reinterpret_cast<const uint16_t*>(ws + w.stashS) : nullptr;
  a.deltaOut = reinterpret_cast<const uint16_t*>(ws + w.deltaOut);
  a.cOut = h->out_act != MLP_ACT_LINEAR ? reinterpret_cast<const float*>(ws + w.cOut) : nullptr;
  a.dY = dY;
  a.partial = reinterpret_cast<float*>(ws + w.partial);
  a.M = M;
  a.M16 = w.M16;
  a.params = param_count(h);
  a.in_dim = h->in_dim;
  a.out_dim = h->out_dim;
  a.act = h->act;
  a.out_act = h->out_act;
  a.ntiles = (int)((M + kBwdgRows - 1) / kBwdgRows);
  a.layH_frags = g.bwd_hidden;
  a.stash_t = stash_t ? 1 : 0;
  int P = 0;
  hipError_t e = launch_backward_fused(h->width, n_mats(h), h->out_dim, seeded, a, s, &P);
  if (e == hipErrorNotSupported) return 1;
  if (e != hipSuccess) return hip_fail(e, "fused backward kernel launch");
  return run_reduce(h, w, ws, M, P, G, loss, nloss, s);
}

int run_wgrad_reduce(const mlp* h, const uint16_t* X, const WsLayout& w, uint8_t* ws, int64_t M,
                     float* G, float* loss, int nloss, hipStream_t s) {
  const int64_t params = param_count(h);
  if (M > 0) {
    WgradArgs a{};
    a.X = X;
    a.stashA = reinterpret_cast<const uint16_t*>(ws + w.stashA);
    a.deltaH = reinterpret_cast<const uint16_t*>(ws + w.deltaH);
    a.deltaOut = reinterpret_cast<const uint16_t*>(ws + w.deltaOut);
    a.partial = reinterpret_cast<float*>(ws + w.partial);
    a.M = M;
    a.M16 = w.M16;
    a.params = params;
    a.in_dim = h->in_dim;
    a.out_dim = h->out_dim;
    a.L = n_mats(h);
    a.P = w.P;
    a.chunks_per_block = w.chunks_per_block;
    hipError_t e = launch_wgrad(h->width, a, s);
    if (e != hipSuccess) return hip_fail(e, "weight-gradient kernel launch");
  }
  return run_reduce(h, w, ws, M, w.P, G, loss, nloss, s);
}

int train_step_impl(const mlp_t* h, const void* packed, const uint16_t* X, const float* T,
                    uint16_t* Y, float* G, float* loss, int64_t M, void* ws_, void* stream);

// Workspace of mlp_train_step_noalloc: one static array per GPU, for callers
// that cannot allocate.  In host code `scratch` only names the array; its
// device address comes from hipGetSymbolAddress, once per device (each GPU
// holds its own copy at its own address), and only that address is passed
// to kernels.
constexpr size_t kScratchBytes = MLP_SCRATCH_BYTES;
__device__ __align__(256) uint8_t scratch[kScratchBytes];

hipError_t scratch_ptr(void** out) {
  static std::mutex mu;
  static std::vector<void*> ptrs;  // per device; null until looked up
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  if ((int)ptrs.size() <= dev) ptrs.resize(dev + 1, nullptr);
  if (!ptrs[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || reinterpret_cast<uintptr_t>(p) % 256 != 0) return hipErrorInvalidSymbol;
    ptrs[dev] = p;
  }
  *out = ptrs[dev];
  return hipSuccess;
}

}  // namespace

namespace ffmlp {

hipError_t device_info(DeviceInfo* out) {
  static std::mutex mu;
  static std::vector<DeviceInfo> cache;
  static std::vector<char> have;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  if ((int)cache.size() <= dev) {
    cache.resize(dev + 1);
    have.resize(dev + 1, 0);
  }
  if (!have[dev]) {
    DeviceInfo d{};
    e = hipDeviceGetAttribute(&d.cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&d.max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e != hipSuccess) return e;
    cache[dev] = d;
    have[dev] = 1;
  }
  *out = cache[dev];
  return hipSuccess;
}

hipError_t kernel_occupancy(const void* kernel, int threads, size_t lds, int* blocks_per_cu) {
  struct Key {
    int dev;
    const void* k;
    size_t lds;
    int threads;
  };
  struct Limit {
    int dev;
    const void* k;
    size_t lds;  // the largest dynamic-LDS limit set so far
  };
  static std::mutex mu;
  static std::vector<std::pair<Key, int>> cache;
  static std::vector<Limit> limits;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  for (const auto& kv : cache)
    if (kv.first.dev == dev && kv.first.k == kernel && kv.first.lds == lds &&
        kv.first.threads == threads) {
      *blocks_per_cu = kv.second;
      return hipSuccess;
    }
  // The limit only ever grows, so configurations cached earlier stay valid.
  Limit* lim = nullptr;
  for (auto& x : limits)
    if (x.dev == dev && x.k == kernel) lim = &x;
  if (!lim || lim->lds < lds) {
    e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    if (lim) lim->lds = lds; else limits.push_back(Limit{dev, kernel, lds});
  }
  int occ = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, threads, lds);
  if (e != hipSuccess) return e;
  if (occ < 1) occ = 1;
  cache.push_back({Key{dev, kernel, lds, threads}, occ});
  *blocks_per_cu = occ;
  return hipSuccess;
}

}  // namespace ffmlp

extern "C" {

const char* mlp_last_error(void) { return g_err.c_str(); }

int mlp_create(int width, int depth, int in_dim, int out_dim, int activation, mlp_t** out) {
  g_err.clear();
  if (!out) return fail(MLP_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (width != 16 && width != 32 && width != 64 && width != 128)
    return fail(MLP_ERR_UNSUPPORTED, "width %d is not one of 16, 32, 64, 128", width);
  if (!valid_act(activation)) return fail(MLP_ERR_UNSUPPORTED, "unknown activation %d", activation);
  if (depth < 0 || depth > MLP_MAX_DEPTH)
    return fail(MLP_ERR_INVALID_ARG, "depth %d outside [0, %d]", depth, (int)MLP_MAX_DEPTH);
  if (in_dim < 1 || in_dim > width)
    return fail(MLP_ERR_INVALID_ARG, "in_dim %d outside [1, %d]", in_dim, width);
  if (out_dim < 1 || out_dim > width)
    return fail(MLP_ERR_INVALID_ARG, "out_dim %d outside [1, %d]", out_dim, width);
  mlp* h = new (std::nothrow) mlp{width, depth, in_dim, out_dim, activation, MLP_ACT_LINEAR};
  if (!h) return fail(MLP_ERR_INVALID_ARG, "out of host memory");
  *out = h;
  return MLP_OK;
}

int mlp_set_output_activation(mlp_t* h, int activation) {
  g_err.clear();
  if (int rc = check_handle(h)) return rc;
  if (!valid_act(activation)) return fail(MLP_ERR_UNSUPPORTED, "unknown activation %d", activation);
  h->out_act = activation;
  return MLP_OK;
}

void mlp_destroy(mlp_t* h) { delete h; }

int64_t mlp_param_count(const mlp_t* h) { return h ? param_count(h) : 0; }

int mlp_layer_shape(const mlp_t* h, int l, int* fan_in, int* fan_out, int64_t* offset) {
  g_err.clear();
  if (int rc = check_handle(h)) return rc;
  if (l < 0 || l >= n_mats(h)) return fail(MLP_ERR_INVALID_ARG, "layer %d outside [0, %d]", l, h->depth);
  int64_t off = 0;
  for (int i = 0; i < l; ++i) off += (int64_t)fan_in_of(h, i) * fan_out_of(h, i);
  if (fan_in) *fan_in = fan_in_of(h, l);
  if (fan_out) *fan_out = fan_out_of(h, l);
  if (offset) *offset = off;
  return MLP_OK;
}

size_t mlp_packed_bytes(const mlp_t* h) {
  if (!h) return 0;
  const PackGeom g = pack_geom(h);
  return (size_t)(g.fwd_total + g.bwd_total + g.bwd0) * 1024;
}

int mlp_pack_weights(const mlp_t* h, const uint16_t* W, void* packed, void* stream) {
  g_err.clear();
  if (int rc = check_handle(h)) return rc;
  if (!W || !packed) return fail(MLP_ERR_INVALID_ARG, "null weight or packed pointer");
  if (!aligned(W, 2) || !aligned(packed, 16))
    return fail(MLP_ERR_INVALID_ARG, "W must be 2-byte and packed 16-byte aligned");
  PackArgs a{};
  a.W = W;
  a.dst = static_cast<uint16_t*>(packed);
  a.width = h->width;
  a.in_dim = h->in_dim;
  a.out_dim = h->out_dim;
  a.L = n_mats(h);
  a.total = (int64_t)(mlp_packed_bytes(h) / 2);
  hipError_t e = launch_pack(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "pack kernel launch");
  return MLP_OK;
}


namespace {

int optim_step(const mlp_t* h, OptArgs a, void* packed, void* stream) {
  if (!a.master || !a.G || !a.W) return fail(MLP_ERR_INVALID_ARG, "null master, G or W");
  if (!aligned(a.master, 4) || !aligned(a.G, 4) || !aligned(a.W, 2) ||
      (a.m && !aligned(a.m, 4)) || (a.v && !aligned(a.v, 4)) || (packed && !aligned(packed, 16)))
    return fail(MLP_ERR_INVALID_ARG, "misaligned pointer (master, m, v, G: 4 bytes; W: 2; packed: 16)");
  if (!std::isfinite(a.lr)) return fail(MLP_ERR_INVALID_ARG, "lr is not finite");
  a.n = param_count(h);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = launch_optim(a, s);
  if (e != hipSuccess) return hip_fail(e, "optimizer kernel launch");
  if (packed) return mlp_pack_weights(h, a.W, packed, stream);
  return MLP_OK;
}

}  // namespace

int mlp_sgd_step(const mlp_t* h, float* master, const float* G, uint16_t* W, void* packed,
                 float lr, void* stream) {
  g_err.clear();
  if (int rc = check_handle(h)) return rc;
  OptArgs a{};
  a.master = master;
  a.G = G;
  a.W = W;
  a.adam = 0;
  a.lr = lr;
  return optim_step(h, a, packed, stream);
}

int mlp_adam_step(const mlp_t* h, float* master, float* m, float* v, const float* G, uint16_t* W,
                  void* packed, float lr, float beta1, float beta2, float eps, int64_t t,
                  void* stream) {
  g_err.clear();
  if (int rc = check_handle(h)) return rc;
  if (!m || !v) return fail(MLP_ERR_INVALID_ARG, "null Adam moment buffer");
  if (t < 1) return fail(MLP_ERR_INVALID_ARG, "Adam step t = %lld < 1", (long long)t);
  if (!(beta1 >= 0.f && beta1 < 1.f) || !(beta2 >= 0.f && beta2 < 1.f) || !(eps > 0.f))
    return fail(MLP_ERR_INVALID_ARG, "need 0 <= beta1, beta2 < 1 and eps > 0");
  OptArgs a{};
  a.master = master;
  a.m = m;
  a.v = v;
  a.G = G;
  a.W = W;
  a.adam = 1;
  a.lr = lr;
  a.beta1 = beta1;
  a.beta2 = beta2;
  a.eps = eps;
  const double bc1 = 1.0 - std::pow((double)beta1, (double)t);
  const double bc2 = 1.0 - std::pow((double)beta2, (double)t);
  a.step_size = (float)((double)lr / bc1);
  a.inv_sqrt_bc2 = (float)(1.0 / std::sqrt(bc2));
  return optim_step(h, a, packed, stream);
}

size_t mlp_workspace_bytes(const mlp_t* h, int64_t M, int mode) {
  if (!h || M < 0 || mode != MLP_MODE_TRAIN) return 0;
  return ws_layout(h, M).total;
}

int mlp_forward(const mlp_t* h, const void* packed, const uint16_t* X, uint16_t* Y, int64_t M,
                void* stash, void* stream) {
  g_err.clear();
  if (int rc = check_handle(h)) return rc;
  if (M < 0) return fail(MLP_ERR_INVALID_ARG, "M = %lld < 0", (long long)M);
  if (M == 0) return MLP_OK;
  if (!packed || !X || !Y) return fail(MLP_ERR_INVALID_ARG, "null packed, X or Y");
  if (!aligned(packed, 16) || !aligned(X, 16) || !aligned(Y, 8))
    return fail(MLP_ERR_INVALID_ARG, "packed and X must be 16-byte, Y 8-byte aligned");
  if (stash && !aligned(stash, 256)) return fail(MLP_ERR_INVALID_ARG, "stash must be 256-byte aligned");
  if (M > ((int64_t)1 << 36)) return fail(MLP_ERR_INVALID_ARG, "M > 2^36");
  hipStream_t s = static_cast<hipStream_t>(stream);
  FwdArgs a = fwd_args(h, packed, X, M);
  a.Y = Y;
  int mode = FWD_INFER;
  if (stash) {
    const WsLayout w = ws_layout(h, M);
    uint8_t* ws = static_cast<uint8_t*>(stash);
    a.stashA = reinterpret_cast<uint16_t*>(ws + w.stashA);
    a.stashS = h->act == MLP_ACT_SINE ? reinterpret_cast<uint16_t*>(ws + w.stashS) : nullptr;
    a.reluMask = h->act == MLP_ACT_RELU ? reinterpret_cast<uint32_t*>(ws + w.reluMask) : nullptr;
    a.cOut = h->out_act != MLP_ACT_LINEAR ? reinterpret_cast<float*>(ws + w.cOut) : nullptr;
    mode = FWD_STASH;
  }
  hipError_t e = launch_forward(h->width, h->act, mode, a, s, nullptr);
  if (e != hipSuccess) return hip_fail(e, "forward kernel launch");
  return MLP_OK;
}

int mlp_backward(const mlp_t* h, const void* packed, const uint16_t* X, const float* dY, float* G,
                 int64_t M, void* ws_, void* stream) {
  return mlp_backward_dx(h, packed, X, dY, G, nullptr, M, ws_, stream);
}

int mlp_backward_dx(const mlp_t* h, const void* packed, const uint16_t* X, const float* dY,
                    float* G, float* dX, int64_t M, void* ws_, void* stream) {
  g_err.clear();
  if (int rc = check_handle(h)) return rc;
  if (M < 0) return fail(MLP_ERR_INVALID_ARG, "M = %lld < 0", (long long)M);
  if (!G || !ws_) return fail(MLP_ERR_INVALID_ARG, "null G or workspace");
  if (M > 0 && (!packed || !X || !dY)) return fail(MLP_ERR_INVALID_ARG, "null packed, X or dY");
  if (!aligned(G, 4) || !aligned(ws_, 256) ||
      (M > 0 && (!aligned(packed, 16) || !aligned(X, 16) || !aligned(dY, 16) || (dX && !aligned(dX, 16)))))
    return fail(MLP_ERR_INVALID_ARG, "misaligned pointer (packed, X, dY, dX: 16 bytes; ws: 256; G: 4)");
  if (M > ((int64_t)1 << 36)) return fail(MLP_ERR_INVALID_ARG, "M > 2^36");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const WsLayout w = ws_layout(h, M);
  uint8_t* ws = static_cast<uint8_t*>(ws_);
  if (!dX && n_mats(h) > 1) {
    const int rc = run_fused_backward(h, packed, X, dY, w, ws, M, G, nullptr, 0, 1, true, s);
    if (rc <= 0) return rc;
  }
  if (M > 0) {
    BwdArgs b = bwd_args(h, packed, w, ws, M);
    b.dY = dY;
    b.dX = dX;
    hipError_t e = launch_backward(h->width, h->act, 1, b, s);
    if (e != hipSuccess) return hip_fail(e, "backward kernel launch");
  }
  return run_wgrad_reduce(h, X, w, ws, M, G, nullptr, 0, s);
}

int mlp_train_step(const mlp_t* h, const void* packed, const uint16_t* X, const float* T,
                   uint16_t* Y, float* G, float* loss, int64_t M, void* ws_, void* stream) {
  g_err.clear();
  return train_step_impl(h, packed, X, T, Y, G, loss, M, ws_, stream);
}

int mlp_train_step_noalloc(const mlp_t* h, const void* packed, const uint16_t* X, const float* T,
                           uint16_t* Y, float* G, float* loss, int64_t M, void* stream) {
  g_err.clear();
  if (int rc = check_handle(h)) return rc;
  if (M >= 0 && M <= ((int64_t)1 << 36)) {
    const size_t need = ws_layout(h, M).total;
    if (need > kScratchBytes)
      return fail(MLP_ERR_WORKSPACE,
                  "a batch of %lld rows needs %zu workspace bytes, more than the %zu of the "
                  "static scratch array",
                  (long long)M, need, kScratchBytes);
  }
  void* ws = nullptr;
  hipError_t e = scratch_ptr(&ws);
  if (e != hipSuccess) return hip_fail(e, "scratch array lookup");
  return train_step_impl(h, packed, X, T, Y, G, loss, M, ws, stream);
}

}  // extern "C"

namespace {

int train_step_impl(const mlp_t* h, const void* packed, const uint16_t* X, const float* T,
                    uint16_t* Y, float* G, float* loss, int64_t M, void* ws_, void* stream) {
  if (int rc = check_handle(h)) return rc;
  if (M < 0) return fail(MLP_ERR_INVALID_ARG, "M = %lld < 0", (long long)M);
  if (!G || !ws_) return fail(MLP_ERR_INVALID_ARG, "null G or workspace");
  if (M > 0 && (!packed || !X || !T)) return fail(MLP_ERR_INVALID_ARG, "null packed, X or T");
  if (!aligned(G, 4) || !aligned(ws_, 256) || (loss && !aligned(loss, 4)) ||
      (M > 0 && (!aligned(packed, 16) || !aligned(X, 16) || !aligned(T, 16) || (Y && !aligned(Y, 8)))))
    return fail(MLP_ERR_INVALID_ARG,
                "misaligned pointer (packed, X, T: 16 bytes; Y: 8; ws: 256; G, loss: 4)");
  if (M > ((int64_t)1 << 36)) return fail(MLP_ERR_INVALID_ARG, "M > 2^36");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const WsLayout w = ws_layout(h, M);
  uint8_t* ws = static_cast<uint8_t*>(ws_);
  int nloss = 0;
  if (M > 0 && train_fused_supported(h->width, n_mats(h))) {
    // Widths 16 and 32: the whole step in one kernel, then the reduce.
    const PackGeom g = pack_geom(h);
    TrainfArgs t{};
    t.packedF = static_cast<const u32x4*>(packed);
    t.packedB = reinterpret_cast<const u32x4*>(static_cast<const uint8_t*>(packed) + (size_t)g.fwd_total * 1024);
    t.X = X;
    t.T = T;
    t.Y = Y;
    t.partial = reinterpret_cast<float*>(ws + w.partial);
    t.lossPart = reinterpret_cast<float*>(ws + w.lossPart);
    t.M = M;
    t.params = param_count(h);
    t.in_dim = h->in_dim;
    t.out_dim = h->out_dim;
    t.out_act = h->out_act;
    t.scale = (float)(2.0 / ((double)M * h->out_dim));
    t.fwd_total = g.fwd_total;
    int P = 0;
    hipError_t e = launch_train_fused(h->width, n_mats(h), h->act, h->out_dim, t, s, &P);
    if (e == hipSuccess) return run_reduce(h, w, ws, M, P, G, loss, P, s);
    if (e != hipErrorNotSupported) return hip_fail(e, "fused training kernel launch");
  }
  if (M > 0) {
    FwdArgs a = fwd_args(h, packed, X, M);
    a.Y = Y;
    a.T = T;
    a.stashA = reinterpret_cast<uint16_t*>(ws + w.stashA);
    a.stashS = h->act == MLP_ACT_SINE ? reinterpret_cast<uint16_t*>(ws + w.stashS) : nullptr;
    // The fused backward at widths up to 64 reads relu' from the stashed
    // activations (which it reads for the weight gradients anyway), so the
    // training forward writes no mask words for it.
    const bool fused = n_mats(h) > 1 &&
                       backward_fused_supported(h->width, n_mats(h), h->act, h->in_dim, h->out_dim);
    const bool masks = h->act == MLP_ACT_RELU && !(fused && h->width <= 64);
    a.reluMask = masks ? reinterpret_cast<uint32_t*>(ws + w.reluMask) : nullptr;
    // At width 128 the fused backward takes the activations transposed
    // (the forward has matrix-core time to spare, the backward does not).
    const bool stash_t = fused && h->width == 128 && masks;
    a.stash_t = stash_t ? 1 : 0;
    a.deltaOut = reinterpret_cast<uint16_t*>(ws + w.deltaOut);
    a.lossPart = reinterpret_cast<float*>(ws + w.lossPart);
    hipError_t e = launch_forward(h->width, h->act, FWD_TRAIN, a, s, &nloss);
    if (e != hipSuccess) return hip_fail(e, "forward kernel launch");
    if (n_mats(h) > 1) {
      const int rc = run_fused_backward(h, packed, X, nullptr, w, ws, M, G, loss, nloss, 0, masks, s, stash_t);
      if (rc <= 0) return rc;
      if (stash_t)  // no other backward reads the transposed stash
        return fail(MLP_ERR_UNSUPPORTED, "fused backward kernel unavailable on this device");
      if (h->act == MLP_ACT_RELU && !masks)  // the unfused backward needs the masks
        return fail(MLP_ERR_UNSUPPORTED, "fused backward kernel unavailable on this device");
      BwdArgs b = bwd_args(h, packed, w, ws, M);
      e = launch_backward(h->width, h->act, 0, b, s);
      if (e != hipSuccess) return hip_fail(e, "backward kernel launch");
    }
  }
  return run_wgrad_reduce(h, X, w, ws, M, G, loss, nloss, s);
}

}  // namespace
