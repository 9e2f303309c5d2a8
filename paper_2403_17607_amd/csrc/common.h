// Internal declarations shared by the kernels and the C-ABI layer.
//
// Register and memory layouts (all built around the gfx950 matrix-core
// instruction v_mfma_f32_16x16x32_bf16, wave64):
//
//  * MFMA operands.  For out[i][n] = sum_p A[i][p] B[p][n] (16x16 output,
//    32 contraction positions p), lane l holds row i = l % 16 of A (column
//    n = l % 16 of B) and eight contraction positions in slots 0..7; the
//    lane group g = l / 16 picks which eight.  A and B use the same
//    (g, slot) -> p assignment, so only the pairing matters: any bijection
//    between (g, slot) and the features being contracted gives the same
//    product.  The fp32 result of lane l holds out[4 g + r][l % 16], r < 4.
//
//  * Transposed layer product.  A layer computes C^T = W^T A^T: the packed
//    weights are the A operand (rows = output features), the activations of
//    16 batch rows are the B operand (columns = batch rows).  The result of
//    a 16-feature "strip" s gives lane (g, i) the features 16 s + 4 g + r of
//    batch row i, exactly where the next layer's B operand wants batch row
//    i.  Two strips (2 kb, 2 kb + 1) form k-block kb of the next layer:
//        slot q < 4  <- feature 32 kb + 4 g + q        (strip 2 kb)
//        slot q >= 4 <- feature 32 kb + 16 + 4 g + q-4 (strip 2 kb + 1)
//    This "chain order" is folded into the packed weights, so activations
//    never move between lanes.  The first layer reads X straight from
//    memory in "input order": slot q of group g <- feature 32 kb + 8 g + q.
//
//  * Packed weights (1 KiB fragments, [strip][k-block][lane][slot] bf16):
//    forward layer l: A[j][p] = W_l[f(p)][j], j = output feature;
//    backward layer l >= 1: A[f][p] = W_l[f][j(p)], f = input feature, for
//    the delta product D_l^T = W_l D_{l+1}^T.  Every layer has the width's
//    k-block count; out-of-range entries are 0.
//
//  * Tile image (stash tensors [M16][F], F a multiple of 16): the fp32 or
//    bf16 result registers of a wave, stored as they are.  Element (m, f)
//    lives at ((m/16 * F/16 + f/16) * 64 + ((f%16)/4) * 16 + m%16) * 4 + f%4.
//    Every 16-row block of a strip is 64 lanes x 4 values, contiguous.
//
//  * ReLU masks ([M16 / 16][64] 32-bit words per hidden activation, ReLU
//    nets only): the word of lane (g, i) for 16-row block b holds, for
//    strip s, [A[16 b + i][16 s + 4 g + r] > 0] in bit 2 s + r / 2 + 16 (r % 2)
//    (r = 0, 2 in the low half, r = 1, 3 in the high half), so one shift
//    and one AND give the 0/1 multipliers of a packed bf16 pair.  The
//    backward pass reads these instead of the bf16 activations.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ffmlp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

enum { ACT_LINEAR = 0, ACT_RELU = 1, ACT_SIGMOID = 2, ACT_SINE = 3 };

// Rows per workgroup tile in the fused forward and backward kernels:
// NT 16-row blocks per wave, NW waves per workgroup.
template <int W> struct TileCfg;
template <> struct TileCfg<16> { static constexpr int NT = 4, NW = 4; };
template <> struct TileCfg<32> { static constexpr int NT = 4, NW = 4; };
template <> struct TileCfg<64> { static constexpr int NT = 4, NW = 4; };
template <> struct TileCfg<128> { static constexpr int NT = 4, NW = 8; };

inline int tile_rows(int width) {
  switch (width) {
    case 16: return TileCfg<16>::NT * TileCfg<16>::NW * 16;
    case 32: return TileCfg<32>::NT * TileCfg<32>::NW * 16;
    case 64: return TileCfg<64>::NT * TileCfg<64>::NW * 16;
    default: return TileCfg<128>::NT * TileCfg<128>::NW * 16;
  }
}

// Weight-gradient kernel geometry: each wave owns a TBK x TBJ block of
// 16x16 output tiles; GK x GJ blocks cover G; KS waves split every chunk of
// the batch; each wave runs KSW 32-row contraction steps per chunk.
template <int W> struct WgCfg;
// The chunk is CH = 32 KS KSW rows, so CH * W / 8 = 2048 16-byte units per
// tensor at every width (eight per thread, all in flight at once).
template <> struct WgCfg<16> { static constexpr int TBK = 1, TBJ = 1, GK = 1, GJ = 1, KS = 4, KSW = 8; };
template <> struct WgCfg<32> { static constexpr int TBK = 2, TBJ = 2, GK = 1, GJ = 1, KS = 4, KSW = 4; };
template <> struct WgCfg<64> { static constexpr int TBK = 2, TBJ = 2, GK = 2, GJ = 2, KS = 1, KSW = 8; };
template <> struct WgCfg<128> { static constexpr int TBK = 4, TBJ = 4, GK = 2, GJ = 2, KS = 1, KSW = 4; };
template <int W> constexpr int wg_chunk() { return 32 * WgCfg<W>::KS * WgCfg<W>::KSW; }
inline int wgrad_chunk(int width) {
  switch (width) {
    case 16: return wg_chunk<16>();
    case 32: return wg_chunk<32>();
    case 64: return wg_chunk<64>();
    default: return wg_chunk<128>();
  }
}

constexpr int kMaxLossParts = 4096;  // upper bound on forward workgroups
constexpr int kWgradTargetBlocks = 1024;

struct FwdArgs {
  const u32x4* packed;  // forward-packed weights, all layers
  const uint16_t* X;    // [M][in_dim]
  uint16_t* Y;          // [M][out_dim] or null (train mode only)
  const float* T;       // [M][out_dim] targets (train mode)
  uint16_t* stashA;     // (L-1) x [M16][W] tile images: a_1 .. a_{L-1}
  uint16_t* stashS;     // same shape, bf16(cos c) of sine layers, or null
  uint16_t* deltaOut;   // [M16][OP] tile image of the output delta (train)
  float* cOut;          // [M16][OP] fp32 tile image of c_{L-1} (stash mode)
  uint32_t* reluMask;   // (L-1) x [M16/16][64] ReLU mask words, or null
  float* lossPart;      // one partial sum per workgroup (train)
  int64_t M, M16;
  int in_dim, out_dim, L, out_act;
  float scale;          // 2 / (M out_dim)
  int ntiles, resident;
  uint32_t lay0_frags, layH_frags, total_frags;  // 1 KiB fragment counts
  int stash_t;          // training forward at width 128 for the fused backward:
                        // stashA holds each strip transposed (see fwd_kernel.h)
};

struct BwdArgs {
  const u32x4* packed;  // backward-packed weights, layers 1 .. L-1
  const uint16_t* stashA;
  const uint16_t* stashS;
  uint16_t* deltaH;     // (L-1) x [M16][W]: delta_0 .. delta_{L-2}
  uint16_t* deltaOut;   // [M16][OP]: delta_{L-1}
  const float* cOut;    // [M16][OP] fp32 (seeded mode, nonlinear output)
  const float* dY;      // [M][out_dim] (seeded mode)
  const uint32_t* reluMask;  // (L-1) x [M16/16][64] ReLU mask words (ReLU nets)
  const u32x4* packed0;  // backward-packed layer 0 (input gradient), read from global
  float* dX;             // [M][in_dim] input gradient, or null
  int64_t M, M16;
  int in_dim, out_dim, L, out_act;
  int ntiles, resident;
  uint32_t layH_frags, total_frags;
};

// Fused backward pass with the weight gradients (bwdg_kernel): the deltas
// never go to HBM; each workgroup keeps fixed slices of every layer's G in
// registers across its row tiles and writes them once, as one partial.
constexpr int kBwdgWaves = 8;        // waves per workgroup, 16 rows each
constexpr int kBwdgRows = 16 * kBwdgWaves;  // rows per tile
constexpr int kBwdgMaxBlocks = 512;  // at most this many partials
constexpr int kBwdgMaxL = 5;         // weight matrices of the largest fused net
struct BwdgArgs {
  const u32x4* packed;       // backward-packed weights, layers 1 .. L-1
  const uint16_t* X;         // [M][in_dim]
  const uint16_t* stashA;    // (L-1) x [M16][W] tile images: a_1 .. a_{L-1}
  const uint32_t* reluMask;  // (L-1) x [M16/16][64] ReLU mask words (ReLU nets)
  const uint16_t* stashS;    // (L-1) x [M16][W] bf16 cos of sine layers, or null
  const uint16_t* deltaOut;  // [M16][OP] output delta (training step)
  const float* cOut;         // [M16][OP] fp32 pre-activation (seeded, nonlinear output)
  const float* dY;           // [M][out_dim] (seeded mode)
  float* partial;            // [gridDim.x][params]
  int64_t M, M16, params;
  int in_dim, out_dim, act, out_act;
  int ntiles;                // kBwdgRows-row tiles
  uint32_t layH_frags;       // 1 KiB fragments of one packed hidden layer
  int stash_t;               // stashA written transposed (FwdArgs::stash_t)
};

// Fused training step (trainf_kernel): the forward pass, the loss, the
// backward pass and the weight gradients of nets of width 16 and 32 in one
// kernel; the hidden activations stay in registers.
constexpr int kTrainfWaves = 8;  // waves per workgroup
constexpr int kTrainfMaxL = 5;   // weight matrices of the largest net
struct TrainfArgs {
  const u32x4* packedF;  // forward-packed weights, layers 0 .. L-1
  const u32x4* packedB;  // backward-packed weights, layers 1 .. L-1
  const uint16_t* X;     // [M][in_dim]
  const float* T;        // [M][out_dim]
  uint16_t* Y;           // [M][out_dim] or null
  float* partial;        // [gridDim.x][params]
  float* lossPart;       // [gridDim.x]
  int64_t M, params;
  int in_dim, out_dim, out_act;
  float scale;           // 2 / (M out_dim)
  int ntiles;            // set by the launcher
  uint32_t fwd_total;    // 1 KiB fragments of the forward-packed layers
};

struct WgradArgs {
  const uint16_t* X;
  const uint16_t* stashA;
  const uint16_t* deltaH;
  const uint16_t* deltaOut;
  float* partial;       // [P][param_count]
  int64_t M, M16, params;
  int in_dim, out_dim, L;
  int P, chunks_per_block;
};

// Fixed-order sum of the P weight-gradient partials: slice y (partials
// [y P / S, (y+1) P / S)) is added in order, then the S slice sums in order
// into G; the same kernel sums the loss partials.
constexpr int kReduceSlices = 16;
struct ReduceArgs {
  const float* partial;  // [P][params]
  float* G;
  int64_t params;
  int P;
  const float* lossPart;
  int nloss;
  float* loss;
  float loss_scale;
};

struct PackArgs {
  const uint16_t* W;  // all weights, concatenated [fan_in][fan_out] matrices
  uint16_t* dst;      // packed buffer: forward layers, then backward layers
  int width, in_dim, out_dim, L;
  int64_t total;      // bf16 elements of the packed buffer
};

struct OptArgs {
  float* master;      // fp32 master weights, updated in place
  float* m;           // Adam first moments (null for SGD)
  float* v;           // Adam second moments (null for SGD)
  const float* G;     // gradients, the weights' layout
  uint16_t* W;        // bf16 copy of the updated master weights
  int64_t n;          // parameter count
  int adam;
  float lr, beta1, beta2, eps;
  float step_size;     // lr / (1 - beta1^t)
  float inv_sqrt_bc2;  // 1 / sqrt(1 - beta2^t)
};

// Host-side launchers (one per translation unit).  They return a HIP error.
hipError_t launch_forward(int width, int act, int mode, const FwdArgs& a,
                          hipStream_t s, int* grid_out);
hipError_t launch_backward(int width, int act, int seeded, const BwdArgs& a,
                           hipStream_t s);
hipError_t launch_wgrad(int width, const WgradArgs& a, hipStream_t s);
// Fused backward pass and weight-gradient partials; *grid_out receives the
// number of partials written.  hipErrorNotSupported when no instantiation
// covers the net (the caller then runs the unfused kernels).
hipError_t launch_backward_fused(int width, int L, int out_dim, int seeded, const BwdgArgs& a,
                                 hipStream_t s, int* grid_out);
// Whether launch_backward_fused covers a net (host-side shape check only).
bool backward_fused_supported(int width, int L, int act, int in_dim, int out_dim);
// Fused training step; *grid_out receives the number of G and loss
// partials written.  hipErrorNotSupported when it does not cover the net.
hipError_t launch_train_fused(int width, int L, int act, int out_dim, const TrainfArgs& a,
                              hipStream_t s, int* grid_out);
// Whether launch_train_fused covers a net (host-side shape check only).
bool train_fused_supported(int width, int L);
hipError_t launch_reduce(const ReduceArgs& a, hipStream_t s);
hipError_t launch_pack(const PackArgs& a, hipStream_t s);
hipError_t launch_optim(const OptArgs& a, hipStream_t s);

// Forward kernel modes.
enum { FWD_INFER = 0, FWD_STASH = 1, FWD_TRAIN = 2 };

struct DeviceInfo {
  int cus;
  int max_lds;  // bytes of LDS one workgroup may use
};
hipError_t device_info(DeviceInfo* out);

// Prepares `kernel` on the current device for `lds` bytes of dynamic LDS
// (raising its limit when needed) and returns how many of its workgroups
// of `threads` fit on one compute unit.  Cached per (device, kernel, lds),
// so repeated launches make no runtime queries.
hipError_t kernel_occupancy(const void* kernel, int threads, size_t lds, int* blocks_per_cu);

}  // namespace ffmlp
