// kernels.hpp -- launch interface of the HIP kernels (gfx950).
//
// All activations are fp32 NCHW over the k*b images of one iteration;
// replica j owns images [j*b, (j+1)*b).  Parameters of replica j start at
// params + j*pstride.  Every launcher enqueues on the given stream and
// returns the hipError_t of the launch.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

namespace cbk {

// Records the message that cb_last_error(NULL) returns (a failure of a call
// made without a context).
void note_error(const std::string& msg);

// Per-launch timing.  When armed, the next kernel launch on this thread
// passes the two events to hipExtLaunchKernel, which stamps them on the
// kernel's own dispatch: the interval is the kernel alone, with no marker
// packets added around it.  Unarmed launches are plain kernel launches,
// which a stream capture records as graph nodes.  Every kernel of this
// library goes through klaunch.
struct LaunchTiming {
  hipEvent_t start = nullptr, stop = nullptr;
};
inline thread_local LaunchTiming g_launch_timing;

template <typename... P, typename... A>
inline void klaunch(void (*kernel)(P...), dim3 grid, dim3 block, uint32_t shm, hipStream_t s,
                    A... args) {
  const LaunchTiming t = g_launch_timing;
  g_launch_timing = LaunchTiming();
  if (t.start)
    hipExtLaunchKernelGGL(kernel, grid, block, shm, s, t.start, t.stop, 0u, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, shm, s, args...);
}

// Raw buffer reads: a wave-uniform descriptor over `bytes` bytes from base
// and a 32-bit byte offset per lane.  An offset at or past `bytes` reads 0
// (the buffer range check), which gives tiles their zero border, and
// loaders their out-of-range elements, with no branch: such lanes use
// OUTSIDE.  `bytes` must stay below 2 GiB.
constexpr uint32_t OUTSIDE = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const float* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), 0, (int)bytes, 0x00020000);
}
// The same descriptor from values the caller knows to be wave-uniform, moved
// to scalar registers first, so that no load has to loop over lanes.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc_u(const float* base, uint32_t bytes) {
  const uint64_t p = reinterpret_cast<uintptr_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)p);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
  return buf_rsrc(reinterpret_cast<const float*>(((uint64_t)hi << 32) | lo),
                  __builtin_amdgcn_readfirstlane(bytes));
}
__device__ __forceinline__ float buf_ld(__amdgpu_buffer_rsrc_t r, uint32_t off_bytes) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off_bytes, 0, 0));
}
typedef float buf_v4f __attribute__((ext_vector_type(4)));
// four consecutive floats; the whole quad reads 0 when it starts at or past `bytes`
__device__ __forceinline__ buf_v4f buf_ld4(__amdgpu_buffer_rsrc_t r, uint32_t off_bytes) {
  return __builtin_bit_cast(buf_v4f, __builtin_amdgcn_raw_buffer_load_b128(r, off_bytes, 0, 0));
}

// Workgroups are handed to the eight XCDs in turn (workgroup w to XCD
// w % 8).  Renumbering them XCD-major gives the workgroups of one XCD a
// contiguous range of ids, so the neighbouring tiles they take share halo
// rows and filters in that XCD's L2.  A bijection on [0, G) for any G.
constexpr int NXCD = 8;
__device__ __forceinline__ int xcd_major(int w, int G) {
  const int x = w % NXCD, i = w / NXCD, q = G / NXCD, r = G % NXCD;
  return x * q + min(x, r) + i;
}

// Geometry of one convolution layer (an FC layer is a 1x1 conv on a 1x1
// image).  b = images per replica, k = replicas.
struct ConvGeom {
  int k, b;
  int Ci, H, W;
  int Co, R, S;
  int st, pad;
  int Ho, Wo;
};

struct ConvFwdArgs {
  ConvGeom g;
  const float* x;     // [k*b][Ci][H][W]
  const float* w;     // replica 0 weights [Co][Ci][R][S]
  const float* bias;  // replica 0 bias [Co] or nullptr
  int64_t pstride;    // elements between replicas' parameters
  float* y;           // [k*b][Co][Ho][Wo]
  int relu;
  // If not null: per-channel partial sums (sum, sum of squares) of the
  // stored outputs of each M tile, [k][Co][tiles_m][2], for the batch norm
  // that consumes y (tiles_m = conv_fwd_tiles_m).
  double* stats;
};

// Residual added to a data gradient (the shortcut of a residual block):
//   ADD_SAME: add src at the same index;
//   ADD_SUBSAMPLE: src is [k*b][Csrc][ceil(H/st)][ceil(W/st)]; dX[n][c][h][w]
//     gets src[n][c][h/st][w/st] when h and w are multiples of st (option-A
//     shortcut read backwards; c < Ci <= Csrc).
enum { ADD_NONE = 0, ADD_SAME = 1, ADD_SUBSAMPLE = 2 };

// A batch norm's output before its residual input and ReLU,
// gamma * (x - mean) * istd + beta, as one fixed sequence of fp32 operations
// (a multiply, then a fused multiply-add), so that a backward kernel that
// recomputes the ReLU decision from x takes exactly the forward's.
__device__ __forceinline__ float bn_affine(float x, float mean, float istd, float ga, float be) {
  return __builtin_fmaf(ga, (x - mean) * istd, be);
}

struct ConvBwdDataArgs {
  ConvGeom g;
  const float* dy;    // [k*b][Co][Ho][Wo]
  const float* w;     // replica 0 weights
  int64_t pstride;
  float* dx;          // [k*b][Ci][H][W]
  int accumulate;     // dx += result instead of dx = result
  const float* mask;  // zero dx where mask <= 0 (a fused ReLU upstream), or nullptr
  const float* add;   // residual gradient, or nullptr
  int add_mode, add_C, add_st;
  // If bn_part is not null, dx is the output gradient of a batch norm; the
  // epilogue also writes that norm's backward partial sums per M tile:
  // with d = dx masked where the norm's ReLU output bn_y is not positive
  // (bn_y null: no mask) and xh = (bn_x - mean) * istd: sum d and sum
  // d*xh, [k][Ci][tiles_m][2].  For a norm with no residual input the
  // caller may also give bn_gamma: the implicit-GEMM epilogue and the
  // direct stride-1 kernels then recompute the ReLU output's sign as
  // bn_affine of bn_x instead of reading bn_y.
  double* bn_part;
  const float* bn_x;
  const float* bn_y;
  const float* bn_mean;
  const float* bn_istd;
  const float* bn_gamma = nullptr;  // replica 0 gamma [Ci], beta at + Ci; pstride apart
  // The mask is that norm's own ReLU output (bn_y null, bn_gamma given):
  // the direct kernels then take the mask's decision as bn_affine of bn_x
  // instead of reading the mask.
  bool mask_from_bn = false;
};

struct ConvBwdWeightArgs {
  ConvGeom g;
  const float* x;     // [k*b][Ci][H][W]
  const float* dy;    // [k*b][Co][Ho][Wo]
  float* dw;          // replica 0 gradient [Co][Ci][R][S] (splits == 1)
  int64_t pstride;
  float* partial;     // [k][splits][Co][Ci*R*S] (splits > 1)
  int splits, chunk;  // contraction (b*Ho*Wo) split into `splits` chunks
};

// Square filters R in {1, 3, 5, 7}, stride 1 or 2; the data gradient is
// built for (R, stride) in {(1,1), (1,2), (3,1), (3,2), (5,1)}.
bool conv_supported(int R, int S, int st, bool need_dx);
// Number of M tiles of the forward / data-gradient GEMMs (the counts of the
// batch-norm partial sums their epilogues write).
int conv_fwd_tiles_m(const ConvGeom& g);
int conv_bwd_data_tiles_m(const ConvGeom& g);
// Split of the weight-gradient contraction; exposed so the host can size scratch.
int conv_bwd_weight_splits(const ConvGeom& g, int* chunk);

// The conv launchers pick a tile shape from the layer's sizes; *name (if
// not null) receives the launched kernel's name, for instrumentation.
hipError_t conv_fwd(const ConvFwdArgs& a, hipStream_t s, const char** name = nullptr);
hipError_t conv_bwd_data(const ConvBwdDataArgs& a, hipStream_t s, const char** name = nullptr);
hipError_t conv_bwd_weight(const ConvBwdWeightArgs& a, hipStream_t s,
                           const char** name = nullptr);
// 3x3 stride-1 pad-1 convolutions on 8/16/32-wide square images with
// channel counts that are multiples of 16 run on a direct kernel (input
// tile staged once in LDS); conv_fwd / conv_bwd_data route there
// themselves.  *_tiles give its number of row tiles per replica (the count
// of batch-norm partial sums its epilogue writes).
bool conv_direct_fwd_ok(const ConvGeom& g);
bool conv_direct_bwd_data_ok(const ConvGeom& g);
int conv_direct_fwd_tiles(const ConvGeom& g);
int conv_direct_bwd_data_tiles(const ConvGeom& g);
// 3x3 stride-2 pad-1 data gradients (dX 16 or 32 wide, channel counts
// multiples of 16) run on a kernel that splits dX by pixel parity
// (conv_bwd_data routes; *_tiles as above).
bool conv_s2_dgrad_ok(const ConvGeom& g);
int conv_s2_dgrad_tiles(const ConvGeom& g);
hipError_t conv_s2_dgrad(const ConvBwdDataArgs& d, hipStream_t s, const char** name = nullptr);
// Their weight gradient has a direct kernel too (conv_bwd_weight routes;
// conv_bwd_weight_splits reports its split).
bool conv_direct_wgrad_ok(const ConvGeom& g);
int conv_direct_wgrad_splits(const ConvGeom& g);
hipError_t conv_direct_wgrad(const ConvBwdWeightArgs& a, hipStream_t s,
                             const char** name = nullptr);
hipError_t conv_direct_fwd(const ConvFwdArgs& a, hipStream_t s, const char** name = nullptr);
hipError_t conv_direct_bwd_data(const ConvBwdDataArgs& a, hipStream_t s,
                                const char** name = nullptr);
// Weight-gradient split reduction of up to MAX_SPLIT_SEGS layers in one
// launch (the table travels as the kernel argument):
//   seg.dw[j*pstride + e] = sum over s of seg.partial[j][s][e], s in order.
constexpr int MAX_SPLIT_SEGS = 80;
struct SplitSeg {
  const float* partial;  // [k][splits][n]
  float* dw;             // replica 0 destination
  int64_t n;
  int splits;
  int block0;            // first 64-element block of this segment
};
template <int S>
struct SplitTableT {
  int nseg = 0, blocks = 0;
  int64_t pstride = 0;
  SplitSeg seg[S];
};
using SplitTable = SplitTableT<MAX_SPLIT_SEGS>;
// Tables of at most this many layers launch with a short kernel argument
// (the full table is 2.6 KB, which the host copies on every launch).
constexpr int SMALL_SPLIT_SEGS = 4;
void split_table_add(SplitTable& t, const float* partial, float* dw, int64_t n, int splits);
hipError_t reduce_splits(const SplitTable& t, int k, hipStream_t s, const char** name = nullptr);
// db[j][c] = sum over replica j's images and pixels of dy[n][c][p].
// With terms (per-image loss terms [k*b]), also mean[j] = the mean of
// replica j's b terms, summed in image order.
hipError_t channel_sum(const float* dy, int k, int b, int C, int HW, float* db,
                       int64_t pstride, hipStream_t s, const float* terms = nullptr,
                       float* mean = nullptr);

// Batch norm with per-replica batch statistics.
enum { RES_NONE = 0, RES_SAME = 1, RES_SUBSAMPLE = 2 };

struct BNArgs {
  int k, b, C, H, W;
  const float* x;       // conv output [k*b][C][H][W]
  float* y;             // output
  const float* gamma;   // replica 0 gamma [C]; beta follows at gamma + C
  int64_t pstride;
  float* mean;          // [k][C] saved for backward
  float* istd;          // [k][C]
  double* part;         // partial sums [k][C][parts][2]
  int parts;            // partials per (replica, channel)
  int chunks;           // blocks per (replica, channel) in the kernels' grids
  int relu;
  const float* res;     // residual input or nullptr
  int res_mode, res_C, res_st, res_H, res_W;
};

struct BNBwdArgs {
  int k, b, C, H, W;
  const float* x;       // conv output (BN input)
  const float* y;       // BN output (for the ReLU mask) or nullptr
  int relu_x = 0;       // y null: the ReLU mask is bn_affine(x) > 0 (no residual input)
  const float* dy;      // gradient at the BN output (before the ReLU mask)
  float* dx;            // gradient at the BN input
  float* dres;          // masked output gradient for the shortcut, or nullptr
  const float* gamma;
  float* dgamma;        // replica 0 gradient of gamma; beta's follows at + C
  int64_t pstride;
  const float* mean;
  const float* istd;
  double* part;         // partial sums [k][C][parts][2]
  int parts;
  int chunks;
};

int bn_chunks(int b, int HW, int C, int k);
// Forward: per-chunk fp64 sums (parts = chunks), then normalise (+ residual,
// ReLU).  The sums can instead come from the producing conv's epilogue.
hipError_t bn_fwd_stats(const BNArgs& a, hipStream_t s);
hipError_t bn_fwd_apply(const BNArgs& a, hipStream_t s, const char** name = nullptr);
// Backward: per-chunk fp64 sums of dy and dy*xhat (parts = chunks), then dx
// and dgamma/dbeta.  The sums can instead come from the epilogue of the
// data-gradient GEMM that wrote dy.
hipError_t bn_bwd_stats(const BNBwdArgs& a, hipStream_t s);
hipError_t bn_bwd_apply(const BNBwdArgs& a, hipStream_t s, const char** name = nullptr);

hipError_t maxpool_fwd(const float* x, int N, int C, int H, int W, int K, int st, int pad,
                       float* y, int Ho, int Wo, int* arg, hipStream_t s);
// dx over the whole input; mask_relu zeroes entries whose input was <= 0.
hipError_t maxpool_bwd(const float* dy, const int* arg, const float* x, int N, int C, int H,
                       int W, int K, int st, int pad, int Ho, int Wo, float* dx, int mask_relu,
                       hipStream_t s);
hipError_t gap_fwd(const float* x, int N, int C, int HW, float* y, hipStream_t s);
hipError_t gap_bwd(const float* dy, int N, int C, int HW, float* dx, hipStream_t s,
                   const char** name = nullptr);
// Mean softmax cross-entropy per replica and its gradient wrt the logits.
// The network head of one image in one launch: global average pool, an FC
// layer with at most HEAD_MAX_CLASSES outputs (no ReLU), softmax
// cross-entropy, then the backward down to the pooled tensor's gradient
// (and the backward partial sums of the batch norm that produced it).
constexpr int HEAD_MAX_C = 1024, HEAD_MAX_CLASSES = 32;
// per image at most HEAD_MAX_PLANE pooled values (HEAD_PASSES float4s per
// thread) and HEAD_MAX_W FC weights (staged in LDS)
constexpr int HEAD_MAX_PLANE = 4096, HEAD_PASSES = HEAD_MAX_PLANE / 1024, HEAD_MAX_W = 4096;
struct HeadArgs {
  int k, b, C, HW, classes;
  const float* y;        // pooled input [k*b][C][HW]
  float* g;              // pooled features [k*b][C] (the FC input, kept for its weight gradient)
  const float* w;        // replica 0 FC weights [classes][C]
  const float* bias;     // replica 0 bias [classes], or nullptr
  int64_t pstride;
  const int32_t* labels; // [k*b]
  float* dlogits;        // [k*b][classes]
  float* loss;           // per image [k*b]; a replica's loss is the mean of its b
  float* dy;             // gradient at the pooled input [k*b][C][HW]
  // If bn_part is set, y is the output of a batch norm (ReLU'd if bn_relu):
  // its backward partial sums per image as in ConvBwdDataArgs, [k][C][b][2].
  double* bn_part;
  int bn_relu;
  const float* bn_x;
  const float* bn_mean;
  const float* bn_istd;
};
// Shapes the head kernel takes: C <= HEAD_MAX_C, 1 <= classes <=
// HEAD_MAX_CLASSES, HW a multiple of 4 with HW/4 a power of two up to 64,
// C*HW <= HEAD_MAX_PLANE, classes*C <= HEAD_MAX_W.
bool head_ok(int C, int HW, int classes);
hipError_t head_fwd_bwd(const HeadArgs& a, hipStream_t s);
hipError_t softmax_xent(const float* logits, const int32_t* labels, int k, int b, int classes,
                        float* dlogits, float* loss, hipStream_t s,
                        const char** name = nullptr);

// The MNIST-shaped LeNet (1 x 28 x 28 images) in two launches: one
// workgroup per image for the forward pass, the loss and the backward data
// path (lenet_image), then each learner's gradient and mean loss
// (lenet_learner).
constexpr int LENET_MAX_CLASSES = 64;
constexpr int LENET_CONV_PARAMS = 150 + 6 + 2400 + 16;  // conv1 w, b, conv2 w, b
// per image, the FC layers' inputs and output gradients:
// p2 (400) | df1 (120) | f1 (120) | df2 (84) | f2 (84) | dlogits (<= 64)
constexpr int LENET_DF1 = 400, LENET_F1 = 520, LENET_DF2 = 640, LENET_F2 = 724,
              LENET_DL = 808, LENET_FC_VEC = 872;
constexpr int LENET_LEARNER_BLOCKS = 260;  // ceil(P / 256) for up to 64 classes
struct LenetArgs {
  int k, b, classes;
  const float* x;        // [k*b][1][28][28]
  const int32_t* labels; // [k*b]
  const float* w;        // replica 0 parameters (pstride apart)
  float* grad;           // replica 0 gradient
  int64_t pstride;
  float* loss;           // per image [k*b]
  float* learner_loss;   // per learner [k]: the mean over its b images
  float* conv_part;      // [k*b][LENET_CONV_PARAMS]: each image's share of the conv gradients
  float* fc_vec;         // [k*b][LENET_FC_VEC]
};
bool lenet_fused_ok(int in_c, int in_h, int in_w, int classes);
hipError_t lenet_image(const LenetArgs& a, hipStream_t s);
hipError_t lenet_learner(const LenetArgs& a, hipStream_t s);

// Fused SMA synchronisation (Algorithm 1).  W, G, Wprev are [k][stride];
// z, zp are [>= P] with P padded to a multiple of 4 elements.
struct SMAArgs {
  float* W;
  const float* G;
  float* Wprev;          // nullptr unless learner momentum is on
  float* z;
  float* zp;
  int k;
  int64_t P4;            // number of float4 columns
  int64_t wstride4, gstride4;
  float alpha, lr, mu, mu_l;
  int correct;           // 0: local step only (no correction, z untouched)
};
hipError_t sma_step(const SMAArgs& a, hipStream_t s, const char** name = nullptr);
// flag[0] = 1 if any of z[0..n) is NaN/Inf (flag must be zeroed first).
hipError_t nonfinite_scan(const float* z, int64_t n, int* flag, hipStream_t s);
hipError_t zero_ints(int* p, int n, hipStream_t s);

}  // namespace cbk
