/*
 * crossbow_sma.h -- C ABI of the MI355X library for synchronous model
 * averaging (SMA) of k learners co-resident on one GPU.
 *
 * Method: Koliousis et al., "Crossbow: Scaling Deep Learning with Small
 * Batch Sizes on Multi-GPU Servers", VLDB 2019 (arXiv 1901.02244),
 * Algorithm 1 in Sec. 3.2.  Each of k learners trains its own replica w_j on
 * its own batch of b images (Sec. 3.1); one synchronisation per iteration
 * corrects every replica towards the central average model z and folds the
 * corrections, with momentum, into z.
 *
 * Conventions for every entry point:
 *   - Return value: CB_OK (0) or a negative CB_E* code; cb_last_error()
 *     gives a message.  After CB_EDEVICE the context is only good for
 *     cb_destroy().
 *   - "_dev" pointers are device memory on the device that was current at
 *     cb_create; "_host" pointers are ordinary host memory.
 *   - Every GPU operation is enqueued on the HIP stream given to cb_create,
 *     in call order.  Calls return once the work is enqueued unless stated
 *     otherwise.  A context is not thread-safe.
 *   - The library never allocates device memory: the caller hands over one
 *     workspace of cb_workspace_bytes() bytes and keeps it alive until
 *     cb_destroy().  The library frees no caller memory.
 *   - Images are fp32 NCHW [k*b][C][H][W]; labels are int32 [k*b].  Learner j
 *     trains on images [j*b, (j+1)*b) (the batch selection of Algorithm 1).
 *   - Parameters are fp32 in one flat vector of P elements, per layer in
 *     forward order: conv weight [Cout][Cin][R][S] then its bias; batch-norm
 *     gamma then beta; FC weight [out][in] then bias.  cb_tensor_info()
 *     describes each tensor.
 */
#ifndef CROSSBOW_SMA_H
#define CROSSBOW_SMA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Version of this interface: raised with every change to a declaration
 * below.  cb_abi_version() returns the value the library was built with;
 * a caller built against another version must not call anything else. */
#define CB_ABI_VERSION 3
int cb_abi_version(void);

typedef struct cb_ctx cb_ctx;

enum {
  CB_OK = 0,
  CB_EINVAL = -1,     /* bad argument or unsupported model description */
  CB_ENOMEM = -2,     /* workspace smaller than cb_workspace_bytes() */
  CB_EDEVICE = -3,    /* a HIP call failed */
  CB_ESTATE = -4,     /* call out of order (e.g. cb_sync with nothing pending) */
  CB_ENONFINITE = -5  /* z holds a NaN or Inf after cb_sync (check_finite set) */
};

/* The three networks of Table 1 that the workloads use (Sec. 5.1). */
enum { CB_ARCH_LENET5 = 1, CB_ARCH_RESNET32 = 2, CB_ARCH_RESNET50 = 3 };

/* Parameter tensor kinds reported by cb_tensor_info(). */
enum { CB_KIND_CONV_W = 0, CB_KIND_BIAS = 1, CB_KIND_BN_GAMMA = 2, CB_KIND_BN_BETA = 3,
       CB_KIND_FC_W = 4 };

typedef struct {
  int32_t arch;             /* CB_ARCH_* */
  int32_t in_c, in_h, in_w; /* image shape */
  int32_t num_classes;
  /* Heavy-ball momentum on each replica, mu_L (Eq. 3 applied per learner):
   * w_j <- w_j - lr*g_j - c_j + mu_L (w_j - w_j_prev).  0 is Algorithm 1 as
   * printed; nonzero costs one more [k][P] array in the workspace. */
  float learner_momentum;
  /* If nonzero, cb_sync() waits for the stream and scans z for NaN/Inf. */
  int32_t check_finite;
} cb_model;

/* Number of parameters P of the network, or CB_EINVAL. */
int64_t cb_num_params(const cb_model* m);

/* Number of parameter tensors, or CB_EINVAL. */
int cb_num_tensors(const cb_model* m);

/* Tensor idx of the flat parameter vector: element offset, CB_KIND_*, rank
 * (1, 2 or 4) and dims (dims4[i] = 1 beyond the rank).  CB_EINVAL if idx is
 * out of range. */
int cb_tensor_info(const cb_model* m, int idx, int64_t* offset, int* kind, int* ndim,
                   int* dims4);

/* Bytes of device workspace that cb_create needs for k learners of batch b
 * (replicas, gradients, z, z_prev, activations, scratch) -- enough for any
 * number of active learners up to k (cb_set_learners); 0 on bad input. */
size_t cb_workspace_bytes(const cb_model* m, int k, int b);

/* Algorithm 1, initialisation: z <- w0, and (readings where the algorithm
 * is silent) z_prev <- w0 and every replica w_j <- w0.
 *   k >= 1 learners (also the capacity for cb_set_learners), b >= 1 images
 *   each; alpha is the correction weight
 *   (about 1/k, Sec. 3.2), lr the learning rate gamma, momentum the Polyak
 *   momentum mu on z; all must be finite.
 *   w0_host: P floats in the order above (copied; the caller keeps it).
 *   workspace_dev: at least cb_workspace_bytes(m, k, b) bytes, 256-byte
 *   aligned.  hip_stream: a hipStream_t (NULL = the default stream).
 * Blocks until w0 is on the device.  On success *out owns no device memory
 * of its own beyond the caller's workspace; it does own a second HIP stream
 * (default priority) and some events, released by cb_destroy. */
int cb_create(const cb_model* m, int k, int b, float alpha, float lr, float momentum,
              const float* w0_host, int64_t n_params, void* workspace_dev, size_t ws_bytes,
              void* hip_stream, cb_ctx** out);

/* The learning tasks of one iteration of Algorithm 1: for every learner j,
 * the gradient of its mean loss over its b images (Eq. 2) at its current
 * replica, by a forward and a backward pass.  Gradients are stored raw;
 * the learning rate is applied by cb_sync.  If the previous cb_step was
 * never synchronised, its gradient is first applied as a local step without
 * correction (a sync interval above one).  inputs_dev / labels_dev must stay
 * unchanged until the work completes.  A label outside [0, classes) makes
 * that learner's loss NaN and contributes no one-hot term.  The weight
 * gradients run on the context's second stream, overlapping the rest of the
 * backward pass; the step's last operation on the caller's stream waits for
 * them, so work the caller enqueues afterwards sees the complete step. */
int cb_step(cb_ctx* c, const float* inputs_dev, const int32_t* labels_dev);

/* The synchronisation of Algorithm 1 for the pending gradients, in one
 * fused pass over all replicas: c_j = alpha (w_j - z) and
 * w_j <- w_j - lr g_j - c_j (+ learner momentum), both from the replica's
 * value before the update; then z <- z + sum_j c_j + mu (z - z_prev) and
 * z_prev <- the old z.  CB_ESTATE if no gradient is pending.  Enqueued
 * asynchronously unless check_finite is set. */
int cb_sync(cb_ctx* c);

/* Waits for all work enqueued on the context's stream. */
int cb_wait(cb_ctx* c);

/* The output z of Algorithm 1: copies P floats to out_host (n must be P).
 * Waits for the stream first. */
int cb_get_central(cb_ctx* c, float* out_host, int64_t n);

/* --- test hooks ------------------------------------------------------- */

/* Replica w_j, z_prev, or learner j's last raw gradient, to the host. */
int cb_get_replica(cb_ctx* c, int j, float* out_host, int64_t n);
int cb_get_prev_central(cb_ctx* c, float* out_host, int64_t n);
int cb_get_grad(cb_ctx* c, int j, float* out_host, int64_t n);

/* Mean loss of each learner from the last cb_step, k floats. */
int cb_get_loss(cb_ctx* c, float* out_host);

/* Synchronisation with gradients supplied by the caller: grads_dev is
 * [k][P] raw gradients on the device (read in place, not copied).  Same
 * update as cb_sync; any gradient pending from cb_step is discarded. */
int cb_sma_apply(cb_ctx* c, const float* grads_dev);

/* A local step with gradients supplied by the caller (the update of a
 * cb_step whose gradient was never synchronised, i.e. a sync interval above
 * one): w_j <- w_j - lr g_j (+ mu_L (w_j - w_j_prev)) for every learner,
 * with no correction; z and z_prev are untouched.  grads_dev as for
 * cb_sma_apply; any gradient pending from cb_step is discarded. */
int cb_local_apply(cb_ctx* c, const float* grads_dev);

/* Overwrites the state from host arrays: W [k][P] replicas, z, z_prev [P];
 * w_prev (learner momentum only) is set equal to W.  Clears any pending
 * gradient.  Blocks until the copies are done. */
int cb_set_state(cb_ctx* c, const float* W_host, const float* z_host, const float* zprev_host);

/* --- control between iterations ----------------------------------------
 * These change the training process between iterations of Algorithm 1 and
 * are enqueued on the context's stream like the rest. */

/* The learning rate gamma for the following updates: the step-wise
 * schedule of Sec. 3.2 changes gamma between iterations.  lr must be
 * finite. */
int cb_set_lr(cb_ctx* c, float lr);

/* Restart of SMA (Sec. 3.2): Algorithm 1 starts again from the latest
 * central model z as its initial model -- every active replica (and its
 * previous value) and z_prev become z.  A gradient pending from an
 * unsynchronised cb_step is dropped. */
int cb_restart(cb_ctx* c);

/* Changes the number of active learners to k, 1 <= k <= the k given to
 * cb_create, between iterations (Sec. 3.4; the tuner of Sec. 4.4 adds a
 * learner at an iteration barrier).  A new learner's replica and its
 * previous value are the latest central model z; removing learners drops
 * the most recently added ones (the paper does not say which).  alpha is
 * the correction weight from now on (about 1/k).  cb_step then takes
 * k*b images.  CB_ESTATE while a gradient is pending (call cb_sync first),
 * CB_EINVAL for k out of range.  Allocates nothing: the workspace was
 * sized for every k up to the capacity. */
int cb_set_learners(cb_ctx* c, int k, float alpha);

/* The number of active learners. */
int cb_learners(const cb_ctx* c);

/* Graph replay of cb_step (on != 0) or direct launches (on == 0, the
 * default).  With replay on, the first cb_step on a given (inputs_dev,
 * labels_dev) pair captures its forward/backward launches from the
 * context's stream into a HIP graph; later steps on the same pair launch
 * that graph, so the host submits one graph instead of each kernel.
 * Results are bitwise those of direct launches.  The buffers themselves
 * are read at replay time, so their contents may change between steps; a
 * graph is kept per pair, at most 8 (the oldest is dropped, after the
 * stream drains).  cb_set_learners drops all graphs; instrumented steps
 * (cb_profile_enable) always launch directly.  Switching off drops all
 * graphs.  Not part of Algorithm 1: launch overhead only. */
int cb_set_graphs(cb_ctx* c, int on);

/* Algorithm 2 (Sec. 3.4), one observation for one GPU: l learners gave
 * throughput t and t_prev was observed before.  Returns l + 1 if t - t_prev
 * exceeds threshold (but at most l_max), l - 1 if t < t_prev (but at least
 * one learner; the algorithm's guard "l > 0" is read as "l > 1"), else l.
 * The caller keeps t as the next t_prev.  Pure host function. */
int cb_tuner_next(int l, double t, double t_prev, double threshold, int l_max);

/* --- operator test hooks ------------------------------------------------
 * One operator of the learning task on caller device buffers, through the
 * same launchers (kernels and tile choices) that cb_step uses, enqueued on
 * `stream` (a hipStream_t).  k replicas of b images; the parameters of
 * replica j start at params + j*pstride (weight, then bias if any; for batch
 * norm gamma then beta), and gradients land in the same layout in grads.
 * Scratch is caller device memory of at least the *_scratch_bytes size.
 * CB_EINVAL for an unsupported shape or a NULL required buffer, CB_ENOMEM
 * for short scratch, CB_EDEVICE if a launch fails. */

/* Scratch for cb_test_conv (split contraction partials); 0 on bad shape. */
size_t cb_test_conv_scratch_bytes(int k, int b, int Ci, int H, int W, int Co, int R, int stride,
                                  int pad);

/* Number of partial sums per (replica, channel) that the forward epilogue
 * writes to cb_test_conv's stats; CB_EINVAL on a bad shape. */
int cb_test_conv_fwd_parts(int k, int b, int Ci, int H, int W, int Co, int R, int stride,
                           int pad);

/* Convolution or FC (a 1x1 conv on 1x1 images), Sec. 2.1 forward pass:
 * y = conv(x, w) + bias, then ReLU if relu.  x [k*b][Ci][H][W],
 * y [k*b][Co][Ho][Wo].  If stats is not NULL, the forward epilogue also
 * writes the per-channel partial sums of the stored y that a following
 * batch norm takes its statistics from, as cb_step uses them:
 * stats [k][Co][parts][2] (fp64; sum of y, sum of y*y; parts =
 * cb_test_conv_fwd_parts()), whose sum over parts is the total over the
 * replica's b images.  If dy is not NULL, also the backward pass: the
 * weight (and bias) gradient into grads and, if dx is not NULL, the input
 * gradient (dy is taken as already masked by any ReLU). */
int cb_test_conv(int k, int b, int Ci, int H, int W, int Co, int R, int stride, int pad,
                 int relu, int has_bias, const float* x, const float* params, int64_t pstride,
                 float* y, double* stats, const float* dy, float* dx, float* grads,
                 void* scratch, size_t scratch_bytes, void* stream);

/* Scratch for the batch-norm hooks; 0 on bad shape. */
size_t cb_test_bn_scratch_bytes(int k, int b, int C, int H, int W);

/* Batch norm with each replica's batch statistics over its b images, then
 * ReLU if relu; mean and istd (1/sqrt(var + 1e-5)) are written as [k][C]. */
int cb_test_bn_fwd(int k, int b, int C, int H, int W, int relu, const float* x,
                   const float* params, int64_t pstride, float* y, float* mean, float* istd,
                   void* scratch, size_t scratch_bytes, void* stream);

/* Backward of cb_test_bn_fwd given its mean and istd: dy is masked where
 * mask_y <= 0 (pass the forward output when the ReLU is on, else NULL), or,
 * with relu_x (mask_y NULL), where the norm's output recomputed from x,
 * fmaf(gamma, (x - mean) * istd, beta), is not positive (the forward's
 * exact decision); dx, and dgamma/dbeta into grads. */
int cb_test_bn_bwd(int k, int b, int C, int H, int W, const float* x, const float* mask_y,
                   int relu_x, const float* dy, const float* params, int64_t pstride,
                   const float* mean, const float* istd, float* dx, float* grads, void* scratch,
                   size_t scratch_bytes, void* stream);

/* Max pool K x K (first strict maximum wins, padded cells never win) on
 * [N][C][H][W]; with dy, its gradient dx (zeroed where x <= 0 if mask_relu).
 * arg_scratch: N*C*Ho*Wo ints of device memory. */
int cb_test_maxpool(int N, int C, int H, int W, int K, int stride, int pad, const float* x,
                    float* y, const float* dy, float* dx, int mask_relu, int* arg_scratch,
                    void* stream);

/* The data gradient of one convolution with every operand its fused
 * epilogue can take, as cb_step uses it: dx = conv_bwd(dy) (+ dx if
 * accumulate) (+ add: ADD_SAME = 1, same shape as dx; ADD_SUBSAMPLE = 2,
 * add is [k*b][add_C][Ho][Wo] and reaches the pixels whose row and column are
 * multiples of stride, channel by channel), zeroed where mask <= 0 (mask
 * may be NULL); then, if bn_part is not NULL, dx is the output gradient of
 * a batch norm with input bn_x and statistics bn_mean / bn_istd [k][Ci]:
 * with d = dx where bn_y > 0 (all of dx if bn_y is NULL) and
 * xh = (bn_x - mean) * istd, per replica and channel the partial sums of d
 * and d*xh are written to bn_part [k][Ci][parts][2] (fp64), parts =
 * cb_test_conv_dgrad_parts(); their sum over parts is the total.  bn_gamma
 * (optional; gamma and beta at bn_gamma + j*pstride + [0, Ci) and [Ci, 2Ci))
 * lets a kernel take a ReLU decision as fmaf(gamma, xh, beta) > 0 instead of
 * reading it: with bn_y, the implicit-GEMM epilogue and the direct stride-1
 * kernels do so for bn_y > 0; without bn_y, mask is taken to be the norm's
 * own ReLU output and the direct stride-1 kernels do so for mask > 0 (the
 * tensor given must agree; bn_gamma with neither bn_y nor mask is
 * CB_EINVAL).  Same kernels and tile choices as cb_step; device pointers
 * 16-byte aligned. */
int cb_test_conv_dgrad_parts(int k, int b, int Ci, int H, int W, int Co, int R, int stride,
                             int pad);
int cb_test_conv_dgrad(int k, int b, int Ci, int H, int W, int Co, int R, int stride, int pad,
                       const float* dy, const float* params, int64_t pstride, float* dx,
                       int accumulate, const float* mask, const float* add, int add_mode,
                       int add_C, const float* bn_x, const float* bn_y, const float* bn_mean,
                       const float* bn_istd, const float* bn_gamma, double* bn_part,
                       void* stream);

/* 1 if the fused network head takes C channels of H x W pixels and
 * `classes` outputs, else 0. */
int cb_test_head_ok(int C, int H, int W, int classes);

/* The fused head of the ResNet workloads as cb_step runs it: global average
 * pool of y [k*b][C][H][W] into features [k*b][C], an FC layer (weights
 * [classes][C] then bias at params + j*pstride), softmax cross-entropy
 * (Eq. 2) with per-image loss terms loss [k*b] (a replica's loss is the
 * mean of its b terms) and logit gradients dlogits [k*b][classes]
 * (softmax - onehot)/b, then the backward pass down to the pooled input:
 * dy [k*b][C][H][W].  If bn_part is not NULL, y is the output of a batch
 * norm with input bn_x and statistics bn_mean / bn_istd [k][C] (ReLU'd if
 * bn_relu): with d = dy where y > 0 (all of dy without the ReLU) and
 * xh = (bn_x - mean) * istd, the per-image sums of d and d*xh per replica
 * and channel go to bn_part [k][C][b][2] (fp64).  Device pointers 16-byte
 * aligned; CB_EINVAL for a shape cb_test_head_ok rejects. */
int cb_test_head(int k, int b, int C, int H, int W, int classes, const float* y,
                 const float* params, int64_t pstride, const int32_t* labels, float* features,
                 float* dlogits, float* loss, float* dy, const float* bn_x,
                 const float* bn_mean, const float* bn_istd, int bn_relu, double* bn_part,
                 void* stream);

/* Mean softmax cross-entropy of each replica's b rows of logits (Eq. 2),
 * loss [k], and its gradient dlogits [k*b][classes]. */
int cb_test_softmax_xent(int k, int b, int classes, const float* logits, const int32_t* labels,
                         float* dlogits, float* loss, void* stream);

/* --- for callers that cannot allocate ----------------------------------
 * For code under HIP graph capture, tight serving loops and harnesses that
 * forbid allocation: cb_test_conv with the scratch of its weight gradient
 * (the split-contraction partials) taken from device memory the library
 * holds instead of from the caller -- a static array of
 * CB_STATIC_SCRATCH_BYTES (enough for every layer of the three workloads),
 * one per GPU, kept until the process ends.  The caller still passes every
 * input and output, as for cb_test_conv.  Allocates nothing (the first call
 * on a device looks up the array's address there).  CB_ENOMEM, with a
 * message from cb_last_error(NULL), if the layer needs more scratch than
 * that (cb_test_conv_scratch_bytes() tells).  The array keeps the last
 * call's contents; nothing it holds is read before the same call writes it.
 * Calls that overlap on one GPU -- on different streams, or from different
 * threads -- share the array and race. */
#define CB_STATIC_SCRATCH_BYTES (32u << 20)
int cb_test_conv_static(int k, int b, int Ci, int H, int W, int Co, int R, int stride, int pad,
                        int relu, int has_bias, const float* x, const float* params,
                        int64_t pstride, float* y, double* stats, const float* dy, float* dx,
                        float* grads, void* stream);

/* --- instrumentation --------------------------------------------------- */

/* While enabled, every kernel launch of the context carries a start/stop
 * hipEvent pair on its own dispatch (hipExtLaunchKernel), and the launch's
 * algorithmic work (FLOPs of the contraction, or bytes the operation must
 * read and write) is recorded with the kernel's name.  Instrumented steps
 * run every kernel on the context's stream (the weight gradients do not
 * overlap the data-gradient chain as they otherwise do), so each recorded
 * duration is the kernel alone. */
int cb_profile_enable(cb_ctx* c, int on);

/* Waits for the stream and folds the records into per-kernel totals
 * (accumulated until cb_profile_clear).  Returns the number of distinct
 * kernels, or a negative CB_E* code. */
int cb_profile_collect(cb_ctx* c);

/* Totals of kernel i < cb_profile_collect(): name (valid until the next
 * collect or clear), launches, summed duration in ms, algorithmic FLOPs and
 * bytes. */
int cb_profile_entry(cb_ctx* c, int i, const char** name, int64_t* launches, double* ms,
                     double* flops, double* bytes);

/* Drops the accumulated totals. */
int cb_profile_clear(cb_ctx* c);

/* Message for the last error on this context ("" if none); valid until the
 * next call on it.  A NULL context gives the last failure of a call made
 * without one (cb_create, cb_test_conv_static). */
const char* cb_last_error(const cb_ctx* c);

/* Frees the context's host-side state; the caller then frees the workspace. */
void cb_destroy(cb_ctx* c);

#ifdef __cplusplus
}
#endif

#endif /* CROSSBOW_SMA_H */
