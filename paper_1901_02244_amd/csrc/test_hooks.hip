// test_hooks.hip -- one operator of the learning task on caller buffers.
//
// These entry points run the same launchers (and so the same kernels and
// tile choices) as cb_step, on device buffers the caller fills, so each
// kernel can be compared with a reference at any shape, including the
// exact layer shapes of the training workloads.  Nothing here allocates:
// scratch comes from the caller, sized by the *_scratch_bytes calls.
#include "crossbow_sma.h"
#include "kernels.hpp"

#include <algorithm>

using namespace cbk;

namespace {

ConvGeom make_geom(int k, int b, int Ci, int H, int W, int Co, int R, int st, int pad) {
  ConvGeom g;
  g.k = k; g.b = b;
  g.Ci = Ci; g.H = H; g.W = W;
  g.Co = Co; g.R = R; g.S = R;
  g.st = st; g.pad = pad;
  g.Ho = (H + 2 * pad - R) / st + 1;
  g.Wo = (W + 2 * pad - R) / st + 1;
  return g;
}

bool geom_ok(int k, int b, int Ci, int H, int W, int Co, int R, int st, int pad) {
  return k >= 1 && b >= 1 && Ci >= 1 && Co >= 1 && H >= R - 2 * pad && W >= R - 2 * pad &&
         pad >= 0 && (H + 2 * pad - R) >= 0;
}

int rc_of(hipError_t e) { return e == hipSuccess ? CB_OK : CB_EDEVICE; }

}  // namespace

extern "C" {

size_t cb_test_conv_scratch_bytes(int k, int b, int Ci, int H, int W, int Co, int R, int stride,
                                  int pad) {
  if (!geom_ok(k, b, Ci, H, W, Co, R, stride, pad)) return 0;
  ConvGeom g = make_geom(k, b, Ci, H, W, Co, R, stride, pad);
  int chunk = 0;
  const int splits = conv_bwd_weight_splits(g, &chunk);
  return (size_t)std::max<int64_t>(16, (int64_t)k * splits * Co * Ci * R * R * 4);
}

int cb_test_conv_fwd_parts(int k, int b, int Ci, int H, int W, int Co, int R, int stride,
                           int pad) {
  if (!geom_ok(k, b, Ci, H, W, Co, R, stride, pad) || !conv_supported(R, R, stride, false))
    return CB_EINVAL;
  return conv_fwd_tiles_m(make_geom(k, b, Ci, H, W, Co, R, stride, pad));
}

int cb_test_conv(int k, int b, int Ci, int H, int W, int Co, int R, int stride, int pad,
                 int relu, int has_bias, const float* x, const float* params, int64_t pstride,
                 float* y, double* stats, const float* dy, float* dx, float* grads,
                 void* scratch, size_t scratch_bytes, void* stream) {
  if (!geom_ok(k, b, Ci, H, W, Co, R, stride, pad) ||
      !conv_supported(R, R, stride, dx != nullptr) || !x || !params || !y)
    return CB_EINVAL;
  if (scratch_bytes < cb_test_conv_scratch_bytes(k, b, Ci, H, W, Co, R, stride, pad))
    return CB_ENOMEM;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const ConvGeom g = make_geom(k, b, Ci, H, W, Co, R, stride, pad);
  const int64_t nw = (int64_t)Co * Ci * R * R;
  ConvFwdArgs f;
  f.g = g;
  f.x = x;
  f.w = params;
  f.bias = has_bias ? params + nw : nullptr;
  f.pstride = pstride;
  f.y = y;
  f.relu = relu;
  f.stats = stats;
  int rc = rc_of(conv_fwd(f, s));
  if (rc || !dy) return rc;
  if (!grads) return CB_EINVAL;
  if (has_bias) {
    rc = rc_of(channel_sum(dy, k, b, Co, g.Ho * g.Wo, grads + nw, pstride, s));
    if (rc) return rc;
  }
  ConvBwdWeightArgs w;
  w.g = g;
  w.x = x;
  w.dy = dy;
  w.dw = grads;
  w.pstride = pstride;
  w.partial = static_cast<float*>(scratch);
  w.splits = conv_bwd_weight_splits(g, &w.chunk);
  rc = rc_of(conv_bwd_weight(w, s));
  if (rc) return rc;
  if (w.splits > 1) {
    SplitTable t;
    t.pstride = pstride;
    split_table_add(t, w.partial, grads, nw, w.splits);
    rc = rc_of(reduce_splits(t, k, s));
  }
  if (rc || !dx) return rc;
  ConvBwdDataArgs d;
  d.g = g;
  d.dy = dy;
  d.w = params;
  d.pstride = pstride;
  d.dx = dx;
  d.accumulate = 0;
  d.mask = nullptr;
  d.add = nullptr;
  d.add_mode = ADD_NONE;
  d.add_C = 0;
  d.add_st = 1;
  d.bn_part = nullptr;
  d.bn_x = d.bn_y = d.bn_mean = d.bn_istd = nullptr;
  return rc_of(conv_bwd_data(d, s));
}

int cb_test_conv_dgrad_parts(int k, int b, int Ci, int H, int W, int Co, int R, int stride,
                             int pad) {
  if (!geom_ok(k, b, Ci, H, W, Co, R, stride, pad) || !conv_supported(R, R, stride, true))
    return CB_EINVAL;
  return conv_bwd_data_tiles_m(make_geom(k, b, Ci, H, W, Co, R, stride, pad));
}

int cb_test_conv_dgrad(int k, int b, int Ci, int H, int W, int Co, int R, int stride, int pad,
                       const float* dy, const float* params, int64_t pstride, float* dx,
                       int accumulate, const float* mask, const float* add, int add_mode,
                       int add_C, const float* bn_x, const float* bn_y, const float* bn_mean,
                       const float* bn_istd, const float* bn_gamma, double* bn_part,
                       void* stream) {
  if (!geom_ok(k, b, Ci, H, W, Co, R, stride, pad) || !conv_supported(R, R, stride, true) ||
      !dy || !params || !dx || add_mode < ADD_NONE || add_mode > ADD_SUBSAMPLE ||
      (add_mode != ADD_NONE && !add) || (bn_part && (!bn_x || !bn_mean || !bn_istd)) ||
      (bn_gamma && !bn_y && !mask))
    return CB_EINVAL;
  ConvBwdDataArgs d;
  d.g = make_geom(k, b, Ci, H, W, Co, R, stride, pad);
  d.dy = dy;
  d.w = params;
  d.pstride = pstride;
  d.dx = dx;
  d.accumulate = accumulate;
  d.mask = mask;
  d.add = add;
  d.add_mode = add_mode;
  d.add_C = add_C;
  d.add_st = stride;
  d.bn_part = bn_part;
  d.bn_x = bn_x;
  d.bn_y = bn_y;
  d.bn_mean = bn_mean;
  d.bn_istd = bn_istd;
  d.bn_gamma = bn_gamma;
  d.mask_from_bn = bn_gamma && !bn_y;
  return rc_of(conv_bwd_data(d, static_cast<hipStream_t>(stream)));
}

size_t cb_test_bn_scratch_bytes(int k, int b, int C, int H, int W) {
  if (k < 1 || b < 1 || C < 1 || H < 1 || W < 1) return 0;
  return (size_t)k * C * bn_chunks(b, H * W, C, k) * 2 * sizeof(double);
}

int cb_test_bn_fwd(int k, int b, int C, int H, int W, int relu, const float* x,
                   const float* params, int64_t pstride, float* y, float* mean, float* istd,
                   void* scratch, size_t scratch_bytes, void* stream) {
  if (k < 1 || b < 1 || C < 1 || H < 1 || W < 1 || !x || !params || !y || !mean || !istd)
    return CB_EINVAL;
  if (scratch_bytes < cb_test_bn_scratch_bytes(k, b, C, H, W)) return CB_ENOMEM;
  hipStream_t s = static_cast<hipStream_t>(stream);
  BNArgs a;
  a.k = k; a.b = b; a.C = C; a.H = H; a.W = W;
  a.x = x; a.y = y;
  a.gamma = params;
  a.pstride = pstride;
  a.mean = mean;
  a.istd = istd;
  a.part = static_cast<double*>(scratch);
  a.chunks = bn_chunks(b, H * W, C, k);
  a.parts = a.chunks;
  a.relu = relu;
  a.res = nullptr;
  a.res_mode = RES_NONE;
  a.res_C = a.res_st = a.res_H = a.res_W = 0;
  int rc = rc_of(bn_fwd_stats(a, s));
  if (rc) return rc;
  return rc_of(bn_fwd_apply(a, s));
}

int cb_test_bn_bwd(int k, int b, int C, int H, int W, const float* x, const float* mask_y,
                   int relu_x, const float* dy, const float* params, int64_t pstride,
                   const float* mean, const float* istd, float* dx, float* grads, void* scratch,
                   size_t scratch_bytes, void* stream) {
  if (k < 1 || b < 1 || C < 1 || H < 1 || W < 1 || !x || !dy || !params || !mean || !istd ||
      !dx || !grads || (mask_y && relu_x))
    return CB_EINVAL;
  if (scratch_bytes < cb_test_bn_scratch_bytes(k, b, C, H, W)) return CB_ENOMEM;
  hipStream_t s = static_cast<hipStream_t>(stream);
  BNBwdArgs a;
  a.k = k; a.b = b; a.C = C; a.H = H; a.W = W;
  a.x = x;
  a.y = mask_y;
  a.relu_x = relu_x != 0;
  a.dy = dy;
  a.dx = dx;
  a.dres = nullptr;
  a.gamma = params;
  a.dgamma = grads;
  a.pstride = pstride;
  a.mean = mean;
  a.istd = istd;
  a.part = static_cast<double*>(scratch);
  a.chunks = bn_chunks(b, H * W, C, k);
  a.parts = a.chunks;
  int rc = rc_of(bn_bwd_stats(a, s));
  if (rc) return rc;
  return rc_of(bn_bwd_apply(a, s));
}

int cb_test_maxpool(int N, int C, int H, int W, int K, int stride, int pad, const float* x,
                    float* y, const float* dy, float* dx, int mask_relu, int* arg_scratch,
                    void* stream) {
  if (N < 1 || C < 1 || K < 1 || stride < 1 || pad < 0 || pad >= K || H + 2 * pad < K ||
      W + 2 * pad < K || !x || !y || !arg_scratch)
    return CB_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int Ho = (H + 2 * pad - K) / stride + 1, Wo = (W + 2 * pad - K) / stride + 1;
  int rc = rc_of(maxpool_fwd(x, N, C, H, W, K, stride, pad, y, Ho, Wo, arg_scratch, s));
  if (rc || !dy) return rc;
  if (!dx) return CB_EINVAL;
  return rc_of(maxpool_bwd(dy, arg_scratch, x, N, C, H, W, K, stride, pad, Ho, Wo, dx, mask_relu,
                           s));
}

int cb_test_head_ok(int C, int H, int W, int classes) {
  return C >= 1 && H >= 1 && W >= 1 && head_ok(C, H * W, classes) ? 1 : 0;
}

int cb_test_head(int k, int b, int C, int H, int W, int classes, const float* y,
                 const float* params, int64_t pstride, const int32_t* labels, float* features,
                 float* dlogits, float* loss, float* dy, const float* bn_x,
                 const float* bn_mean, const float* bn_istd, int bn_relu, double* bn_part,
                 void* stream) {
  if (k < 1 || b < 1 || !cb_test_head_ok(C, H, W, classes) || !y || !params || !labels ||
      !features || !dlogits || !loss || !dy || (bn_part && (!bn_x || !bn_mean || !bn_istd)))
    return CB_EINVAL;
  HeadArgs a;
  a.k = k; a.b = b; a.C = C; a.HW = H * W; a.classes = classes;
  a.y = y;
  a.g = features;
  a.w = params;
  a.bias = params + (int64_t)classes * C;
  a.pstride = pstride;
  a.labels = labels;
  a.dlogits = dlogits;
  a.loss = loss;
  a.dy = dy;
  a.bn_part = bn_part;
  a.bn_relu = bn_relu;
  a.bn_x = bn_part ? bn_x : nullptr;
  a.bn_mean = bn_part ? bn_mean : nullptr;
  a.bn_istd = bn_part ? bn_istd : nullptr;
  return rc_of(head_fwd_bwd(a, static_cast<hipStream_t>(stream)));
}

int cb_test_softmax_xent(int k, int b, int classes, const float* logits, const int32_t* labels,
                         float* dlogits, float* loss, void* stream) {
  if (k < 1 || b < 1 || classes < 1 || !logits || !labels || !dlogits || !loss) return CB_EINVAL;
  return rc_of(softmax_xent(logits, labels, k, b, classes, dlogits, loss,
                            static_cast<hipStream_t>(stream)));
}

}  // extern "C"
