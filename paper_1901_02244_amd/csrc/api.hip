// api.hip -- runtime and C ABI (include/crossbow_sma.h).
//
// A context holds one SMA job of k learners on one GPU (Algorithm 1,
// Sec. 3.2).  cb_create turns the network description into a fixed list of
// replica-batched operators (the learning task of Sec. 4.2, here one launch
// per operator for all learners instead of one task per learner stream),
// carves the caller's workspace, and uploads w0.  cb_step enqueues the
// forward and backward passes of all learners; cb_sync enqueues the fused
// SMA kernel.  Everything runs in order on the caller's stream.
#include "crossbow_sma.h"
#include "kernels.hpp"

#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

using namespace cbk;

namespace {

constexpr int64_t ALIGN = 256;
inline int64_t align_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

enum OpKind { OP_CONV, OP_BN, OP_MAXPOOL, OP_GAP, OP_XENT };

struct Tensor {
  int C = 0, H = 0, W = 0;
  int64_t act = -1, grad = -1;  // byte offsets into the workspace
  bool relu_fused = false;      // produced by a conv/FC with a fused ReLU
  int consumers = 0;
};

struct Op {
  OpKind kind;
  int in = -1, out = -1;
  // conv / FC
  int Ci = 0, Co = 0, R = 1, st = 1, pad = 0, H = 0, W = 0, Ho = 0, Wo = 0;
  bool bias = false, relu = false, need_dx = true;
  int64_t w_off = -1, b_off = -1;   // parameter offsets (elements)
  int splits = 1, chunk = 0;
  int64_t part_off = -1;            // this layer's weight-gradient split partials
  bool emit_stats = false;          // epilogue writes BN partial sums
  int bnb = -1;                     // data-gradient epilogue feeds this BN's backward sums
  // batch norm
  int C = 0;
  int64_t g_off = -1;
  int res = -1, res_mode = RES_NONE, res_st = 1;
  int64_t mean = -1, istd = -1, dres = -1;
  int chunks = 1;
  int parts = 0;                    // > 0: statistics come from the producing conv
  int bwd_parts = 0;                // > 0: backward sums come from the next conv's dx
  // pooling
  int K = 0;
  int64_t arg = -1;
  // backward routing decided at plan time
  bool dx_accumulate = false, dx_mask = false;
  int add_mode = ADD_NONE, add_C = 0, add_st = 1;
  int64_t add_buf = -1;
  // fused head: a pool, FC and softmax cross-entropy run as one kernel
  // (launched at the pool; the FC keeps its weight gradient)
  bool head = false;
  int head_fc = -1, head_bn = -1;   // at the pool: the FC op, the batch norm feeding the pool
};

struct ParamInfo {
  int64_t offset;
  int kind, ndim, dims[4];
};

struct Plan {
  cb_model m{};
  int k = 0, b = 0;
  int kcap = 0;  // replicas the parameter state is laid out for (k <= kcap)
  std::vector<Tensor> t;
  std::vector<Op> ops;
  std::vector<ParamInfo> params;
  int64_t P = 0, Pp = 0;
  int input = -1, logits = -1;
  bool loss_per_image = false;  // the loss buffer holds k*b per-image terms (fused head)
  // The MNIST-shaped LeNet runs as two fused launches (lenet.hip) instead of
  // the operator list; its scratch: per-image loss terms, conv gradient
  // shares and FC vectors.
  bool lenet_fused = false;
  int64_t off_lenet_loss = -1, off_lenet_conv = -1, off_lenet_fc = -1;
  // workspace layout (bytes)
  int64_t off_W = 0, off_G = 0, off_Z = 0, off_Zp = 0, off_Wprev = -1;
  int64_t off_loss = 0, off_flag = 0, off_bnpart = 0;
  int64_t off_loss_mean = -1;  // with per-image terms: each replica's mean [k]
  int64_t total = 0;
};

// ------------------------------------------------------------------ builder
struct Builder {
  Plan& p;
  explicit Builder(Plan& pl) : p(pl) {}

  int tensor(int C, int H, int W) {
    Tensor x;
    x.C = C; x.H = H; x.W = W;
    p.t.push_back(x);
    return (int)p.t.size() - 1;
  }
  int64_t param(int kind, int ndim, int d0, int d1 = 1, int d2 = 1, int d3 = 1) {
    ParamInfo pi;
    pi.offset = p.P;
    pi.kind = kind;
    pi.ndim = ndim;
    pi.dims[0] = d0; pi.dims[1] = d1; pi.dims[2] = d2; pi.dims[3] = d3;
    p.params.push_back(pi);
    p.P += (int64_t)d0 * d1 * d2 * d3;
    return pi.offset;
  }
  int conv(int in, int Co, int R, int st, int pad, bool bias, bool relu, bool fc = false) {
    const Tensor x = p.t[in];
    Op o;
    o.kind = OP_CONV;
    o.in = in;
    o.Ci = fc ? x.C * x.H * x.W : x.C;
    o.H = fc ? 1 : x.H;
    o.W = fc ? 1 : x.W;
    o.Co = Co; o.R = R; o.st = st; o.pad = pad; o.bias = bias; o.relu = relu;
    o.Ho = (o.H + 2 * pad - R) / st + 1;
    o.Wo = (o.W + 2 * pad - R) / st + 1;
    o.w_off = fc ? param(CB_KIND_FC_W, 2, Co, o.Ci) : param(CB_KIND_CONV_W, 4, Co, o.Ci, R, R);
    if (bias) o.b_off = param(CB_KIND_BIAS, 1, Co);
    o.need_dx = in != p.input;
    o.out = tensor(Co, o.Ho, o.Wo);
    p.t[o.out].relu_fused = relu;
    p.t[in].consumers++;
    p.ops.push_back(o);
    return o.out;
  }
  int bn(int in, bool relu, int res = -1, int res_mode = RES_NONE, int res_st = 1) {
    const Tensor x = p.t[in];
    Op o;
    o.kind = OP_BN;
    o.in = in;
    o.C = x.C; o.H = x.H; o.W = x.W;
    o.relu = relu;
    o.g_off = param(CB_KIND_BN_GAMMA, 1, x.C);
    param(CB_KIND_BN_BETA, 1, x.C);
    o.res = res; o.res_mode = res_mode; o.res_st = res_st;
    o.out = tensor(x.C, x.H, x.W);
    p.t[in].consumers++;
    if (res >= 0) p.t[res].consumers++;
    p.ops.push_back(o);
    return o.out;
  }
  int maxpool(int in, int K, int st, int pad) {
    const Tensor x = p.t[in];
    Op o;
    o.kind = OP_MAXPOOL;
    o.in = in;
    o.C = x.C; o.H = x.H; o.W = x.W; o.K = K; o.st = st; o.pad = pad;
    o.Ho = (x.H + 2 * pad - K) / st + 1;
    o.Wo = (x.W + 2 * pad - K) / st + 1;
    o.out = tensor(x.C, o.Ho, o.Wo);
    p.t[in].consumers++;
    p.ops.push_back(o);
    return o.out;
  }
  int gap(int in) {
    const Tensor x = p.t[in];
    Op o;
    o.kind = OP_GAP;
    o.in = in;
    o.C = x.C; o.H = x.H; o.W = x.W;
    o.out = tensor(x.C, 1, 1);
    p.t[in].consumers++;
    p.ops.push_back(o);
    return o.out;
  }
  void xent(int in) {
    Op o;
    o.kind = OP_XENT;
    o.in = in;
    p.t[in].consumers++;
    p.ops.push_back(o);
    p.logits = in;
  }
};

// The networks of Table 1 used by the workloads; shapes as declared in the
// library header's model notes (LeNet with a padded first conv, ResNet-32
// with option-A shortcuts, ResNet-50 v1 with stride on the first 1x1).
bool build_lenet(Builder& B) {
  const cb_model& m = B.p.m;
  if (m.in_h % 4 || m.in_w % 4 || m.in_h < 12 || m.in_w < 12) return false;
  if ((m.in_h / 2 - 4) % 2 || (m.in_w / 2 - 4) % 2) return false;
  int x = B.p.input;
  x = B.conv(x, 6, 5, 1, 2, true, true);
  x = B.maxpool(x, 2, 2, 0);
  x = B.conv(x, 16, 5, 1, 0, true, true);
  x = B.maxpool(x, 2, 2, 0);
  x = B.conv(x, 120, 1, 1, 0, true, true, true);
  x = B.conv(x, 84, 1, 1, 0, true, true, true);
  x = B.conv(x, m.num_classes, 1, 1, 0, true, false, true);
  B.xent(x);
  return true;
}

bool build_resnet32(Builder& B) {
  const cb_model& m = B.p.m;
  if (m.in_h % 4 || m.in_w % 4 || m.in_h < 4 || m.in_w < 4) return false;
  int x = B.conv(B.p.input, 16, 3, 1, 1, false, false);
  x = B.bn(x, true);
  int cin = 16;
  for (int stage = 0; stage < 3; ++stage) {
    const int cout = 16 << stage;
    for (int i = 0; i < 5; ++i) {
      const int st = (stage > 0 && i == 0) ? 2 : 1;
      int a = B.conv(x, cout, 3, st, 1, false, false);
      a = B.bn(a, true);
      a = B.conv(a, cout, 3, 1, 1, false, false);
      x = B.bn(a, true, x, st == 1 ? RES_SAME : RES_SUBSAMPLE, st);
      cin = cout;
    }
  }
  (void)cin;
  x = B.gap(x);
  x = B.conv(x, m.num_classes, 1, 1, 0, true, false, true);
  B.xent(x);
  return true;
}

bool build_resnet50(Builder& B) {
  const cb_model& m = B.p.m;
  if (m.in_h % 32 || m.in_w % 32 || m.in_h < 32 || m.in_w < 32) return false;
  int x = B.conv(B.p.input, 64, 7, 2, 3, false, false);
  x = B.bn(x, true);
  x = B.maxpool(x, 3, 2, 1);
  static const int depth[4] = {3, 4, 6, 3};
  for (int stage = 0; stage < 4; ++stage) {
    const int w = 64 << stage, cout = 4 * w;
    for (int i = 0; i < depth[stage]; ++i) {
      const int st = (stage > 0 && i == 0) ? 2 : 1;
      int a = B.conv(x, w, 1, st, 0, false, false);
      a = B.bn(a, true);
      a = B.conv(a, w, 3, 1, 1, false, false);
      a = B.bn(a, true);
      a = B.conv(a, cout, 1, 1, 0, false, false);
      if (i == 0) {
        // projection shortcut; its BN adds the main path and applies the ReLU
        a = B.bn(a, false);
        int pr = B.conv(x, cout, 1, st, 0, false, false);
        x = B.bn(pr, true, a, RES_SAME, 1);
      } else {
        x = B.bn(a, true, x, RES_SAME, 1);
      }
    }
  }
  x = B.gap(x);
  x = B.conv(x, m.num_classes, 1, 1, 0, true, false, true);
  B.xent(x);
  return true;
}

ConvGeom geom(const Plan& p, const Op& o) {
  ConvGeom g;
  g.k = p.k; g.b = p.b;
  g.Ci = o.Ci; g.H = o.H; g.W = o.W;
  g.Co = o.Co; g.R = o.R; g.S = o.R;
  g.st = o.st; g.pad = o.pad; g.Ho = o.Ho; g.Wo = o.Wo;
  return g;
}

// Builds the operator list, the backward routing and the workspace layout
// for k active learners.  The parameter state (W, G, z, z_prev, w_prev)
// comes first and is laid out for kcap replicas, so plans for any k <= kcap
// put it at the same place.  Returns false for an unsupported model.
bool make_plan(const cb_model* m, int k, int b, Plan& p, int kcap = 0) {
  p = Plan();
  if (!m || k < 1 || b < 1 || m->in_c < 1 || m->num_classes < 1) return false;
  if (kcap < k) kcap = k;
  p.m = *m;
  p.k = k;
  p.kcap = kcap;
  p.b = b;
  Builder B(p);
  p.input = B.tensor(m->in_c, m->in_h, m->in_w);
  bool ok = false;
  switch (m->arch) {
    case CB_ARCH_LENET5: ok = build_lenet(B); break;
    case CB_ARCH_RESNET32: ok = build_resnet32(B); break;
    case CB_ARCH_RESNET50: ok = build_resnet50(B); break;
    default: ok = false;
  }
  if (!ok) return false;
  p.Pp = align_up(p.P, 64);
  p.lenet_fused = m->arch == CB_ARCH_LENET5 &&
                  lenet_fused_ok(m->in_c, m->in_h, m->in_w, m->num_classes);

  // backward routing: visit ops in reverse, track which gradients exist
  std::vector<char> written(p.t.size(), 0);
  struct Pending { int mode = ADD_NONE, C = 0, st = 1, op = -1; };
  std::vector<Pending> pend(p.t.size());
  for (int i = (int)p.ops.size() - 1; i >= 0; --i) {
    Op& o = p.ops[i];
    switch (o.kind) {
      case OP_XENT: written[o.in] = 1; break;
      case OP_GAP:
      case OP_MAXPOOL:
        if (written[o.in]) return false;  // single consumer expected
        o.dx_mask = p.t[o.in].relu_fused;
        written[o.in] = 1;
        break;
      case OP_BN:
        if (written[o.in]) return false;
        written[o.in] = 1;
        if (o.res >= 0) {
          if (p.t[o.res].consumers == 1) {
            written[o.res] = 1;  // dres is the residual's whole gradient
          } else {
            pend[o.res].mode = o.res_mode == RES_SAME ? ADD_SAME : ADD_SUBSAMPLE;
            pend[o.res].C = o.C;
            pend[o.res].st = o.res_st;
            pend[o.res].op = i;
          }
        }
        break;
      case OP_CONV:
        if (!o.need_dx) break;
        o.dx_accumulate = written[o.in];
        if (pend[o.in].mode != ADD_NONE) {
          o.add_mode = pend[o.in].mode;
          o.add_C = pend[o.in].C;
          o.add_st = pend[o.in].st;
          o.add_buf = pend[o.in].op;  // op index for now; byte offset below
          pend[o.in].mode = ADD_NONE;
        }
        if (p.t[o.in].relu_fused) {
          if (p.t[o.in].consumers != 1) return false;
          o.dx_mask = true;
        }
        written[o.in] = 1;
        break;
    }
  }

  // workspace layout
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    const int64_t o = off;
    off = align_up(off + bytes, ALIGN);
    return o;
  };
  const int64_t kp = (int64_t)kcap * p.Pp * 4;
  p.off_W = take(kp);
  p.off_G = take(kp);
  p.off_Z = take(p.Pp * 4);
  p.off_Zp = take(p.Pp * 4);
  if (m->learner_momentum != 0.f) p.off_Wprev = take(kp);
  const int64_t N = (int64_t)k * b;
  if (p.lenet_fused) {
    for (Op& o : p.ops) o.splits = 1;
    p.off_lenet_loss = take(N * 4);
    p.off_lenet_conv = take(N * LENET_CONV_PARAMS * 4);
    p.off_lenet_fc = take(N * LENET_FC_VEC * 4);
    p.off_bnpart = take(16);
    p.off_loss = take((int64_t)k * 4);
    p.off_flag = take(16);
    p.total = off;
    return true;
  }
  for (size_t i = 0; i < p.t.size(); ++i) {
    Tensor& x = p.t[i];
    const int64_t bytes = N * x.C * x.H * x.W * 4;
    if ((int)i == p.input) continue;  // the caller's images
    x.act = take(bytes);
    x.grad = take(bytes);
  }
  // a batch norm right after the conv that produces its input takes its
  // statistics from that conv's epilogue
  for (size_t i = 1; i < p.ops.size(); ++i) {
    Op& o = p.ops[i];
    Op& prev = p.ops[i - 1];
    if (o.kind == OP_BN && prev.kind == OP_CONV && prev.out == o.in) {
      prev.emit_stats = true;
      o.parts = conv_fwd_tiles_m(geom(p, prev));
    }
  }
  // a batch norm whose output gradient is written last by the data
  // gradient of the very next conv takes its backward sums from that
  // conv's epilogue (nothing else touches the partial-sum scratch between
  // the two)
  {
    std::vector<int> writer(p.t.size(), -1);
    for (int i = (int)p.ops.size() - 1; i >= 0; --i) {
      const Op& o = p.ops[i];
      if ((o.kind == OP_CONV && o.need_dx) || o.kind == OP_GAP || o.kind == OP_MAXPOOL ||
          o.kind == OP_BN)
        writer[o.in] = i;
      if (o.kind == OP_BN && o.res >= 0 && p.t[o.res].consumers == 1) writer[o.res] = i;
    }
    for (size_t i = 0; i + 1 < p.ops.size(); ++i) {
      Op& o = p.ops[i];
      Op& w = p.ops[i + 1];
      if (o.kind == OP_BN && writer[o.out] == (int)i + 1 && w.kind == OP_CONV && w.need_dx &&
          w.in == o.out && !w.dx_mask) {
        w.bnb = (int)i;
        o.bwd_parts = conv_bwd_data_tiles_m(geom(p, w));
      }
    }
  }
  // The head -- global average pool, an FC layer with few classes and no
  // ReLU, softmax cross-entropy -- runs as one kernel per image, which also
  // writes the backward sums of the batch norm feeding the pool (one part
  // per image).
  for (size_t i = 0; i + 2 < p.ops.size(); ++i) {
    Op& gp = p.ops[i];
    Op& fc = p.ops[i + 1];
    Op& xe = p.ops[i + 2];
    if (gp.kind != OP_GAP || fc.kind != OP_CONV || xe.kind != OP_XENT) continue;
    if (fc.in != gp.out || xe.in != fc.out || fc.R != 1 || fc.H != 1 || fc.W != 1 || fc.relu ||
        !fc.bias || !fc.need_dx || !head_ok(gp.C, gp.H * gp.W, fc.Co) ||
        p.t[gp.out].consumers != 1 || p.t[fc.out].consumers != 1)
      continue;
    gp.head = fc.head = xe.head = true;
    gp.head_fc = (int)i + 1;
    p.loss_per_image = true;
    if (i > 0) {
      Op& bn = p.ops[i - 1];
      if (bn.kind == OP_BN && bn.out == gp.in && p.t[gp.in].consumers == 1 && bn.bwd_parts == 0) {
        bn.bwd_parts = b;
        gp.head_bn = (int)i - 1;
      }
    }
  }
  int64_t bnpart = 0;
  for (size_t i = 0; i < p.ops.size(); ++i) {
    Op& o = p.ops[i];
    if (o.kind == OP_CONV) {
      if (!conv_supported(o.R, o.R, o.st, o.need_dx)) return false;
      ConvGeom g = geom(p, o);
      o.splits = conv_bwd_weight_splits(g, &o.chunk);
      // every layer keeps its own partials: one launch reduces them all
      // after the backward pass
      if (o.splits > 1) o.part_off = take((int64_t)k * o.splits * o.Co * o.Ci * o.R * o.R * 4);
    } else if (o.kind == OP_BN) {
      o.mean = take((int64_t)k * o.C * 4);
      o.istd = take((int64_t)k * o.C * 4);
      o.chunks = bn_chunks(b, o.H * o.W, o.C, k);
      bnpart = std::max<int64_t>(
          bnpart, (int64_t)k * o.C * std::max(std::max(o.chunks, o.parts), o.bwd_parts) * 2 * 8);
      if (o.res >= 0) {
        const Tensor& r = p.t[o.res];
        if (r.consumers == 1) o.dres = r.grad;
        else o.dres = take(N * o.C * o.H * o.W * 4);
      }
    } else if (o.kind == OP_MAXPOOL) {
      o.arg = take(N * o.C * o.Ho * o.Wo * 4);
    }
  }
  for (Op& o : p.ops)
    if (o.kind == OP_CONV && o.add_mode != ADD_NONE) o.add_buf = p.ops[o.add_buf].dres;
  p.off_bnpart = take(std::max<int64_t>(bnpart, 16));
  p.off_loss = take((int64_t)k * b * 4);
  if (p.loss_per_image) p.off_loss_mean = take((int64_t)k * 4);
  p.off_flag = take(16);
  p.total = off;
  return true;
}

}  // namespace

struct ProfRec {
  hipEvent_t a, b;
  const char* name;
  double flops, bytes;
};

struct ProfAgg {
  std::string name;
  int64_t launches = 0;
  double ms = 0, flops = 0, bytes = 0;
};

// Weight gradients go to the side stream FORK_GROUP layers at a time behind
// one fork event: each fork is an event record on the caller's stream and a
// barrier packet on the side stream (ResNet-32, k=4, b=32: one fork per
// layer 90.3k images/s, per two layers 93.1k, per three 93.2k, per four
// 92.5k; with the lighter weight-gradient grids, three layers per fork
// matched two at k=4 b=32 and were 2% faster at k=1..4, b=16).
constexpr int FORK_GROUP = 3;

struct cb_ctx {
  Plan p;
  char* ws = nullptr;
  size_t ws_bytes = 0;
  hipStream_t stream = nullptr;
  int device = 0;
  float alpha = 0, lr = 0, mu = 0;
  bool pending = false;
  std::string err;
  // instrumentation: events around every launch while enabled
  bool prof = false;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> evpool;
  std::vector<ProfAgg> agg;
  // weight-gradient split reductions of all layers, one launch per table
  std::vector<SplitTable> split_tables;
  std::vector<double> split_bytes;
  std::vector<int> split_after;  // per table: the operator whose weight gradient completes it
  bool split_per_layer = false;   // one table per layer
  int first_conv = -1;            // the first conv operator (the backward pass ends with it)
  std::vector<char> flush_at;     // per operator: its layer closes a side-stream group
  // Weight gradients run on a second stream of the library's own (default
  // priority), forked in groups of layers whose output gradients are
  // final and joined before the step ends, so they overlap the
  // data-gradient chain.
  hipStream_t side = nullptr;
  std::vector<hipEvent_t> fork_ev;  // per operator (conv layers only)
  hipEvent_t join_ev = nullptr;
  // Graph replay: the launches of one forward/backward pass, captured once
  // per (inputs, labels) pair as a HIP graph and replayed by later steps on
  // the same buffers; the host then submits one graph instead of every
  // kernel.  Least recently captured graphs are dropped beyond
  // GRAPH_CACHE pairs.
  static constexpr size_t GRAPH_CACHE = 8;
  struct StepGraph {
    const void* x;
    const void* y;
    hipGraph_t g;
    hipGraphExec_t e;
  };
  bool graphs = false;
  std::vector<StepGraph> step_graphs;
  hipStream_t cap = nullptr;  // capture stream (default priority)

  void drop_graphs() {
    if (step_graphs.empty()) return;
    (void)hipStreamSynchronize(stream);
    for (auto& sg : step_graphs) {
      (void)hipGraphExecDestroy(sg.e);
      (void)hipGraphDestroy(sg.g);
    }
    step_graphs.clear();
  }

  ~cb_ctx() {
    drop_graphs();
    if (cap) (void)hipStreamDestroy(cap);
    if (side) {
      (void)hipStreamSynchronize(side);
      (void)hipStreamDestroy(side);
    }
    for (auto e : fork_ev)
      if (e) (void)hipEventDestroy(e);
    if (join_ev) (void)hipEventDestroy(join_ev);
    for (auto& r : recs) {
      (void)hipEventDestroy(r.a);
      (void)hipEventDestroy(r.b);
    }
    for (auto e : evpool) (void)hipEventDestroy(e);
  }

  template <class T>
  T* at(int64_t off) const { return reinterpret_cast<T*>(ws + off); }
  float* W() const { return at<float>(p.off_W); }
  float* G() const { return at<float>(p.off_G); }
  float* Z() const { return at<float>(p.off_Z); }
  float* Zp() const { return at<float>(p.off_Zp); }
  float* Wprev() const { return p.off_Wprev >= 0 ? at<float>(p.off_Wprev) : nullptr; }
};

namespace {

std::string g_create_error;

}  // namespace

void cbk::note_error(const std::string& msg) { g_create_error = msg; }

namespace {

int fail(cb_ctx* c, int code, const std::string& msg) {
  if (c) c->err = msg;
  else g_create_error = msg;
  return code;
}

#define CB_HIP(c, call)                                                        \
  do {                                                                         \
    hipError_t e_ = (call);                                                    \
    if (e_ != hipSuccess)                                                      \
      return fail(c, CB_EDEVICE, std::string(#call) + ": " + hipGetErrorString(e_)); \
  } while (0)

hipEvent_t prof_event(cb_ctx* c) {
  hipEvent_t e = nullptr;
  if (!c->evpool.empty()) {
    e = c->evpool.back();
    c->evpool.pop_back();
  } else if (hipEventCreate(&e) != hipSuccess) {
    e = nullptr;
  }
  return e;
}

// Times the one kernel launch made inside the scope when instrumentation is
// on: the events ride on that kernel's dispatch (see klaunch).
struct ProfScope {
  cb_ctx* c;
  hipEvent_t a = nullptr, b = nullptr;
  explicit ProfScope(cb_ctx* cc) : c(cc) {
    if (!c->prof) return;
    a = prof_event(c);
    b = a ? prof_event(c) : nullptr;
    if (a && b) {
      g_launch_timing.start = a;
      g_launch_timing.stop = b;
    }
  }
  void done(const char* name, double flops, double bytes) {
    if (!a || !b) return;
    if (g_launch_timing.start == a) {  // nothing was launched: give the events back
      g_launch_timing = LaunchTiming();
      c->evpool.push_back(a);
      c->evpool.push_back(b);
    } else {
      c->recs.push_back(ProfRec{a, b, name, flops, bytes});
    }
    a = b = nullptr;
  }
  ~ProfScope() {
    if (a && b && g_launch_timing.start == a) g_launch_timing = LaunchTiming();
    if (a && b) {
      c->evpool.push_back(a);
      c->evpool.push_back(b);
    }
  }
};

// One instrumented launch; `call` may overwrite nm_ with the name of the
// kernel variant it launched.
#define CB_LAUNCH(c, name, flops, bytes, call) \
  do {                                         \
    ProfScope ps_(c);                          \
    const char* nm_ = (name);                  \
    CB_HIP(c, call);                           \
    ps_.done(nm_, flops, bytes);               \
  } while (0)

// The MNIST-shaped LeNet: one launch per image for the forward and
// backward data path, one for the learners' gradients and losses.
int enqueue_lenet(cb_ctx* c, const float* x, const int32_t* labels, hipStream_t s) {
  const Plan& p = c->p;
  LenetArgs a;
  a.k = p.k; a.b = p.b; a.classes = p.m.num_classes;
  a.x = x;
  a.labels = labels;
  a.w = c->W();
  a.grad = c->G();
  a.pstride = p.Pp;
  a.loss = c->at<float>(p.off_lenet_loss);
  a.learner_loss = c->at<float>(p.off_loss);
  a.conv_part = c->at<float>(p.off_lenet_conv);
  a.fc_vec = c->at<float>(p.off_lenet_fc);
  const double N = (double)p.k * p.b, C = p.m.num_classes;
  // multiply-adds per image: conv1 and conv2 forward, the FC layers forward
  // and backward, conv2's data gradient, conv2's and conv1's weight shares
  const double fc = 400.0 * 120 + 120.0 * 84 + 84.0 * C;
  const double macs = 117600.0 + 240000.0 + 2.0 * fc + 240000.0 + 240000.0 + 117600.0;
  const double img_bytes = 4.0 * (784.0 + 1 + (double)LENET_CONV_PARAMS + LENET_FC_VEC);
  CB_LAUNCH(c, "lenet_image_k", 2.0 * macs * N, N * img_bytes + 4.0 * p.k * p.P,
            lenet_image(a, s));
  // the learners' FC weight gradients (sums over b images of outer products)
  CB_LAUNCH(c, "lenet_learner_k", 2.0 * fc * N,
            4.0 * (N * ((double)LENET_CONV_PARAMS + LENET_FC_VEC + 1) + p.k * (double)p.P + p.k),
            lenet_learner(a, s));
  return CB_OK;
}

int enqueue_step(cb_ctx* c, const float* x, const int32_t* labels, hipStream_t s) {
  const Plan& p = c->p;
  if (p.lenet_fused) return enqueue_lenet(c, x, labels, s);
  const int k = p.k, b = p.b, N = k * b;
  auto act = [&](int t) -> float* { return t == p.input ? const_cast<float*>(x) : c->at<float>(p.t[t].act); };
  auto grd = [&](int t) -> float* { return c->at<float>(p.t[t].grad); };
  float* W = c->W();
  float* G = c->G();

  // forward, all learners in every launch
  for (size_t oi = 0; oi < p.ops.size(); ++oi) {
    const Op& o = p.ops[oi];
    switch (o.kind) {
      case OP_CONV: {
        if (o.head) break;  // inside the fused head
        ConvFwdArgs a;
        a.g = geom(p, o);
        a.x = act(o.in);
        a.w = W + o.w_off;
        a.bias = o.bias ? W + o.b_off : nullptr;
        a.pstride = p.Pp;
        a.y = act(o.out);
        a.relu = o.relu;
        a.stats = o.emit_stats ? c->at<double>(p.off_bnpart) : nullptr;
        const double flops = 2.0 * N * o.Ho * o.Wo * o.Co * o.Ci * o.R * o.R;
        const double bytes = 4.0 * ((double)N * o.Ci * o.H * o.W + (double)k * o.Co * o.Ci * o.R * o.R +
                                    (double)N * o.Co * o.Ho * o.Wo);
        ProfScope ps(c);
        const char* nm = "conv_fwd_k";
        CB_HIP(c, conv_fwd(a, s, &nm));
        ps.done(nm, flops, bytes);
        break;
      }
      case OP_BN: {
        BNArgs a;
        a.k = k; a.b = b; a.C = o.C; a.H = o.H; a.W = o.W;
        a.x = act(o.in);
        a.y = act(o.out);
        a.gamma = W + o.g_off;
        a.pstride = p.Pp;
        a.mean = c->at<float>(o.mean);
        a.istd = c->at<float>(o.istd);
        a.part = c->at<double>(p.off_bnpart);
        a.chunks = o.chunks;
        a.parts = o.parts > 0 ? o.parts : o.chunks;
        a.relu = o.relu;
        a.res = o.res >= 0 ? act(o.res) : nullptr;
        a.res_mode = o.res >= 0 ? o.res_mode : RES_NONE;
        a.res_C = o.res >= 0 ? p.t[o.res].C : 0;
        a.res_st = o.res_st;
        a.res_H = o.res >= 0 ? p.t[o.res].H : 0;
        a.res_W = o.res >= 0 ? p.t[o.res].W : 0;
        const double n = (double)N * o.C * o.H * o.W;
        const double res = a.res_mode == RES_SAME ? n
                           : a.res_mode == RES_SUBSAMPLE ? (double)N * a.res_C * o.H * o.W : 0.0;
        if (o.parts == 0) CB_LAUNCH(c, "bn_stats_k", 0.0, 4.0 * n, bn_fwd_stats(a, s));
        CB_LAUNCH(c, "bn_apply_k", 0.0, 4.0 * (2.0 * n + res), bn_fwd_apply(a, s, &nm_));
        break;
      }
      case OP_MAXPOOL:
        CB_LAUNCH(c, "maxpool_fwd_k", 0.0,
                  4.0 * N * o.C * ((double)o.H * o.W + 2.0 * o.Ho * o.Wo),
                  maxpool_fwd(act(o.in), N, o.C, o.H, o.W, o.K, o.st, o.pad, act(o.out), o.Ho,
                              o.Wo, c->at<int>(o.arg), s));
        break;
      case OP_GAP: {
        if (!o.head) {
          CB_LAUNCH(c, "gap_fwd_k", 0.0, 4.0 * N * o.C * (o.H * o.W + 1.0),
                    gap_fwd(act(o.in), N, o.C, o.H * o.W, act(o.out), s));
          break;
        }
        const Op& fc = p.ops[o.head_fc];
        HeadArgs a;
        a.k = k; a.b = b; a.C = o.C; a.HW = o.H * o.W; a.classes = fc.Co;
        a.y = act(o.in);
        a.g = act(o.out);
        a.w = W + fc.w_off;
        a.bias = fc.bias ? W + fc.b_off : nullptr;
        a.pstride = p.Pp;
        a.labels = labels;
        a.dlogits = grd(fc.out);
        a.loss = c->at<float>(p.off_loss);
        a.dy = grd(o.in);
        a.bn_part = nullptr;
        a.bn_relu = 0;
        a.bn_x = a.bn_mean = a.bn_istd = nullptr;
        if (o.head_bn >= 0) {
          const Op& bn = p.ops[o.head_bn];
          a.bn_part = c->at<double>(p.off_bnpart);
          a.bn_relu = bn.relu;
          a.bn_x = act(bn.in);
          a.bn_mean = c->at<float>(bn.mean);
          a.bn_istd = c->at<float>(bn.istd);
        }
        // the pooled tensor (read twice), its gradient, the norm's x, the
        // FC weights, features, logit gradients
        const double plane = (double)N * o.C * o.H * o.W;
        const double bytes = 4.0 * (plane * (2.0 + (o.head_bn >= 0 ? 1.0 : 0.0)) +
                                    (double)k * fc.Co * o.C + (double)N * (o.C + 2.0 * fc.Co + 2.0));
        // the FC's forward and data-gradient contractions
        const double flops = 4.0 * N * o.C * fc.Co;
        CB_LAUNCH(c, "head_k", flops, bytes, head_fwd_bwd(a, s));
        break;
      }
      case OP_XENT:
        if (o.head) break;  // inside the fused head
        CB_LAUNCH(c, "softmax_xent_k", 0.0, 4.0 * N * (2.0 * p.m.num_classes + 1),
                  softmax_xent(act(o.in), labels, k, b, p.m.num_classes, grd(o.in),
                               c->at<float>(p.off_loss), s, &nm_));
        break;
    }
  }
  // Weight gradients, one layer's: bias sums, the weight gradient, and
  // the split reductions that layer completes.
  auto wgrad = [&](int idx, hipStream_t ss) -> int {
    const Op& o = p.ops[idx];
    const ConvGeom g = geom(p, o);
    const double flops = 2.0 * N * o.Ho * o.Wo * o.Co * o.Ci * o.R * o.R;
    const double wn = (double)o.Co * o.Ci * o.R * o.R;
    const double xin = (double)N * o.Ci * o.H * o.W, yout = (double)N * o.Co * o.Ho * o.Wo;
    if (o.bias) {
      // the fused head's FC also reduces the per-image loss terms to each
      // replica's mean loss
      const bool terms = o.head && p.loss_per_image;
      CB_LAUNCH(c, "channel_sum_k", 0.0, 4.0 * (yout + (terms ? N + k : 0)),
                channel_sum(grd(o.out), k, b, o.Co, o.Ho * o.Wo, G + o.b_off, p.Pp, ss,
                            terms ? c->at<float>(p.off_loss) : nullptr,
                            terms ? c->at<float>(p.off_loss_mean) : nullptr));
    }
    ConvBwdWeightArgs w;
    w.g = g;
    w.x = act(o.in);
    w.dy = grd(o.out);
    w.dw = G + o.w_off;
    w.pstride = p.Pp;
    w.partial = o.splits > 1 ? c->at<float>(o.part_off) : nullptr;
    w.splits = o.splits;
    w.chunk = o.chunk;
    {
      ProfScope ps(c);
      const char* nm = "conv_bwd_weight_k";
      CB_HIP(c, conv_bwd_weight(w, ss, &nm));
      ps.done(nm, flops, 4.0 * (xin + yout + k * wn));
    }
    for (size_t t = 0; t < c->split_tables.size(); ++t)
      if (c->split_after[t] == idx)
        CB_LAUNCH(c, "reduce_splits_k", 0.0, c->split_bytes[t],
                  reduce_splits(c->split_tables[t], k, ss, &nm_));
    return CB_OK;
  };
  // Layers whose dY is final wait in `pending` and go to the side stream
  // together behind one fork event, in the groups of FORK_GROUP layers
  // that flush_at marks.
  std::vector<int> pending;
  auto flush = [&](int at) -> int {
    if (pending.empty()) return CB_OK;
    CB_HIP(c, hipEventRecord(c->fork_ev[at], s));
    CB_HIP(c, hipStreamWaitEvent(c->side, c->fork_ev[at], 0));
    for (int idx : pending)
      if (int rc = wgrad(idx, c->side)) return rc;
    pending.clear();
    return CB_OK;
  };
  // backward in reverse operator order
  for (int i = (int)p.ops.size() - 1; i >= 0; --i) {
    const Op& o = p.ops[i];
    switch (o.kind) {
      case OP_XENT: break;
      case OP_GAP:
        if (o.head) break;  // done by the fused head
        CB_LAUNCH(c, "gap_bwd_k", 0.0, 4.0 * N * o.C * (o.H * o.W + 1.0),
                  gap_bwd(grd(o.out), N, o.C, o.H * o.W, grd(o.in), s, &nm_));
        break;
      case OP_MAXPOOL:
        CB_LAUNCH(c, "maxpool_bwd_k", 0.0,
                  4.0 * N * o.C * (2.0 * o.Ho * o.Wo + (1.0 + o.dx_mask) * o.H * o.W),
                  maxpool_bwd(grd(o.out), c->at<int>(o.arg), act(o.in), N, o.C, o.H, o.W, o.K,
                              o.st, o.pad, o.Ho, o.Wo, grd(o.in), o.dx_mask, s));
        break;
      case OP_BN: {
        BNBwdArgs a;
        a.k = k; a.b = b; a.C = o.C; a.H = o.H; a.W = o.W;
        a.x = act(o.in);
        // without a residual input the ReLU mask is recomputed from x
        // (read anyway) instead of read from y
        a.relu_x = o.relu && o.res < 0;
        a.y = (o.relu && !a.relu_x) ? act(o.out) : nullptr;
        a.dy = grd(o.out);
        a.dx = grd(o.in);
        a.dres = o.res >= 0 ? c->at<float>(o.dres) : nullptr;
        a.gamma = W + o.g_off;
        a.dgamma = G + o.g_off;
        a.pstride = p.Pp;
        a.mean = c->at<float>(o.mean);
        a.istd = c->at<float>(o.istd);
        a.part = c->at<double>(p.off_bnpart);
        a.chunks = o.chunks;
        a.parts = o.bwd_parts > 0 ? o.bwd_parts : o.chunks;
        const double n = (double)N * o.C * o.H * o.W;
        const double mask = a.y ? 1.0 : 0.0, dres = o.res >= 0 ? 1.0 : 0.0;
        if (o.bwd_parts == 0)
          CB_LAUNCH(c, "bn_bwd_stats_k", 0.0, 4.0 * n * (2.0 + mask), bn_bwd_stats(a, s));
        CB_LAUNCH(c, "bn_bwd_apply_k", 0.0, 4.0 * n * (3.0 + mask + dres), bn_bwd_apply(a, s, &nm_));
        break;
      }
      case OP_CONV: {
        const ConvGeom g = geom(p, o);
        const double flops = 2.0 * N * o.Ho * o.Wo * o.Co * o.Ci * o.R * o.R;
        const double wn = (double)o.Co * o.Ci * o.R * o.R;
        const double xin = (double)N * o.Ci * o.H * o.W, yout = (double)N * o.Co * o.Ho * o.Wo;
        // dY of this layer is final here: its weight (and bias) gradient,
        // which reads dY and the layer's input and writes only this layer's
        // slice of G and its own split partials, can go to the side stream
        // (with instrumentation on, everything stays on the caller's stream,
        // so each measured duration is the kernel alone).  The first
        // layer's ends the step with nothing left to overlap: with per-layer
        // reductions it stays on the caller's stream, saving a fork and the
        // join's wait (1%), and so do the layers still waiting for a full
        // group (fewer than FORK_GROUP), which would otherwise be forked
        // off just before the join (ResNet-32 k=4 b=32: 94.8k -> 95.7k
        // images/s; keeping the last 5 or 8 layers there instead measured
        // 2.5-5% slower).
        if (c->prof) {
          if (int rc = wgrad(i, s)) return rc;
        } else if (c->split_per_layer && i == c->first_conv) {
          for (int idx : pending)
            if (int rc = wgrad(idx, s)) return rc;
          pending.clear();
          if (int rc = wgrad(i, s)) return rc;
        } else {
          pending.push_back(i);
          if (c->flush_at[i])
            if (int rc = flush(i)) return rc;
        }
        if (o.need_dx && !o.head) {  // a head FC's dx comes from the fused head
          ConvBwdDataArgs d;
          d.g = g;
          d.dy = grd(o.out);
          d.w = W + o.w_off;
          d.pstride = p.Pp;
          d.dx = grd(o.in);
          d.accumulate = o.dx_accumulate;
          d.mask = o.dx_mask ? act(o.in) : nullptr;
          d.add = o.add_mode != ADD_NONE ? c->at<float>(o.add_buf) : nullptr;
          d.add_mode = o.add_mode;
          d.add_C = o.add_C;
          d.add_st = o.add_st;
          d.bn_part = nullptr;
          d.bn_x = d.bn_y = d.bn_mean = d.bn_istd = nullptr;
          if (o.bnb >= 0) {
            const Op& bn = p.ops[o.bnb];
            d.bn_part = c->at<double>(p.off_bnpart);
            d.bn_x = act(bn.in);
            d.bn_y = bn.relu ? act(bn.out) : nullptr;
            d.bn_mean = c->at<float>(bn.mean);
            d.bn_istd = c->at<float>(bn.istd);
            // without a residual input the norm's ReLU output can be
            // recomputed from bn_x (the implicit-GEMM epilogue does)
            if (bn.relu && bn.res < 0) d.bn_gamma = W + bn.g_off;
            // When that ReLU output is this layer's input, the ReLU mask has
            // already zeroed dX wherever it is not positive: the batch norm's
            // own ReLU test would repeat it on the same tensor.
            if (d.bn_y == d.mask) {
              d.bn_y = nullptr;
              d.mask_from_bn = d.bn_gamma != nullptr;
            }
          }
          ProfScope ps(c);
          const char* nm = "conv_bwd_data_k";
          CB_HIP(c, conv_bwd_data(d, s, &nm));
          // every tensor the kernel and its fused epilogue must move once: dY,
          // the filters, dX (read too when accumulating), the ReLU mask
          // (unless the direct kernel recomputes it), the residual gradient
          // and the next batch norm's x (and y for its ReLU)
          const bool mask_read =
              o.dx_mask && !(d.mask_from_bn && conv_direct_bwd_data_ok(g));
          double moved = yout + k * wn + xin * (1.0 + o.dx_accumulate + mask_read);
          if (o.add_mode == ADD_SAME) moved += xin;
          if (o.add_mode == ADD_SUBSAMPLE)
            moved += (double)N * o.add_C * (o.H / o.add_st) * (o.W / o.add_st);
          // (y is not read where the ReLU decision is recomputed from x:
          // the direct stride-1 and implicit-GEMM kernels, given gamma)
          const bool y_read = d.bn_y && !(d.bn_gamma && (conv_direct_bwd_data_ok(g) ||
                                                          !conv_s2_dgrad_ok(g)));
          if (d.bn_part) moved += xin * (y_read ? 2.0 : 1.0);
          ps.done(nm, flops, 4.0 * moved);
        }
        break;
      }
    }
  }
  if (!pending.empty())
    if (int rc = flush(pending.back())) return rc;
  // join: G is complete, and nothing reads this step's buffers any more
  if (!c->prof) {
    CB_HIP(c, hipEventRecord(c->join_ev, c->side));
    CB_HIP(c, hipStreamWaitEvent(s, c->join_ev, 0));
  }
  return CB_OK;
}

int enqueue_sma(cb_ctx* c, const float* G, int64_t gstride, int correct) {
  SMAArgs a;
  a.W = c->W();
  a.G = G;
  a.Wprev = c->Wprev();
  a.z = c->Z();
  a.zp = c->Zp();
  a.k = c->p.k;
  a.P4 = (c->p.P + 3) / 4;  // stays inside a [k][P] gradient array when P % 4 == 0
  a.wstride4 = c->p.Pp / 4;
  a.gstride4 = gstride / 4;
  a.alpha = c->alpha;
  a.lr = c->lr;
  a.mu = c->mu;
  a.mu_l = c->p.m.learner_momentum;
  a.correct = correct;
  const double P = (double)c->p.P, k = c->p.k;
  double bytes = correct ? 4.0 * P * (3.0 * k + 4.0) : 4.0 * P * 3.0 * k;
  if (a.Wprev) bytes += 8.0 * k * P;
  CB_LAUNCH(c, correct ? "sma_k" : "sma_k<local step>", 0.0, bytes, sma_step(a, c->stream, &nm_));
  return CB_OK;
}

// One forward/backward pass as a graph replay on the context's stream: the
// graph of this (inputs, labels) pair if there is one, else the pass
// captured and instantiated first.  The capture runs on a stream of the
// library's own (the caller's may be the null stream, which cannot be
// captured); the side stream joins the capture through the fork events and
// is joined back before it ends.  Capturing launches nothing.
int replay_step(cb_ctx* c, const float* x, const int32_t* labels) {
  for (auto& sg : c->step_graphs)
    if (sg.x == x && sg.y == labels) {
      CB_HIP(c, hipGraphLaunch(sg.e, c->stream));
      return CB_OK;
    }
  if (c->step_graphs.size() >= cb_ctx::GRAPH_CACHE) {
    CB_HIP(c, hipStreamSynchronize(c->stream));
    (void)hipGraphExecDestroy(c->step_graphs.front().e);
    (void)hipGraphDestroy(c->step_graphs.front().g);
    c->step_graphs.erase(c->step_graphs.begin());
  }
  if (!c->cap) CB_HIP(c, hipStreamCreateWithFlags(&c->cap, hipStreamNonBlocking));
  CB_HIP(c, hipStreamBeginCapture(c->cap, hipStreamCaptureModeRelaxed));
  const int rc = enqueue_step(c, x, labels, c->cap);
  hipGraph_t g = nullptr;
  const hipError_t e = hipStreamEndCapture(c->cap, &g);  // ends the capture on every path
  if (rc != CB_OK) {
    if (g) (void)hipGraphDestroy(g);
    return rc;
  }
  CB_HIP(c, e);
  hipGraphExec_t ex = nullptr;
  const hipError_t ei = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
  if (ei != hipSuccess) {
    (void)hipGraphDestroy(g);
    CB_HIP(c, ei);
  }
  c->step_graphs.push_back(cb_ctx::StepGraph{x, labels, g, ex});
  CB_HIP(c, hipGraphLaunch(ex, c->stream));
  return CB_OK;
}

int check_finite(cb_ctx* c) {
  int* flag = c->at<int>(c->p.off_flag);
  CB_HIP(c, zero_ints(flag, 1, c->stream));
  CB_HIP(c, nonfinite_scan(c->Z(), c->p.P, flag, c->stream));
  int h = 0;
  CB_HIP(c, hipMemcpyAsync(&h, flag, sizeof(int), hipMemcpyDeviceToHost, c->stream));
  CB_HIP(c, hipStreamSynchronize(c->stream));
  if (h) return fail(c, CB_ENONFINITE, "central model holds NaN or Inf");
  return CB_OK;
}

int enter(cb_ctx* c) {
  if (!c) return CB_EINVAL;
  c->err.clear();
  CB_HIP(c, hipSetDevice(c->device));
  return CB_OK;
}

}  // namespace

extern "C" {

int64_t cb_num_params(const cb_model* m) {
  Plan p;
  if (!make_plan(m, 1, 1, p)) return CB_EINVAL;
  return p.P;
}

int cb_num_tensors(const cb_model* m) {
  Plan p;
  if (!make_plan(m, 1, 1, p)) return CB_EINVAL;
  return (int)p.params.size();
}

int cb_tensor_info(const cb_model* m, int idx, int64_t* offset, int* kind, int* ndim,
                   int* dims4) {
  Plan p;
  if (!make_plan(m, 1, 1, p) || idx < 0 || idx >= (int)p.params.size()) return CB_EINVAL;
  const ParamInfo& pi = p.params[idx];
  *offset = pi.offset;
  *kind = pi.kind;
  *ndim = pi.ndim;
  for (int i = 0; i < 4; ++i) dims4[i] = pi.dims[i];
  return CB_OK;
}

}  // extern "C"

namespace {

// The split-reduction tables of the current plan (one segment per layer
// whose weight gradient is split).
// The layers' split reductions, grouped: a group's reduction is launched on
// the second stream right after the last of its weight gradients (in
// backward order), so every group's but the last overlaps the rest of the
// backward pass instead of waiting for its end.  From 64 input images of
// 32 x 32 per step (k*b*H*W input pixels), one group per layer: that
// measured fastest (ResNet-32 k=4 b=32 2.6% and k=8..16 b=16 5% faster than
// one reduction after the backward pass, k=4 and 6 at b=16 5-6%; ResNet-50
// 1.5%).  With less work the weight gradients are short and the extra
// launches would crowd the second stream (ResNet-32 k = 1 at b = 16 loses
// 1.5%), so all layers form one group, reduced after the last weight
// gradient.
void build_split_tables(cb_ctx* c) {
  c->split_tables.clear();
  c->split_bytes.clear();
  c->split_after.clear();
  if (c->p.lenet_fused) {  // no split partials on the fused LeNet path
    c->split_per_layer = false;
    c->first_conv = -1;
    c->flush_at.assign(c->p.ops.size(), 0);
    return;
  }
  const int nops = (int)c->p.ops.size();
  const bool per_layer =
      (int64_t)c->p.k * c->p.b * c->p.m.in_h * c->p.m.in_w >= (int64_t)64 * 32 * 32;
  c->split_per_layer = per_layer;
  c->first_conv = -1;
  for (int i = 0; i < nops && c->first_conv < 0; ++i)
    if (c->p.ops[i].kind == OP_CONV) c->first_conv = i;
  // Side-stream groups: conv layers in backward order, FORK_GROUP at a time
  // (with per-layer reductions, the first layer runs on the caller's
  // stream instead and belongs to none).
  c->flush_at.assign(nops, 0);
  int in_group = 0;
  for (int i = nops - 1; i >= 0; --i) {
    if (c->p.ops[i].kind != OP_CONV || (per_layer && i == c->first_conv)) continue;
    if (++in_group == FORK_GROUP) {
      c->flush_at[i] = 1;
      in_group = 0;
    }
  }
  auto add = [&](int i) {
    const Op& o = c->p.ops[i];
    const int64_t wn = (int64_t)o.Co * o.Ci * o.R * o.R;
    split_table_add(c->split_tables.back(), c->at<float>(o.part_off), c->G() + o.w_off, wn,
                    o.splits);
    c->split_bytes.back() += 4.0 * c->p.k * wn * (o.splits + 1.0);
  };
  auto open = [&]() {
    c->split_tables.emplace_back();
    c->split_tables.back().pstride = c->p.Pp;
    c->split_bytes.push_back(0.0);
    c->split_after.push_back(-1);
  };
  if (per_layer) {
    // one table per layer, reduced right after its weight gradient (one
    // table per side-stream group instead, reduced after the group's last
    // weight gradient, measured 3.7% slower at ResNet-32 k=4 b=32)
    for (int i = 0; i < nops; ++i) {
      if (c->p.ops[i].kind != OP_CONV || c->p.ops[i].splits <= 1) continue;
      open();
      add(i);
      c->split_after.back() = i;
    }
    return;
  }
  // all layers in as few tables as fit, reduced after the backward pass
  for (int i = 0; i < nops; ++i) {
    const Op& o = c->p.ops[i];
    if (o.kind != OP_CONV || o.splits <= 1) continue;
    if (c->split_tables.empty() || c->split_tables.back().nseg == MAX_SPLIT_SEGS) {
      open();
      c->split_after.back() = i;  // the table's first layer: its last weight gradient
    }
    add(i);
  }
}

}  // namespace

extern "C" {

size_t cb_workspace_bytes(const cb_model* m, int k, int b) {
  // enough for every number of active learners up to k (cb_set_learners)
  int64_t most = 0;
  for (int kk = 1; kk <= k; ++kk) {
    Plan p;
    if (!make_plan(m, kk, b, p, k)) return 0;
    most = std::max(most, p.total);
  }
  return (size_t)most;
}

int cb_create(const cb_model* m, int k, int b, float alpha, float lr, float momentum,
              const float* w0_host, int64_t n_params, void* workspace_dev, size_t ws_bytes,
              void* hip_stream, cb_ctx** out) {
  if (!out) return fail(nullptr, CB_EINVAL, "out is NULL");
  *out = nullptr;
  if (!std::isfinite(alpha) || !std::isfinite(lr) || !std::isfinite(momentum) ||
      (m && !std::isfinite(m->learner_momentum)))
    return fail(nullptr, CB_EINVAL, "alpha, lr, momentum and learner_momentum must be finite");
  cb_ctx* c = new cb_ctx();
  if (!make_plan(m, k, b, c->p)) {
    delete c;
    return fail(nullptr, CB_EINVAL, "unsupported model description, k or b");
  }
  if (!w0_host || n_params != c->p.P) {
    delete c;
    return fail(nullptr, CB_EINVAL, "w0 is NULL or n_params differs from the model's count");
  }
  if (!workspace_dev || reinterpret_cast<uintptr_t>(workspace_dev) % ALIGN) {
    delete c;
    return fail(nullptr, CB_EINVAL, "workspace is NULL or not 256-byte aligned");
  }
  if (ws_bytes < cb_workspace_bytes(m, k, b)) {
    delete c;
    return fail(nullptr, CB_ENOMEM, "workspace smaller than cb_workspace_bytes()");
  }
  c->ws = static_cast<char*>(workspace_dev);
  c->stream = static_cast<hipStream_t>(hip_stream);
  c->ws_bytes = ws_bytes;
  build_split_tables(c);
  c->alpha = alpha;
  c->lr = lr;
  c->mu = momentum;
  int rc = CB_OK;
  auto dev = [&](hipError_t e, const char* what) {
    if (e != hipSuccess && rc == CB_OK) {
      g_create_error = std::string(what) + ": " + hipGetErrorString(e);
      rc = CB_EDEVICE;
    }
  };
  dev(hipGetDevice(&c->device), "hipGetDevice");
  dev(hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking), "hipStreamCreate");
  c->fork_ev.assign(c->p.ops.size(), nullptr);
  for (size_t i = 0; i < c->p.ops.size(); ++i)
    if (c->p.ops[i].kind == OP_CONV)
      dev(hipEventCreateWithFlags(&c->fork_ev[i], hipEventDisableTiming), "hipEventCreate");
  dev(hipEventCreateWithFlags(&c->join_ev, hipEventDisableTiming), "hipEventCreate");
  const Plan& p = c->p;
  const size_t pbytes = (size_t)p.P * 4;
  // w0 is host memory the caller may free after this call, so the copies
  // are waited for before returning
  dev(hipMemcpyAsync(c->Z(), w0_host, pbytes, hipMemcpyHostToDevice, c->stream), "upload w0");
  dev(hipMemcpyAsync(c->Zp(), c->Z(), pbytes, hipMemcpyDeviceToDevice, c->stream), "z_prev");
  for (int j = 0; j < k; ++j) {
    dev(hipMemcpyAsync(c->W() + (int64_t)j * p.Pp, c->Z(), pbytes, hipMemcpyDeviceToDevice,
                       c->stream), "replica init");
    if (c->Wprev())
      dev(hipMemcpyAsync(c->Wprev() + (int64_t)j * p.Pp, c->Z(), pbytes,
                         hipMemcpyDeviceToDevice, c->stream), "replica init");
  }
  dev(hipStreamSynchronize(c->stream), "hipStreamSynchronize");
  if (rc != CB_OK) {
    delete c;
    return rc;
  }
  *out = c;
  return CB_OK;
}

int cb_step(cb_ctx* c, const float* inputs_dev, const int32_t* labels_dev) {
  int rc = enter(c);
  if (rc) return rc;
  if (!inputs_dev || !labels_dev) return fail(c, CB_EINVAL, "inputs or labels is NULL");
  if (c->pending) {
    rc = enqueue_sma(c, c->G(), c->p.Pp, 0);  // unsynced gradient: local step
    if (rc) return rc;
  }
  rc = (c->graphs && !c->prof) ? replay_step(c, inputs_dev, labels_dev)
                               : enqueue_step(c, inputs_dev, labels_dev, c->stream);
  if (rc) return rc;
  c->pending = true;
  return CB_OK;
}

int cb_sync(cb_ctx* c) {
  int rc = enter(c);
  if (rc) return rc;
  if (!c->pending) return fail(c, CB_ESTATE, "cb_sync: no gradient pending");
  rc = enqueue_sma(c, c->G(), c->p.Pp, 1);
  if (rc) return rc;
  c->pending = false;
  if (c->p.m.check_finite) return check_finite(c);
  return CB_OK;
}

int cb_wait(cb_ctx* c) {
  int rc = enter(c);
  if (rc) return rc;
  CB_HIP(c, hipStreamSynchronize(c->stream));
  return CB_OK;
}

static int copy_out(cb_ctx* c, const float* src, float* out_host, int64_t n, int64_t want) {
  int rc = enter(c);
  if (rc) return rc;
  if (!out_host || n != want) return fail(c, CB_EINVAL, "output is NULL or n is wrong");
  CB_HIP(c, hipMemcpyAsync(out_host, src, (size_t)n * 4, hipMemcpyDeviceToHost, c->stream));
  CB_HIP(c, hipStreamSynchronize(c->stream));
  return CB_OK;
}

int cb_get_central(cb_ctx* c, float* out_host, int64_t n) {
  if (!c) return CB_EINVAL;
  return copy_out(c, c->Z(), out_host, n, c->p.P);
}

int cb_get_prev_central(cb_ctx* c, float* out_host, int64_t n) {
  if (!c) return CB_EINVAL;
  return copy_out(c, c->Zp(), out_host, n, c->p.P);
}

int cb_get_replica(cb_ctx* c, int j, float* out_host, int64_t n) {
  if (!c) return CB_EINVAL;
  if (j < 0 || j >= c->p.k) return fail(c, CB_EINVAL, "replica index out of range");
  return copy_out(c, c->W() + (int64_t)j * c->p.Pp, out_host, n, c->p.P);
}

int cb_get_grad(cb_ctx* c, int j, float* out_host, int64_t n) {
  if (!c) return CB_EINVAL;
  if (j < 0 || j >= c->p.k) return fail(c, CB_EINVAL, "replica index out of range");
  return copy_out(c, c->G() + (int64_t)j * c->p.Pp, out_host, n, c->p.P);
}

int cb_get_loss(cb_ctx* c, float* out_host) {
  if (!c) return CB_EINVAL;
  const Plan& p = c->p;
  // with the fused head, the FC's bias-gradient kernel wrote each replica's
  // mean of its per-image terms
  const int64_t off = p.loss_per_image ? p.off_loss_mean : p.off_loss;
  return copy_out(c, c->at<float>(off), out_host, p.k, p.k);
}

int cb_abi_version(void) { return CB_ABI_VERSION; }

}  // extern "C"

namespace {

// The update of Algorithm 1 (correct = 1) or a local step (correct = 0)
// with caller gradients [k][P].
int apply_grads(cb_ctx* c, const float* grads_dev, int correct) {
  int rc = enter(c);
  if (rc) return rc;
  if (!grads_dev) return fail(c, CB_EINVAL, "grads is NULL");
  const Plan& p = c->p;
  const bool aligned = p.P % 4 == 0 && reinterpret_cast<uintptr_t>(grads_dev) % 16 == 0;
  if (aligned) {
    rc = enqueue_sma(c, grads_dev, p.P, correct);
  } else {
    CB_HIP(c, hipMemcpy2DAsync(c->G(), (size_t)p.Pp * 4, grads_dev, (size_t)p.P * 4,
                               (size_t)p.P * 4, p.k, hipMemcpyDeviceToDevice, c->stream));
    rc = enqueue_sma(c, c->G(), p.Pp, correct);
  }
  if (rc) return rc;
  c->pending = false;
  if (correct && p.m.check_finite) return check_finite(c);
  return CB_OK;
}

}  // namespace

extern "C" {

int cb_sma_apply(cb_ctx* c, const float* grads_dev) { return apply_grads(c, grads_dev, 1); }

int cb_local_apply(cb_ctx* c, const float* grads_dev) { return apply_grads(c, grads_dev, 0); }

int cb_set_state(cb_ctx* c, const float* W_host, const float* z_host, const float* zprev_host) {
  int rc = enter(c);
  if (rc) return rc;
  if (!W_host || !z_host || !zprev_host) return fail(c, CB_EINVAL, "state pointer is NULL");
  const Plan& p = c->p;
  const size_t pb = (size_t)p.P * 4;
  CB_HIP(c, hipMemcpy2DAsync(c->W(), (size_t)p.Pp * 4, W_host, pb, pb, p.k,
                             hipMemcpyHostToDevice, c->stream));
  if (c->Wprev())
    CB_HIP(c, hipMemcpy2DAsync(c->Wprev(), (size_t)p.Pp * 4, W_host, pb, pb, p.k,
                               hipMemcpyHostToDevice, c->stream));
  CB_HIP(c, hipMemcpyAsync(c->Z(), z_host, pb, hipMemcpyHostToDevice, c->stream));
  CB_HIP(c, hipMemcpyAsync(c->Zp(), zprev_host, pb, hipMemcpyHostToDevice, c->stream));
  CB_HIP(c, hipStreamSynchronize(c->stream));
  c->pending = false;
  return CB_OK;
}

int cb_set_lr(cb_ctx* c, float lr) {
  int rc = enter(c);
  if (rc) return rc;
  if (!std::isfinite(lr)) return fail(c, CB_EINVAL, "lr must be finite");
  c->lr = lr;
  return CB_OK;
}

int cb_restart(cb_ctx* c) {
  int rc = enter(c);
  if (rc) return rc;
  const Plan& p = c->p;
  const size_t pb = (size_t)p.P * 4;
  for (int j = 0; j < p.k; ++j) {
    CB_HIP(c, hipMemcpyAsync(c->W() + (int64_t)j * p.Pp, c->Z(), pb, hipMemcpyDeviceToDevice,
                             c->stream));
    if (c->Wprev())
      CB_HIP(c, hipMemcpyAsync(c->Wprev() + (int64_t)j * p.Pp, c->Z(), pb,
                               hipMemcpyDeviceToDevice, c->stream));
  }
  CB_HIP(c, hipMemcpyAsync(c->Zp(), c->Z(), pb, hipMemcpyDeviceToDevice, c->stream));
  c->pending = false;
  return CB_OK;
}

int cb_set_learners(cb_ctx* c, int k, float alpha) {
  int rc = enter(c);
  if (rc) return rc;
  if (c->pending) return fail(c, CB_ESTATE, "cb_set_learners: a gradient is pending (sync first)");
  if (k < 1 || k > c->p.kcap)
    return fail(c, CB_EINVAL, "k must be between 1 and the capacity given to cb_create");
  if (!std::isfinite(alpha)) return fail(c, CB_EINVAL, "alpha must be finite");
  Plan np;
  if (!make_plan(&c->p.m, k, c->p.b, np, c->p.kcap) || (size_t)np.total > c->ws_bytes ||
      np.off_W != c->p.off_W || np.off_Z != c->p.off_Z)
    return fail(c, CB_EINVAL, "cb_set_learners: no plan for this k in the workspace");
  // new learners start from the latest central model, with zero velocity
  const size_t pb = (size_t)c->p.P * 4;
  for (int j = c->p.k; j < k; ++j) {
    CB_HIP(c, hipMemcpyAsync(c->W() + (int64_t)j * c->p.Pp, c->Z(), pb,
                             hipMemcpyDeviceToDevice, c->stream));
    if (c->Wprev())
      CB_HIP(c, hipMemcpyAsync(c->Wprev() + (int64_t)j * c->p.Pp, c->Z(), pb,
                               hipMemcpyDeviceToDevice, c->stream));
  }
  c->drop_graphs();  // captured with the old plan
  c->p = std::move(np);
  c->alpha = alpha;
  build_split_tables(c);
  return CB_OK;
}

int cb_learners(const cb_ctx* c) { return c ? c->p.k : CB_EINVAL; }

int cb_tuner_next(int l, double t, double t_prev, double threshold, int l_max) {
  if (t - t_prev > threshold) return l < l_max ? l + 1 : l;
  if (t < t_prev && l > 1) return l - 1;
  return l;
}

int cb_set_graphs(cb_ctx* c, int on) {
  int rc = enter(c);
  if (rc) return rc;
  c->graphs = on != 0;
  if (!c->graphs) c->drop_graphs();
  return CB_OK;
}

int cb_profile_enable(cb_ctx* c, int on) {
  int rc = enter(c);
  if (rc) return rc;
  c->prof = on != 0;
  return CB_OK;
}

int cb_profile_collect(cb_ctx* c) {
  int rc = enter(c);
  if (rc) return rc;
  CB_HIP(c, hipStreamSynchronize(c->stream));
  for (const ProfRec& r : c->recs) {
    float ms = 0.f;
    CB_HIP(c, hipEventElapsedTime(&ms, r.a, r.b));
    ProfAgg* g = nullptr;
    for (auto& x : c->agg)
      if (x.name == r.name) g = &x;
    if (!g) {
      c->agg.push_back(ProfAgg());
      g = &c->agg.back();
      g->name = r.name;
    }
    g->launches += 1;
    g->ms += ms;
    g->flops += r.flops;
    g->bytes += r.bytes;
    c->evpool.push_back(r.a);
    c->evpool.push_back(r.b);
  }
  c->recs.clear();
  return (int)c->agg.size();
}

int cb_profile_entry(cb_ctx* c, int i, const char** name, int64_t* launches, double* ms,
                     double* flops, double* bytes) {
  if (!c || i < 0 || i >= (int)c->agg.size()) return CB_EINVAL;
  const ProfAgg& g = c->agg[i];
  *name = g.name.c_str();
  *launches = g.launches;
  *ms = g.ms;
  *flops = g.flops;
  *bytes = g.bytes;
  return CB_OK;
}

int cb_profile_clear(cb_ctx* c) {
  if (!c) return CB_EINVAL;
  c->agg.clear();
  return CB_OK;
}

const char* cb_last_error(const cb_ctx* c) {
  return c ? c->err.c_str() : g_create_error.c_str();
}

void cb_destroy(cb_ctx* c) { delete c; }

}  // extern "C"
