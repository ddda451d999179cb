/*
 * cbref.c -- CPU oracle for one SMA iteration of k learners (Crossbow,
 * Koliousis et al., VLDB 2019, arXiv 1901.02244).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, single-threaded
 * reference that the HIP path is checked against.  Only the tests, the smoke
 * check and the CPU-baseline leg of the benchmark may load it.  It shares no
 * code, header, table or constant with the GPU library: its network
 * descriptions, parameter layout, layer math and SMA update are all written
 * out here again from the paper.
 *
 * Precision: every tensor is held in double.  Inputs and the initial model
 * arrive as fp32 and are widened exactly.  The one place where floating
 * point decides an integer -- which cell of a max-pool window wins -- is
 * decided on the fp32-rounded values, the precision the GPU kernels store.
 *
 * What is computed (each function below cites its passage):
 *   - mini-batch gradient of the mean loss over a learner's batch
 *     (Sec. 2.1, Eq. 1 and Eq. 2), by back-propagation (Sec. 2.1);
 *   - Algorithm 1 (Sec. 3.2): per learner j a gradient g_j = lr * grad,
 *     a correction c_j = alpha (w_j - z), the replica update
 *     w_j <- w_j - g_j - c_j; then z <- z + sum_j c_j + mu (z - z_prev) and
 *     z_prev <- the z from before that update;
 *   - the three networks of Table 1 that the workloads use (LeNet,
 *     ResNet-32, ResNet-50).
 *
 * Readings where the paper is silent (the same list is kept with the design
 * notes of the repository):
 *   - z_prev starts equal to w0 (zero initial velocity); the algorithm leaves
 *     it empty.  Every replica starts equal to w0.
 *   - g_j and c_j are both taken at the replica's value from before the
 *     update, as the algorithm writes them.
 *   - gradients are stored raw; the learning rate is applied in the update.
 *   - optional learner momentum mu_L (default 0, i.e. Algorithm 1 as
 *     printed): w_j <- w_j - g_j - c_j + mu_L (w_j - w_j_prev), the heavy-ball
 *     form of Eq. 3 applied to each replica.
 *   - a step whose gradient was never synchronised is applied as a local
 *     update without correction (sync interval larger than one) before the
 *     next gradient is taken.
 *   - loss: softmax cross-entropy averaged over the learner's b images
 *     (Eq. 2).  Weight decay 0.
 *   - batch norm uses batch statistics per learner over its own images
 *     (learners are independent), eps = 1e-5, biased variance; gamma and beta
 *     are parameters and are averaged like any other.
 *   - LeNet: conv5x5x6 pad 2, ReLU, max 2x2/2, conv5x5x16 pad 0, ReLU,
 *     max 2x2/2, FC 400-120 ReLU, FC 120-84 ReLU, FC 84-10; biases on every
 *     conv and FC.
 *   - ResNet-32: conv3x3x16-BN-ReLU, 3 stages x 5 basic blocks (16/32/64),
 *     stride 2 in the first block of stages 2 and 3, shortcut option A: the
 *     block input subsampled by 2 fills the first Cin channels, the rest are
 *     zero; ReLU after the add; global average pool; FC with bias; no conv
 *     bias.
 *   - ResNet-50: v1 bottlenecks [3,4,6,3], widths 64..512, stride on the
 *     first 1x1 conv of a stage, projection shortcut (1x1 conv + BN) in the
 *     first block of each stage; 7x7/2 pad 3 stem, max 3x3/2 pad 1; global
 *     average pool; FC with bias; no conv bias.
 *   - max-pool: padded cells never win; the first maximum in row-major window
 *     order wins (strict greater-than).  ReLU'(0) = 0.
 *   - parameter order: layers in forward order; conv weight
 *     [Cout][Cin][R][S] then its bias; BN gamma then beta; FC weight
 *     [out][in] then bias.  In a ResNet-50 block the projection shortcut
 *     comes after the main path.
 */
#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define CBREF_ARCH_LENET5 1
#define CBREF_ARCH_RESNET32 2
#define CBREF_ARCH_RESNET50 3

#define KIND_CONV_W 0
#define KIND_BIAS 1
#define KIND_BN_GAMMA 2
#define KIND_BN_BETA 3
#define KIND_FC_W 4

#define BN_EPS 1e-5
#define MAX_TENSORS 256

typedef struct {
  int32_t arch, in_c, in_h, in_w, num_classes;
} cbref_model;

/* ------------------------------------------------------------------ */
/* Parameter layout                                                    */
/* ------------------------------------------------------------------ */

typedef struct {
  int64_t offset, numel;
  int kind, ndim, dims[4];
} TensorInfo;

typedef struct {
  int ci, co, r, s, st, pad, has_bias;
  int64_t w_off, b_off;
} Conv;

typedef struct {
  int c;
  int64_t g_off, b_off;
} BN;

typedef struct {
  int in, out;
  int64_t w_off, b_off;
} FC;

typedef struct {
  Conv a, b;
  BN ba, bb;
  int cin, cout, st;
} Basic; /* ResNet-32 block */

typedef struct {
  Conv c1, c2, c3, proj;
  BN b1, b2, b3, bproj;
  int has_proj, st;
} Bottle; /* ResNet-50 block */

typedef struct {
  cbref_model m;
  int ntensors;
  TensorInfo t[MAX_TENSORS];
  int64_t nparams;
  /* LeNet */
  Conv l_c1, l_c2;
  FC l_f1, l_f2, l_f3;
  /* ResNets */
  Conv stem;
  BN stem_bn;
  int nblocks;
  Basic basic[15];
  Bottle bottle[16];
  FC fc;
} Net;

static void add_tensor(Net* n, int kind, int ndim, int d0, int d1, int d2, int d3,
                       int64_t* off) {
  TensorInfo* t = &n->t[n->ntensors++];
  int dims[4] = {d0, d1, d2, d3};
  t->kind = kind;
  t->ndim = ndim;
  t->numel = 1;
  for (int i = 0; i < 4; ++i) {
    t->dims[i] = i < ndim ? dims[i] : 1;
    if (i < ndim) t->numel *= dims[i];
  }
  t->offset = n->nparams;
  *off = n->nparams;
  n->nparams += t->numel;
}

static Conv make_conv(Net* n, int ci, int co, int r, int st, int pad, int has_bias) {
  Conv c;
  c.ci = ci; c.co = co; c.r = r; c.s = r; c.st = st; c.pad = pad; c.has_bias = has_bias;
  add_tensor(n, KIND_CONV_W, 4, co, ci, r, r, &c.w_off);
  c.b_off = -1;
  if (has_bias) add_tensor(n, KIND_BIAS, 1, co, 1, 1, 1, &c.b_off);
  return c;
}

static BN make_bn(Net* n, int c) {
  BN b;
  b.c = c;
  add_tensor(n, KIND_BN_GAMMA, 1, c, 1, 1, 1, &b.g_off);
  add_tensor(n, KIND_BN_BETA, 1, c, 1, 1, 1, &b.b_off);
  return b;
}

static FC make_fc(Net* n, int in, int out) {
  FC f;
  f.in = in; f.out = out;
  add_tensor(n, KIND_FC_W, 2, out, in, 1, 1, &f.w_off);
  add_tensor(n, KIND_BIAS, 1, out, 1, 1, 1, &f.b_off);
  return f;
}

/* Returns 0 on success, -1 if the model description is not supported. */
static int build_net(const cbref_model* m, Net* n) {
  memset(n, 0, sizeof(*n));
  n->m = *m;
  if (m->in_c < 1 || m->num_classes < 1) return -1;
  if (m->arch == CBREF_ARCH_LENET5) {
    /* conv pad 2 keeps H; pool halves; conv 5x5 pad 0 takes 4; pool halves */
    if (m->in_h % 4 || m->in_w % 4 || m->in_h < 12 || m->in_w < 12) return -1;
    int h2 = m->in_h / 2 - 4, w2 = m->in_w / 2 - 4;
    if (h2 % 2 || w2 % 2) return -1;
    n->l_c1 = make_conv(n, m->in_c, 6, 5, 1, 2, 1);
    n->l_c2 = make_conv(n, 6, 16, 5, 1, 0, 1);
    n->l_f1 = make_fc(n, 16 * (h2 / 2) * (w2 / 2), 120);
    n->l_f2 = make_fc(n, 120, 84);
    n->l_f3 = make_fc(n, 84, m->num_classes);
    return 0;
  }
  if (m->arch == CBREF_ARCH_RESNET32) {
    if (m->in_h % 4 || m->in_w % 4 || m->in_h < 4 || m->in_w < 4) return -1;
    n->stem = make_conv(n, m->in_c, 16, 3, 1, 1, 0);
    n->stem_bn = make_bn(n, 16);
    int cin = 16, nb = 0;
    for (int stage = 0; stage < 3; ++stage) {
      int cout = 16 << stage;
      for (int i = 0; i < 5; ++i) {
        Basic* b = &n->basic[nb++];
        b->cin = cin; b->cout = cout; b->st = (stage > 0 && i == 0) ? 2 : 1;
        b->a = make_conv(n, cin, cout, 3, b->st, 1, 0);
        b->ba = make_bn(n, cout);
        b->b = make_conv(n, cout, cout, 3, 1, 1, 0);
        b->bb = make_bn(n, cout);
        cin = cout;
      }
    }
    n->nblocks = nb;
    n->fc = make_fc(n, 64, m->num_classes);
    return 0;
  }
  if (m->arch == CBREF_ARCH_RESNET50) {
    if (m->in_h % 32 || m->in_w % 32 || m->in_h < 32 || m->in_w < 32) return -1;
    n->stem = make_conv(n, m->in_c, 64, 7, 2, 3, 0);
    n->stem_bn = make_bn(n, 64);
    static const int depth[4] = {3, 4, 6, 3};
    int cin = 64, nb = 0;
    for (int stage = 0; stage < 4; ++stage) {
      int w = 64 << stage, cout = 4 * w;
      for (int i = 0; i < depth[stage]; ++i) {
        Bottle* b = &n->bottle[nb++];
        b->st = (stage > 0 && i == 0) ? 2 : 1;
        b->has_proj = (i == 0);
        b->c1 = make_conv(n, cin, w, 1, b->st, 0, 0);
        b->b1 = make_bn(n, w);
        b->c2 = make_conv(n, w, w, 3, 1, 1, 0);
        b->b2 = make_bn(n, w);
        b->c3 = make_conv(n, w, cout, 1, 1, 0, 0);
        b->b3 = make_bn(n, cout);
        if (b->has_proj) {
          b->proj = make_conv(n, cin, cout, 1, b->st, 0, 0);
          b->bproj = make_bn(n, cout);
        }
        cin = cout;
      }
    }
    n->nblocks = nb;
    n->fc = make_fc(n, 2048, m->num_classes);
    return 0;
  }
  return -1;
}

/* ------------------------------------------------------------------ */
/* Layer math (Sec. 2.1: forward pass, loss, backward pass)            */
/* ------------------------------------------------------------------ */

/* Decision margin: the smallest distance, relative to the layer's RMS, of
 * any value on which a ReLU or a max-pool decision turns.  A decision whose
 * margin is within rounding can go either way in another precision; the
 * tests use this to know which inputs make every decision unambiguous.
 * Each computation is single-threaded; the running minimum (like all the
 * bookkeeping below) belongs to the calling thread, reset by the API, so
 * independent calls may run on different threads. */
static _Thread_local double g_margin = INFINITY;

static void note_margin(double m) {
  if (m < g_margin) g_margin = m;
}

/* Decisions of one forward pass.  Every ReLU and every max pool is a
 * "site", numbered in forward order from 0.  A ReLU decision is element
 * idx of the site's tensor (kept iff its input is positive); a max-pool
 * decision is output idx of the site (the cell that wins its window).
 * When a decision's value lies within rounding of the point where it
 * turns, the other outcome is also a correct result at that precision.
 * The API can list such decisions (relative margin below delta, with the
 * runner-up cell as the alternative outcome for a max pool) and can compute
 * the gradient with chosen decisions taken the other way.  A flipped ReLU
 * outputs 0, or the magnitude of its input, instead of its usual output (a
 * change within the margin), so that later decisions see the flip; a
 * flipped max pool keeps its forward value (the two cells differ by less
 * than the margin) and routes the gradient to the alternative cell. */
#define MAX_SITES 256

typedef struct {
  int nsites;
  const void* site_key[MAX_SITES]; /* ReLU: its output tensor; max pool: its winners */
  /* listing (delta > 0) */
  double delta;
  int cap, count;
  int* d_site;
  int64_t *d_idx, *d_alt;
  double* d_rel;
  /* decisions taken the other way */
  int nflip;
  const int* f_site;
  const int64_t *f_idx, *f_alt;
} Decisions;

static _Thread_local Decisions g_dec;

static int new_site(const void* key) {
  if (g_dec.nsites >= MAX_SITES) return -1;
  g_dec.site_key[g_dec.nsites] = key;
  return g_dec.nsites++;
}

static int find_site(const void* key) {
  for (int s = g_dec.nsites - 1; s >= 0; --s)
    if (g_dec.site_key[s] == key) return s;
  return -1;
}

static void note_decision(int site, int64_t idx, int64_t alt, double rel) {
  if (site < 0 || !(rel < g_dec.delta)) return;
  if (g_dec.count < g_dec.cap) {
    g_dec.d_site[g_dec.count] = site;
    g_dec.d_idx[g_dec.count] = idx;
    g_dec.d_alt[g_dec.count] = alt;
    g_dec.d_rel[g_dec.count] = rel;
  }
  g_dec.count++;
}

/* Batch-norm conditioning: the largest, over channels, of
 * sqrt(var + mean^2) / sqrt(var + eps), the factor by which a relative
 * error in the norm's input grows in its output.  Over very few values a
 * channel can have a spread far below its mean, and then fp32 inputs carry
 * little of the normalised output's precision. */
static _Thread_local double g_bn_cond = 0.0;

static double* dalloc(size_t n) {
  double* p = (double*)calloc(n ? n : 1, sizeof(double));
  if (!p) abort();
  return p;
}

static int out_dim(int in, int r, int st, int pad) { return (in + 2 * pad - r) / st + 1; }

/* The outputs o in [0, n_out) whose input cell o*st - pad + r lies inside
 * [0, n_in): returned as the half-open range [*lo, *hi).  The loops below
 * visit exactly the (output, tap) pairs the definition sums over. */
static void valid_range(int n_out, int n_in, int st, int pad, int r, int* lo, int* hi) {
  int a = 0, b = n_out;
  while (a < b && a * st - pad + r < 0) ++a;
  while (b > a && (b - 1) * st - pad + r >= n_in) --b;
  *lo = a;
  *hi = b;
}

/* Convolution, the definition: y[n][co][oh][ow] = bias[co] +
 * sum over (ci, r, s) of x[n][ci][oh*st-pad+r][ow*st-pad+s] * w[co][ci][r][s],
 * out-of-range input cells contributing nothing.  The loops are arranged so
 * that the innermost one runs over independent outputs; every output still
 * adds its terms in (ci, r, s) order. */
#define MAX_TAPS 16

/* Valid output ranges for every tap index r < R of one spatial axis. */
static void tap_ranges(int n_out, int n_in, int st, int pad, int R, int* lo, int* hi) {
  for (int r = 0; r < R; ++r) valid_range(n_out, n_in, st, pad, r, &lo[r], &hi[r]);
}

static void conv_fwd(const Conv* c, const double* w, const double* x, int N, int H, int W,
                     double* y, int Ho, int Wo) {
  const double* wt = w + c->w_off;
  int rlo[MAX_TAPS], rhi[MAX_TAPS], slo[MAX_TAPS], shi[MAX_TAPS];
  tap_ranges(Ho, H, c->st, c->pad, c->r, rlo, rhi);
  tap_ranges(Wo, W, c->st, c->pad, c->s, slo, shi);
  for (int n = 0; n < N; ++n)
    for (int co = 0; co < c->co; ++co) {
      double* yp = y + ((size_t)n * c->co + co) * Ho * Wo;
      double b0 = c->has_bias ? w[c->b_off + co] : 0.0;
      for (int i = 0; i < Ho * Wo; ++i) yp[i] = b0;
      for (int ci = 0; ci < c->ci; ++ci) {
        const double* xp = x + ((size_t)n * c->ci + ci) * H * W;
        for (int r = 0; r < c->r; ++r)
          for (int s = 0; s < c->s; ++s) {
            double wv = wt[(((size_t)co * c->ci + ci) * c->r + r) * c->s + s];
            int oh0 = rlo[r], oh1 = rhi[r], ow0 = slo[s], ow1 = shi[s];
            for (int oh = oh0; oh < oh1; ++oh) {
              const double* xr = xp + (oh * c->st - c->pad + r) * W - c->pad + s;
              double* yr = yp + oh * Wo;
              for (int ow = ow0; ow < ow1; ++ow) yr[ow] += xr[ow * c->st] * wv;
            }
          }
      }
    }
}

/* Gradients of conv_fwd.  dw and db are accumulated over the batch
 * (caller zeroes them); dx (if not NULL) is overwritten. */
static void conv_bwd(const Conv* c, const double* w, const double* x, int N, int H, int W,
                     const double* dy, int Ho, int Wo, double* dx, double* g) {
  const double* wt = w + c->w_off;
  int rlo[MAX_TAPS], rhi[MAX_TAPS], slo[MAX_TAPS], shi[MAX_TAPS];
  tap_ranges(Ho, H, c->st, c->pad, c->r, rlo, rhi);
  tap_ranges(Wo, W, c->st, c->pad, c->s, slo, shi);
  double* dw = g + c->w_off;
  if (c->has_bias) {
    double* db = g + c->b_off;
    for (int co = 0; co < c->co; ++co) {
      double acc = 0.0;
      for (int n = 0; n < N; ++n) {
        const double* dp = dy + ((size_t)n * c->co + co) * Ho * Wo;
        for (int i = 0; i < Ho * Wo; ++i) acc += dp[i];
      }
      db[co] += acc;
    }
  }
  /* dW[co][ci][r][s] = sum over (n, oh, ow) of dy[n][co][oh][ow] * x[n][ci][ih][iw] */
  for (int co = 0; co < c->co; ++co)
    for (int ci = 0; ci < c->ci; ++ci)
      for (int r = 0; r < c->r; ++r)
        for (int s = 0; s < c->s; ++s) {
          double acc = 0.0;
          int oh0 = rlo[r], oh1 = rhi[r], ow0 = slo[s], ow1 = shi[s];
          for (int n = 0; n < N; ++n) {
            const double* dp = dy + ((size_t)n * c->co + co) * Ho * Wo;
            const double* xp = x + ((size_t)n * c->ci + ci) * H * W;
            for (int oh = oh0; oh < oh1; ++oh) {
              const double* xr = xp + (oh * c->st - c->pad + r) * W - c->pad + s;
              const double* dr = dp + oh * Wo;
              for (int ow = ow0; ow < ow1; ++ow) acc += dr[ow] * xr[ow * c->st];
            }
          }
          dw[(((size_t)co * c->ci + ci) * c->r + r) * c->s + s] += acc;
        }
  if (!dx) return;
  /* dX[n][ci][ih][iw] = sum over (co, r, s) with ih = oh*st-pad+r, iw = ... of
   * dy[n][co][oh][ow] * w[co][ci][r][s]; written as a scatter over (oh, ow). */
  memset(dx, 0, sizeof(double) * (size_t)N * c->ci * H * W);
  for (int n = 0; n < N; ++n)
    for (int ci = 0; ci < c->ci; ++ci) {
      double* xp = dx + ((size_t)n * c->ci + ci) * H * W;
      for (int co = 0; co < c->co; ++co) {
        const double* dp = dy + ((size_t)n * c->co + co) * Ho * Wo;
        for (int r = 0; r < c->r; ++r)
          for (int s = 0; s < c->s; ++s) {
            double wv = wt[(((size_t)co * c->ci + ci) * c->r + r) * c->s + s];
            int oh0 = rlo[r], oh1 = rhi[r], ow0 = slo[s], ow1 = shi[s];
            for (int oh = oh0; oh < oh1; ++oh) {
              double* xr = xp + (oh * c->st - c->pad + r) * W - c->pad + s;
              const double* dr = dp + oh * Wo;
              for (int ow = ow0; ow < ow1; ++ow) xr[ow * c->st] += dr[ow] * wv;
            }
          }
      }
    }
}

/* Fully connected: y[n][o] = b[o] + sum_i W[o][i] x[n][i]. */
static void fc_fwd(const FC* f, const double* w, const double* x, int N, double* y) {
  for (int n = 0; n < N; ++n)
    for (int o = 0; o < f->out; ++o) {
      double acc = w[f->b_off + o];
      for (int i = 0; i < f->in; ++i) acc += w[f->w_off + (size_t)o * f->in + i] * x[(size_t)n * f->in + i];
      y[(size_t)n * f->out + o] = acc;
    }
}

static void fc_bwd(const FC* f, const double* w, const double* x, int N, const double* dy,
                   double* dx, double* g) {
  for (int o = 0; o < f->out; ++o) {
    double acc = 0.0;
    for (int n = 0; n < N; ++n) acc += dy[(size_t)n * f->out + o];
    g[f->b_off + o] += acc;
    for (int i = 0; i < f->in; ++i) {
      double a = 0.0;
      for (int n = 0; n < N; ++n) a += dy[(size_t)n * f->out + o] * x[(size_t)n * f->in + i];
      g[f->w_off + (size_t)o * f->in + i] += a;
    }
  }
  if (!dx) return;
  for (int n = 0; n < N; ++n)
    for (int i = 0; i < f->in; ++i) {
      double a = 0.0;
      for (int o = 0; o < f->out; ++o) a += dy[(size_t)n * f->out + o] * w[f->w_off + (size_t)o * f->in + i];
      dx[(size_t)n * f->in + i] = a;
    }
}

/* Batch norm with the statistics of this batch: per channel c,
 * mean = E[x], var = E[(x - mean)^2] over (n, h, w),
 * y = gamma (x - mean) / sqrt(var + eps) + beta. */
static void bn_fwd(const BN* b, const double* w, const double* x, int N, int HW, double* y,
                   double* mean, double* istd) {
  const double cnt = (double)N * HW;
  for (int c = 0; c < b->c; ++c) {
    double s = 0.0;
    for (int n = 0; n < N; ++n) {
      const double* p = x + ((size_t)n * b->c + c) * HW;
      for (int i = 0; i < HW; ++i) s += p[i];
    }
    double mu = s / cnt, v = 0.0;
    for (int n = 0; n < N; ++n) {
      const double* p = x + ((size_t)n * b->c + c) * HW;
      for (int i = 0; i < HW; ++i) v += (p[i] - mu) * (p[i] - mu);
    }
    v /= cnt;
    double is = 1.0 / sqrt(v + BN_EPS);
    double cond = sqrt(v + mu * mu) * is;
    if (cond > g_bn_cond) g_bn_cond = cond;
    double ga = w[b->g_off + c], be = w[b->b_off + c];
    for (int n = 0; n < N; ++n) {
      const double* p = x + ((size_t)n * b->c + c) * HW;
      double* q = y + ((size_t)n * b->c + c) * HW;
      for (int i = 0; i < HW; ++i) q[i] = ga * (p[i] - mu) * is + be;
    }
    mean[c] = mu;
    istd[c] = is;
  }
}

/* Derivative of bn_fwd, batch statistics included:
 * dbeta = sum dy, dgamma = sum dy*xhat,
 * dx = gamma*istd*(dy - dbeta/m - xhat*dgamma/m). */
static void bn_bwd(const BN* b, const double* w, const double* x, int N, int HW,
                   const double* mean, const double* istd, const double* dy, double* dx,
                   double* g) {
  const double cnt = (double)N * HW;
  for (int c = 0; c < b->c; ++c) {
    double sdy = 0.0, sdyx = 0.0;
    for (int n = 0; n < N; ++n) {
      const double* p = x + ((size_t)n * b->c + c) * HW;
      const double* d = dy + ((size_t)n * b->c + c) * HW;
      for (int i = 0; i < HW; ++i) {
        sdy += d[i];
        sdyx += d[i] * (p[i] - mean[c]) * istd[c];
      }
    }
    g[b->g_off + c] += sdyx;
    g[b->b_off + c] += sdy;
    double k = w[b->g_off + c] * istd[c];
    for (int n = 0; n < N; ++n) {
      const double* p = x + ((size_t)n * b->c + c) * HW;
      const double* d = dy + ((size_t)n * b->c + c) * HW;
      double* q = dx + ((size_t)n * b->c + c) * HW;
      for (int i = 0; i < HW; ++i) {
        double xh = (p[i] - mean[c]) * istd[c];
        q[i] = k * (d[i] - sdy / cnt - xh * sdyx / cnt);
      }
    }
  }
}



/* In place: y <- max(y, 0).  A decision listed to be taken the other way
 * outputs 0 where the input is positive, and the input's magnitude (a
 * positive value within the margin of 0) where it is not, so that the
 * decisions downstream see it -- a max pool over ReLU outputs then lets
 * that cell win a window of zeros, as the other precision does. */
static void relu_inplace(double* y, size_t n) {
  const int site = new_site(y);
  double ss = 0.0, mn = INFINITY;
  for (size_t i = 0; i < n; ++i) {
    ss += y[i] * y[i];
    if (fabs(y[i]) < mn) mn = fabs(y[i]);
  }
  if (n && ss > 0.0) {
    const double rms = sqrt(ss / n);
    note_margin(mn / rms);
    if (g_dec.delta > 0.0)
      for (size_t i = 0; i < n; ++i) note_decision(site, (int64_t)i, -1, fabs(y[i]) / rms);
  }
  double* flipped = NULL;
  if (site >= 0 && g_dec.nflip) {
    flipped = dalloc((size_t)g_dec.nflip);
    for (int f = 0; f < g_dec.nflip; ++f)
      if (g_dec.f_site[f] == site && g_dec.f_idx[f] >= 0 && (size_t)g_dec.f_idx[f] < n) {
        const double v = y[g_dec.f_idx[f]];
        flipped[f] = v > 0.0 ? 0.0 : (-v > 0.0 ? -v : DBL_MIN);
      }
  }
  for (size_t i = 0; i < n; ++i)
    if (!(y[i] > 0.0)) y[i] = 0.0;
  if (flipped) {
    for (int f = 0; f < g_dec.nflip; ++f)
      if (g_dec.f_site[f] == site && g_dec.f_idx[f] >= 0 && (size_t)g_dec.f_idx[f] < n)
        y[g_dec.f_idx[f]] = flipped[f];
    free(flipped);
  }
}

/* dy <- dy where the layer's output was positive, else 0 (ReLU'(0) = 0). */
static void relu_mask(double* dy, const double* out, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!(out[i] > 0.0)) dy[i] = 0.0;
}

/* Max pool K x K, stride st, padding pad.  The winner of a window is the
 * first cell, in row-major order, whose fp32-rounded value is strictly
 * greater than every earlier one; padded cells never win. */
static void maxpool_fwd(const double* x, int N, int C, int H, int W, int K, int st, int pad,
                        double* y, int Ho, int Wo, int* arg) {
  const int site = new_site(arg);
  double ss = 0.0, gap = INFINITY;
  for (size_t i = 0; i < (size_t)N * C * H * W; ++i) ss += x[i] * x[i];
  const double rms = ss > 0.0 ? sqrt(ss / ((double)N * C * H * W)) : 0.0;
  for (size_t nc = 0; nc < (size_t)N * C; ++nc)
    for (int oh = 0; oh < Ho; ++oh)
      for (int ow = 0; ow < Wo; ++ow) {
        int best = -1;
        float bv = 0.0f;
        for (int r = 0; r < K; ++r)
          for (int s = 0; s < K; ++s) {
            int ih = oh * st - pad + r, iw = ow * st - pad + s;
            if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
            float v = (float)x[nc * H * W + ih * W + iw];
            if (best < 0 || v > bv) {
              best = ih * W + iw;
              bv = v;
            }
          }
        y[nc * Ho * Wo + oh * Wo + ow] = x[nc * H * W + best];
        arg[nc * Ho * Wo + oh * Wo + ow] = best;
        /* margin: gap to the runner-up, when the winner is positive (a
         * non-positive winner's gradient is cut by the ReLU before it) */
        if (bv > 0.0f)
          for (int r = 0; r < K; ++r)
            for (int s = 0; s < K; ++s) {
              int ih = oh * st - pad + r, iw = ow * st - pad + s;
              if (ih < 0 || ih >= H || iw < 0 || iw >= W || ih * W + iw == best) continue;
              double d = x[nc * H * W + best] - x[nc * H * W + ih * W + iw];
              if (d < gap) gap = d;
              if (g_dec.delta > 0.0 && rms > 0.0)
                note_decision(site, (int64_t)(nc * Ho * Wo + oh * Wo + ow), ih * W + iw,
                              d / rms);
            }
      }
  size_t n = (size_t)N * C * H * W;
  if (n && ss > 0.0 && gap < INFINITY) note_margin(gap / sqrt(ss / n));
  /* windows whose winner is to be taken the other way: the gradient goes
   * to the alternative cell, the forward value stays */
  if (site >= 0)
    for (int f = 0; f < g_dec.nflip; ++f)
      if (g_dec.f_site[f] == site && g_dec.f_idx[f] >= 0 &&
          g_dec.f_idx[f] < (int64_t)N * C * Ho * Wo && g_dec.f_alt[f] >= 0 &&
          g_dec.f_alt[f] < (int64_t)H * W)
        arg[g_dec.f_idx[f]] = (int)g_dec.f_alt[f];
}

static void maxpool_bwd(const double* dy, const int* arg, int N, int C, int H, int W, int Ho,
                        int Wo, double* dx) {
  memset(dx, 0, sizeof(double) * (size_t)N * C * H * W);
  for (size_t nc = 0; nc < (size_t)N * C; ++nc)
    for (int i = 0; i < Ho * Wo; ++i) dx[nc * H * W + arg[nc * Ho * Wo + i]] += dy[nc * Ho * Wo + i];
}

/* Global average pool over H x W. */
static void gap_fwd(const double* x, int N, int C, int HW, double* y) {
  for (size_t nc = 0; nc < (size_t)N * C; ++nc) {
    double s = 0.0;
    for (int i = 0; i < HW; ++i) s += x[nc * HW + i];
    y[nc] = s / HW;
  }
}

static void gap_bwd(const double* dy, int N, int C, int HW, double* dx) {
  for (size_t nc = 0; nc < (size_t)N * C; ++nc)
    for (int i = 0; i < HW; ++i) dx[nc * HW + i] = dy[nc] / HW;
}

/* Mean softmax cross-entropy over the N images of the batch (Eq. 2 with
 * the per-sample loss -log softmax(o)_y), and its gradient
 * (softmax(o) - onehot(y)) / N with respect to the logits. */
static double xent(const double* o, const int32_t* y, int N, int C, double* d) {
  double tot = 0.0;
  for (int n = 0; n < N; ++n) {
    const double* p = o + (size_t)n * C;
    double mx = p[0];
    for (int c = 1; c < C; ++c)
      if (p[c] > mx) mx = p[c];
    double se = 0.0;
    for (int c = 0; c < C; ++c) se += exp(p[c] - mx);
    double lse = mx + log(se);
    tot += lse - p[y[n]];
    for (int c = 0; c < C; ++c) d[(size_t)n * C + c] = (exp(p[c] - lse) - (c == y[n] ? 1.0 : 0.0)) / N;
  }
  return tot / N;
}

/* ------------------------------------------------------------------ */
/* Networks: loss and gradient for one learner's batch                 */
/* ------------------------------------------------------------------ */

/* LeNet (Table 1).  Returns the mean loss; g (if not NULL) receives the
 * gradient, overwritten. */
static double lenet_grad(const Net* net, const double* w, const double* x, const int32_t* y,
                         int N, double* g) {
  const cbref_model* m = &net->m;
  int H = m->in_h, W = m->in_w;
  int H1 = H, W1 = W, H1p = H1 / 2, W1p = W1 / 2;
  int H2 = H1p - 4, W2 = W1p - 4, H2p = H2 / 2, W2p = W2 / 2;
  double* a1 = dalloc((size_t)N * 6 * H1 * W1);
  double* p1 = dalloc((size_t)N * 6 * H1p * W1p);
  int* g1 = (int*)calloc((size_t)N * 6 * H1p * W1p, sizeof(int));
  double* a2 = dalloc((size_t)N * 16 * H2 * W2);
  double* p2 = dalloc((size_t)N * 16 * H2p * W2p);
  int* g2 = (int*)calloc((size_t)N * 16 * H2p * W2p, sizeof(int));
  double* f1 = dalloc((size_t)N * 120);
  double* f2 = dalloc((size_t)N * 84);
  double* o = dalloc((size_t)N * m->num_classes);
  double* d_o = dalloc((size_t)N * m->num_classes);

  conv_fwd(&net->l_c1, w, x, N, H, W, a1, H1, W1);
  relu_inplace(a1, (size_t)N * 6 * H1 * W1);
  maxpool_fwd(a1, N, 6, H1, W1, 2, 2, 0, p1, H1p, W1p, g1);
  conv_fwd(&net->l_c2, w, p1, N, H1p, W1p, a2, H2, W2);
  relu_inplace(a2, (size_t)N * 16 * H2 * W2);
  maxpool_fwd(a2, N, 16, H2, W2, 2, 2, 0, p2, H2p, W2p, g2);
  fc_fwd(&net->l_f1, w, p2, N, f1);
  relu_inplace(f1, (size_t)N * 120);
  fc_fwd(&net->l_f2, w, f1, N, f2);
  relu_inplace(f2, (size_t)N * 84);
  fc_fwd(&net->l_f3, w, f2, N, o);
  double loss = xent(o, y, N, m->num_classes, d_o);

  if (g) {
    memset(g, 0, sizeof(double) * net->nparams);
    double* d_f2 = dalloc((size_t)N * 84);
    double* d_f1 = dalloc((size_t)N * 120);
    double* d_p2 = dalloc((size_t)N * 16 * H2p * W2p);
    double* d_a2 = dalloc((size_t)N * 16 * H2 * W2);
    double* d_p1 = dalloc((size_t)N * 6 * H1p * W1p);
    double* d_a1 = dalloc((size_t)N * 6 * H1 * W1);
    fc_bwd(&net->l_f3, w, f2, N, d_o, d_f2, g);
    relu_mask(d_f2, f2, (size_t)N * 84);
    fc_bwd(&net->l_f2, w, f1, N, d_f2, d_f1, g);
    relu_mask(d_f1, f1, (size_t)N * 120);
    fc_bwd(&net->l_f1, w, p2, N, d_f1, d_p2, g);
    maxpool_bwd(d_p2, g2, N, 16, H2, W2, H2p, W2p, d_a2);
    relu_mask(d_a2, a2, (size_t)N * 16 * H2 * W2);
    conv_bwd(&net->l_c2, w, p1, N, H1p, W1p, d_a2, H2, W2, d_p1, g);
    maxpool_bwd(d_p1, g1, N, 6, H1, W1, H1p, W1p, d_a1);
    relu_mask(d_a1, a1, (size_t)N * 6 * H1 * W1);
    conv_bwd(&net->l_c1, w, x, N, H, W, d_a1, H1, W1, NULL, g);
    free(d_f2); free(d_f1); free(d_p2); free(d_a2); free(d_p1); free(d_a1);
  }
  free(a1); free(p1); free(g1); free(a2); free(p2); free(g2);
  free(f1); free(f2); free(o); free(d_o);
  return loss;
}

/* One conv followed by batch norm, with the tensors the backward pass
 * needs: the conv output (pre-norm) and the per-channel statistics. */
typedef struct {
  int C, H, W;
  double *conv, *out, *mean, *istd;
} CBState;

static void cb_fwd(const Conv* c, const BN* b, const double* w, const double* x, int N, int H,
                   int W, CBState* st, int relu) {
  st->C = c->co;
  st->H = out_dim(H, c->r, c->st, c->pad);
  st->W = out_dim(W, c->s, c->st, c->pad);
  size_t n = (size_t)N * st->C * st->H * st->W;
  st->conv = dalloc(n);
  st->out = dalloc(n);
  st->mean = dalloc(st->C);
  st->istd = dalloc(st->C);
  conv_fwd(c, w, x, N, H, W, st->conv, st->H, st->W);
  bn_fwd(b, w, st->conv, N, st->H * st->W, st->out, st->mean, st->istd);
  if (relu) relu_inplace(st->out, n);
}

static void cb_free(CBState* st) {
  free(st->conv); free(st->out); free(st->mean); free(st->istd);
  memset(st, 0, sizeof(*st));
}

/* Backward through batch norm and the conv.  dout is the gradient at the
 * norm's output (already masked by the ReLU if there is one); it is only
 * read.  dx (if not NULL) receives the gradient at the conv input. */
static void cb_bwd(const Conv* c, const BN* b, const double* w, const double* x, int N, int H,
                   int W, CBState* st, double* dout, double* dx, double* g) {
  size_t n = (size_t)N * st->C * st->H * st->W;
  double* dconv = dalloc(n);
  bn_bwd(b, w, st->conv, N, st->H * st->W, st->mean, st->istd, dout, dconv, g);
  conv_bwd(c, w, x, N, H, W, dconv, st->H, st->W, dx, g);
  free(dconv);
}

/* ResNet-32 for CIFAR-sized inputs (Table 1; basic blocks, option-A
 * shortcut as described at the top of this file). */
static double resnet32_grad(const Net* net, const double* w, const double* x, const int32_t* y,
                            int N, double* g) {
  const cbref_model* m = &net->m;
  CBState stem;
  cb_fwd(&net->stem, &net->stem_bn, w, x, N, m->in_h, m->in_w, &stem, 1);
  CBState sa[15], sb[15];
  double* outs[15];
  const double* cur = stem.out;
  int H = stem.H, W = stem.W;
  for (int i = 0; i < 15; ++i) {
    const Basic* bl = &net->basic[i];
    cb_fwd(&bl->a, &bl->ba, w, cur, N, H, W, &sa[i], 1);
    cb_fwd(&bl->b, &bl->bb, w, sa[i].out, N, sa[i].H, sa[i].W, &sb[i], 0);
    int Ho = sb[i].H, Wo = sb[i].W;
    double* o = dalloc((size_t)N * bl->cout * Ho * Wo);
    for (int n = 0; n < N; ++n)
      for (int c = 0; c < bl->cout; ++c)
        for (int h = 0; h < Ho; ++h)
          for (int ww = 0; ww < Wo; ++ww) {
            double sc = 0.0;
            if (c < bl->cin)
              sc = cur[(((size_t)n * bl->cin + c) * H + h * bl->st) * W + ww * bl->st];
            size_t idx = (((size_t)n * bl->cout + c) * Ho + h) * Wo + ww;
            o[idx] = sb[i].out[idx] + sc;
          }
    relu_inplace(o, (size_t)N * bl->cout * Ho * Wo);
    outs[i] = o;
    cur = o;
    H = Ho; W = Wo;
  }
  double* pooled = dalloc((size_t)N * 64);
  gap_fwd(cur, N, 64, H * W, pooled);
  double* o = dalloc((size_t)N * m->num_classes);
  double* d_o = dalloc((size_t)N * m->num_classes);
  fc_fwd(&net->fc, w, pooled, N, o);
  double loss = xent(o, y, N, m->num_classes, d_o);

  if (g) {
    memset(g, 0, sizeof(double) * net->nparams);
    double* d_pool = dalloc((size_t)N * 64);
    fc_bwd(&net->fc, w, pooled, N, d_o, d_pool, g);
    double* dcur = dalloc((size_t)N * 64 * H * W);
    gap_bwd(d_pool, N, 64, H * W, dcur);
    free(d_pool);
    for (int i = 14; i >= 0; --i) {
      const Basic* bl = &net->basic[i];
      const double* in = i ? outs[i - 1] : stem.out;
      int Hi = i ? sb[i - 1].H : stem.H, Wi = i ? sb[i - 1].W : stem.W;
      int Ho = sb[i].H, Wo = sb[i].W;
      size_t nout = (size_t)N * bl->cout * Ho * Wo;
      relu_mask(dcur, outs[i], nout); /* gradient at the pre-activation sum */
      double* dmid = dalloc((size_t)N * bl->cout * sa[i].H * sa[i].W);
      cb_bwd(&bl->b, &bl->bb, w, sa[i].out, N, sa[i].H, sa[i].W, &sb[i], dcur, dmid, g);
      relu_mask(dmid, sa[i].out, (size_t)N * bl->cout * sa[i].H * sa[i].W);
      double* din = dalloc((size_t)N * bl->cin * Hi * Wi);
      cb_bwd(&bl->a, &bl->ba, w, in, N, Hi, Wi, &sa[i], dmid, din, g);
      free(dmid);
      /* shortcut: the subsampled input went to the first cin channels */
      for (int n = 0; n < N; ++n)
        for (int c = 0; c < bl->cin; ++c)
          for (int h = 0; h < Ho; ++h)
            for (int ww = 0; ww < Wo; ++ww)
              din[(((size_t)n * bl->cin + c) * Hi + h * bl->st) * Wi + ww * bl->st] +=
                  dcur[(((size_t)n * bl->cout + c) * Ho + h) * Wo + ww];
      free(dcur);
      dcur = din;
    }
    relu_mask(dcur, stem.out, (size_t)N * 16 * stem.H * stem.W);
    cb_bwd(&net->stem, &net->stem_bn, w, x, N, m->in_h, m->in_w, &stem, dcur, NULL, g);
    free(dcur);
  }
  for (int i = 0; i < 15; ++i) {
    cb_free(&sa[i]); cb_free(&sb[i]); free(outs[i]);
  }
  cb_free(&stem);
  free(pooled); free(o); free(d_o);
  return loss;
}

/* ResNet-50 (Table 1; v1 bottlenecks as described at the top). */
static double resnet50_grad(const Net* net, const double* w, const double* x, const int32_t* y,
                            int N, double* g) {
  const cbref_model* m = &net->m;
  CBState stem;
  cb_fwd(&net->stem, &net->stem_bn, w, x, N, m->in_h, m->in_w, &stem, 1);
  int Hp = out_dim(stem.H, 3, 2, 1), Wp = out_dim(stem.W, 3, 2, 1);
  double* pool = dalloc((size_t)N * 64 * Hp * Wp);
  int* parg = (int*)calloc((size_t)N * 64 * Hp * Wp, sizeof(int));
  maxpool_fwd(stem.out, N, 64, stem.H, stem.W, 3, 2, 1, pool, Hp, Wp, parg);
  int nb = net->nblocks;
  CBState s1[16], s2[16], s3[16], sp[16];
  double* outs[16];
  int Hs[17], Ws[17], Cs[17];
  const double* cur = pool;
  Hs[0] = Hp; Ws[0] = Wp; Cs[0] = 64;
  for (int i = 0; i < nb; ++i) {
    const Bottle* bl = &net->bottle[i];
    cb_fwd(&bl->c1, &bl->b1, w, cur, N, Hs[i], Ws[i], &s1[i], 1);
    cb_fwd(&bl->c2, &bl->b2, w, s1[i].out, N, s1[i].H, s1[i].W, &s2[i], 1);
    cb_fwd(&bl->c3, &bl->b3, w, s2[i].out, N, s2[i].H, s2[i].W, &s3[i], 0);
    size_t n = (size_t)N * s3[i].C * s3[i].H * s3[i].W;
    double* o = dalloc(n);
    if (bl->has_proj) {
      cb_fwd(&bl->proj, &bl->bproj, w, cur, N, Hs[i], Ws[i], &sp[i], 0);
      for (size_t e = 0; e < n; ++e) o[e] = s3[i].out[e] + sp[i].out[e];
    } else {
      memset(&sp[i], 0, sizeof(sp[i]));
      for (size_t e = 0; e < n; ++e) o[e] = s3[i].out[e] + cur[e];
    }
    relu_inplace(o, n);
    outs[i] = o;
    cur = o;
    Hs[i + 1] = s3[i].H; Ws[i + 1] = s3[i].W; Cs[i + 1] = s3[i].C;
  }
  int H = Hs[nb], W = Ws[nb];
  double* pooled = dalloc((size_t)N * 2048);
  gap_fwd(cur, N, 2048, H * W, pooled);
  double* o = dalloc((size_t)N * m->num_classes);
  double* d_o = dalloc((size_t)N * m->num_classes);
  fc_fwd(&net->fc, w, pooled, N, o);
  double loss = xent(o, y, N, m->num_classes, d_o);

  if (g) {
    memset(g, 0, sizeof(double) * net->nparams);
    double* d_pool = dalloc((size_t)N * 2048);
    fc_bwd(&net->fc, w, pooled, N, d_o, d_pool, g);
    double* dcur = dalloc((size_t)N * 2048 * H * W);
    gap_bwd(d_pool, N, 2048, H * W, dcur);
    free(d_pool);
    for (int i = nb - 1; i >= 0; --i) {
      const Bottle* bl = &net->bottle[i];
      const double* in = i ? outs[i - 1] : pool;
      size_t nout = (size_t)N * Cs[i + 1] * Hs[i + 1] * Ws[i + 1];
      size_t nin = (size_t)N * Cs[i] * Hs[i] * Ws[i];
      relu_mask(dcur, outs[i], nout);
      double* din = dalloc(nin);
      /* shortcut branch */
      if (bl->has_proj) {
        cb_bwd(&bl->proj, &bl->bproj, w, in, N, Hs[i], Ws[i], &sp[i], dcur, din, g);
      } else {
        memcpy(din, dcur, sizeof(double) * nin);
      }
      /* main branch, last conv first */
      double* d2 = dalloc((size_t)N * s2[i].C * s2[i].H * s2[i].W);
      cb_bwd(&bl->c3, &bl->b3, w, s2[i].out, N, s2[i].H, s2[i].W, &s3[i], dcur, d2, g);
      relu_mask(d2, s2[i].out, (size_t)N * s2[i].C * s2[i].H * s2[i].W);
      double* d1 = dalloc((size_t)N * s1[i].C * s1[i].H * s1[i].W);
      cb_bwd(&bl->c2, &bl->b2, w, s1[i].out, N, s1[i].H, s1[i].W, &s2[i], d2, d1, g);
      free(d2);
      relu_mask(d1, s1[i].out, (size_t)N * s1[i].C * s1[i].H * s1[i].W);
      double* d0 = dalloc(nin);
      cb_bwd(&bl->c1, &bl->b1, w, in, N, Hs[i], Ws[i], &s1[i], d1, d0, g);
      free(d1);
      for (size_t e = 0; e < nin; ++e) din[e] += d0[e];
      free(d0);
      free(dcur);
      dcur = din;
    }
    double* dstem = dalloc((size_t)N * 64 * stem.H * stem.W);
    maxpool_bwd(dcur, parg, N, 64, stem.H, stem.W, Hp, Wp, dstem);
    free(dcur);
    relu_mask(dstem, stem.out, (size_t)N * 64 * stem.H * stem.W);
    cb_bwd(&net->stem, &net->stem_bn, w, x, N, m->in_h, m->in_w, &stem, dstem, NULL, g);
    free(dstem);
  }
  for (int i = 0; i < nb; ++i) {
    cb_free(&s1[i]); cb_free(&s2[i]); cb_free(&s3[i]);
    if (net->bottle[i].has_proj) cb_free(&sp[i]);
    free(outs[i]);
  }
  cb_free(&stem);
  free(pool); free(parg); free(pooled); free(o); free(d_o);
  return loss;
}

static double net_grad(const Net* net, const double* w, const double* x, const int32_t* y,
                       int N, double* g) {
  g_dec.nsites = 0;
  switch (net->m.arch) {
    case CBREF_ARCH_LENET5: return lenet_grad(net, w, x, y, N, g);
    case CBREF_ARCH_RESNET32: return resnet32_grad(net, w, x, y, N, g);
    default: return resnet50_grad(net, w, x, y, N, g);
  }
}

/* ------------------------------------------------------------------ */
/* Exported: layout and a learner's loss and gradient                  */
/* ------------------------------------------------------------------ */

int64_t cbref_num_params(const cbref_model* m) {
  Net* n = (Net*)malloc(sizeof(Net));
  int64_t p = build_net(m, n) ? -1 : n->nparams;
  free(n);
  return p;
}

int cbref_num_tensors(const cbref_model* m) {
  Net* n = (Net*)malloc(sizeof(Net));
  int t = build_net(m, n) ? -1 : n->ntensors;
  free(n);
  return t;
}

/* Describes parameter tensor idx: offset, kind, rank and dims. */
int cbref_tensor_info(const cbref_model* m, int idx, int64_t* offset, int* kind, int* ndim,
                      int* dims4) {
  Net* n = (Net*)malloc(sizeof(Net));
  int rc = -1;
  if (!build_net(m, n) && idx >= 0 && idx < n->ntensors) {
    *offset = n->t[idx].offset;
    *kind = n->t[idx].kind;
    *ndim = n->t[idx].ndim;
    for (int i = 0; i < 4; ++i) dims4[i] = n->t[idx].dims[i];
    rc = 0;
  }
  free(n);
  return rc;
}

/* Mean loss of one learner's batch of N images (x: N x C x H x W fp32,
 * y: N labels) at parameters w (double), and, if g is not NULL, its
 * gradient (Eq. 2).  Returns 0, or -1 on a bad model or label. */
int cbref_learner_grad(const cbref_model* m, const double* w, const float* x,
                       const int32_t* y, int N, double* g, double* loss) {
  Net* net = (Net*)malloc(sizeof(Net));
  if (build_net(m, net) || N < 1) {
    free(net);
    return -1;
  }
  for (int n = 0; n < N; ++n)
    if (y[n] < 0 || y[n] >= m->num_classes) {
      free(net);
      return -1;
    }
  size_t nx = (size_t)N * m->in_c * m->in_h * m->in_w;
  double* xd = dalloc(nx);
  for (size_t i = 0; i < nx; ++i) xd[i] = x[i];
  *loss = net_grad(net, w, xd, y, N, g);
  free(xd);
  free(net);
  return 0;
}

/* Smallest relative decision margin of the forward pass of one learner's
 * batch (see g_margin) and, if bn_cond is not NULL, its largest batch-norm
 * conditioning factor (see g_bn_cond).  Returns 0, or -1 on a bad model or
 * label. */
int cbref_learner_margin(const cbref_model* m, const double* w, const float* x,
                         const int32_t* y, int N, double* margin, double* bn_cond) {
  double loss;
  g_margin = INFINITY;
  g_bn_cond = 0.0;
  int rc = cbref_learner_grad(m, w, x, y, N, NULL, &loss);
  *margin = g_margin;
  if (bn_cond) *bn_cond = g_bn_cond;
  return rc;
}

/* The decisions of the forward pass of one learner's batch whose relative
 * margin is below delta (see Decisions above): for each, its site, its
 * index, the alternative outcome (the runner-up cell of a max-pool window,
 * -1 for a ReLU) and its relative margin, in the order the forward pass
 * meets them.  At most cap are written; *count receives how many there
 * are.  Returns 0, or -1 on a bad model, label or argument. */
int cbref_learner_decisions(const cbref_model* m, const double* w, const float* x,
                            const int32_t* y, int N, double delta, int cap, int* site,
                            int64_t* idx, int64_t* alt, double* rel, int* count) {
  if (!(delta > 0.0) || cap < 0 || (cap > 0 && (!site || !idx || !alt || !rel))) return -1;
  double loss;
  memset(&g_dec, 0, sizeof(g_dec));
  g_dec.delta = delta;
  g_dec.cap = cap;
  g_dec.d_site = site;
  g_dec.d_idx = idx;
  g_dec.d_alt = alt;
  g_dec.d_rel = rel;
  int rc = cbref_learner_grad(m, w, x, y, N, NULL, &loss);
  *count = g_dec.count;
  memset(&g_dec, 0, sizeof(g_dec));
  return rc;
}

/* Loss and gradient of one learner's batch (as cbref_learner_grad) with
 * the nflip listed decisions taken the other way in the backward pass:
 * site[i], idx[i] and alt[i] as cbref_learner_decisions reports them.
 * Returns 0, or -1 on a bad model or label. */
int cbref_learner_grad_flipped(const cbref_model* m, const double* w, const float* x,
                               const int32_t* y, int N, int nflip, const int* site,
                               const int64_t* idx, const int64_t* alt, double* g,
                               double* loss) {
  if (nflip < 0 || (nflip > 0 && (!site || !idx || !alt))) return -1;
  memset(&g_dec, 0, sizeof(g_dec));
  g_dec.nflip = nflip;
  g_dec.f_site = site;
  g_dec.f_idx = idx;
  g_dec.f_alt = alt;
  int rc = cbref_learner_grad(m, w, x, y, N, g, loss);
  memset(&g_dec, 0, sizeof(g_dec));
  return rc;
}

/* ------------------------------------------------------------------ */
/* Synchronous model averaging (Algorithm 1, Sec. 3.2)                 */
/* ------------------------------------------------------------------ */

typedef struct cbref_ctx {
  Net net;
  int k, b;
  double alpha, lr, mu, mu_l;
  int64_t P;
  double *W, *Wprev, *G, *Z, *Zp, *loss;
  int pending; /* a gradient taken by step() has not been applied */
} cbref_ctx;

/* Initialisation (Algorithm 1, first two assignments): z = w0; z_prev is
 * read as w0; every replica (and its previous value) starts at w0. */
cbref_ctx* cbref_create(const cbref_model* m, const float* w0, int64_t n, int k, int b,
                        double alpha, double lr, double mu, double mu_l) {
  if (k < 1 || b < 1) return NULL;
  cbref_ctx* c = (cbref_ctx*)calloc(1, sizeof(cbref_ctx));
  if (build_net(m, &c->net) || c->net.nparams != n) {
    free(c);
    return NULL;
  }
  c->k = k; c->b = b; c->alpha = alpha; c->lr = lr; c->mu = mu; c->mu_l = mu_l;
  c->P = n;
  c->W = dalloc((size_t)k * n);
  c->Wprev = dalloc((size_t)k * n);
  c->G = dalloc((size_t)k * n);
  c->Z = dalloc(n);
  c->Zp = dalloc(n);
  c->loss = dalloc(k);
  for (int64_t e = 0; e < n; ++e) {
    c->Z[e] = w0[e];
    c->Zp[e] = w0[e];
    for (int j = 0; j < k; ++j) c->W[(size_t)j * n + e] = c->Wprev[(size_t)j * n + e] = w0[e];
  }
  return c;
}

void cbref_destroy(cbref_ctx* c) {
  if (!c) return;
  free(c->W); free(c->Wprev); free(c->G); free(c->Z); free(c->Zp); free(c->loss);
  free(c);
}

/* One synchronisation of Algorithm 1 on n parameters of k replicas held as
 * [k][n] arrays (W, Wprev, G) and [n] arrays (Z, Zp):
 *   c_j = alpha (w_j - z)            from the replica before its update,
 *   w_j <- w_j - lr g_j - c_j + mu_L (w_j - w_j_prev),   w_j_prev <- old w_j,
 *   z <- z + sum_j c_j + mu (z - z_prev),                z_prev <- old z,
 * the sum taken in replica order.  With correct == 0 the correction is left
 * out and z is not touched (a local step of a learner). */
void cbref_sma_update(int k, int64_t n, double* W, double* Wprev, const double* G, double* Z,
                      double* Zp, double alpha, double lr, double mu, double mu_l, int correct) {
  for (int64_t e = 0; e < n; ++e) {
    double s = 0.0;
    for (int j = 0; j < k; ++j) {
      size_t i = (size_t)j * n + e;
      double w = W[i];
      double cj = correct ? alpha * (w - Z[e]) : 0.0;
      double wn = w - lr * G[i] - cj + mu_l * (w - Wprev[i]);
      Wprev[i] = w;
      W[i] = wn;
      s += cj;
    }
    if (correct) {
      double z = Z[e];
      Z[e] = z + s + mu * (z - Zp[e]);
      Zp[e] = z;
    }
  }
}

/* Gradients of all k learners on one iteration's batch; learner j takes
 * images [j*b, (j+1)*b) (the select step of Algorithm 1).  A gradient
 * from an earlier step() that was never synchronised is applied first as
 * a local step. */
int cbref_step(cbref_ctx* c, const float* x, const int32_t* y) {
  if (c->pending)
    cbref_sma_update(c->k, c->P, c->W, c->Wprev, c->G, c->Z, c->Zp, c->alpha, c->lr, c->mu,
                     c->mu_l, 0);
  const cbref_model* m = &c->net.m;
  size_t img = (size_t)m->in_c * m->in_h * m->in_w;
  for (int j = 0; j < c->k; ++j) {
    double l;
    int rc = cbref_learner_grad(m, c->W + (size_t)j * c->P, x + (size_t)j * c->b * img,
                                y + (size_t)j * c->b, c->b, c->G + (size_t)j * c->P, &l);
    if (rc) return rc;
    c->loss[j] = l;
  }
  c->pending = 1;
  return 0;
}

/* The synchronisation of Algorithm 1: corrections from the pre-update
 * replicas, replica updates, then z <- z + sum_j c_j + mu (z - z_prev)
 * and z_prev <- the old z.  Returns -4 if no gradient is pending. */
int cbref_sync(cbref_ctx* c) {
  if (!c->pending) return -4;
  cbref_sma_update(c->k, c->P, c->W, c->Wprev, c->G, c->Z, c->Zp, c->alpha, c->lr, c->mu,
                   c->mu_l, 1);
  c->pending = 0;
  return 0;
}

/* A new learning rate gamma for the following updates (the step-wise
 * schedule of Sec. 3.2: gamma may change between iterations). */
int cbref_set_lr(cbref_ctx* c, double lr) {
  c->lr = lr;
  return 0;
}

/* Restart of SMA (Sec. 3.2): Algorithm 1 starts again with the latest
 * central model as its initial model, so every replica, its previous
 * value and z_prev become z (zero velocity).  A gradient still pending
 * from an unsynchronised step is dropped. */
int cbref_restart(cbref_ctx* c) {
  for (int64_t e = 0; e < c->P; ++e) {
    const double z = c->Z[e];
    c->Zp[e] = z;
    for (int j = 0; j < c->k; ++j) c->W[(size_t)j * c->P + e] = c->Wprev[(size_t)j * c->P + e] = z;
  }
  c->pending = 0;
  return 0;
}

/* Changes the number of learners between iterations (Sec. 3.4 / 4.4): a
 * new learner's replica is initialised with the latest central model z
 * (and so is its previous value); removing learners drops the most recently
 * added ones.  alpha is the correction factor used from now on.  Returns
 * -4 while a gradient is pending, -1 for k < 1. */
int cbref_set_learners(cbref_ctx* c, int k, double alpha) {
  if (k < 1) return -1;
  if (c->pending) return -4;
  const int64_t n = c->P;
  double* W = dalloc((size_t)k * n);
  double* Wprev = dalloc((size_t)k * n);
  double* G = dalloc((size_t)k * n);
  double* loss = dalloc(k);
  for (int j = 0; j < k; ++j)
    for (int64_t e = 0; e < n; ++e) {
      const size_t i = (size_t)j * n + e;
      W[i] = j < c->k ? c->W[i] : c->Z[e];
      Wprev[i] = j < c->k ? c->Wprev[i] : c->Z[e];
    }
  free(c->W); free(c->Wprev); free(c->G); free(c->loss);
  c->W = W; c->Wprev = Wprev; c->G = G; c->loss = loss;
  c->k = k;
  c->alpha = alpha;
  return 0;
}

/* Algorithm 2 (Sec. 3.4), one observation: l learners gave throughput t;
 * t_prev is the throughput observed before.  Returns l + 1 if the increase
 * exceeds the threshold, l - 1 if throughput fell (never below one
 * learner), l otherwise; the caller then keeps t as the next t_prev.
 * l_max bounds the increase (the capacity the caller provisioned). */
int cbref_tuner_next(int l, double t, double t_prev, double threshold, int l_max) {
  if (t - t_prev > threshold) return l < l_max ? l + 1 : l;
  if (t < t_prev && l > 1) return l - 1;
  return l;
}

/* Test hook: take grads [k][P] as the learners' raw gradients, then sync. */
int cbref_sma_apply(cbref_ctx* c, const double* grads) {
  memcpy(c->G, grads, sizeof(double) * (size_t)c->k * c->P);
  c->pending = 1;
  return cbref_sync(c);
}

/* Test hook: overwrite the state.  W and (optionally) Wprev are [k][P]. */
int cbref_set_state(cbref_ctx* c, const double* W, const double* Wprev, const double* Z,
                    const double* Zp) {
  memcpy(c->W, W, sizeof(double) * (size_t)c->k * c->P);
  memcpy(c->Wprev, Wprev ? Wprev : W, sizeof(double) * (size_t)c->k * c->P);
  memcpy(c->Z, Z, sizeof(double) * c->P);
  memcpy(c->Zp, Zp, sizeof(double) * c->P);
  c->pending = 0;
  return 0;
}

int cbref_get_central(const cbref_ctx* c, double* out) {
  memcpy(out, c->Z, sizeof(double) * c->P);
  return 0;
}

int cbref_get_prev_central(const cbref_ctx* c, double* out) {
  memcpy(out, c->Zp, sizeof(double) * c->P);
  return 0;
}

int cbref_get_replica(const cbref_ctx* c, int j, double* out) {
  if (j < 0 || j >= c->k) return -1;
  memcpy(out, c->W + (size_t)j * c->P, sizeof(double) * c->P);
  return 0;
}

int cbref_get_grad(const cbref_ctx* c, int j, double* out) {
  if (j < 0 || j >= c->k) return -1;
  memcpy(out, c->G + (size_t)j * c->P, sizeof(double) * c->P);
  return 0;
}

int cbref_get_loss(const cbref_ctx* c, double* out) {
  memcpy(out, c->loss, sizeof(double) * c->k);
  return 0;
}

/* Layer primitives exposed so that tests can pin each against a library
 * routine.  Shapes follow the structs above; parameters come from w. */
void cbref_conv2d(const double* x, int N, int Ci, int H, int W, const double* wt,
                  const double* bias, int Co, int R, int st, int pad, double* y,
                  double* dy_in, double* dx, double* dw, double* db) {
  if (R < 1 || R > MAX_TAPS) return;
  /* Build a throw-away parameter vector [weight | bias]. */
  Conv c = {Ci, Co, R, R, st, pad, bias != NULL, 0, (int64_t)Co * Ci * R * R};
  size_t nw = (size_t)Co * Ci * R * R;
  double* w = dalloc(nw + Co);
  memcpy(w, wt, sizeof(double) * nw);
  if (bias) memcpy(w + nw, bias, sizeof(double) * Co);
  int Ho = out_dim(H, R, st, pad), Wo = out_dim(W, R, st, pad);
  conv_fwd(&c, w, x, N, H, W, y, Ho, Wo);
  if (dy_in) {
    double* g = dalloc(nw + Co);
    conv_bwd(&c, w, x, N, H, W, dy_in, Ho, Wo, dx, g);
    memcpy(dw, g, sizeof(double) * nw);
    if (bias && db) memcpy(db, g + nw, sizeof(double) * Co);
    free(g);
  }
  free(w);
}

void cbref_batchnorm(const double* x, int N, int C, int HW, const double* gamma,
                     const double* beta, double* y, const double* dy, double* dx,
                     double* dgamma, double* dbeta) {
  BN b = {C, 0, C};
  double* w = dalloc(2 * (size_t)C);
  memcpy(w, gamma, sizeof(double) * C);
  memcpy(w + C, beta, sizeof(double) * C);
  double* mean = dalloc(C);
  double* istd = dalloc(C);
  bn_fwd(&b, w, x, N, HW, y, mean, istd);
  if (dy) {
    double* g = dalloc(2 * (size_t)C);
    bn_bwd(&b, w, x, N, HW, mean, istd, dy, dx, g);
    memcpy(dgamma, g, sizeof(double) * C);
    memcpy(dbeta, g + C, sizeof(double) * C);
    free(g);
  }
  free(w); free(mean); free(istd);
}

void cbref_maxpool(const double* x, int N, int C, int H, int W, int K, int st, int pad,
                   double* y, const double* dy, double* dx) {
  int Ho = out_dim(H, K, st, pad), Wo = out_dim(W, K, st, pad);
  int* arg = (int*)calloc((size_t)N * C * Ho * Wo, sizeof(int));
  maxpool_fwd(x, N, C, H, W, K, st, pad, y, Ho, Wo, arg);
  if (dy) maxpool_bwd(dy, arg, N, C, H, W, Ho, Wo, dx);
  free(arg);
}

/* Sampled elements of a convolution and its gradients, each computed
 * alone from the definition (for checks at sizes where the full tensors
 * are too slow).  Inputs are fp32 as stored; sums run in double.
 *   what 0: y[n][co][oh][ow]  = bias[co] + sum_(ci,r,s) x * w     (q = n,co,oh,ow)
 *   what 1: dW[co][ci][r][s]  = sum_(n,oh,ow) dy * x               (q = co,ci,r,s)
 *   what 2: dX[n][ci][ih][iw] = sum_(co,r,s) dy * w over the taps
 *           with oh*st = ih + pad - r, ow*st = iw + pad - s        (q = n,ci,ih,iw)
 * q holds 4 indices per sample. */
void cbref_conv_samples(int what, const float* x, const float* dy, const float* w,
                        const float* bias, int N, int Ci, int H, int W, int Co, int R, int st,
                        int pad, const int32_t* q, int nsamples, double* out) {
  int Ho = out_dim(H, R, st, pad), Wo = out_dim(W, R, st, pad);
  for (int t = 0; t < nsamples; ++t) {
    const int32_t* e = q + 4 * t;
    double acc = 0.0;
    if (what == 0) {
      int n = e[0], co = e[1], oh = e[2], ow = e[3];
      acc = bias ? bias[co] : 0.0;
      for (int ci = 0; ci < Ci; ++ci)
        for (int r = 0; r < R; ++r)
          for (int s = 0; s < R; ++s) {
            int ih = oh * st - pad + r, iw = ow * st - pad + s;
            if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
            acc += (double)x[(((size_t)n * Ci + ci) * H + ih) * W + iw] *
                   (double)w[(((size_t)co * Ci + ci) * R + r) * R + s];
          }
    } else if (what == 1) {
      int co = e[0], ci = e[1], r = e[2], s = e[3];
      for (int n = 0; n < N; ++n)
        for (int oh = 0; oh < Ho; ++oh) {
          int ih = oh * st - pad + r;
          if (ih < 0 || ih >= H) continue;
          for (int ow = 0; ow < Wo; ++ow) {
            int iw = ow * st - pad + s;
            if (iw < 0 || iw >= W) continue;
            acc += (double)dy[(((size_t)n * Co + co) * Ho + oh) * Wo + ow] *
                   (double)x[(((size_t)n * Ci + ci) * H + ih) * W + iw];
          }
        }
    } else {
      int n = e[0], ci = e[1], ih = e[2], iw = e[3];
      for (int co = 0; co < Co; ++co)
        for (int r = 0; r < R; ++r)
          for (int s = 0; s < R; ++s) {
            int th = ih + pad - r, tw = iw + pad - s;
            if (th < 0 || tw < 0 || th % st || tw % st) continue;
            int oh = th / st, ow = tw / st;
            if (oh >= Ho || ow >= Wo) continue;
            acc += (double)dy[(((size_t)n * Co + co) * Ho + oh) * Wo + ow] *
                   (double)w[(((size_t)co * Ci + ci) * R + r) * R + s];
          }
    }
    out[t] = acc;
  }
}

double cbref_softmax_xent(const double* logits, const int32_t* y, int N, int C, double* dlogits) {
  double* d = dalloc((size_t)N * C);
  double l = xent(logits, y, N, C, d);
  if (dlogits) memcpy(dlogits, d, sizeof(double) * (size_t)N * C);
  free(d);
  return l;
}
