/*
 * oracle_sanitize.c -- drives every exported function of the CPU oracle
 * (oracle/cbref.c) at tiny sizes, for a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer (test_oracle_sanitizers.py compiles and runs
 * it).  It checks no values: the point is that no call reads or writes out
 * of bounds, leaks, or hits undefined behaviour.  Inputs come from a fixed
 * linear congruential sequence.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef struct {
  int32_t arch, in_c, in_h, in_w, num_classes;
} cbref_model;
typedef struct cbref_ctx cbref_ctx;

int64_t cbref_num_params(const cbref_model* m);
int cbref_num_tensors(const cbref_model* m);
int cbref_tensor_info(const cbref_model* m, int idx, int64_t* offset, int* kind, int* ndim,
                      int* dims4);
int cbref_learner_grad(const cbref_model* m, const double* w, const float* x, const int32_t* y,
                       int N, double* g, double* loss);
int cbref_learner_margin(const cbref_model* m, const double* w, const float* x,
                         const int32_t* y, int N, double* margin, double* bn_cond);
int cbref_learner_decisions(const cbref_model* m, const double* w, const float* x,
                            const int32_t* y, int N, double delta, int cap, int* site,
                            int64_t* idx, int64_t* alt, double* rel, int* count);
int cbref_learner_grad_flipped(const cbref_model* m, const double* w, const float* x,
                               const int32_t* y, int N, int nflip, const int* site,
                               const int64_t* idx, const int64_t* alt, double* g, double* loss);
cbref_ctx* cbref_create(const cbref_model* m, const float* w0, int64_t n, int k, int b,
                        double alpha, double lr, double mu, double mu_l);
void cbref_destroy(cbref_ctx* c);
void cbref_sma_update(int k, int64_t n, double* W, double* Wprev, const double* G, double* Z,
                      double* Zp, double alpha, double lr, double mu, double mu_l, int correct);
int cbref_step(cbref_ctx* c, const float* x, const int32_t* y);
int cbref_sync(cbref_ctx* c);
int cbref_set_lr(cbref_ctx* c, double lr);
int cbref_restart(cbref_ctx* c);
int cbref_set_learners(cbref_ctx* c, int k, double alpha);
int cbref_tuner_next(int l, double t, double t_prev, double threshold, int l_max);
int cbref_sma_apply(cbref_ctx* c, const double* grads);
int cbref_set_state(cbref_ctx* c, const double* W, const double* Wprev, const double* Z,
                    const double* Zp);
int cbref_get_central(const cbref_ctx* c, double* out);
int cbref_get_prev_central(const cbref_ctx* c, double* out);
int cbref_get_replica(const cbref_ctx* c, int j, double* out);
int cbref_get_grad(const cbref_ctx* c, int j, double* out);
int cbref_get_loss(const cbref_ctx* c, double* out);
void cbref_conv2d(const double* x, int N, int Ci, int H, int W, const double* wt,
                  const double* bias, int Co, int R, int st, int pad, double* y, double* dy_in,
                  double* dx, double* dw, double* db);
void cbref_batchnorm(const double* x, int N, int C, int HW, const double* gamma,
                     const double* beta, double* y, const double* dy, double* dx,
                     double* dgamma, double* dbeta);
void cbref_maxpool(const double* x, int N, int C, int H, int W, int K, int st, int pad,
                   double* y, const double* dy, double* dx);
void cbref_conv_samples(int what, const float* x, const float* dy, const float* w,
                        const float* bias, int N, int Ci, int H, int W, int Co, int R, int st,
                        int pad, const int32_t* q, int nsamples, double* out);
double cbref_softmax_xent(const double* logits, const int32_t* y, int N, int C, double* dlogits);

static uint64_t lcg = 88172645463325252ull;
static double rnd(void) { /* uniform in [-1, 1) */
  lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
  return (double)(lcg >> 11) / 4503599627370496.0 - 1.0;
}
static double* dvec(size_t n, double s) {
  double* p = malloc(sizeof(double) * (n ? n : 1));
  for (size_t i = 0; i < n; ++i) p[i] = s * rnd();
  return p;
}
static float* fvec(size_t n, double s) {
  float* p = malloc(sizeof(float) * (n ? n : 1));
  for (size_t i = 0; i < n; ++i) p[i] = (float)(s * rnd());
  return p;
}
static int32_t* labels(int n, int classes) {
  int32_t* p = malloc(sizeof(int32_t) * n);
  for (int i = 0; i < n; ++i) p[i] = (int32_t)((rnd() + 1.0) * 0.5 * classes) % classes;
  return p;
}

#define CHECK(cond)                                                    \
  do {                                                                 \
    if (!(cond)) {                                                     \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      return 1;                                                        \
    }                                                                  \
  } while (0)

static int one_net(cbref_model m, int b, int with_job) {
  const int64_t P = cbref_num_params(&m);
  CHECK(P > 0);
  const int nt = cbref_num_tensors(&m);
  for (int i = 0; i < nt; ++i) {
    int64_t off;
    int kind, nd, dims[4];
    CHECK(cbref_tensor_info(&m, i, &off, &kind, &nd, dims) == 0);
  }
  int64_t off;
  int kind, nd, dims[4];
  CHECK(cbref_tensor_info(&m, nt, &off, &kind, &nd, dims) != 0);
  const size_t img = (size_t)m.in_c * m.in_h * m.in_w;
  double* w = dvec((size_t)P, 0.3);
  float* x = fvec(img * b, 1.0);
  int32_t* y = labels(b, m.num_classes);
  double* g = malloc(sizeof(double) * P);
  double loss, margin, cond;
  CHECK(cbref_learner_grad(&m, w, x, y, b, g, &loss) == 0 && isfinite(loss));
  CHECK(cbref_learner_margin(&m, w, x, y, b, &margin, &cond) == 0);
  int site[64], count = 0;
  int64_t idx[64], alt[64];
  double rel[64];
  CHECK(cbref_learner_decisions(&m, w, x, y, b, 0.05, 64, site, idx, alt, rel, &count) == 0);
  const int n = count < 64 ? count : 64;
  CHECK(cbref_learner_grad_flipped(&m, w, x, y, b, n, site, idx, alt, g, &loss) == 0);
  if (!with_job) {
    free(w); free(x); free(y); free(g);
    return 0;
  }
  /* an SMA job of 3 learners: steps, an unsynchronised step, resizing,
   * restart, a learning-rate change, caller gradients and state */
  float* w0 = fvec((size_t)P, 0.3);
  float* xs = fvec(img * 3 * b, 1.0);
  int32_t* ys = labels(3 * b, m.num_classes);
  cbref_ctx* c = cbref_create(&m, w0, P, 3, b, 1.0 / 3, 0.01, 0.9, 0.5);
  CHECK(c);
  CHECK(cbref_sync(c) != 0);
  CHECK(cbref_step(c, xs, ys) == 0 && cbref_sync(c) == 0);
  CHECK(cbref_step(c, xs, ys) == 0 && cbref_step(c, xs, ys) == 0 && cbref_sync(c) == 0);
  CHECK(cbref_set_learners(c, 2, 0.5) == 0);
  CHECK(cbref_step(c, xs, ys) == 0 && cbref_sync(c) == 0);
  CHECK(cbref_set_learners(c, 3, 1.0 / 3) == 0);
  CHECK(cbref_set_learners(c, 0, 1.0) != 0);
  CHECK(cbref_restart(c) == 0 && cbref_set_lr(c, 0.02) == 0);
  double* G = dvec((size_t)3 * P, 0.1);
  CHECK(cbref_sma_apply(c, G) == 0);
  double* W = dvec((size_t)3 * P, 0.3);
  double* Z = dvec((size_t)P, 0.3);
  CHECK(cbref_set_state(c, W, NULL, Z, Z) == 0);
  double* out = malloc(sizeof(double) * P);
  double lossv[3];
  CHECK(cbref_get_central(c, out) == 0 && cbref_get_prev_central(c, out) == 0);
  CHECK(cbref_get_replica(c, 2, out) == 0 && cbref_get_grad(c, 2, out) == 0);
  CHECK(cbref_get_replica(c, 3, out) != 0);
  CHECK(cbref_get_loss(c, lossv) == 0);
  cbref_destroy(c);
  free(w); free(x); free(y); free(g); free(w0); free(xs); free(ys); free(G); free(W); free(Z);
  free(out);
  return 0;
}

int main(void) {
  cbref_model lenet = {1, 1, 28, 28, 10}, r32 = {2, 3, 8, 8, 10}, r50 = {3, 3, 32, 32, 12};
  if (one_net(lenet, 2, 1) || one_net(r32, 2, 1) || one_net(r50, 2, 0)) return 1;
  cbref_model bad = {9, 1, 28, 28, 10};
  CHECK(cbref_num_params(&bad) < 0);
  /* layer primitives and the update on their own */
  {
    const int N = 2, Ci = 3, H = 7, Co = 5, R = 3;
    double *x = dvec(N * Ci * H * H, 1), *wt = dvec(Co * Ci * R * R, 1), *bias = dvec(Co, 1);
    const int Ho = (H + 2 - R) / 2 + 1;
    double *y = dvec(N * Co * Ho * Ho, 0), *dy = dvec(N * Co * Ho * Ho, 1);
    double *dx = dvec(N * Ci * H * H, 0), *dw = dvec(Co * Ci * R * R, 0), *db = dvec(Co, 0);
    cbref_conv2d(x, N, Ci, H, H, wt, bias, Co, R, 2, 1, y, dy, dx, dw, db);
    float *xf = fvec(N * Ci * H * H, 1), *wf = fvec(Co * Ci * R * R, 1), *dyf = fvec(N * Co * Ho * Ho, 1);
    int32_t q[8] = {0, 1, 2, 2, 1, 2, 0, 1}; /* valid for every `what` */
    double s[2];
    for (int what = 0; what < 3; ++what)
      cbref_conv_samples(what, xf, dyf, wf, NULL, N, Ci, H, H, Co, R, 2, 1, q, 2, s);
    double *g = dvec(Ci, 1), *be = dvec(Ci, 1), *yb = dvec(N * Ci * H * H, 0), *dyb = dvec(N * Ci * H * H, 1);
    double *dxb = dvec(N * Ci * H * H, 0), *dg = dvec(Ci, 0), *dbe = dvec(Ci, 0);
    cbref_batchnorm(x, N, Ci, H * H, g, be, yb, dyb, dxb, dg, dbe);
    const int Hp = (H + 2 - 3) / 2 + 1;
    double *yp = dvec(N * Ci * Hp * Hp, 0), *dyp = dvec(N * Ci * Hp * Hp, 1), *dxp = dvec(N * Ci * H * H, 0);
    cbref_maxpool(x, N, Ci, H, H, 3, 2, 1, yp, dyp, dxp);
    double *lo = dvec(4 * 6, 3), *dl = dvec(4 * 6, 0);
    int32_t yy[4] = {0, 5, 2, 3};
    CHECK(isfinite(cbref_softmax_xent(lo, yy, 4, 6, dl)));
    double *Wu = dvec(3 * 9, 1), *Wp = dvec(3 * 9, 1), *Gu = dvec(3 * 9, 1), *Zu = dvec(9, 1), *Zpu = dvec(9, 1);
    cbref_sma_update(3, 9, Wu, Wp, Gu, Zu, Zpu, 0.3, 0.1, 0.9, 0.5, 1);
    cbref_sma_update(3, 9, Wu, Wp, Gu, Zu, Zpu, 0.3, 0.1, 0.9, 0.5, 0);
    CHECK(cbref_tuner_next(3, 10.0, 5.0, 1.0, 8) == 4 && cbref_tuner_next(1, 1.0, 5.0, 1.0, 8) == 1);
    free(x); free(wt); free(bias); free(y); free(dy); free(dx); free(dw); free(db); free(xf);
    free(wf); free(dyf); free(g); free(be); free(yb); free(dyb); free(dxb); free(dg); free(dbe);
    free(yp); free(dyp); free(dxp); free(lo); free(dl); free(Wu); free(Wp); free(Gu); free(Zu);
    free(Zpu);
  }
  puts("oracle ran clean under the sanitizers");
  return 0;
}
