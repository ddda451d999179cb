// layers.hip -- the memory-bound layers of a learner's forward and backward
// pass (Sec. 2.1), batched over all k learners of the GPU.
//
// Batch norm uses each learner's own batch statistics (learners are
// independent, Sec. 3.1).  Every reduction runs in a fixed order (per-thread
// partial, wave butterfly, then the four waves in order; partials across
// blocks are combined in block order), so results are bitwise reproducible.
// Statistics are accumulated in fp64.
#include "kernels.hpp"

#include <algorithm>

namespace cbk {
namespace {

constexpr double BN_EPS = 1e-5;

inline unsigned cdiv(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }
inline bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_sum_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Sum of two doubles over a 256-thread block, fixed order; result in all threads.
__device__ __forceinline__ void block_sum2(double& a, double& b, double* red) {
  a = wave_sum_d(a);
  b = wave_sum_d(b);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
    red[w] = a;
    red[4 + w] = b;
  }
  __syncthreads();
  a = (red[0] + red[1]) + (red[2] + red[3]);
  b = (red[4] + red[5]) + (red[6] + red[7]);
}

// The elements of (replica j, channel c) are e in [0, b*HW): image e / HW of
// the replica, pixel e % HW.  Block `chunk` owns e in [e0, e1).
struct ChanIter {
  int img, p;
  __device__ ChanIter(int e, int HW) : img(e / HW), p(e - (e / HW) * HW) {}
  __device__ void step(int d, int HW) {
    p += d;
    while (p >= HW) {
      p -= HW;
      ++img;
    }
  }
};

__global__ __launch_bounds__(256) void bn_stats_k(BNArgs a) {
  __shared__ double red[8];
  const int chunk = blockIdx.x, c = blockIdx.y, j = blockIdx.z;
  const int HW = a.H * a.W, n = a.b * HW;
  const int per = (n + a.chunks - 1) / a.chunks;
  const int e0 = chunk * per, e1 = min(n, e0 + per);
  double s = 0.0, ss = 0.0;
  const float* X = a.x + ((int64_t)j * a.b * a.C + c) * HW;
  ChanIter it(e0 + threadIdx.x, HW);
  for (int e = e0 + threadIdx.x; e < e1; e += 256, it.step(256, HW)) {
    const double v = X[(int64_t)it.img * a.C * HW + it.p];
    s += v;
    ss += v * v;
  }
  block_sum2(s, ss, red);
  if (threadIdx.x == 0) {
    double* p = a.part + (((int64_t)j * a.C + c) * a.chunks + chunk) * 2;
    p[0] = s;
    p[1] = ss;
  }
}

__global__ __launch_bounds__(256) void bn_apply_k(BNArgs a) {
  __shared__ double red[8];
  const int chunk = blockIdx.x, c = blockIdx.y, j = blockIdx.z;
  const int HW = a.H * a.W, n = a.b * HW;
  const int per = (n + a.chunks - 1) / a.chunks;
  const int e0 = chunk * per, e1 = min(n, e0 + per);
  // the partial sums of this (replica, channel), combined in a fixed order
  const double* p = a.part + ((int64_t)j * a.C + c) * a.parts * 2;
  double s = 0.0, ss = 0.0;
  for (int i = threadIdx.x; i < a.parts; i += 256) {
    s += p[2 * i];
    ss += p[2 * i + 1];
  }
  block_sum2(s, ss, red);
  const double mean = s / n;
  const double var = fmax(ss / n - mean * mean, 0.0);
  const float mf = (float)mean, isf = (float)(1.0 / sqrt(var + BN_EPS));
  if (chunk == 0 && threadIdx.x == 0) {
    a.mean[j * a.C + c] = mf;
    a.istd[j * a.C + c] = isf;
  }
  const float* gam = a.gamma + (int64_t)j * a.pstride;
  const float ga = gam[c], be = gam[a.C + c];
  const int64_t base = ((int64_t)j * a.b * a.C + c) * HW;
  const float* X = a.x + base;
  float* Y = a.y + base;
  ChanIter it(e0 + threadIdx.x, HW);
  for (int e = e0 + threadIdx.x; e < e1; e += 256, it.step(256, HW)) {
    const int64_t off = (int64_t)it.img * a.C * HW + it.p;
    float v = bn_affine(X[off], mf, isf, ga, be);
    if (a.res_mode == RES_SAME) {
      v += a.res[base + off];
    } else if (a.res_mode == RES_SUBSAMPLE) {
      if (c < a.res_C) {
        const int oh = it.p / a.W, ow = it.p - oh * a.W;
        const int img = j * a.b + it.img;
        v += a.res[(((int64_t)img * a.res_C + c) * a.res_H + oh * a.res_st) * a.res_W +
                   ow * a.res_st];
      }
    }
    if (a.relu) v = v > 0.f ? v : 0.f;
    Y[off] = v;
  }
}

__global__ __launch_bounds__(256) void bn_bwd_stats_k(BNBwdArgs a) {
  __shared__ double red[8];
  const int chunk = blockIdx.x, c = blockIdx.y, j = blockIdx.z;
  const int HW = a.H * a.W, n = a.b * HW;
  const int per = (n + a.chunks - 1) / a.chunks;
  const int e0 = chunk * per, e1 = min(n, e0 + per);
  const float mf = a.mean[j * a.C + c], isf = a.istd[j * a.C + c];
  const float ga = a.gamma[(int64_t)j * a.pstride + c];
  const float be = a.gamma[(int64_t)j * a.pstride + a.C + c];
  const int64_t base = ((int64_t)j * a.b * a.C + c) * HW;
  double s = 0.0, sx = 0.0;
  ChanIter it(e0 + threadIdx.x, HW);
  for (int e = e0 + threadIdx.x; e < e1; e += 256, it.step(256, HW)) {
    const int64_t off = base + (int64_t)it.img * a.C * HW + it.p;
    float d = a.dy[off];
    if (a.y && !(a.y[off] > 0.f)) d = 0.f;
    if (!a.y && a.relu_x && !(bn_affine(a.x[off], mf, isf, ga, be) > 0.f)) d = 0.f;
    const float xh = (a.x[off] - mf) * isf;
    s += d;
    sx += (double)d * xh;
  }
  block_sum2(s, sx, red);
  if (threadIdx.x == 0) {
    double* p = a.part + (((int64_t)j * a.C + c) * a.chunks + chunk) * 2;
    p[0] = s;
    p[1] = sx;
  }
}

__global__ __launch_bounds__(256) void bn_bwd_apply_k(BNBwdArgs a) {
  __shared__ double red[8];
  const int chunk = blockIdx.x, c = blockIdx.y, j = blockIdx.z;
  const int HW = a.H * a.W, n = a.b * HW;
  const int per = (n + a.chunks - 1) / a.chunks;
  const int e0 = chunk * per, e1 = min(n, e0 + per);
  const double* p = a.part + ((int64_t)j * a.C + c) * a.parts * 2;
  double s = 0.0, sx = 0.0;
  for (int i = threadIdx.x; i < a.parts; i += 256) {
    s += p[2 * i];
    sx += p[2 * i + 1];
  }
  block_sum2(s, sx, red);
  const float mf = a.mean[j * a.C + c], isf = a.istd[j * a.C + c];
  const float ga = a.gamma[(int64_t)j * a.pstride + c];
  const float be = a.gamma[(int64_t)j * a.pstride + a.C + c];
  if (chunk == 0 && threadIdx.x == 0) {
    a.dgamma[(int64_t)j * a.pstride + c] = (float)sx;
    a.dgamma[(int64_t)j * a.pstride + a.C + c] = (float)s;
  }
  const float k1 = ga * isf, mdy = (float)(s / n), mdyx = (float)(sx / n);
  const int64_t base = ((int64_t)j * a.b * a.C + c) * HW;
  ChanIter it(e0 + threadIdx.x, HW);
  for (int e = e0 + threadIdx.x; e < e1; e += 256, it.step(256, HW)) {
    const int64_t off = base + (int64_t)it.img * a.C * HW + it.p;
    float d = a.dy[off];
    if (a.y && !(a.y[off] > 0.f)) d = 0.f;
    if (!a.y && a.relu_x && !(bn_affine(a.x[off], mf, isf, ga, be) > 0.f)) d = 0.f;
    const float xh = (a.x[off] - mf) * isf;
    a.dx[off] = k1 * (d - mdy - xh * mdyx);
    if (a.dres) a.dres[off] = d;
  }
}

// Vector forms of the two apply kernels, for planes of a multiple of 4
// pixels with 16-byte aligned tensors: each thread moves float4s, U of them
// per round, and the first round's loads are issued before the block sums
// the partials, so the two latencies overlap.  Same arithmetic per element
// as the scalar forms.
typedef float v4f __attribute__((ext_vector_type(4)));
constexpr int BN_U = 4;

struct Quad {
  int off;   // element offset of the quad from the (replica, channel) base
  int p;     // pixel of its first element
  int img;   // image within the replica
  bool ok;
};

// Quad q of a (replica, channel): image q / HW4, pixel 4 (q % HW4).  Planes
// whose quad count is a power of two (sh >= 0) divide by shifting.
__device__ __forceinline__ Quad quad_at(int q, int q1, int HW4, int sh, int CHW) {
  Quad r;
  r.ok = q < q1;
  const int qq = r.ok ? q : 0;
  if (sh >= 0) {
    r.img = qq >> sh;
    r.p = (qq & (HW4 - 1)) * 4;
  } else {
    r.img = qq / HW4;
    r.p = (qq - r.img * HW4) * 4;
  }
  r.off = r.img * CHW + r.p;
  return r;
}

__device__ __forceinline__ int pow2_shift(int n) { return (n & (n - 1)) == 0 ? __builtin_ctz(n) : -1; }

__global__ __launch_bounds__(256) void bn_apply_v4_k(BNArgs a) {
  __shared__ double red[8];
  const int chunk = blockIdx.x, c = blockIdx.y, j = blockIdx.z;
  const int HW = a.H * a.W, HW4 = HW >> 2, n4 = a.b * HW4, CHW = a.C * HW;
  const int sh = pow2_shift(HW4);
  const int per = (n4 + a.chunks - 1) / a.chunks;
  const int q0 = chunk * per, q1 = min(n4, q0 + per);
  const int64_t base = ((int64_t)j * a.b * a.C + c) * HW;
  const float* X = a.x + base;
  float* Y = a.y + base;
  Quad qd[BN_U];
  v4f xv[BN_U], rv[BN_U];
  int qb = q0 + threadIdx.x;
  auto load = [&]() {
#pragma unroll
    for (int u = 0; u < BN_U; ++u) {
      qd[u] = quad_at(qb + u * 256, q1, HW4, sh, CHW);
      if (qd[u].ok) {
        xv[u] = *reinterpret_cast<const v4f*>(X + qd[u].off);
        if (a.res_mode == RES_SAME) rv[u] = *reinterpret_cast<const v4f*>(a.res + base + qd[u].off);
      }
    }
  };
  load();
  const double* p = a.part + ((int64_t)j * a.C + c) * a.parts * 2;
  double s = 0.0, ss = 0.0;
  for (int i = threadIdx.x; i < a.parts; i += 256) {
    s += p[2 * i];
    ss += p[2 * i + 1];
  }
  block_sum2(s, ss, red);
  const int n = a.b * HW;
  const double mean = s / n;
  const double var = fmax(ss / n - mean * mean, 0.0);
  const float mf = (float)mean, isf = (float)(1.0 / sqrt(var + BN_EPS));
  if (chunk == 0 && threadIdx.x == 0) {
    a.mean[j * a.C + c] = mf;
    a.istd[j * a.C + c] = isf;
  }
  const float* gam = a.gamma + (int64_t)j * a.pstride;
  const float ga = gam[c], be = gam[a.C + c];
  while (true) {
#pragma unroll
    for (int u = 0; u < BN_U; ++u) {
      if (!qd[u].ok) continue;
      v4f v;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = bn_affine(xv[u][i], mf, isf, ga, be);
      if (a.res_mode == RES_SAME) {
        v += rv[u];
      } else if (a.res_mode == RES_SUBSAMPLE && c < a.res_C) {
        const int img = j * a.b + qd[u].img;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int pp = qd[u].p + i, oh = pp / a.W, ow = pp - oh * a.W;
          v[i] += a.res[(((int64_t)img * a.res_C + c) * a.res_H + oh * a.res_st) * a.res_W +
                        ow * a.res_st];
        }
      }
      if (a.relu)
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = v[i] > 0.f ? v[i] : 0.f;
      *reinterpret_cast<v4f*>(Y + qd[u].off) = v;
    }
    qb += BN_U * 256;
    if (qb >= q1) break;
    load();
  }
}

__global__ __launch_bounds__(256) void bn_bwd_apply_v4_k(BNBwdArgs a) {
  __shared__ double red[8];
  const int chunk = blockIdx.x, c = blockIdx.y, j = blockIdx.z;
  const int HW = a.H * a.W, HW4 = HW >> 2, n4 = a.b * HW4, CHW = a.C * HW;
  const int sh = pow2_shift(HW4);
  const int per = (n4 + a.chunks - 1) / a.chunks;
  const int q0 = chunk * per, q1 = min(n4, q0 + per);
  const int64_t base = ((int64_t)j * a.b * a.C + c) * HW;
  Quad qd[BN_U];
  v4f dv[BN_U], yv[BN_U], xv[BN_U];
  int qb = q0 + threadIdx.x;
  auto load = [&]() {
#pragma unroll
    for (int u = 0; u < BN_U; ++u) {
      qd[u] = quad_at(qb + u * 256, q1, HW4, sh, CHW);
      if (qd[u].ok) {
        const int64_t o = base + qd[u].off;
        dv[u] = *reinterpret_cast<const v4f*>(a.dy + o);
        xv[u] = *reinterpret_cast<const v4f*>(a.x + o);
        if (a.y) yv[u] = *reinterpret_cast<const v4f*>(a.y + o);
      }
    }
  };
  load();
  const double* p = a.part + ((int64_t)j * a.C + c) * a.parts * 2;
  double s = 0.0, sx = 0.0;
  for (int i = threadIdx.x; i < a.parts; i += 256) {
    s += p[2 * i];
    sx += p[2 * i + 1];
  }
  block_sum2(s, sx, red);
  const int n = a.b * HW;
  const float mf = a.mean[j * a.C + c], isf = a.istd[j * a.C + c];
  const float ga = a.gamma[(int64_t)j * a.pstride + c];
  const float be = a.gamma[(int64_t)j * a.pstride + a.C + c];
  if (chunk == 0 && threadIdx.x == 0) {
    a.dgamma[(int64_t)j * a.pstride + c] = (float)sx;
    a.dgamma[(int64_t)j * a.pstride + a.C + c] = (float)s;
  }
  const float k1 = ga * isf, mdy = (float)(s / n), mdyx = (float)(sx / n);
  while (true) {
#pragma unroll
    for (int u = 0; u < BN_U; ++u) {
      if (!qd[u].ok) continue;
      v4f d = dv[u], dx;
      if (a.y) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (!(yv[u][i] > 0.f)) d[i] = 0.f;
      } else if (a.relu_x) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (!(bn_affine(xv[u][i], mf, isf, ga, be) > 0.f)) d[i] = 0.f;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float xh = (xv[u][i] - mf) * isf;
        dx[i] = k1 * (d[i] - mdy - xh * mdyx);
      }
      const int64_t o = base + qd[u].off;
      *reinterpret_cast<v4f*>(a.dx + o) = dx;
      if (a.dres) *reinterpret_cast<v4f*>(a.dres + o) = d;
    }
    qb += BN_U * 256;
    if (qb >= q1) break;
    load();
  }
}

// Max pool: the first cell (row-major) whose value is strictly greater than
// all earlier ones wins; padded cells never win.
// Grid: x over the (image, channel) planes, y over 256-pixel blocks of a
// plane, so that a thread splits only its in-plane index (32-bit).
__global__ __launch_bounds__(256) void maxpool_fwd_k(const float* x, int NC, int H, int W, int K,
                                                     int st, int pad, float* y, int Ho, int Wo,
                                                     int* arg) {
  const int cello = blockIdx.y * 256 + threadIdx.x;
  if (cello >= Ho * Wo) return;
  const int64_t nc = blockIdx.x;
  const int oh = cello / Wo, ow = cello - oh * Wo;
  const int64_t o = nc * Ho * Wo + cello;
  const float* xp = x + nc * H * W;
  int best = -1;
  float bv = 0.f;
  for (int r = 0; r < K; ++r) {
    const int ih = oh * st - pad + r;
    if (ih < 0 || ih >= H) continue;
    for (int s = 0; s < K; ++s) {
      const int iw = ow * st - pad + s;
      if (iw < 0 || iw >= W) continue;
      const float v = xp[ih * W + iw];
      if (best < 0 || v > bv) {
        best = ih * W + iw;
        bv = v;
      }
    }
  }
  y[o] = bv;
  arg[o] = best;
}

// Gradient of max pool, gathered per input cell over the windows that can
// contain it (no atomics): windows visited in row-major order.
__global__ __launch_bounds__(256) void maxpool_bwd_k(const float* dy, const int* arg,
                                                     const float* x, int NC, int H, int W, int K,
                                                     int st, int pad, int Ho, int Wo, float* dx,
                                                     int mask_relu) {
  const int cell = blockIdx.y * 256 + threadIdx.x;
  if (cell >= H * W) return;
  const int64_t nc = blockIdx.x;
  const int ih = cell / W, iw = cell - ih * W;
  const int64_t i = nc * H * W + cell;
  // windows oh with oh*st - pad <= ih <= oh*st - pad + K - 1
  const int oh_lo = max(0, (ih + pad - K + st) / st), oh_hi = min(Ho - 1, (ih + pad) / st);
  const int ow_lo = max(0, (iw + pad - K + st) / st), ow_hi = min(Wo - 1, (iw + pad) / st);
  float s = 0.f;
  for (int oh = oh_lo; oh <= oh_hi; ++oh)
    for (int ow = ow_lo; ow <= ow_hi; ++ow) {
      const int64_t o = (nc * Ho + oh) * Wo + ow;
      if (arg[o] == cell) s += dy[o];
    }
  if (mask_relu && !(x[i] > 0.f)) s = 0.f;
  dx[i] = s;
}

// The same two kernels over tiles of rows, through LDS: a workgroup stages
// the rows its windows cover with coalesced reads, then visits the windows
// there in the same order (identical results).  POOL_LDS floats of LDS.
constexpr int POOL_LDS = 4096;

// Forward: output rows [oh0, oh0 + toh) of plane blockIdx.x.
__global__ __launch_bounds__(256) void maxpool_fwd_rows_k(const float* x, int H, int W, int K,
                                                          int st, int pad, float* y, int Ho,
                                                          int Wo, int* arg, int toh) {
  __shared__ float xs[POOL_LDS];
  const int64_t nc = blockIdx.x;
  const int oh0 = blockIdx.y * toh, oh1 = min(Ho, oh0 + toh);
  const int ih_lo = max(0, oh0 * st - pad), ih_hi = min(H, (oh1 - 1) * st - pad + K);
  const float* xp = x + nc * H * W + ih_lo * W;
  const int n = max(0, ih_hi - ih_lo) * W;
  for (int e = threadIdx.x; e < n; e += 256) xs[e] = xp[e];
  __syncthreads();
  const int cells = (oh1 - oh0) * Wo;
  for (int q = threadIdx.x; q < cells; q += 256) {
    const int r0 = q / Wo, ow = q - r0 * Wo, oh = oh0 + r0;
    int best = -1;
    float bv = 0.f;
    for (int r = 0; r < K; ++r) {
      const int ih = oh * st - pad + r;
      if (ih < 0 || ih >= H) continue;
      for (int s = 0; s < K; ++s) {
        const int iw = ow * st - pad + s;
        if (iw < 0 || iw >= W) continue;
        const float v = xs[(ih - ih_lo) * W + iw];
        if (best < 0 || v > bv) {
          best = ih * W + iw;
          bv = v;
        }
      }
    }
    const int64_t o = (nc * Ho + oh) * Wo + ow;
    y[o] = bv;
    arg[o] = best;
  }
}

// Backward: input rows [ih0, ih0 + tih) of plane blockIdx.x; the window rows
// that can contain them are staged (gradient and argmax), half of the LDS
// each.
__global__ __launch_bounds__(256) void maxpool_bwd_rows_k(const float* dy, const int* arg,
                                                          const float* x, int H, int W, int K,
                                                          int st, int pad, int Ho, int Wo,
                                                          float* dx, int mask_relu, int tih) {
  __shared__ float ds[POOL_LDS / 2];
  __shared__ int as[POOL_LDS / 2];
  const int64_t nc = blockIdx.x;
  const int ih0 = blockIdx.y * tih, ih1 = min(H, ih0 + tih);
  const int oh_lo = max(0, (ih0 + pad - K + st) / st), oh_hi = min(Ho - 1, (ih1 - 1 + pad) / st);
  const int n = max(0, oh_hi - oh_lo + 1) * Wo;
  const int64_t ob = (nc * Ho + oh_lo) * Wo;
  for (int e = threadIdx.x; e < n; e += 256) {
    ds[e] = dy[ob + e];
    as[e] = arg[ob + e];
  }
  __syncthreads();
  const int cells = (ih1 - ih0) * W;
  for (int q = threadIdx.x; q < cells; q += 256) {
    const int r0 = q / W, iw = q - r0 * W, ih = ih0 + r0;
    const int cell = ih * W + iw;
    const int a_lo = max(0, (ih + pad - K + st) / st), a_hi = min(Ho - 1, (ih + pad) / st);
    const int w_lo = max(0, (iw + pad - K + st) / st), w_hi = min(Wo - 1, (iw + pad) / st);
    float s = 0.f;
    for (int oh = a_lo; oh <= a_hi; ++oh)
      for (int ow = w_lo; ow <= w_hi; ++ow) {
        const int e = (oh - oh_lo) * Wo + ow;
        if (as[e] == cell) s += ds[e];
      }
    const int64_t i = nc * H * W + cell;
    if (mask_relu && !(x[i] > 0.f)) s = 0.f;
    dx[i] = s;
  }
}

// Global average pool: one wave per (image, channel) plane, lanes over its
// pixels (coalesced), a fixed-order wave reduction.
__global__ __launch_bounds__(256) void gap_fwd_k(const float* x, int64_t NC, int HW, float* y) {
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= NC) return;
  const float* p = x + i * HW;
  float s = 0.f;
  for (int e = lane; e < HW; e += 64) s += p[e];
  s = wave_sum_f(s);
  if (lane == 0) y[i] = s / HW;
}

// Its gradient: every pixel of a plane gets the plane's output gradient / HW.
__global__ __launch_bounds__(256) void gap_bwd_k(const float* dy, int64_t n, int HW, float* dx) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  dx[i] = dy[i / HW] / HW;
}

// The same for planes of a multiple of 4 pixels, four pixels per thread.
__global__ __launch_bounds__(256) void gap_bwd_v4_k(const float* dy, int64_t n4, int HW4, int HW,
                                                    float* dx) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n4) return;
  const float v = dy[i / HW4] / HW;
  *reinterpret_cast<v4f*>(dx + 4 * i) = v4f{v, v, v, v};
}

// One block per learner: mean over its b images of -log softmax(o)_y and
// the gradient (softmax(o) - onehot(y)) / b (Eq. 2).
// 16 waves per learner; wave w takes rows w, w+16, ...  A row's logits are
// read once into registers (lane l holds classes l, l+64, ...; up to
// XENT_REG_CLASSES, beyond which the later passes read them again); its
// max and sum of exponentials are wave reductions (no block barriers).  The
// waves' fp64 loss partials, each summed in row order, are combined in
// wave order.
constexpr int XENT_WAVES = 16, XENT_CPL = 16, XENT_REG_CLASSES = 64 * XENT_CPL;
__global__ __launch_bounds__(64 * XENT_WAVES) void softmax_xent_k(const float* logits,
                                                                  const int32_t* labels, int b,
                                                                  int classes, float* dlogits,
                                                                  float* loss) {
  __shared__ double red[XENT_WAVES];
  const int j = blockIdx.x, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const bool in_regs = classes <= XENT_REG_CLASSES;
  double tot = 0.0;
  for (int i = w; i < b; i += XENT_WAVES) {
    const int64_t row = (int64_t)(j * b + i) * classes;
    const float* o = logits + row;
    const int y = labels[j * b + i];
    float v[XENT_CPL];
    float mx = -INFINITY;
    if (in_regs) {
#pragma unroll
      for (int u = 0; u < XENT_CPL; ++u) {
        const int c = lane + 64 * u;
        v[u] = c < classes ? o[c] : -INFINITY;
      }
#pragma unroll
      for (int u = 0; u < XENT_CPL; ++u) mx = fmaxf(mx, v[u]);
    } else {
      for (int c = lane; c < classes; c += 64) mx = fmaxf(mx, o[c]);
    }
    mx = wave_max_f(mx);
    float se = 0.f;
    if (in_regs) {
#pragma unroll
      for (int u = 0; u < XENT_CPL; ++u)
        if (lane + 64 * u < classes) se += expf(v[u] - mx);
    } else {
      for (int c = lane; c < classes; c += 64) se += expf(o[c] - mx);
    }
    se = wave_sum_f(se);
    const float lse = mx + logf(se);
    const bool yok = (unsigned)y < (unsigned)classes;
    if (in_regs) {
#pragma unroll
      for (int u = 0; u < XENT_CPL; ++u) {
        const int c = lane + 64 * u;
        if (c < classes) dlogits[row + c] = (expf(v[u] - lse) - (c == y ? 1.f : 0.f)) / b;
      }
    } else {
      for (int c = lane; c < classes; c += 64)
        dlogits[row + c] = (expf(o[c] - lse) - (c == y ? 1.f : 0.f)) / b;
    }
    if (lane == 0) tot += yok ? (double)(lse - o[y]) : (double)NAN;
  }
  if (lane == 0) red[w] = tot;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int q = 0; q < XENT_WAVES; ++q) t += red[q];
    loss[j] = (float)(t / b);
  }
}

constexpr int XENT_ROW_CLASSES = 32;
__global__ __launch_bounds__(256) void softmax_xent_rows_k(const float* logits,
                                                           const int32_t* labels, int b,
                                                           int classes, float* dlogits,
                                                           float* loss) {
  __shared__ double red[4];
  const int j = blockIdx.x, w = threadIdx.x >> 6;
  double tot = 0.0;
  for (int i = threadIdx.x; i < b; i += 256) {
    const int64_t row = (int64_t)(j * b + i) * classes;
    const float* o = logits + row;
    float mx = -INFINITY;
    for (int c = 0; c < classes; ++c) mx = fmaxf(mx, o[c]);
    float se = 0.f;
    for (int c = 0; c < classes; ++c) se += expf(o[c] - mx);
    const float lse = mx + logf(se);
    const int y = labels[j * b + i];
    const bool yok = (unsigned)y < (unsigned)classes;
    for (int c = 0; c < classes; ++c)
      dlogits[row + c] = (expf(o[c] - lse) - (c == y ? 1.f : 0.f)) / b;
    tot += yok ? (double)(lse - o[y]) : (double)NAN;
  }
  tot = wave_sum_d(tot);
  if ((threadIdx.x & 63) == 0) red[w] = tot;
  __syncthreads();
  if (threadIdx.x == 0) loss[j] = (float)((((red[0] + red[1]) + red[2]) + red[3]) / b);
}

// The head of one image, block (n, j).  A channel's HW pixels are HW/4
// float4s, one per thread of a group of TPC = HW/4 lanes (a power of two up
// to 64), so a pass covers 256/TPC channels with every load in flight, and
// a channel's sums combine by xor butterfly within its group.  Logits: a
// wave per class, lanes over channels.  Softmax cross-entropy: wave 0, a
// lane per class (the same arithmetic per row as softmax_xent_rows_k).
// Features' gradient: a thread per channel, in class order.  Then the pool
// backward with the batch norm's partial sums (fp64).
__device__ __forceinline__ float group_sum_f(float v, int tpc) {
  for (int o = 1; o < tpc; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ double group_sum_d(double v, int tpc) {
  for (int o = 1; o < tpc; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__global__ __launch_bounds__(256) void head_k(HeadArgs a) {
  __shared__ float gs[HEAD_MAX_C], dgs[HEAD_MAX_C], ls[HEAD_MAX_CLASSES];
  __shared__ float wsh[HEAD_MAX_W], bsh[HEAD_MAX_CLASSES], msh[HEAD_MAX_C], ish[HEAD_MAX_C];
  const int n = blockIdx.x, j = blockIdx.y, row = j * a.b + n;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int tpc = a.HW >> 2, cpp = 256 / tpc;  // threads per channel, channels per pass
  const int cg = threadIdx.x / tpc, q = threadIdx.x - cg * tpc;
  const int64_t plane0 = (int64_t)row * a.C * a.HW;
  const float* Y = a.y + plane0;
  // every global read goes out first: the pooled plane and the norm's x
  // (at most HEAD_PASSES float4s per thread), the FC weights and bias, the
  // norm's statistics, the label
  v4f yv[HEAD_PASSES], xv[HEAD_PASSES];
#pragma unroll
  for (int r = 0; r < HEAD_PASSES; ++r) {
    const int c = cg + r * cpp;
    if (c < a.C) {
      const int64_t idx = (int64_t)c * a.HW + 4 * q;
      yv[r] = *reinterpret_cast<const v4f*>(Y + idx);
      if (a.bn_part) xv[r] = *reinterpret_cast<const v4f*>(a.bn_x + plane0 + idx);
    }
  }
  const float* Wf = a.w + (int64_t)j * a.pstride;
  for (int e = threadIdx.x; e < a.classes * a.C; e += 256) wsh[e] = Wf[e];
  if ((int)threadIdx.x < a.classes)
    bsh[threadIdx.x] = a.bias ? a.bias[(int64_t)j * a.pstride + threadIdx.x] : 0.f;
  if (a.bn_part)
    for (int c = threadIdx.x; c < a.C; c += 256) {
      msh[c] = a.bn_mean[j * a.C + c];
      ish[c] = a.bn_istd[j * a.C + c];
    }
  const int label = a.labels[row];
#pragma unroll
  for (int r = 0; r < HEAD_PASSES; ++r) {
    const int c = cg + r * cpp;
    if (c >= a.C) continue;  // whole channel groups, so group_sum stays within active lanes
    const float s = group_sum_f(((yv[r][0] + yv[r][1]) + yv[r][2]) + yv[r][3], tpc);
    if (q == 0) {
      gs[c] = s / a.HW;
      a.g[(int64_t)row * a.C + c] = s / a.HW;
    }
  }
  __syncthreads();
  for (int o = w; o < a.classes; o += 4) {
    float s = 0.f;
    for (int c = lane; c < a.C; c += 64) s += wsh[o * a.C + c] * gs[c];
    s = wave_sum_f(s);
    if (lane == 0) ls[o] = a.bias ? s + bsh[o] : s;
  }
  __syncthreads();
  if (w == 0) {
    const bool on = lane < a.classes;
    const float o = on ? ls[lane] : -INFINITY;
    const float mx = wave_max_f(o);
    const float lse = mx + logf(wave_sum_f(on ? expf(o - mx) : 0.f));
    const bool yok = (unsigned)label < (unsigned)a.classes;
    if (lane == 0) a.loss[row] = yok ? lse - ls[label] : NAN;
    __builtin_amdgcn_wave_barrier();
    if (on) {
      const float d = (expf(o - lse) - (lane == label ? 1.f : 0.f)) / a.b;
      ls[lane] = d;
      a.dlogits[(int64_t)row * a.classes + lane] = d;
    }
  }
  __syncthreads();
  for (int c = threadIdx.x; c < a.C; c += 256) {
    float s = 0.f;
    for (int o = 0; o < a.classes; ++o) s += ls[o] * wsh[o * a.C + c];
    dgs[c] = s;
  }
  __syncthreads();
  float* DY = a.dy + plane0;
#pragma unroll
  for (int r = 0; r < HEAD_PASSES; ++r) {
    const int c = cg + r * cpp;
    if (c >= a.C) continue;
    const float d0 = dgs[c] / a.HW;
    *reinterpret_cast<v4f*>(DY + (int64_t)c * a.HW + 4 * q) = v4f{d0, d0, d0, d0};
    if (!a.bn_part) continue;  // uniform
    const float bm = msh[c], bi = ish[c];
    double s1 = 0.0, s2 = 0.0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float d = (!a.bn_relu || yv[r][i] > 0.f) ? d0 : 0.f;
      s1 += (double)d;
      s2 += (double)d * ((xv[r][i] - bm) * bi);
    }
    s1 = group_sum_d(s1, tpc);
    s2 = group_sum_d(s2, tpc);
    if (q == 0) {
      double* pq = a.bn_part + (((int64_t)j * a.C + c) * a.b + n) * 2;
      pq[0] = s1;
      pq[1] = s2;
    }
  }
}

}  // namespace

bool head_ok(int C, int HW, int classes) {
  const int tpc = HW / 4;
  return C <= HEAD_MAX_C && classes >= 1 && classes <= HEAD_MAX_CLASSES && HW % 4 == 0 &&
         tpc >= 1 && tpc <= 64 && (tpc & (tpc - 1)) == 0 && (int64_t)C * HW <= HEAD_MAX_PLANE &&
         classes * C <= HEAD_MAX_W;
}

hipError_t head_fwd_bwd(const HeadArgs& a, hipStream_t s) {
  if (!head_ok(a.C, a.HW, a.classes) || !al16(a.y) || !al16(a.dy) || !al16(a.bn_x))
    return hipErrorInvalidValue;
  klaunch(head_k, dim3(a.b, a.k), dim3(256), 0, s, a);
  return hipGetLastError();
}

// Workgroups per (replica, channel): enough for 512 over the launch, and
// for large planes at least one per 8192 values, so that no workgroup runs a
// long serial loop (ResNet-50's 56 x 56 stage: 1 -> 12 for 256 channels,
// its batch-norm statistics 101 -> 58 us per launch).
int bn_chunks(int b, int HW, int C, int k) {
  const int n = b * HW;
  int chunks = (int)std::max<int64_t>(cdiv(512, (int64_t)C * k), n / 8192);
  chunks = std::min(chunks, (int)cdiv(n, 1024));
  return std::max(1, chunks);
}

hipError_t bn_fwd_stats(const BNArgs& a, hipStream_t s) {
  klaunch(bn_stats_k, dim3(a.chunks, a.C, a.k), dim3(256), 0, s, a);
  return hipGetLastError();
}


hipError_t bn_fwd_apply(const BNArgs& a, hipStream_t s, const char** name) {
  if ((a.H * a.W) % 4 == 0 && al16(a.x) && al16(a.y) && (a.res_mode != RES_SAME || al16(a.res))) {
    if (name) *name = "bn_apply_v4_k";
    klaunch(bn_apply_v4_k, dim3(a.chunks, a.C, a.k), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  if (name) *name = "bn_apply_k";
  klaunch(bn_apply_k, dim3(a.chunks, a.C, a.k), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t bn_bwd_stats(const BNBwdArgs& a, hipStream_t s) {
  klaunch(bn_bwd_stats_k, dim3(a.chunks, a.C, a.k), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t bn_bwd_apply(const BNBwdArgs& a, hipStream_t s, const char** name) {
  if ((a.H * a.W) % 4 == 0 && al16(a.x) && al16(a.y) && al16(a.dy) && al16(a.dx) &&
      al16(a.dres)) {
    if (name) *name = "bn_bwd_apply_v4_k";
    klaunch(bn_bwd_apply_v4_k, dim3(a.chunks, a.C, a.k), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  if (name) *name = "bn_bwd_apply_k";
  klaunch(bn_bwd_apply_k, dim3(a.chunks, a.C, a.k), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t maxpool_fwd(const float* x, int N, int C, int H, int W, int K, int st, int pad,
                       float* y, int Ho, int Wo, int* arg, hipStream_t s) {
  const int64_t n = (int64_t)N * C * Ho * Wo;
  if (n == 0) return hipSuccess;
  // output rows per tile: as many as keep the input rows they cover within
  // the LDS staging buffer, at most 16
  const int room = POOL_LDS / W - K;
  const int toh = room < 0 ? 0 : std::min(std::min(Ho, 16), room / st + 1);
  if (toh >= 1) {
    klaunch(maxpool_fwd_rows_k, dim3((unsigned)(N * C), cdiv(Ho, toh)), dim3(256), 0, s, x, H, W,
            K, st, pad, y, Ho, Wo, arg, toh);
    return hipGetLastError();
  }
  klaunch(maxpool_fwd_k, dim3((unsigned)(N * C), cdiv((int64_t)Ho * Wo, 256)), dim3(256), 0, s, x, N * C, H, W, K, st,
                     pad, y, Ho, Wo, arg);
  return hipGetLastError();
}

hipError_t maxpool_bwd(const float* dy, const int* arg, const float* x, int N, int C, int H,
                       int W, int K, int st, int pad, int Ho, int Wo, float* dx, int mask_relu,
                       hipStream_t s) {
  const int64_t n = (int64_t)N * C * H * W;
  if (n == 0) return hipSuccess;
  // input rows per tile: at most 32, and the window rows they reach,
  // (tih + K - 2) / st + 2 at most, within half the LDS staging buffer
  int tih = std::min(H, 32);
  while (tih >= 1 && ((tih + K - 2) / st + 2) * Wo > POOL_LDS / 2) --tih;
  if (tih >= 1) {
    klaunch(maxpool_bwd_rows_k, dim3((unsigned)(N * C), cdiv(H, tih)), dim3(256), 0, s, dy, arg, x,
            H, W, K, st, pad, Ho, Wo, dx, mask_relu, tih);
    return hipGetLastError();
  }
  klaunch(maxpool_bwd_k, dim3((unsigned)(N * C), cdiv((int64_t)H * W, 256)), dim3(256), 0, s, dy, arg, x, N * C, H, W,
                     K, st, pad, Ho, Wo, dx, mask_relu);
  return hipGetLastError();
}

hipError_t gap_fwd(const float* x, int N, int C, int HW, float* y, hipStream_t s) {
  const int64_t nc = (int64_t)N * C;
  klaunch(gap_fwd_k, dim3(cdiv(nc, 4)), dim3(256), 0, s, x, nc, HW, y);
  return hipGetLastError();
}

hipError_t gap_bwd(const float* dy, int N, int C, int HW, float* dx, hipStream_t s,
                   const char** name) {
  const int64_t n = (int64_t)N * C * HW;
  if (name) *name = "gap_bwd_k";
  if (HW % 4 == 0 && al16(dx)) {
    if (name) *name = "gap_bwd_v4_k";
    klaunch(gap_bwd_v4_k, dim3(cdiv(n / 4, 256)), dim3(256), 0, s, dy, n / 4, HW / 4, HW, dx);
    return hipGetLastError();
  }
  klaunch(gap_bwd_k, dim3(cdiv(n, 256)), dim3(256), 0, s, dy, n, HW, dx);
  return hipGetLastError();
}

hipError_t softmax_xent(const float* logits, const int32_t* labels, int k, int b, int classes,
                        float* dlogits, float* loss, hipStream_t s, const char** name) {
  if (classes <= XENT_ROW_CLASSES) {
    if (name) *name = "softmax_xent_rows_k";
    klaunch(softmax_xent_rows_k, dim3(k), dim3(256), 0, s, logits, labels, b, classes, dlogits,
            loss);
  } else {
    if (name) *name = "softmax_xent_k";
    klaunch(softmax_xent_k, dim3(k), dim3(64 * XENT_WAVES), 0, s, logits, labels, b, classes, dlogits,
            loss);
  }
  return hipGetLastError();
}

}  // namespace cbk
