// lenet.hip -- the learning task of the MNIST-shaped LeNet in two launches.
//
// LeNet on 28 x 28 single-channel images (Table 1's MNIST workload) is tiny:
// one image's forward and backward pass is ~1 M multiply-adds, so the
// operator-by-operator path spends its time in ~25 kernel boundaries per
// iteration.  Here one workgroup per image keeps every activation of its
// image in LDS and runs the whole forward pass, the loss (Eq. 2), the whole
// backward data path and that image's share of the convolution weight
// gradients (lenet_image_k); a second launch forms each learner's gradient:
// the convolution shares summed over the learner's images in image order,
// the FC weight gradients as sums over the images of outer products of the
// stored FC inputs and output gradients, and the learner's mean loss
// (lenet_learner_k).  The network is the one the library describes for
// LeNet: conv 5x5x6 pad 2, ReLU, max 2x2/2, conv 5x5x16, ReLU, max 2x2/2,
// FC 400-120 ReLU, FC 120-84 ReLU, FC 84-classes, softmax cross-entropy.
// Max pooling takes the first strict maximum of its window in row-major
// order; ReLU'(0) = 0.  Every sum runs in a fixed order (deterministic).
#include "kernels.hpp"

namespace cbk {
namespace {

constexpr int IMG = 28, PADW = 32;                 // input and its 2-pixel-padded copy
constexpr int C1 = 6, A1 = IMG * IMG, P1W = 14, P1 = P1W * P1W;
constexpr int C2 = 16, A2W = 10, A2 = A2W * A2W, P2W = 5, P2 = P2W * P2W;
constexpr int F0 = C2 * P2, F1 = 120, F2 = 84;     // 400 -> 120 -> 84 -> classes
constexpr int NW1 = C1 * 25, NW2 = C2 * C1 * 25;   // conv weights
constexpr int THREADS = 1024;
constexpr int D2P = A2W + 8;          // padded da2 plane width (18)
constexpr int R1PARTS = 7, R1ROWS = IMG / R1PARTS;  // conv1 weight shares: 7 slices of 4 rows
constexpr int D1PARTS = 8;  // conv2 data gradient: 8 parts of the output channels
typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4f mfma4(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// First strict maximum of a 2 x 2 window (row-major), its position 0..3.
__device__ __forceinline__ int win_arg(float v0, float v1, float v2, float v3, float* best) {
  int a = 0;
  float b = v0;
  if (v1 > b) { b = v1; a = 1; }
  if (v2 > b) { b = v2; a = 2; }
  if (v3 > b) { b = v3; a = 3; }
  *best = b;
  return a;
}

// FC weights pass through one LDS buffer: W1 (120 x 400) in three slabs of
// 40 rows, W2 and W3 whole.  All threads copy a slab with 16-byte loads, so
// the whole slab is in flight at once instead of each output's row being a
// chain of dependent L2 round trips.
constexpr int SLAB_ROWS = 40, SLAB = SLAB_ROWS * F0;  // 16000 floats (64 KB)
static_assert(F2 * F1 <= SLAB && LENET_MAX_CLASSES * F2 <= SLAB, "FC weights fit the slab");

// A slab is copied in two halves, with 16-byte loads (n a multiple of 4, src
// 16-byte aligned): fetch issues the global reads into registers (at most PFQ
// float4s a thread) and put writes them to LDS later, so that a slab's reads
// overlap the work before its use (the first slab's the convolutions, each
// later one's the use of the slab before it).
constexpr int PFQ = (SLAB / 4 + THREADS - 1) / THREADS;
__device__ __forceinline__ void fetch(v4f (&r)[PFQ], const float* src, int n) {
  const v4f* s4 = reinterpret_cast<const v4f*>(src);
#pragma unroll
  for (int u = 0; u < PFQ; ++u) {
    const int e = threadIdx.x + u * THREADS;
    if (e < (n >> 2)) r[u] = s4[e];
  }
}
__device__ __forceinline__ void put(float* dst, const v4f (&r)[PFQ], int n) {
  v4f* d4 = reinterpret_cast<v4f*>(dst);
#pragma unroll
  for (int u = 0; u < PFQ; ++u) {
    const int e = threadIdx.x + u * THREADS;
    if (e < (n >> 2)) d4[e] = r[u];
  }
}

// y[o0 + r] = bias[o0 + r] + sum_i W[r][i] x[i] for the nrows rows of W in
// LDS (row length NIN, 16-byte aligned rows and x); ReLU if relu.
template <int NIN>
__device__ __forceinline__ void fc_rows(const float* W, const float* bias, const float* x, int o0,
                                        int nrows, bool relu, float* y) {
  // 16 lanes per row, four rows per wave at a time: lane l of a row takes the
  // input quads l, l + 16, ..., reads all of them and their weights first,
  // then sums the inputs in that order; a 16-lane xor butterfly combines the
  // lanes (4 steps instead of a 64-lane sum's 6, for four rows at once)
  static_assert(NIN % 4 == 0, "rows of whole quads");
  constexpr int NQ = NIN / 4, NQL = (NQ + 15) / 16;  // quads per row, per lane
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, l16 = lane & 15;
  for (int r0 = w * 4; r0 < nrows; r0 += THREADS / 16) {
    const int r = r0 + (lane >> 4);
    float s = 0.f;
    if (r < nrows) {
      v4f wv[NQL], xv[NQL];
#pragma unroll
      for (int i = 0; i < NQL; ++i)
        if (l16 + 16 * i < NQ) {
          wv[i] = *reinterpret_cast<const v4f*>(W + r * NIN + 4 * (l16 + 16 * i));
          xv[i] = *reinterpret_cast<const v4f*>(x + 4 * (l16 + 16 * i));
        }
#pragma unroll
      for (int i = 0; i < NQL; ++i)
        if (l16 + 16 * i < NQ)
#pragma unroll
          for (int c = 0; c < 4; ++c) s += wv[i][c] * xv[i][c];
    }
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) s += __shfl_xor(s, o, 16);
    if (l16 == 0 && r < nrows) {
      s += bias[o0 + r];
      y[o0 + r] = relu ? (s > 0.f ? s : 0.f) : s;
    }
  }
}

__global__ __launch_bounds__(THREADS) void lenet_image_k(LenetArgs a) {
  __shared__ float xs[PADW * PADW];
  __shared__ float w1[NW1], b1[C1], w2[NW2], b2[C2];
  __shared__ float a1[C1 * A1], p1[C1 * P1];
  __shared__ float a2[C2 * A2];
  __shared__ __attribute__((aligned(16))) float p2[F0];
  __shared__ unsigned char g1[C1 * P1], g2[F0];
  __shared__ __attribute__((aligned(16))) float f1[F1];
  __shared__ __attribute__((aligned(16))) float f2[F2];
  __shared__ float lg[LENET_MAX_CLASSES];
  __shared__ float fbs[F1 + F2 + LENET_MAX_CLASSES];  // the FC biases
  __shared__ int koff2[NW2 / C2];  // conv2 tap k = (c, r, s): its offset in p1
  // conv2's filters again as [co][tap][8 input channels, 6 used]: the data
  // gradient reads a tap's six weights as two vector loads
  __shared__ __attribute__((aligned(16))) float w2t[C2 * 25 * 8];
  __shared__ float dl[LENET_MAX_CLASSES], df2[F2], df1[F1], dp2[F0];
  __shared__ float da2[C2 * A2], dp1[C1 * P1];
  __shared__ __attribute__((aligned(16))) float wb[SLAB];
  // once the FC weights are done with, their buffer holds da2 with a
  // 4-pixel zero border, the two halves of conv2's data gradient and the
  // seven slices of conv1's weight shares
  float* const da2p = wb;
  float* const pdp1 = wb + C2 * D2P * D2P;
  float* const part1 = pdp1 + D1PARTS * C1 * P1;
  static_assert(C2 * D2P * D2P + D1PARTS * C1 * P1 + R1PARTS * (NW1 + C1) <= SLAB, "aliases fit");
  const int tid = threadIdx.x;
  const int n = blockIdx.x, j = n / a.b;  // image n belongs to learner j
  const float* Wj = a.w + (int64_t)j * a.pstride;
  const float* x = a.x + (int64_t)n * A1;
  const int C = a.classes;
  const float* fw1 = Wj + NW1 + C1 + NW2 + C2;
  const float* fb1 = fw1 + F1 * F0;
  const float* fw2 = fb1 + F1;
  const float* fb2 = fw2 + F2 * F1;
  const float* fw3 = fb2 + F2;
  const float* fb3 = fw3 + C * F2;

  // ---- forward -------------------------------------------------------
  for (int e = tid; e < PADW * PADW; e += THREADS) {
    const int r = e / PADW - 2, c = e % PADW - 2;
    xs[e] = (r >= 0 && r < IMG && c >= 0 && c < IMG) ? x[r * IMG + c] : 0.f;
  }
  for (int e = tid; e < NW1 + C1 + NW2 + C2; e += THREADS) {
    const float v = Wj[e];
    if (e < NW1) w1[e] = v;
    else if (e < NW1 + C1) b1[e - NW1] = v;
    else if (e < NW1 + C1 + NW2) {
      const int f = e - NW1 - C1;
      w2[f] = v;
      w2t[((f / 150) * 25 + f % 25) * 8 + (f % 150) / 25] = v;
    }
    else b2[e - NW1 - C1 - NW2] = v;
  }
  // the FC biases and the label are read here too, off the FC chain
  for (int e = tid; e < F1 + F2 + C; e += THREADS)
    fbs[e] = e < F1 ? fb1[e] : (e < F1 + F2 ? fb2[e - F1] : fb3[e - F1 - F2]);
  for (int e = tid; e < NW2 / C2; e += THREADS)
    koff2[e] = (e / 25) * P1 + ((e % 25) / 5) * P1W + e % 5;
  const int label = a.labels[n];
  v4f pf[PFQ];
  fetch(pf, fw1, SLAB);  // FC1's first slab, in flight through the convolutions
  __syncthreads();
  for (int pix = tid; pix < A1; pix += THREADS) {  // conv1 + bias + ReLU, a thread per pixel
    const int y = pix / IMG, xx = pix % IMG;
    float v[25];
#pragma unroll
    for (int t = 0; t < 25; ++t) v[t] = xs[(y + t / 5) * PADW + xx + t % 5];
#pragma unroll
    for (int co = 0; co < C1; ++co) {
      float s = 0.f;
#pragma unroll
      for (int t = 0; t < 25; ++t) s += w1[co * 25 + t] * v[t];
      s += b1[co];
      a1[co * A1 + pix] = s > 0.f ? s : 0.f;
    }
  }
  __syncthreads();
  for (int o = tid; o < C1 * P1; o += THREADS) {  // max pool 2x2/2
    const int c = o / P1, py = (o % P1) / P1W, px = o % P1W;
    const float* v = a1 + c * A1 + 2 * py * IMG + 2 * px;
    float b;
    g1[o] = (unsigned char)win_arg(v[0], v[1], v[IMG], v[IMG + 1], &b);
    p1[o] = b;
  }
  __syncthreads();
  // conv2 + bias + ReLU on fp32 MFMA: rows = the 100 output pixels (7 tiles
  // of 16, a wave each), columns = the 16 output channels, contraction over
  // the 150 taps k = (c, r, s) in 38 steps of 4 (k >= 150 reads 0)
  if ((tid >> 6) < (A2 + 15) / 16) {
    constexpr int K2 = NW2 / C2;
    const int lane = tid & 63, tile = tid >> 6;
    const int m = tile * 16 + (lane & 15), co = lane & 15, kq = lane >> 4;
    const bool mok = m < A2;
    const int pb = mok ? (m / A2W) * P1W + m % A2W : 0;
    v4f acc = {0.f, 0.f, 0.f, 0.f};
    // ten steps' operands read before their MFMAs, so that their LDS
    // reads (the tap table, then the input) are in flight together
    constexpr int NT2 = (K2 + 3) / 4, BT = 10;
    for (int t0 = 0; t0 < NT2; t0 += BT) {
      float av[BT], bv[BT];
#pragma unroll
      for (int u = 0; u < BT; ++u) {
        const int k = 4 * (t0 + u) + kq;
        const bool kok = k < K2;
        const int kc = kok ? k : 0;
        av[u] = (mok && kok) ? p1[pb + koff2[kc]] : 0.f;
        bv[u] = kok ? w2[co * K2 + kc] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < BT; ++u)
        if (t0 + u < NT2) acc = mfma4(av[u], bv[u], acc);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int mm = tile * 16 + kq * 4 + i;
      const float s = acc[i] + b2[co];
      if (mm < A2) a2[co * A2 + mm] = s > 0.f ? s : 0.f;
    }
  }
  __syncthreads();
  for (int o = tid; o < F0; o += THREADS) {  // max pool 2x2/2
    const int c = o / P2, py = (o % P2) / P2W, px = o % P2W;
    const float* v = a2 + c * A2 + 2 * py * A2W + 2 * px;
    float b;
    g2[o] = (unsigned char)win_arg(v[0], v[1], v[A2W], v[A2W + 1], &b);
    p2[o] = b;
  }
  __syncthreads();
  for (int o0 = 0; o0 < F1; o0 += SLAB_ROWS) {  // FC1 + ReLU, by slabs
    put(wb, pf, SLAB);
    __syncthreads();
    // the next slab (or W2) is read while this one is used
    if (o0 + SLAB_ROWS < F1) fetch(pf, fw1 + (o0 + SLAB_ROWS) * F0, SLAB);
    else fetch(pf, fw2, F2 * F1);
    fc_rows<F0>(wb, fbs, p2, o0, SLAB_ROWS, true, f1);
    __syncthreads();
  }
  put(wb, pf, F2 * F1);  // FC2 + ReLU
  __syncthreads();
  fetch(pf, fw3, C * F2);
  fc_rows<F1>(wb, fbs + F1, f1, 0, F2, true, f2);
  __syncthreads();
  put(wb, pf, C * F2);  // FC3 (kept in LDS for its data gradient)
  __syncthreads();
  fetch(pf, fw2, F2 * F1);  // for the backward pass
  fc_rows<F2>(wb, fbs + F1 + F2, f2, 0, C, false, lg);
  __syncthreads();
  // softmax cross-entropy of this image: the loss term and (softmax -
  // onehot) / b; a label out of range gives a NaN term and no one-hot
  if (tid < 64) {
    const bool on = tid < C;
    const float o = on ? lg[tid] : -INFINITY;
    const float mx = wave_max(o);
    const float lse = mx + logf(wave_sum(on ? expf(o - mx) : 0.f));
    const bool yok = (unsigned)label < (unsigned)C;
    if (tid == 0) a.loss[n] = yok ? lse - lg[label] : NAN;
    if (on) dl[tid] = (expf(o - lse) - (tid == label ? 1.f : 0.f)) / a.b;
  }
  __syncthreads();

  // ---- backward ------------------------------------------------------
  for (int i = tid; i < F2; i += THREADS) {
    float s = 0.f;
    for (int o = 0; o < C; ++o) s += dl[o] * wb[o * F2 + i];
    df2[i] = f2[i] > 0.f ? s : 0.f;
  }
  __syncthreads();
  put(wb, pf, F2 * F1);
  __syncthreads();
  fetch(pf, fw1, SLAB);
  for (int i = tid; i < F1; i += THREADS) {
    float s = 0.f;
    for (int o = 0; o < F2; ++o) s += df2[o] * wb[o * F1 + i];
    df1[i] = f1[i] > 0.f ? s : 0.f;
  }
  for (int i = tid; i < F0; i += THREADS) dp2[i] = 0.f;
  for (int o0 = 0; o0 < F1; o0 += SLAB_ROWS) {  // dp2 = W1^T df1, slab by slab in order
    __syncthreads();
    put(wb, pf, SLAB);
    __syncthreads();
    if (o0 + SLAB_ROWS < F1) fetch(pf, fw1 + (o0 + SLAB_ROWS) * F0, SLAB);
    for (int i = tid; i < F0; i += THREADS) {
      float s = dp2[i];
      for (int r = 0; r < SLAB_ROWS; ++r) s += df1[o0 + r] * wb[r * F0 + i];
      dp2[i] = s;
    }
  }
  __syncthreads();
  for (int e = tid; e < C2 * D2P * D2P; e += THREADS) {  // pool2 backward, ReLU mask
    const int c = e / (D2P * D2P), y = (e % (D2P * D2P)) / D2P - 4, xx = e % D2P - 4;
    float d = 0.f;
    if (y >= 0 && y < A2W && xx >= 0 && xx < A2W) {
      const int o = c * P2 + (y >> 1) * P2W + (xx >> 1), pos = (y & 1) * 2 + (xx & 1);
      const int a = c * A2 + y * A2W + xx;
      d = (g2[o] == pos && a2[a] > 0.f) ? dp2[o] : 0.f;
      da2[a] = d;
    }
    da2p[e] = d;
  }
  __syncthreads();
  // conv2 data gradient: dp1[c][iy][ix] = sum over co, r, q of
  // da2[co][iy - r][ix - q] w2[co][c][r][q]; a thread per pair of
  // horizontally adjacent input pixels and an eighth of the output
  // channels, all six input channels, so that the pair shares its 5 x 6
  // window reads and each tap's weight loads; the eighths summed in order
  for (int t0 = tid; t0 < D1PARTS * (P1 / 2); t0 += THREADS) {
    const int pp = t0 % (P1 / 2), qt = t0 / (P1 / 2);
    const int iy = pp / (P1W / 2) + 4, ix = 2 * (pp % (P1W / 2)) + 4;
    float acc0[C1] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, acc1[C1] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int co = qt * (C2 / D1PARTS); co < (qt + 1) * (C2 / D1PARTS); ++co) {
      float v[5][6];  // da2 rows iy - r, columns ix - 4 .. ix + 1
#pragma unroll
      for (int r = 0; r < 5; ++r)
#pragma unroll
        for (int u = 0; u < 6; ++u) v[r][u] = da2p[co * D2P * D2P + (iy - r) * D2P + ix - 4 + u];
#pragma unroll
      for (int t = 0; t < 25; ++t) {
        const int r = t / 5, q = t % 5;
        const float* wt = w2t + (co * 25 + t) * 8;
        const v4f wa = *reinterpret_cast<const v4f*>(wt);
        const v4f wc = *reinterpret_cast<const v4f*>(wt + 4);
        const float x0 = v[r][4 - q], x1 = v[r][5 - q];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          acc0[c] += wa[c] * x0;
          acc1[c] += wa[c] * x1;
        }
        acc0[4] += wc[0] * x0;
        acc0[5] += wc[1] * x0;
        acc1[4] += wc[0] * x1;
        acc1[5] += wc[1] * x1;
      }
    }
    const int pix = (iy - 4) * P1W + ix - 4;
#pragma unroll
    for (int c = 0; c < C1; ++c) {
      pdp1[qt * C1 * P1 + c * P1 + pix] = acc0[c];
      pdp1[qt * C1 * P1 + c * P1 + pix + 1] = acc1[c];
    }
  }
  __syncthreads();
  for (int e = tid; e < C1 * P1; e += THREADS) {
    float s = pdp1[e];
#pragma unroll
    for (int q = 1; q < D1PARTS; ++q) s += pdp1[q * C1 * P1 + e];
    dp1[e] = s;
  }
  __syncthreads();
  for (int e = tid; e < C1 * A1; e += THREADS) {  // pool1 backward, ReLU mask (in a1)
    const int c = e / A1, y = (e % A1) / IMG, xx = e % IMG;
    const int o = c * P1 + (y >> 1) * P1W + (xx >> 1), pos = (y & 1) * 2 + (xx & 1);
    a1[e] = (g1[o] == pos && a1[e] > 0.f) ? dp1[o] : 0.f;
  }
  __syncthreads();

  // ---- this image's share of the convolution weight gradients ---------
  float* cw = a.conv_part + (int64_t)n * LENET_CONV_PARAMS;
  // conv2: dW[co][c][r][q] = sum over y, x of da2[co][y][x] p1[c][y+r][x+q];
  // a thread per (co, c, r) computes the five q, row by row
  for (int t = tid; t < C2 * C1 * 5 + C2; t += THREADS) {
    if (t < C2 * C1 * 5) {
      const int co = t / 30, c = (t % 30) / 5, r = t % 5;
      float acc[5] = {0.f, 0.f, 0.f, 0.f, 0.f};
      for (int y = 0; y < A2W; ++y) {
        float d[A2W], pr[P1W];
#pragma unroll
        for (int xx = 0; xx < A2W; ++xx) d[xx] = da2[co * A2 + y * A2W + xx];
#pragma unroll
        for (int xx = 0; xx < P1W; ++xx) pr[xx] = p1[c * P1 + (y + r) * P1W + xx];
#pragma unroll
        for (int q = 0; q < 5; ++q)
#pragma unroll
          for (int xx = 0; xx < A2W; ++xx) acc[q] += d[xx] * pr[xx + q];
      }
#pragma unroll
      for (int q = 0; q < 5; ++q) cw[NW1 + C1 + co * 150 + c * 25 + r * 5 + q] = acc[q];
    } else {
      const int co = t - C2 * C1 * 5;
      float s = 0.f;
      for (int e = 0; e < A2; ++e) s += da2[co * A2 + e];
      cw[NW1 + C1 + NW2 + co] = s;
    }
  }
  // conv1: dW[co][r][q] over 28 x 28 pixels, in seven slices of four rows
  // summed in order; a thread per (slice, co, r) computes the five q
  for (int t = tid; t < R1PARTS * (C1 * 5 + C1); t += THREADS) {
    const int part = t / (C1 * 5 + C1), u = t % (C1 * 5 + C1);
    const int y0 = part * R1ROWS;
    if (u < C1 * 5) {
      const int co = u / 5, r = u % 5;
      float acc[5] = {0.f, 0.f, 0.f, 0.f, 0.f};
      for (int y = y0; y < y0 + R1ROWS; ++y) {
        float d[IMG], xr[PADW];
#pragma unroll
        for (int xx = 0; xx < IMG; ++xx) d[xx] = a1[co * A1 + y * IMG + xx];
#pragma unroll
        for (int xx = 0; xx < PADW; ++xx) xr[xx] = xs[(y + r) * PADW + xx];
#pragma unroll
        for (int q = 0; q < 5; ++q)
#pragma unroll
          for (int xx = 0; xx < IMG; ++xx) acc[q] += d[xx] * xr[xx + q];
      }
#pragma unroll
      for (int q = 0; q < 5; ++q) part1[part * (NW1 + C1) + co * 25 + r * 5 + q] = acc[q];
    } else {
      const int co = u - C1 * 5;
      float s = 0.f;
      for (int e = y0 * IMG; e < (y0 + R1ROWS) * IMG; ++e) s += a1[co * A1 + e];
      part1[part * (NW1 + C1) + NW1 + co] = s;
    }
  }
  // the FC layers' inputs and output gradients, for their weight gradients
  float* fv = a.fc_vec + (int64_t)n * LENET_FC_VEC;
  for (int e = tid; e < LENET_FC_VEC; e += THREADS) {
    float v = 0.f;
    if (e < LENET_DF1) v = p2[e];
    else if (e < LENET_F1) v = df1[e - LENET_DF1];
    else if (e < LENET_DF2) v = f1[e - LENET_F1];
    else if (e < LENET_F2) v = df2[e - LENET_DF2];
    else if (e < LENET_DL) v = f2[e - LENET_F2];
    else if (e - LENET_DL < C) v = dl[e - LENET_DL];
    fv[e] = v;
  }
  __syncthreads();
  for (int u = tid; u < NW1 + C1; u += THREADS) {
    float s = part1[u];
#pragma unroll
    for (int part = 1; part < R1PARTS; ++part) s += part1[part * (NW1 + C1) + u];
    cw[u] = s;
  }
}

// Learner j's gradient: blockIdx.y = j; each thread several parameters.
__global__ __launch_bounds__(256) void lenet_learner_k(LenetArgs a) {
  const int j = blockIdx.y, C = a.classes;
  const int64_t P = LENET_CONV_PARAMS + (int64_t)F1 * F0 + F1 + F2 * F1 + F2 + C * F2 + C;
  float* g = a.grad + (int64_t)j * a.pstride;
  const float* cw = a.conv_part + (int64_t)j * a.b * LENET_CONV_PARAMS;
  const float* fv = a.fc_vec + (int64_t)j * a.b * LENET_FC_VEC;
  const int64_t o_fw1 = LENET_CONV_PARAMS, o_fb1 = o_fw1 + F1 * F0, o_fw2 = o_fb1 + F1,
                o_fb2 = o_fw2 + F2 * F1, o_fw3 = o_fb2 + F2, o_fb3 = o_fw3 + C * F2;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < P; e += (int64_t)gridDim.x * 256) {
    // (one parameter per thread: the grid covers P)
    float s = 0.f;
    if (e < LENET_CONV_PARAMS) {
      // eight images' shares in flight at a time, added in image order
      for (int i0 = 0; i0 < a.b; i0 += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          v[u] = i0 + u < a.b ? cw[(int64_t)(i0 + u) * LENET_CONV_PARAMS + e] : 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (i0 + u < a.b) s += v[u];
      }
    } else {
      // dW[o][in] = sum over images of dy[o] * x[in]; db[o] = sum of dy[o]
      int dyo, xo = -1;
      if (e < o_fb1) { dyo = LENET_DF1 + (int)((e - o_fw1) / F0); xo = (int)((e - o_fw1) % F0); }
      else if (e < o_fw2) { dyo = LENET_DF1 + (int)(e - o_fb1); }
      else if (e < o_fb2) { dyo = LENET_DF2 + (int)((e - o_fw2) / F1); xo = LENET_F1 + (int)((e - o_fw2) % F1); }
      else if (e < o_fw3) { dyo = LENET_DF2 + (int)(e - o_fb2); }
      else if (e < o_fb3) { dyo = LENET_DL + (int)((e - o_fw3) / F2); xo = LENET_F2 + (int)((e - o_fw3) % F2); }
      else { dyo = LENET_DL + (int)(e - o_fb3); }
      // eight images' terms in flight at a time, added in image order
      for (int i0 = 0; i0 < a.b; i0 += 8) {
        float dy[8], xv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const float* v = fv + (int64_t)(i0 + u) * LENET_FC_VEC;
          const bool in = i0 + u < a.b;
          dy[u] = in ? v[dyo] : 0.f;
          xv[u] = in && xo >= 0 ? v[xo] : 1.f;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (i0 + u < a.b) s += xo >= 0 ? dy[u] * xv[u] : dy[u];
      }
    }
    g[e] = s;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    double l = 0.0;
    for (int i = 0; i < a.b; ++i) l += (double)a.loss[(int64_t)j * a.b + i];
    a.learner_loss[j] = (float)(l / a.b);
  }
}

}  // namespace

bool lenet_fused_ok(int in_c, int in_h, int in_w, int classes) {
  return in_c == 1 && in_h == IMG && in_w == IMG && classes >= 1 && classes <= LENET_MAX_CLASSES;
}

hipError_t lenet_image(const LenetArgs& a, hipStream_t s) {
  if (!lenet_fused_ok(1, IMG, IMG, a.classes) || a.k < 1 || a.b < 1) return hipErrorInvalidValue;
  klaunch(lenet_image_k, dim3((unsigned)(a.k * a.b)), dim3(THREADS), 0, s, a);
  return hipGetLastError();
}

hipError_t lenet_learner(const LenetArgs& a, hipStream_t s) {
  if (!lenet_fused_ok(1, IMG, IMG, a.classes) || a.k < 1 || a.b < 1) return hipErrorInvalidValue;
  klaunch(lenet_learner_k, dim3(LENET_LEARNER_BLOCKS, (unsigned)a.k), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace cbk
