// conv_gemm.hip -- replica-batched convolution (and FC) as implicit GEMM on
// the fp32 matrix cores of gfx950 (v_mfma_f32_16x16x4f32).
//
// Sec. 2.1: training a learner is a forward pass and a backward pass
// through its layers; for a convolution these are three contractions:
//   forward      Y[m][n]  = sum_k A[m][k] W[n][k],  m=(img,oh,ow), n=co, k=(ci,r,s)
//   data grad    dX[m][n] = sum_k dY~[m][k] W'[k][n], m=(img,ih,iw), n=ci, k=(co,r,s)
//   weight grad  dW[n][k] = sum_m dY[m][n] A[m][k],  contracted over the
//                                                      b*Ho*Wo pixels of a learner
// Every learner has its own weights, so the grid's z axis runs over the k
// replicas: one launch covers all learners and fills the CUs even when each
// learner's batch is small (Sec. 3.1: learners train independently).
//
// Tiling: 256 threads (4 wave64s), LDS stages of BK contraction steps
// stored with k contiguous, so each 16x16x4 MFMA operand group is one
// ds_read_b128; within a group of 16 steps the contraction index seen by
// lane l at sub-step kk is 4*(l/16) + kk for both operands.  Global loads
// for the next stage are in flight while the current stage is multiplied
// (two LDS buffers, one barrier per stage).  The filter size R is a template
// parameter, so splitting a contraction index into (channel, r, s) is
// multiply-shift arithmetic; in the A-operand loaders that index is
// wave-uniform and the split runs on the scalar unit.
#include "kernels.hpp"

#include <algorithm>
#include <string>

namespace cbk {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v2f __attribute__((ext_vector_type(2)));
constexpr int OUT_OF_RANGE = -(1 << 29);

__device__ __forceinline__ v4f mfma4(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// The GEMM grids (x: M tiles, y: N tiles, z: replica, or replica and
// split) renumbered XCD-major with the N tiles fastest: the tiles of one M
// tile, which read the same rows of the left operand, and then the
// neighbouring M tiles of the same z run on one XCD and share its L2.
struct GemmTile {
  int mt, nt, z;
};
__device__ __forceinline__ GemmTile gemm_tile() {
  const int gx = gridDim.x, gy = gridDim.y;
  const int t = xcd_major(blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z), gx * gy * gridDim.z);
  GemmTile r;
  r.nt = t % gy;
  const int rest = t / gy;
  r.mt = rest % gx;
  r.z = rest / gx;
  return r;
}

// One LDS stage: As[rows][BK+4], Bs[cols][BK+4], both k-contiguous.
template <int TM, int TN, int BK>
__device__ __forceinline__ void mma_stage(const float* As, const float* Bs, int wm0, int wn0,
                                          int lane, v4f (&acc)[TM][TN]) {
  constexpr int LDK = BK + 4;
  const int r = lane & 15, q = (lane >> 4) * 4;
#pragma unroll
  for (int g = 0; g < BK; g += 16) {
    v4f av[TM], bv[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
      av[i] = *reinterpret_cast<const v4f*>(As + (wm0 + i * 16 + r) * LDK + g + q);
#pragma unroll
    for (int i = 0; i < TN; ++i)
      bv[i] = *reinterpret_cast<const v4f*>(Bs + (wn0 + i * 16 + r) * LDK + g + q);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) acc[a][b] = mfma4(av[a][kk], bv[b][kk], acc[a][b]);
  }
}

__device__ __forceinline__ float relu0(float v) { return v > 0.f ? v : 0.f; }

__device__ __forceinline__ double shfl_xor_d(double v, int o) { return __shfl_xor(v, o, 64); }

// ---------------------------------------------------------------- forward
// CF (Ci a multiple of BK): the contraction runs over k = (channel block of
// BK, r, s, channel in the block) instead of (ci, r, s), the same sum in
// another order (the same order for 1x1 filters).  A stage of BK steps then
// shares one tap (r, s), so its window check and tap offset are computed
// once per stage, and a thread's steps are consecutive channels (one plane
// apart in X, RS floats apart in W); the R*R taps of a channel block follow
// each other, so its planes stay in L2 across them.
template <int BM, int BN, int WM, int WN, int R, int BK, bool CF = false>
__global__ __launch_bounds__(256) void conv_fwd_k(ConvFwdArgs a) {
  constexpr int RS = R * R;
  constexpr int LDK = BK + 4;
  constexpr int TM = BM / (WM * 16), TN = BN / (WN * 16);
  constexpr int TPR = 256 / BM;   // threads sharing one output row
  constexpr int KPT = BK / TPR;   // contraction steps each of them loads
  constexpr int QPR = BK / 4;     // float4 groups per B row
  constexpr int BQ = BN * QPR;
  constexpr int BPT = (BQ + 255) / 256;
  __shared__ __attribute__((aligned(16))) float As[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) float Bs[2][BN * LDK];

  const ConvGeom g = a.g;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const GemmTile tl = gemm_tile();
  const int j = tl.z;
  const int HW = g.H * g.W, HoWo = g.Ho * g.Wo;
  const int M = g.b * HoWo, N = g.Co, K = g.Ci * RS;
  const int m0 = tl.mt * BM, n0 = tl.nt * BN;
  const float* X = a.x + (int64_t)j * g.b * g.Ci * HW;
  const float* Wt = a.w + (int64_t)j * a.pstride;

  const int am = tid % BM;
  const int akq = __builtin_amdgcn_readfirstlane(tid / BM);
  // The lane's output pixel: element offset of its window corner (ih0, iw0)
  // and, as bit masks, the window rows and columns that lie inside the
  // image (none past the last pixel).  Every load below is a buffer load
  // whose offset is OUTSIDE where the element is zero, so the loaders have
  // no branches.
  int xb = 0;
  uint32_t rmask = 0, cmask = 0;
  {
    const int m = m0 + am;
    if (m < M) {
      const int img = m / HoWo, p = m - img * HoWo, oh = p / g.Wo, ow = p - oh * g.Wo;
      const int ih0 = oh * g.st - g.pad, iw0 = ow * g.st - g.pad;
      xb = img * g.Ci * HW + ih0 * g.W + iw0;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if ((unsigned)(ih0 + r) < (unsigned)g.H) rmask |= 1u << r;
        if ((unsigned)(iw0 + r) < (unsigned)g.W) cmask |= 1u << r;
      }
    }
  }
  const uint32_t xbytes = (uint32_t)((int64_t)g.b * g.Ci * HW * 4);
  const uint32_t wbytes = (uint32_t)((int64_t)N * K * 4);
  // filter rows as 16-byte quads when every quad is aligned and whole
  const bool wq = (K & 3) == 0 && (reinterpret_cast<uintptr_t>(a.w) & 15) == 0;
  float ra[KPT];
  float rb[BPT][4];

  auto loadA = [&](int k0, float (&ra)[KPT]) {
    const auto xsrc = buf_rsrc_u(X, xbytes);
    if constexpr (CF) {
      const int t = k0 / BK, blk = t / RS, rs = t - blk * RS, r = rs / R, s = rs - r * R;
      const int c0 = blk * BK + akq * KPT;  // wave-uniform
      const uint32_t in = (rmask >> r) & (cmask >> s) & 1u;
      const uint32_t a0 = in ? (uint32_t)(xb + c0 * HW + r * g.W + s) * 4u : OUTSIDE;
#pragma unroll
      for (int i = 0; i < KPT; ++i) ra[i] = buf_ld(xsrc, a0 + (uint32_t)(i * HW) * 4u);
      return;
    }
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int k = k0 + akq * KPT + i;  // wave-uniform
      const int ci = k / RS, rs = k - ci * RS, r = rs / R, s = rs - r * R;
      const int koff = __builtin_amdgcn_readfirstlane(ci * HW + r * g.W + s);
      const uint32_t in = (rmask >> r) & (cmask >> s) & (k < K ? 1u : 0u);
      const uint32_t off = (uint32_t)(xb + koff) * 4u;
      ra[i] = buf_ld(xsrc, (in & 1u) ? off : OUTSIDE);
    }
  };
  auto loadB = [&](int k0, float (&rb)[BPT][4]) {
    const auto wsrc = buf_rsrc_u(Wt, wbytes);
    if constexpr (CF) {
      const int t = k0 / BK, blk = t / RS, rs = t - blk * RS, c0 = blk * BK;
#pragma unroll
      for (int u = 0; u < BPT; ++u) {
        const int idx = tid + u * 256, n = n0 + idx / QPR, ci = c0 + 4 * (idx % QPR);
        const uint32_t b0 = idx < BQ && n < N ? (uint32_t)(n * K + ci * RS + rs) * 4u : OUTSIDE;
        if (RS == 1 && wq) {
          const buf_v4f v = buf_ld4(wsrc, b0);
#pragma unroll
          for (int i = 0; i < 4; ++i) rb[u][i] = v[i];
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) rb[u][i] = buf_ld(wsrc, b0 + 4u * i * RS);
        }
      }
      return;
    }
#pragma unroll
    for (int u = 0; u < BPT; ++u) {
      const int idx = tid + u * 256, n = n0 + idx / QPR, kq = k0 + 4 * (idx % QPR);
      const bool row = idx < BQ && n < N;
      const uint32_t off = (uint32_t)(n * K + kq) * 4u;
      if (wq) {
        const buf_v4f v = buf_ld4(wsrc, row && kq < K ? off : OUTSIDE);
#pragma unroll
        for (int i = 0; i < 4; ++i) rb[u][i] = v[i];
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) rb[u][i] = buf_ld(wsrc, row && kq + i < K ? off + 4u * i : OUTSIDE);
      }
    }
  };
  auto store = [&](int buf, const float (&ra)[KPT], const float (&rb)[BPT][4]) {
#pragma unroll
    for (int q = 0; q < KPT / 4; ++q)
      *reinterpret_cast<v4f*>(&As[buf][am * LDK + akq * KPT + 4 * q]) =
          v4f{ra[4 * q], ra[4 * q + 1], ra[4 * q + 2], ra[4 * q + 3]};
#pragma unroll
    for (int u = 0; u < BPT; ++u) {
      const int idx = tid + u * 256;
      if (idx < BQ)
        *reinterpret_cast<v4f*>(&Bs[buf][(idx / QPR) * LDK + 4 * (idx % QPR)]) =
            v4f{rb[u][0], rb[u][1], rb[u][2], rb[u][3]};
    }
  };

  v4f acc[TM][TN];
#pragma unroll
  for (int x = 0; x < TM; ++x)
#pragma unroll
    for (int y = 0; y < TN; ++y) acc[x][y] = v4f{0.f, 0.f, 0.f, 0.f};
  const int wm = wave % WM, wm0 = wm * TM * 16, wn0 = (wave / WM) * TN * 16;
  const int T = (K + BK - 1) / BK;
  loadA(0, ra);
  loadB(0, rb);
  store(0, ra, rb);
  __syncthreads();
  for (int t = 0; t < T; ++t) {
    const int cur = t & 1;
    if (t + 1 < T) {
      loadA((t + 1) * BK, ra);
      loadB((t + 1) * BK, rb);
    }
    mma_stage<TM, TN, BK>(As[cur], Bs[cur], wm0, wn0, lane, acc);
    if (t + 1 < T) store(cur ^ 1, ra, rb);
    __syncthreads();
  }

  const float* bias = a.bias ? a.bias + (int64_t)j * a.pstride : nullptr;
  float* Y = a.y + (int64_t)j * g.b * N * HoWo;
  const bool vec = (HoWo & 3) == 0 && (reinterpret_cast<uintptr_t>(Y) & 15) == 0;
  double s1[TN], s2[TN];  // per-column sums of the stored outputs (BN statistics)
#pragma unroll
  for (int y = 0; y < TN; ++y) s1[y] = s2[y] = 0.0;
#pragma unroll
  for (int x = 0; x < TM; ++x)
#pragma unroll
    for (int y = 0; y < TN; ++y) {
      const int n = n0 + wn0 + y * 16 + (lane & 15);
      const int mb = m0 + wm0 + x * 16 + (lane >> 4) * 4;
      if (n >= N || mb >= M) continue;
      const float bv = bias ? bias[n] : 0.f;
      int img = mb / HoWo, p = mb - img * HoWo;
      if (vec) {
        // the lane's four pixels are consecutive in one plane
        v4f v = acc[x][y];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float e = v[i] + bv;
          if (a.relu) e = relu0(e);
          v[i] = e;
          s1[y] += (double)e;
          s2[y] += (double)e * e;
        }
        *reinterpret_cast<v4f*>(&Y[((int64_t)img * N + n) * HoWo + p]) = v;
        continue;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (mb + i < M) {
          float v = acc[x][y][i] + bv;
          if (a.relu) v = relu0(v);
          Y[((int64_t)img * N + n) * HoWo + p] = v;
          s1[y] += (double)v;
          s2[y] += (double)v * v;
        }
        if (++p == HoWo) {
          p = 0;
          ++img;
        }
      }
    }
  if (!a.stats) return;
  // Per-channel partial sums of this tile for the batch norm that follows:
  // lanes with the same column combine by an xor butterfly, then the WM
  // waves of a column strip in wave order.  Written to
  // stats[j][n][M tile][0..1].
  __shared__ double red[WM][BN][2];
#pragma unroll
  for (int y = 0; y < TN; ++y) {
    double u = s1[y], v = s2[y];
    u += shfl_xor_d(u, 16);
    v += shfl_xor_d(v, 16);
    u += shfl_xor_d(u, 32);
    v += shfl_xor_d(v, 32);
    if (lane < 16) {
      red[wm][wn0 + y * 16 + lane][0] = u;
      red[wm][wn0 + y * 16 + lane][1] = v;
    }
  }
  __syncthreads();
  if (tid < BN && n0 + tid < N) {
    double u = 0.0, v = 0.0;
#pragma unroll
    for (int w = 0; w < WM; ++w) {
      u += red[w][tid][0];
      v += red[w][tid][1];
    }
    double* o = a.stats + (((int64_t)j * N + n0 + tid) * gridDim.x + tl.mt) * 2;
    o[0] = u;
    o[1] = v;
  }
}

// ------------------------------------------------------------ data grad
// SP (1x1, stride 2, even H and W): only the dX pixels (2oh, 2ow) receive a
// contribution, so the GEMM runs over the Ho x Wo grid (a quarter of the
// MFMA work) and the epilogue writes the 2x2 block of each grid point: the
// contraction at (2oh, 2ow), zero at the other three, every pixel through
// the same accumulate / add / mask / batch-norm epilogue.
// CF (stride 1 or the grid-only form, Co a multiple of BK): the contraction
// runs over k = (channel block, r, s, co in the block), as in the forward
// kernel.
template <int BM, int BN, int WM, int WN, int R, int ST, int BK, bool SP = false, bool CF = false>
__global__ __launch_bounds__(256) void conv_bwd_data_k(ConvBwdDataArgs a) {
  static_assert(!SP || (R == 1 && ST == 2), "the grid-only form is the 1x1 stride-2 case");
  static_assert(!CF || ST == 1 || SP, "the tap-major loaders read dY at stride 1");
  constexpr int RS = R * R;
  constexpr int LDK = BK + 4;
  constexpr int TM = BM / (WM * 16), TN = BN / (WN * 16);
  constexpr int TPR = 256 / BM;
  constexpr int KPT = BK / TPR;
  constexpr int QPR = BK / 4;
  constexpr int BQ = BN * QPR;
  constexpr int BPT = (BQ + 255) / 256;
  __shared__ __attribute__((aligned(16))) float As[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) float Bs[2][BN * LDK];

  const ConvGeom g = a.g;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const GemmTile tl = gemm_tile();
  const int j = tl.z;
  const int HW = g.H * g.W, HoWo = g.Ho * g.Wo;
  const int M = SP ? g.b * HoWo : g.b * HW, N = g.Ci, K = g.Co * RS;
  const int m0 = tl.mt * BM, n0 = tl.nt * BN;
  const float* DY = a.dy + (int64_t)j * g.b * g.Co * HoWo;
  const float* Wt = a.w + (int64_t)j * a.pstride;

  const int am = tid % BM;
  const int akq = __builtin_amdgcn_readfirstlane(tid / BM);
  int thp = OUT_OF_RANGE, twp = OUT_OF_RANGE, yb = 0;
  {
    const int m = m0 + am;
    if (m < M) {
      if (SP) {  // m is a grid point: dY pixel m % HoWo of image m / HoWo
        const int img = m / HoWo;
        thp = twp = 0;
        yb = img * g.Co * HoWo + (m - img * HoWo);
      } else {
        const int img = m / HW, p = m - img * HW, ih = p / g.W, iw = p - ih * g.W;
        thp = ih + g.pad;
        twp = iw + g.pad;
        yb = img * g.Co * HoWo;
      }
    }
  }
  float ra[KPT];
  float rb[BPT][4];
  // tap-major loaders: the lane's dY window as row and column masks (tap
  // (r, s) reads dY row thp - r, column twp - s), every load a buffer load
  // that reads 0 at OUTSIDE
  uint32_t rmask = 0, cmask = 0;
  int ybase = 0;
  if (CF && m0 + am < M) {
    if (SP) {
      rmask = cmask = 1u;
      ybase = yb;
    } else {
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if ((unsigned)(thp - r) < (unsigned)g.Ho) rmask |= 1u << r;
        if ((unsigned)(twp - r) < (unsigned)g.Wo) cmask |= 1u << r;
      }
      ybase = yb + thp * g.Wo + twp;
    }
  }
  const uint32_t dybytes = (uint32_t)((int64_t)g.b * g.Co * HoWo * 4);
  const uint32_t wbytes = (uint32_t)((int64_t)g.Co * N * RS * 4);

  auto loadA = [&](int k0, float (&ra)[KPT]) {
    if constexpr (CF) {
      const auto ysrc = buf_rsrc_u(DY, dybytes);
      const int t = k0 / BK, blk = t / RS, rs = t - blk * RS, r = rs / R, s = rs - r * R;
      const int c0 = blk * BK + akq * KPT;  // wave-uniform
      const uint32_t in = (rmask >> r) & (cmask >> s) & 1u;
      const uint32_t a0 = in ? (uint32_t)(ybase + c0 * HoWo - r * g.Wo - s) * 4u : OUTSIDE;
#pragma unroll
      for (int i = 0; i < KPT; ++i) ra[i] = buf_ld(ysrc, a0 + (uint32_t)(i * HoWo) * 4u);
      return;
    }
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int k = k0 + akq * KPT + i;  // wave-uniform
      float v = 0.f;
      if (SP) {
        if (k < K && thp == 0) v = DY[yb + k * HoWo];
      } else if (k < K) {
        const int co = k / RS, rs = k - co * RS, r = rs / R, s = rs - r * R;
        const int th = thp - r, tw = twp - s;
        if (ST == 1) {
          if ((unsigned)th < (unsigned)g.Ho && (unsigned)tw < (unsigned)g.Wo)
            v = DY[yb + co * HoWo + th * g.Wo + tw];
        } else {
          if ((unsigned)th < (unsigned)(ST * g.Ho) && (unsigned)tw < (unsigned)(ST * g.Wo) &&
              th % ST == 0 && tw % ST == 0)
            v = DY[yb + co * HoWo + (th / ST) * g.Wo + tw / ST];
        }
      }
      ra[i] = v;
    }
  };
  auto loadB = [&](int k0, float (&rb)[BPT][4]) {
    if constexpr (CF) {
      // W'[k][n] = W[co][n][r][s]: a quad is four consecutive co, N*RS apart
      const auto wsrc = buf_rsrc_u(Wt, wbytes);
      const int t = k0 / BK, blk = t / RS, rs = t - blk * RS, c0 = blk * BK;
#pragma unroll
      for (int u = 0; u < BPT; ++u) {
        const int idx = tid + u * 256, n = n0 + idx / QPR, co = c0 + 4 * (idx % QPR);
        const uint32_t b0 = idx < BQ && n < N ? (uint32_t)((co * N + n) * RS + rs) * 4u : OUTSIDE;
#pragma unroll
        for (int i = 0; i < 4; ++i) rb[u][i] = buf_ld(wsrc, b0 + (uint32_t)(i * N * RS) * 4u);
      }
      return;
    }
#pragma unroll
    for (int u = 0; u < BPT; ++u) {
      const int idx = tid + u * 256, n = n0 + idx / QPR, kq = k0 + 4 * (idx % QPR);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v = 0.f;
        const int k = kq + i, co = k / RS, rs = k - co * RS;
        if (idx < BQ && n < N && k < K) v = Wt[((int64_t)co * N + n) * RS + rs];
        rb[u][i] = v;
      }
    }
  };
  auto store = [&](int buf, const float (&ra)[KPT], const float (&rb)[BPT][4]) {
#pragma unroll
    for (int q = 0; q < KPT / 4; ++q)
      *reinterpret_cast<v4f*>(&As[buf][am * LDK + akq * KPT + 4 * q]) =
          v4f{ra[4 * q], ra[4 * q + 1], ra[4 * q + 2], ra[4 * q + 3]};
#pragma unroll
    for (int u = 0; u < BPT; ++u) {
      const int idx = tid + u * 256;
      if (idx < BQ)
        *reinterpret_cast<v4f*>(&Bs[buf][(idx / QPR) * LDK + 4 * (idx % QPR)]) =
            v4f{rb[u][0], rb[u][1], rb[u][2], rb[u][3]};
    }
  };

  v4f acc[TM][TN];
#pragma unroll
  for (int x = 0; x < TM; ++x)
#pragma unroll
    for (int y = 0; y < TN; ++y) acc[x][y] = v4f{0.f, 0.f, 0.f, 0.f};
  const int wm0 = (wave % WM) * TM * 16, wn0 = (wave / WM) * TN * 16;
  const int T = (K + BK - 1) / BK;
  loadA(0, ra);
  loadB(0, rb);
  store(0, ra, rb);
  __syncthreads();
  for (int t = 0; t < T; ++t) {
    const int cur = t & 1;
    if (t + 1 < T) {
      loadA((t + 1) * BK, ra);
      loadB((t + 1) * BK, rb);
    }
    mma_stage<TM, TN, BK>(As[cur], Bs[cur], wm0, wn0, lane, acc);
    if (t + 1 < T) store(cur ^ 1, ra, rb);
    __syncthreads();
  }

  float* DX = a.dx + (int64_t)j * g.b * N * HW;
  const float* MSK = a.mask ? a.mask + (int64_t)j * g.b * N * HW : nullptr;
  // the subsampled source keeps every st-th row and column: ceil(H / st) x ceil(W / st)
  const int sst = a.add_st > 0 ? a.add_st : 1;
  const int Hs = (g.H + sst - 1) / sst, Ws = (g.W + sst - 1) / sst;
  const float* ADD = a.add;
  if (ADD)
    ADD += (a.add_mode == ADD_SAME) ? (int64_t)j * g.b * N * HW
                                    : (int64_t)j * g.b * a.add_C * Hs * Ws;
  const bool bn = a.bn_part != nullptr;
  const float* BX = bn ? a.bn_x + (int64_t)j * g.b * N * HW : nullptr;
  // the norm's ReLU output recomputed from its input where gamma is given
  // (one tensor fewer to read), else read
  const float* BG = (bn && a.bn_y && a.bn_gamma) ? a.bn_gamma + (int64_t)j * a.pstride : nullptr;
  const float* BY = (bn && a.bn_y && !BG) ? a.bn_y + (int64_t)j * g.b * N * HW : nullptr;
  // float4 epilogue when a lane's four pixels never straddle two planes and
  // every tensor it touches per pixel is 16-byte aligned
  const uintptr_t align = reinterpret_cast<uintptr_t>(DX) | reinterpret_cast<uintptr_t>(MSK) |
                          reinterpret_cast<uintptr_t>(BX) | reinterpret_cast<uintptr_t>(BY) |
                          (a.add_mode == ADD_SAME ? reinterpret_cast<uintptr_t>(ADD) : 0);
  const bool vec = (HW & 3) == 0 && (align & 15) == 0;
  // grid-only form: four consecutive grid points share a grid row
  const bool sp_vec = SP && (g.Wo & 3) == 0 && (align & 15) == 0;
  double s1[TN], s2[TN];
#pragma unroll
  for (int y = 0; y < TN; ++y) s1[y] = s2[y] = 0.0;
#pragma unroll
  for (int x = 0; x < TM; ++x)
#pragma unroll
    for (int y = 0; y < TN; ++y) {
      const int n = n0 + wn0 + y * 16 + (lane & 15);
      const int mb = m0 + wm0 + x * 16 + (lane >> 4) * 4;
      if (n >= N || mb >= M) continue;
      int img = mb / HW, p = mb - img * HW;
      float bm = 0.f, bi = 0.f, bg = 0.f, bb = 0.f;
      if (bn) {
        bm = a.bn_mean[j * N + n];
        bi = a.bn_istd[j * N + n];
      }
      if (BG) {
        bg = BG[n];
        bb = BG[N + n];
      }
      if (SP && sp_vec) {
        // the lane's four grid points (oh, ow .. ow + 3) lie in one grid row:
        // dX rows 2oh and 2oh + 1, 8 consecutive pixels each from column
        // 2ow, moved as two float4s per row.  Pixel 2ow + q of row 2oh holds
        // the contraction of point q / 2 when q is even; every other pixel
        // starts at 0.  The same epilogue as below, element for element.
        const int im = mb / HoWo, pp = mb - im * HoWo, oh = pp / g.Wo, ow = pp - oh * g.Wo;
#pragma unroll
        for (int r2 = 0; r2 < 2; ++r2) {
          const int ih = 2 * oh + r2;
          const int64_t idx = (((int64_t)im * N + n) * g.H + ih) * g.W + 2 * ow;
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int64_t e = idx + 4 * h;
            v4f v = {r2 == 0 ? acc[x][y][2 * h] : 0.f, 0.f, r2 == 0 ? acc[x][y][2 * h + 1] : 0.f, 0.f};
            if (a.accumulate) v += *reinterpret_cast<const v4f*>(DX + e);
            if (a.add_mode == ADD_SAME) {
              v += *reinterpret_cast<const v4f*>(ADD + e);
            } else if (a.add_mode == ADD_SUBSAMPLE && ih % a.add_st == 0) {
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const int iw = 2 * ow + 4 * h + q;
                if (iw % a.add_st == 0)
                  v[q] += ADD[(((int64_t)im * a.add_C + n) * Hs + ih / a.add_st) * Ws + iw / a.add_st];
              }
            }
            if (MSK) {
              const v4f mk = *reinterpret_cast<const v4f*>(MSK + e);
#pragma unroll
              for (int q = 0; q < 4; ++q)
                if (!(mk[q] > 0.f)) v[q] = 0.f;
            }
            *reinterpret_cast<v4f*>(DX + e) = v;
            if (bn) {
              const v4f bx = *reinterpret_cast<const v4f*>(BX + e);
              v4f by = {1.f, 1.f, 1.f, 1.f};
              if (BY) by = *reinterpret_cast<const v4f*>(BY + e);
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const bool on = BY ? by[q] > 0.f : BG ? bn_affine(bx[q], bm, bi, bg, bb) > 0.f : true;
                const float d = on ? v[q] : 0.f;
                const float xh = (bx[q] - bm) * bi;
                s1[y] += (double)d;
                s2[y] += (double)d * xh;
              }
            }
          }
        }
        continue;
      }
      if (SP) {
        // grid point m: dX rows 2oh and 2oh + 1, columns 2ow and 2ow + 1,
        // two pixels (8 bytes) per row; the lane's four grid points are
        // consecutive, so (image, oh, ow) is stepped rather than divided out
        int im = mb / HoWo, pp = mb - im * HoWo, oh = pp / g.Wo, ow = pp - oh * g.Wo;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (mb + i >= M) break;
          if (i > 0 && ++ow == g.Wo) {
            ow = 0;
            if (++oh == g.Ho) {
              oh = 0;
              ++im;
            }
          }
#pragma unroll
          for (int r2 = 0; r2 < 2; ++r2) {
            const int ih = 2 * oh + r2;
            const int64_t idx = (((int64_t)im * N + n) * g.H + ih) * g.W + 2 * ow;
            v2f v = {r2 == 0 ? acc[x][y][i] : 0.f, 0.f};
            if (a.accumulate) v += *reinterpret_cast<const v2f*>(DX + idx);
            if (a.add_mode == ADD_SAME) {
              v += *reinterpret_cast<const v2f*>(ADD + idx);
            } else if (a.add_mode == ADD_SUBSAMPLE) {
#pragma unroll
              for (int c2 = 0; c2 < 2; ++c2) {
                const int iw = 2 * ow + c2;
                if (ih % a.add_st == 0 && iw % a.add_st == 0)
                  v[c2] += ADD[(((int64_t)im * a.add_C + n) * Hs + ih / a.add_st) * Ws + iw / a.add_st];
              }
            }
            if (MSK) {
              const v2f mk = *reinterpret_cast<const v2f*>(MSK + idx);
#pragma unroll
              for (int c2 = 0; c2 < 2; ++c2)
                if (!(mk[c2] > 0.f)) v[c2] = 0.f;
            }
            *reinterpret_cast<v2f*>(DX + idx) = v;
            if (bn) {
              const v2f bx = *reinterpret_cast<const v2f*>(BX + idx);
              v2f by = {1.f, 1.f};
              if (BY) by = *reinterpret_cast<const v2f*>(BY + idx);
#pragma unroll
              for (int c2 = 0; c2 < 2; ++c2) {
                const bool on = BY ? by[c2] > 0.f : BG ? bn_affine(bx[c2], bm, bi, bg, bb) > 0.f : true;
                const float d = on ? v[c2] : 0.f;
                const float xh = (bx[c2] - bm) * bi;
                s1[y] += (double)d;
                s2[y] += (double)d * xh;
              }
            }
          }
        }
        continue;
      }
      if (vec) {
        // the lane's four pixels are consecutive in one plane: float4 access
        const int64_t idx = ((int64_t)img * N + n) * HW + p;
        v4f v = acc[x][y];
        if (a.accumulate) v += *reinterpret_cast<const v4f*>(DX + idx);
        if (a.add_mode == ADD_SAME) {
          v += *reinterpret_cast<const v4f*>(ADD + idx);
        } else if (a.add_mode == ADD_SUBSAMPLE) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int pp = p + i, ih = pp / g.W, iw = pp - ih * g.W;
            if (ih % a.add_st == 0 && iw % a.add_st == 0)
              v[i] += ADD[(((int64_t)img * a.add_C + n) * Hs + ih / a.add_st) * Ws + iw / a.add_st];
          }
        }
        if (MSK) {
          const v4f mk = *reinterpret_cast<const v4f*>(MSK + idx);
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (!(mk[i] > 0.f)) v[i] = 0.f;
        }
        *reinterpret_cast<v4f*>(DX + idx) = v;
        if (bn) {
          const v4f bx = *reinterpret_cast<const v4f*>(BX + idx);
          v4f by = {1.f, 1.f, 1.f, 1.f};
          if (BY) by = *reinterpret_cast<const v4f*>(BY + idx);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const bool on = BY ? by[i] > 0.f : BG ? bn_affine(bx[i], bm, bi, bg, bb) > 0.f : true;
            const float d = on ? v[i] : 0.f;
            const float xh = (bx[i] - bm) * bi;
            s1[y] += (double)d;
            s2[y] += (double)d * xh;
          }
        }
        continue;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (mb + i < M) {
          const int64_t idx = ((int64_t)img * N + n) * HW + p;
          float v = acc[x][y][i];
          if (a.accumulate) v += DX[idx];
          if (a.add_mode == ADD_SAME) {
            v += ADD[idx];
          } else if (a.add_mode == ADD_SUBSAMPLE) {
            const int ih = p / g.W, iw = p - ih * g.W;
            if (ih % a.add_st == 0 && iw % a.add_st == 0)
              v += ADD[(((int64_t)img * a.add_C + n) * Hs + ih / a.add_st) * Ws + iw / a.add_st];
          }
          if (MSK && !(MSK[idx] > 0.f)) v = 0.f;
          DX[idx] = v;
          if (bn) {
            const bool on = BY ? BY[idx] > 0.f : BG ? bn_affine(BX[idx], bm, bi, bg, bb) > 0.f : true;
            const float d = on ? v : 0.f;
            const float xh = (BX[idx] - bm) * bi;
            s1[y] += (double)d;
            s2[y] += (double)d * xh;
          }
        }
        if (++p == HW) {
          p = 0;
          ++img;
        }
      }
    }
  if (!bn) return;
  // per-channel partial sums of this tile, combined in a fixed order (lanes
  // of a column by xor butterfly, then the WM waves of a column strip)
  __shared__ double red[WM][BN][2];
  const int wm = wave % WM;
#pragma unroll
  for (int y = 0; y < TN; ++y) {
    double u = s1[y], w = s2[y];
    u += shfl_xor_d(u, 16);
    w += shfl_xor_d(w, 16);
    u += shfl_xor_d(u, 32);
    w += shfl_xor_d(w, 32);
    if (lane < 16) {
      red[wm][wn0 + y * 16 + lane][0] = u;
      red[wm][wn0 + y * 16 + lane][1] = w;
    }
  }
  __syncthreads();
  if (tid < BN && n0 + tid < N) {
    double u = 0.0, w = 0.0;
#pragma unroll
    for (int q = 0; q < WM; ++q) {
      u += red[q][tid][0];
      w += red[q][tid][1];
    }
    double* o = a.bn_part + (((int64_t)j * N + n0 + tid) * gridDim.x + tl.mt) * 2;
    o[0] = u;
    o[1] = w;
  }
}

// ---------------------------------------------------------- weight grad
// Stages of BK pixels; thread (pl, rg) loads pixel pl of the stage for the
// dY rows rg, rg+RG, ... and the im2col rows (ci, r, s) rg, rg+RG, ...
template <int BM, int BN, int WM, int WN, int R, int BK>
__global__ __launch_bounds__(256) void conv_bwd_weight_k(ConvBwdWeightArgs a) {
  constexpr int RS = R * R;
  constexpr int LDK = BK + 4;
  constexpr int TM = BM / (WM * 16), TN = BN / (WN * 16);
  constexpr int RG = 256 / BK;            // row groups
  constexpr int RA = BM / RG, RB = BN / RG;
  static_assert(RA >= 1 && RB >= 1, "tile smaller than the row groups");
  __shared__ __attribute__((aligned(16))) float As[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) float Bs[2][BN * LDK];

  const ConvGeom g = a.g;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const GemmTile tl = gemm_tile();
  const int j = tl.z / a.splits, split = tl.z - j * a.splits;
  const int HW = g.H * g.W, HoWo = g.Ho * g.Wo;
  const int Mo = g.Co, No = g.Ci * RS, L = g.b * HoWo;
  const int L0 = split * a.chunk, L1 = min(L, L0 + a.chunk);
  const int m0 = tl.mt * BM, n0 = tl.nt * BN;
  const float* X = a.x + (int64_t)j * g.b * g.Ci * HW;
  const float* DY = a.dy + (int64_t)j * g.b * g.Co * HoWo;

  const int pl = tid % BK, rg = tid / BK;
  // pixel this thread loads in the current stage, kept as (img, oh, ow)
  int pix = L0 + pl;
  int img = pix / HoWo, rem = pix - img * HoWo, oh = rem / g.Wo, ow = rem - oh * g.Wo;
  // (offset, r, s) of this thread's weight-gradient columns kk = (ci, r, s)
  int tx[RB], tr[RB], ts[RB];
#pragma unroll
  for (int i = 0; i < RB; ++i) {
    const int kk = n0 + rg + RG * i;
    const int ci = kk / RS, rs = kk - ci * RS, r = rs / R, s = rs - r * R;
    tx[i] = ci * HW + r * g.W + s;
    tr[i] = kk < No ? r : OUT_OF_RANGE;
    ts[i] = s;
  }
  float ra[RA], rb[RB];

  auto load = [&]() {
    const bool ok = pix < L1;
    const int yb = img * g.Co * HoWo + oh * g.Wo + ow;
    const int ih0 = oh * g.st - g.pad, iw0 = ow * g.st - g.pad;
    const int xb = img * g.Ci * HW + ih0 * g.W + iw0;
#pragma unroll
    for (int i = 0; i < RA; ++i) {
      const int co = m0 + rg + RG * i;
      ra[i] = (ok && co < Mo) ? DY[yb + co * HoWo] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      float v = 0.f;
      if (ok && (unsigned)(ih0 + tr[i]) < (unsigned)g.H && (unsigned)(iw0 + ts[i]) < (unsigned)g.W)
        v = X[xb + tx[i]];
      rb[i] = v;
    }
  };
  auto advance = [&]() {
    pix += BK;
    ow += BK;
    while (ow >= g.Wo) {
      ow -= g.Wo;
      if (++oh == g.Ho) {
        oh = 0;
        ++img;
      }
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < RA; ++i) As[buf][(rg + RG * i) * LDK + pl] = ra[i];
#pragma unroll
    for (int i = 0; i < RB; ++i) Bs[buf][(rg + RG * i) * LDK + pl] = rb[i];
  };

  v4f acc[TM][TN];
#pragma unroll
  for (int x = 0; x < TM; ++x)
#pragma unroll
    for (int y = 0; y < TN; ++y) acc[x][y] = v4f{0.f, 0.f, 0.f, 0.f};
  const int wm0 = (wave % WM) * TM * 16, wn0 = (wave / WM) * TN * 16;
  const int T = (L1 - L0 + BK - 1) / BK;
  load();
  store(0);
  __syncthreads();
  for (int t = 0; t < T; ++t) {
    const int cur = t & 1;
    if (t + 1 < T) {
      advance();
      load();
    }
    mma_stage<TM, TN, BK>(As[cur], Bs[cur], wm0, wn0, lane, acc);
    if (t + 1 < T) store(cur ^ 1);
    __syncthreads();
  }

  float* out = a.splits == 1 ? a.dw + (int64_t)j * a.pstride
                             : a.partial + (int64_t)(j * a.splits + split) * Mo * No;
#pragma unroll
  for (int x = 0; x < TM; ++x)
#pragma unroll
    for (int y = 0; y < TN; ++y) {
      const int n = n0 + wn0 + y * 16 + (lane & 15);
      const int mb = m0 + wm0 + x * 16 + (lane >> 4) * 4;
      if (n >= No) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (mb + i < Mo) out[(int64_t)(mb + i) * No + n] = acc[x][y][i];
    }
}

// Split reduction of several layers in one launch:
//   dw[j][e] = sum over s of partial[j][s][e], s in order,
// for every segment of the table.  A block covers 64 elements of one
// segment and one replica; its 4 waves take the splits in 4 contiguous
// runs (loads U at a time, adds in order), combined in run order.
template <int S>
__global__ __launch_bounds__(256) void reduce_splits_k(SplitTableT<S> t) {
  __shared__ float red[4][64];
  const int bx = blockIdx.x, j = blockIdx.y, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int lo = 0, hi = t.nseg - 1;  // the last segment whose first block is <= bx
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (t.seg[mid].block0 <= bx) lo = mid;
    else hi = mid - 1;
  }
  const float* part = t.seg[lo].partial;
  float* dw = t.seg[lo].dw;
  const int64_t n = t.seg[lo].n;
  const int splits = t.seg[lo].splits;
  const int64_t e = (int64_t)(bx - t.seg[lo].block0) * 64 + lane;
  const int per = (splits + 3) / 4, s0 = w * per, s1 = min(splits, s0 + per);
  float s = 0.f;
  if (e < n) {
    const float* p = part + (int64_t)j * splits * n + e;
    constexpr int U = 8;
    int i = s0;
    for (; i + U <= s1; i += U) {
      float v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = p[(int64_t)(i + u) * n];
#pragma unroll
      for (int u = 0; u < U; ++u) s += v[u];
    }
    for (; i < s1; ++i) s += p[(int64_t)i * n];
  }
  red[w][lane] = s;
  __syncthreads();
  if (w == 0 && e < n)
    dw[(int64_t)j * t.pstride + e] = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Fully connected layers (a 1x1 convolution on 1x1 images) with few inputs
// per output: the tile machinery of the implicit GEMM costs more than the
// arithmetic there.
// Forward: one wave per output y[n][co] = sum_ci x[n][ci] w[co][ci] (+ b),
// lanes over ci, a fixed-order wave sum.
__global__ __launch_bounds__(256) void fc_fwd_k(const float* x, const float* w, const float* bias,
                                                int64_t pstride, int b, int Ci, int Co, int relu,
                                                float* y) {
  const int lane = threadIdx.x & 63;
  const int64_t o = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // over k*b*Co outputs
  const int j = blockIdx.y;
  if (o >= (int64_t)b * Co) return;
  const int n = (int)(o / Co), co = (int)(o - (int64_t)n * Co);
  const float* X = x + ((int64_t)j * b + n) * Ci;
  const float* Wr = w + (int64_t)j * pstride + (int64_t)co * Ci;
  float s = 0.f;
  for (int ci = lane; ci < Ci; ci += 64) s += X[ci] * Wr[ci];
  s = wave_sum(s);
  if (lane == 0) {
    if (bias) s += bias[(int64_t)j * pstride + co];
    if (relu) s = s > 0.f ? s : 0.f;
    y[((int64_t)j * b + n) * Co + co] = s;
  }
}

// Data gradient: one thread per dX[n][ci] = sum_co dY[n][co] w[co][ci], in
// co order; then accumulate and the ReLU mask as in the GEMM epilogue.
__global__ __launch_bounds__(256) void fc_dgrad_k(const float* dy, const float* w, int64_t pstride,
                                                  int b, int Ci, int Co, int accumulate,
                                                  const float* mask, float* dx) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;  // over b*Ci of replica j
  const int j = blockIdx.y;
  if (i >= (int64_t)b * Ci) return;
  const int n = (int)(i / Ci), ci = (int)(i - (int64_t)n * Ci);
  const float* D = dy + ((int64_t)j * b + n) * Co;
  const float* Wt = w + (int64_t)j * pstride + ci;
  float s = 0.f;
  for (int co = 0; co < Co; ++co) s += D[co] * Wt[(int64_t)co * Ci];
  const int64_t g = ((int64_t)j * b + n) * Ci + ci;
  if (accumulate) s += dx[g];
  if (mask && !(mask[g] > 0.f)) s = 0.f;
  dx[g] = s;
}

// Fully connected layers of at most 64 images per replica that the kernels
// above do not take (wider layers): one workgroup per 16 outputs (forward)
// or 16 inputs (data gradient) of a replica and all its images, on fp32
// MFMA.  The 8 waves split the contraction into 8 ranges of whole 16-step
// groups, and their partial tiles are summed in wave order through LDS.
// The fragments come straight from memory: in each group a lane takes four
// consecutive steps (16 bytes of an image row; the contraction length is a
// multiple of 4, so the four are all in range or all out) and the matching
// four weights.  Out-of-range reads use OUTSIDE and read 0.
constexpr int FCM_WAVES = 8;

template <int MF>
__device__ __forceinline__ void fcm_reduce(v4f (&acc)[MF], v4f (*red)[MF][64], int wave,
                                           int lane) {
#pragma unroll
  for (int f = 0; f < MF; ++f) red[wave][f][lane] = acc[f];
  __syncthreads();
  if (wave == 0)
#pragma unroll
    for (int f = 0; f < MF; ++f) {
      v4f t = red[0][f][lane];
      for (int q = 1; q < FCM_WAVES; ++q) t += red[q][f][lane];
      acc[f] = t;
    }
}

// Forward: y[n][co] = sum_ci x[n][ci] w[co][ci] (+ bias, ReLU); MF = image
// fragments of 16.
template <int MF>
__global__ __launch_bounds__(64 * FCM_WAVES) void fc_fwd_mfma_k(const float* x, const float* w,
                                                                const float* bias,
                                                                int64_t pstride, int b, int Ci,
                                                                int Co, int relu, float* y) {
  __shared__ v4f red[FCM_WAVES][MF][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, l16 = lane & 15;
  const int q = (lane >> 4) * 4, j = blockIdx.y, co = blockIdx.x * 16 + l16;
  const __amdgpu_buffer_rsrc_t xr = buf_rsrc_u(x + (int64_t)j * b * Ci, (uint32_t)(b * Ci) * 4u);
  const __amdgpu_buffer_rsrc_t wr = buf_rsrc_u(w + (int64_t)j * pstride, (uint32_t)(Co * Ci) * 4u);
  const int groups = (Ci + 15) / 16, per = (groups + FCM_WAVES - 1) / FCM_WAVES;
  const int g0 = wave * per, g1 = min(groups, g0 + per);
  v4f acc[MF];
#pragma unroll
  for (int f = 0; f < MF; ++f) acc[f] = v4f{0.f, 0.f, 0.f, 0.f};
  for (int g = g0; g < g1; ++g) {
    const int k = g * 16 + q;  // the lane's first step
    v4f av[MF];
    float bv[4];
#pragma unroll
    for (int f = 0; f < MF; ++f) {
      const int n = f * 16 + l16;
      av[f] = buf_ld4(xr, (k < Ci && n < b) ? (uint32_t)(n * Ci + k) * 4u : OUTSIDE);
    }
    const uint32_t wo = (k < Ci && co < Co) ? (uint32_t)(co * Ci + k) * 4u : OUTSIDE;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) bv[kk] = buf_ld(wr, wo == OUTSIDE ? OUTSIDE : wo + 4u * kk);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int f = 0; f < MF; ++f) acc[f] = mfma4(av[f][kk], bv[kk], acc[f]);
  }
  fcm_reduce<MF>(acc, red, wave, lane);
  if (wave != 0 || co >= Co) return;
  const float bb = bias ? bias[(int64_t)j * pstride + co] : 0.f;
#pragma unroll
  for (int f = 0; f < MF; ++f)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int n = f * 16 + q + i;
      if (n >= b) continue;
      float v = acc[f][i] + bb;
      if (relu) v = v > 0.f ? v : 0.f;
      y[((int64_t)j * b + n) * Co + co] = v;
    }
}

// Data gradient: dx[n][ci] = sum_co dy[n][co] w[co][ci], then accumulate
// and the ReLU mask as in the GEMM epilogue.
template <int MF>
__global__ __launch_bounds__(64 * FCM_WAVES) void fc_dgrad_mfma_k(const float* dy, const float* w,
                                                                  int64_t pstride, int b, int Ci,
                                                                  int Co, int accumulate,
                                                                  const float* mask, float* dx) {
  __shared__ v4f red[FCM_WAVES][MF][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, l16 = lane & 15;
  const int q = (lane >> 4) * 4, j = blockIdx.y, ci = blockIdx.x * 16 + l16;
  const __amdgpu_buffer_rsrc_t dr = buf_rsrc_u(dy + (int64_t)j * b * Co, (uint32_t)(b * Co) * 4u);
  const __amdgpu_buffer_rsrc_t wr = buf_rsrc_u(w + (int64_t)j * pstride, (uint32_t)(Co * Ci) * 4u);
  const int groups = (Co + 15) / 16, per = (groups + FCM_WAVES - 1) / FCM_WAVES;
  const int g0 = wave * per, g1 = min(groups, g0 + per);
  v4f acc[MF];
#pragma unroll
  for (int f = 0; f < MF; ++f) acc[f] = v4f{0.f, 0.f, 0.f, 0.f};
  for (int g = g0; g < g1; ++g) {
    const int k = g * 16 + q;  // the lane's first output channel
    v4f av[MF];
    float bv[4];
#pragma unroll
    for (int f = 0; f < MF; ++f) {
      const int n = f * 16 + l16;
      av[f] = buf_ld4(dr, (k < Co && n < b) ? (uint32_t)(n * Co + k) * 4u : OUTSIDE);
    }
    const uint32_t wo = (k < Co && ci < Ci) ? (uint32_t)(k * Ci + ci) * 4u : OUTSIDE;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      bv[kk] = buf_ld(wr, wo == OUTSIDE ? OUTSIDE : wo + (uint32_t)(kk * Ci) * 4u);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int f = 0; f < MF; ++f) acc[f] = mfma4(av[f][kk], bv[kk], acc[f]);
  }
  fcm_reduce<MF>(acc, red, wave, lane);
  if (wave != 0 || ci >= Ci) return;
#pragma unroll
  for (int f = 0; f < MF; ++f)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int n = f * 16 + q + i;
      if (n >= b) continue;
      const int64_t gi = ((int64_t)j * b + n) * Ci + ci;
      float v = acc[f][i];
      if (accumulate) v += dx[gi];
      if (mask && !(mask[gi] > 0.f)) v = 0.f;
      dx[gi] = v;
    }
}

// db[j][c]: one block per (c, j), fixed-order reduction.
__global__ __launch_bounds__(256) void channel_sum_k(const float* dy, int b, int C, int HW,
                                                     float* db, int64_t pstride,
                                                     const float* terms, float* mean) {
  __shared__ float red[4];
  const int c = blockIdx.x, j = blockIdx.y;
  const int n = b * HW;
  float s = 0.f;
  for (int e = threadIdx.x; e < n; e += 256) {
    const int img = e / HW, p = e - img * HW;
    s += dy[((int64_t)(j * b + img) * C + c) * HW + p];
  }
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) db[(int64_t)j * pstride + c] = (red[0] + red[1]) + (red[2] + red[3]);
  if (terms && c == 0 && threadIdx.x == 0) {
    // the replica's mean loss (Eq. 2) from its b per-image terms, in order
    double t = 0.0;
    for (int i = 0; i < b; ++i) t += (double)terms[(int64_t)j * b + i];
    mean[j] = (float)(t / b);
  }
}

inline unsigned cdiv(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }

// Name of one kernel instantiation, as the profiler shows its template.
template <int KIND, int BM, int BN, int WM, int WN, int R, int ST, int BK>
const char* tile_name() {
  // KIND 3: the grid-only data gradient (SP = true)
  static const char* base[4] = {"conv_fwd_k", "conv_bwd_data_k", "conv_bwd_weight_k",
                                "conv_bwd_data_k"};
  static const std::string n = std::string(base[KIND]) + "<" + std::to_string(BM) + ", " +
                               std::to_string(BN) + ", " + std::to_string(WM) + ", " +
                               std::to_string(WN) + ", " + std::to_string(R) +
                               (ST ? ", " + std::to_string(ST) : "") + ", " +
                               std::to_string(BK) + (KIND == 3 ? ", true>" : ">");
  return n.c_str();
}

// LDS stage depth: 32 contraction steps, 16 for tiles of 128 rows or more
// (the 1x1 stride-2 grid-only data gradient from 256 rows: its 128-row
// tiles measured slower with 16).  The shallow stage halves the LDS of a
// 128 x 64 tile (32 KB), so five workgroups share a CU instead of two, and
// one workgroup's epilogue traffic overlaps the others' MFMAs (ResNet-50
// k=2 b=32: 1x1 data gradients 147 -> 130 us, 1x1 forward 104 -> 96 us, 3x3
// data gradients 252 -> 228 us; with the tap-major loaders the 3x3 forward
// 211 -> 206 us).
template <int BM, bool SP = false>
constexpr int stage_k() { return BM >= 256 || (BM >= 128 && !SP) ? 16 : 32; }

template <int BM, int BN, int WM, int WN, int R>
hipError_t launch_fwd(const ConvFwdArgs& a, hipStream_t s, const char** name) {
  constexpr int BK = stage_k<BM>();
  const int M = a.g.b * a.g.Ho * a.g.Wo;
  dim3 grid(cdiv(M, BM), cdiv(a.g.Co, BN), a.g.k);
  if (a.g.Ci % BK == 0) {
    klaunch((conv_fwd_k<BM, BN, WM, WN, R, BK, true>), grid, dim3(256), 0, s, a);
    if (name) {
      static const std::string n = std::string(tile_name<0, BM, BN, WM, WN, R, 0, BK>()) + " tap-major";
      *name = n.c_str();
    }
    return hipGetLastError();
  }
  klaunch((conv_fwd_k<BM, BN, WM, WN, R, BK>), grid, dim3(256), 0, s, a);
  if (name) *name = tile_name<0, BM, BN, WM, WN, R, 0, BK>();
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, int R, int ST, bool SP = false>
hipError_t launch_bwd_data(const ConvBwdDataArgs& a, hipStream_t s, const char** name) {
  constexpr int BK = stage_k<BM, SP>();
  const int M = SP ? a.g.b * a.g.Ho * a.g.Wo : a.g.b * a.g.H * a.g.W;
  dim3 grid(cdiv(M, BM), cdiv(a.g.Ci, BN), a.g.k);
  if constexpr (ST == 1 || SP) {
    if (a.g.Co % BK == 0) {
      klaunch((conv_bwd_data_k<BM, BN, WM, WN, R, ST, BK, SP, true>), grid, dim3(256), 0, s, a);
      if (name) {
        static const std::string n =
            std::string(SP ? tile_name<3, BM, BN, WM, WN, R, ST, BK>() : tile_name<1, BM, BN, WM, WN, R, ST, BK>()) +
            " tap-major";
        *name = n.c_str();
      }
      return hipGetLastError();
    }
  }
  klaunch((conv_bwd_data_k<BM, BN, WM, WN, R, ST, BK, SP>), grid, dim3(256), 0, s, a);
  if (name) *name = SP ? tile_name<3, BM, BN, WM, WN, R, ST, BK>() : tile_name<1, BM, BN, WM, WN, R, ST, BK>();
  return hipGetLastError();
}

constexpr int WG_BK = 32;  // pixels per stage of the weight gradient

// 128-row tiles stage 16 pixels (30 KB of LDS, five workgroups per CU);
// the others 32.  Split chunks are whole multiples of WG_BK either way.
template <int BM, int BN, int WM, int WN, int R>
hipError_t launch_bwd_weight(const ConvBwdWeightArgs& a, hipStream_t s, const char** name) {
  constexpr int BK = BM >= 128 ? 16 : WG_BK;
  dim3 grid(cdiv(a.g.Co, BM), cdiv(a.g.Ci * R * R, BN), a.g.k * a.splits);
  klaunch((conv_bwd_weight_k<BM, BN, WM, WN, R, BK>), grid, dim3(256), 0, s, a);
  if (name) *name = tile_name<2, BM, BN, WM, WN, R, 0, BK>();
  return hipGetLastError();
}

// Output rows per weight-gradient tile: 128 for 1x1 filters from 128 output
// channels (its waves hold 64 x 32 outputs, half the LDS reads per MFMA of
// 32 x 32; ResNet-50's 1x1 weight gradients 98 -> 93 us per launch, while
// its 3x3 ones measured 236 -> 305 us and keep 64).
int bwd_weight_bm(int Co, int R) {
  return Co <= 16 ? 16 : (Co <= 32 ? 32 : (Co < 128 || R > 1 ? 64 : 128));
}

// Enough workgroups to give every CU at least two.
constexpr int64_t MIN_WGS = 512;

// Output-tile choice for the forward / data-gradient GEMM (M x N per
// replica): the biggest tile of the N class that still yields MIN_WGS
// workgroups over all replicas, else the smallest.  For N > 32 the
// 128 x 64 tile is kept down to MIN_WGS / 4 workgroups: its waves hold
// 64 x 32 outputs and read half the LDS bytes per MFMA of the 64 x 64
// tile's 32 x 32, which at 3-4 workgroups per CU is the limit (ResNet-50
// k=2 b=32: the 14 x 14 and 7 x 7 stages' 3 x 3 convolutions 325-375 ->
// 210-250 us, the step 30.8 -> 29.3 ms).  Returns 0..5:
//   0 (256,16)  1 (64,16)  2 (128,32)  3 (64,32)  4 (128,64)  5 (64,64)
int pick_tile(int64_t M, int N, int k) {
  auto wgs = [&](int bm, int bn) { return (int64_t)cdiv(M, bm) * cdiv(N, bn) * k; };
  if (N <= 16) return wgs(256, 16) >= MIN_WGS ? 0 : 1;
  if (N <= 32) return wgs(128, 32) >= MIN_WGS ? 2 : 3;
  if (wgs(128, 64) >= MIN_WGS / 4) return 4;
  // under one workgroup per CU even at 64 x 64: 16-column tiles (same rows)
  return wgs(64, 64) >= MIN_WGS / 2 ? 5 : 1;
}

int tile_rows(int t) {
  static const int rows[6] = {256, 64, 128, 64, 128, 64};
  return rows[t];
}

template <int R>
hipError_t fwd_r(const ConvFwdArgs& a, hipStream_t s, const char** name) {
  switch (pick_tile((int64_t)a.g.b * a.g.Ho * a.g.Wo, a.g.Co, a.g.k)) {
    case 0: return launch_fwd<256, 16, 4, 1, R>(a, s, name);
    case 1: return launch_fwd<64, 16, 4, 1, R>(a, s, name);
    case 2: return launch_fwd<128, 32, 4, 1, R>(a, s, name);
    case 3: return launch_fwd<64, 32, 4, 1, R>(a, s, name);
    case 4: return launch_fwd<128, 64, 2, 2, R>(a, s, name);
    default: return launch_fwd<64, 64, 2, 2, R>(a, s, name);
  }
}

template <int R, int ST, bool SP = false>
hipError_t bwd_data_r(const ConvBwdDataArgs& a, hipStream_t s, const char** name) {
  const int64_t M = SP ? (int64_t)a.g.b * a.g.Ho * a.g.Wo : (int64_t)a.g.b * a.g.H * a.g.W;
  switch (pick_tile(M, a.g.Ci, a.g.k)) {
    case 0: return launch_bwd_data<256, 16, 4, 1, R, ST, SP>(a, s, name);
    case 1: return launch_bwd_data<64, 16, 4, 1, R, ST, SP>(a, s, name);
    case 2: return launch_bwd_data<128, 32, 4, 1, R, ST, SP>(a, s, name);
    case 3: return launch_bwd_data<64, 32, 4, 1, R, ST, SP>(a, s, name);
    case 4: return launch_bwd_data<128, 64, 2, 2, R, ST, SP>(a, s, name);
    default: return launch_bwd_data<64, 64, 2, 2, R, ST, SP>(a, s, name);
  }
}

// The 1x1 stride-2 data gradient on the Ho x Wo grid only (see
// conv_bwd_data_k): even planes, 8-byte aligned pixel pairs.
bool s2_grid_ok(const ConvGeom& g) {
  return g.R == 1 && g.S == 1 && g.st == 2 && g.pad == 0 && g.H % 2 == 0 && g.W % 2 == 0 &&
         g.Ho == g.H / 2 && g.Wo == g.W / 2;
}

template <int R>
hipError_t bwd_weight_r(const ConvBwdWeightArgs& a, hipStream_t s, const char** name) {
  switch (bwd_weight_bm(a.g.Co, R)) {
    case 16: return launch_bwd_weight<16, 64, 1, 4, R>(a, s, name);
    case 32: return launch_bwd_weight<32, 64, 2, 2, R>(a, s, name);
    case 64: return launch_bwd_weight<64, 64, 2, 2, R>(a, s, name);
    default: return launch_bwd_weight<128, 64, 2, 2, R>(a, s, name);
  }
}

}  // namespace

inline bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }
inline bool al8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7) == 0; }

int conv_fwd_tiles_m(const ConvGeom& g) {
  if (conv_direct_fwd_ok(g)) return conv_direct_fwd_tiles(g);
  const int64_t M = (int64_t)g.b * g.Ho * g.Wo;
  return (int)cdiv(M, tile_rows(pick_tile(M, g.Co, g.k)));
}

int conv_bwd_data_tiles_m(const ConvGeom& g) {
  if (conv_direct_bwd_data_ok(g)) return conv_direct_bwd_data_tiles(g);
  if (conv_s2_dgrad_ok(g)) return conv_s2_dgrad_tiles(g);
  const int64_t M = s2_grid_ok(g) ? (int64_t)g.b * g.Ho * g.Wo : (int64_t)g.b * g.H * g.W;
  return (int)cdiv(M, tile_rows(pick_tile(M, g.Ci, g.k)));
}

int conv_bwd_weight_splits(const ConvGeom& g, int* chunk) {
  if (conv_direct_wgrad_ok(g)) {
    *chunk = 0;
    return conv_direct_wgrad_splits(g);
  }
  const int L = g.b * g.Ho * g.Wo;
  const int bm = bwd_weight_bm(g.Co, g.R);
  const int64_t tiles = (int64_t)cdiv(g.Co, bm) * cdiv(g.Ci * g.R * g.S, 64) * g.k;
  // about 1024 workgroups (512 of the 128-row tiles: the same partials)
  const int64_t target = bm >= 128 ? 512 : 1024;
  int splits = (int)std::max<int64_t>(1, std::min<int64_t>(cdiv(L, 2 * WG_BK), cdiv(target, tiles)));
  int c = (int)cdiv(L, splits);
  c = (c + WG_BK - 1) / WG_BK * WG_BK;
  *chunk = c;
  return (int)cdiv(L, c);
}

bool conv_supported(int R, int S, int st, bool need_dx) {
  if (R != S || st < 1 || st > 2) return false;
  if (R == 1 || R == 3) return true;
  if (R == 5) return !need_dx || st == 1;
  if (R == 7) return !need_dx;
  return false;
}

// The FC kernels take layers with at most FC_MAX_K inputs per output
// (forward) or FC_MAX_DK outputs per input (data gradient), without fused
// BN partials.
constexpr int FC_MAX_K = 1024, FC_MAX_DK = 256;

bool fc_layer(const ConvGeom& g) {
  return g.R == 1 && g.S == 1 && g.H == 1 && g.W == 1 && g.st == 1 && g.pad == 0;
}

// The MFMA FC kernels: at most 64 images per replica, a contraction length
// (klen) that is a multiple of 4, and every operand within the 32-bit byte
// offsets of one buffer descriptor.
bool fc_mfma_ok(const ConvGeom& g, int klen, int other) {
  return fc_layer(g) && g.b >= 1 && g.b <= 64 && klen % 4 == 0 &&
         (int64_t)klen * other * 4 < (int64_t)OUTSIDE && (int64_t)g.b * klen * 4 < (int64_t)OUTSIDE;
}
int fc_mfma_frags(int b) { return b <= 16 ? 1 : (b <= 32 ? 2 : 4); }

hipError_t conv_fwd(const ConvFwdArgs& a, hipStream_t s, const char** name) {
  if (fc_layer(a.g) && !a.stats && a.g.Ci <= FC_MAX_K) {
    const int64_t outs = (int64_t)a.g.b * a.g.Co;
    klaunch(fc_fwd_k, dim3(cdiv(outs, 4), a.g.k), dim3(256), 0, s, a.x, a.w, a.bias, a.pstride,
            a.g.b, a.g.Ci, a.g.Co, a.relu, a.y);
    if (name) *name = "fc_fwd_k";
    return hipGetLastError();
  }
  if (fc_mfma_ok(a.g, a.g.Ci, a.g.Co) && !a.stats && al16(a.x)) {
    const dim3 grid(cdiv(a.g.Co, 16), a.g.k), block(64 * FCM_WAVES);
    const int mf = fc_mfma_frags(a.g.b);
    if (name) *name = mf == 1 ? "fc_fwd_mfma_k<1>" : mf == 2 ? "fc_fwd_mfma_k<2>" : "fc_fwd_mfma_k<4>";
    if (mf == 1)
      klaunch(fc_fwd_mfma_k<1>, grid, block, 0, s, a.x, a.w, a.bias, a.pstride, a.g.b, a.g.Ci, a.g.Co, a.relu, a.y);
    else if (mf == 2)
      klaunch(fc_fwd_mfma_k<2>, grid, block, 0, s, a.x, a.w, a.bias, a.pstride, a.g.b, a.g.Ci, a.g.Co, a.relu, a.y);
    else
      klaunch(fc_fwd_mfma_k<4>, grid, block, 0, s, a.x, a.w, a.bias, a.pstride, a.g.b, a.g.Ci, a.g.Co, a.relu, a.y);
    return hipGetLastError();
  }
  // the direct kernel moves its outputs in 16-byte pieces (workspace
  // tensors are 256-byte aligned, so layers of a plan always qualify)
  if (conv_direct_fwd_ok(a.g) && al16(a.y)) return conv_direct_fwd(a, s, name);
  switch (a.g.R) {
    case 1: return fwd_r<1>(a, s, name);
    case 3: return fwd_r<3>(a, s, name);
    case 5: return fwd_r<5>(a, s, name);
    case 7: return fwd_r<7>(a, s, name);
    default: return hipErrorInvalidValue;
  }
}

hipError_t conv_bwd_data(const ConvBwdDataArgs& a, hipStream_t s, const char** name) {
  if (fc_layer(a.g) && !a.bn_part && a.add_mode == ADD_NONE && a.g.Co <= FC_MAX_DK) {
    klaunch(fc_dgrad_k, dim3(cdiv((int64_t)a.g.b * a.g.Ci, 256), a.g.k), dim3(256), 0, s, a.dy,
            a.w, a.pstride, a.g.b, a.g.Ci, a.g.Co, a.accumulate, a.mask, a.dx);
    if (name) *name = "fc_dgrad_k";
    return hipGetLastError();
  }
  if (fc_mfma_ok(a.g, a.g.Co, a.g.Ci) && !a.bn_part && a.add_mode == ADD_NONE && al16(a.dy)) {
    const dim3 grid(cdiv(a.g.Ci, 16), a.g.k), block(64 * FCM_WAVES);
    const int mf = fc_mfma_frags(a.g.b);
    if (name)
      *name = mf == 1 ? "fc_dgrad_mfma_k<1>" : mf == 2 ? "fc_dgrad_mfma_k<2>" : "fc_dgrad_mfma_k<4>";
    if (mf == 1)
      klaunch(fc_dgrad_mfma_k<1>, grid, block, 0, s, a.dy, a.w, a.pstride, a.g.b, a.g.Ci, a.g.Co, a.accumulate, a.mask, a.dx);
    else if (mf == 2)
      klaunch(fc_dgrad_mfma_k<2>, grid, block, 0, s, a.dy, a.w, a.pstride, a.g.b, a.g.Ci, a.g.Co, a.accumulate, a.mask, a.dx);
    else
      klaunch(fc_dgrad_mfma_k<4>, grid, block, 0, s, a.dy, a.w, a.pstride, a.g.b, a.g.Ci, a.g.Co, a.accumulate, a.mask, a.dx);
    return hipGetLastError();
  }
  const bool vec_ok = al16(a.dx) && al16(a.mask) && al16(a.bn_x) && al16(a.bn_y) && al16(a.add);
  if (conv_direct_bwd_data_ok(a.g) && vec_ok) return conv_direct_bwd_data(a, s, name);
  if (conv_s2_dgrad_ok(a.g) && vec_ok && (a.add_mode != ADD_SUBSAMPLE || a.add_st == 2))
    return conv_s2_dgrad(a, s, name);
  const int key = a.g.R * 10 + a.g.st;
  switch (key) {
    case 11: return bwd_data_r<1, 1>(a, s, name);
    case 12:
      if (s2_grid_ok(a.g)) {
        // the batch-norm partials are laid out for the grid's tiles
        if (!(al8(a.dx) && al8(a.mask) && al8(a.bn_x) && al8(a.bn_y) &&
              (a.add_mode != ADD_SAME || al8(a.add))))
          return hipErrorInvalidValue;
        return bwd_data_r<1, 2, true>(a, s, name);
      }
      return bwd_data_r<1, 2>(a, s, name);
    case 31: return bwd_data_r<3, 1>(a, s, name);
    case 32: return bwd_data_r<3, 2>(a, s, name);
    case 51: return bwd_data_r<5, 1>(a, s, name);
    default: return hipErrorInvalidValue;
  }
}

hipError_t conv_bwd_weight(const ConvBwdWeightArgs& a, hipStream_t s, const char** name) {
  if (conv_direct_wgrad_ok(a.g))  // reads dY in 16-byte pieces
    return al16(a.dy) ? conv_direct_wgrad(a, s, name) : hipErrorInvalidValue;
  switch (a.g.R) {
    case 1: return bwd_weight_r<1>(a, s, name);
    case 3: return bwd_weight_r<3>(a, s, name);
    case 5: return bwd_weight_r<5>(a, s, name);
    case 7: return bwd_weight_r<7>(a, s, name);
    default: return hipErrorInvalidValue;
  }
}

static_assert(SMALL_SPLIT_SEGS == 4 && MAX_SPLIT_SEGS == 80, "the kernel names below");
hipError_t reduce_splits(const SplitTable& t, int k, hipStream_t s, const char** name) {
  if (t.nseg < 1 || t.nseg > MAX_SPLIT_SEGS) return hipErrorInvalidValue;
  if (t.nseg <= SMALL_SPLIT_SEGS) {
    SplitTableT<SMALL_SPLIT_SEGS> u;
    u.nseg = t.nseg;
    u.blocks = t.blocks;
    u.pstride = t.pstride;
    for (int i = 0; i < t.nseg; ++i) u.seg[i] = t.seg[i];
    klaunch(reduce_splits_k<SMALL_SPLIT_SEGS>, dim3(u.blocks, k), dim3(256), 0, s, u);
    if (name) *name = "reduce_splits_k<4>";
  } else {
    klaunch(reduce_splits_k<MAX_SPLIT_SEGS>, dim3(t.blocks, k), dim3(256), 0, s, t);
    if (name) *name = "reduce_splits_k<80>";
  }
  return hipGetLastError();
}

void split_table_add(SplitTable& t, const float* partial, float* dw, int64_t n, int splits) {
  SplitSeg& g = t.seg[t.nseg++];
  g.partial = partial;
  g.dw = dw;
  g.n = n;
  g.splits = splits;
  g.block0 = t.blocks;
  t.blocks += (int)cdiv(n, 64);
}

hipError_t channel_sum(const float* dy, int k, int b, int C, int HW, float* db, int64_t pstride,
                       hipStream_t s, const float* terms, float* mean) {
  klaunch(channel_sum_k, dim3(C, k), dim3(256), 0, s, dy, b, C, HW, db, pstride, terms, mean);
  return hipGetLastError();
}

}  // namespace cbk
