// conv_direct.hip -- 3x3, stride 1, pad 1 convolutions (forward and data
// gradient) with the input tile staged once in LDS.
//
// The implicit GEMM gathers every input pixel nine times (once per filter
// tap) from the caches.  Here a workgroup computes TH full output rows of one
// image for BN output channels: it stages CC input channels of the TH+2
// rows (with a zero border) in LDS, then every filter tap is an LDS read at a
// constant offset from the lane's pixel.  The contraction runs on
// v_mfma_f32_16x16x4f32: per MFMA the four lane groups (lane / 16) take four
// consecutive input channels of the same tap; 16 consecutive output pixels
// are the rows of the 16x16 block and 16 output channels its columns.
//
// The data gradient of such a convolution (Sec. 2.1, backward pass) is the
// same operation on dY with the filter transposed in its channels and
// rotated by 180 degrees, which the weight loader applies (FLIP).
//
// Grid: x = row tiles of one replica (b * H / TH), y = output-channel tiles,
// z = replica.  Epilogues match the implicit GEMM's: bias, ReLU and the
// batch-norm partial sums of the forward; accumulate, residual add, ReLU
// mask and the batch-norm backward partial sums of the data gradient.
#include "kernels.hpp"

#include <string>

namespace cbk {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4f mfma4(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ double shfl_xor_d(double v, int o) { return __shfl_xor(v, o, 64); }

// Channel stride of the LDS input tile, rounded so that the four lane groups
// of a wave fall in distinct 16-bank ranges.
constexpr int pad_cs(int n) { return ((n + 47) / 64) * 64 + 16; }

struct DirectArgs {
  int k, b, H;           // replicas, images per replica, image height (= width WW)
  int Cin, Cout;         // channels of the operand read and of the result
  const float* in;       // [k*b][Cin][H][W]: x (forward) or dY (data gradient)
  const float* w;        // replica 0 filter [Co][Ci][3][3] of the convolution
  int64_t pstride;
  float* out;            // [k*b][Cout][H][W]
  // forward epilogue
  const float* bias;
  int relu;
  double* stats;
  // data-gradient epilogue (see ConvBwdDataArgs)
  int accumulate;
  const float* mask;
  const float* add;
  int add_mode, add_C, add_st;
  double* bn_part;
  const float* bn_x;
  const float* bn_y;
  const float* bn_mean;
  const float* bn_istd;
};

template <int WW, int TH, int BN, int CC, bool FLIP>
__global__ __launch_bounds__(256) void conv3x3_k(DirectArgs a) {
  constexpr int WP = WW + 2, HR = TH + 2;
  constexpr int CS = pad_cs(HR * WP);     // LDS channel stride of the input tile
  constexpr int M = TH * WW;              // output pixels per tile
  constexpr int TM = M / 64;              // 16-pixel blocks per wave (waves split M)
  constexpr int TN = BN / 16;
  // Filter tile in LDS: [tap][ci][BN].  With BN = 32, odd input channels
  // keep their two 16-column halves swapped, so the four lane groups of a
  // read (four consecutive ci) do not pair up on the same banks.
  constexpr int SWZ = BN == 32 ? 16 : 0;
  constexpr int NX = CC * HR * WP;        // input-tile elements per chunk
  constexpr int NXT = (NX + 255) / 256;
  constexpr int NW = 9 * CC * BN;         // filter elements per chunk
  constexpr int NWT = (NW + 255) / 256;
  static_assert(TM >= 1 && M % 64 == 0, "tile must cover whole 64-pixel wave strips");
  __shared__ __attribute__((aligned(16))) float xs[2][CC * CS];
  __shared__ __attribute__((aligned(16))) float ws[2][9 * CC * BN];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, kq = lane >> 4;
  const int j = blockIdx.z, H = a.H, HW = H * WW;
  const int tiles_img = H / TH;
  const int img = blockIdx.x / tiles_img, oh0 = (blockIdx.x - img * tiles_img) * TH;
  const int co0 = blockIdx.y * BN;
  const int n_img = j * a.b + img;
  const float* IN = a.in + (int64_t)n_img * a.Cin * HW;
  const float* Wt = a.w + (int64_t)j * a.pstride;
  const int nchunk = a.Cin / CC;

  float rx[NXT], rw[NWT];
  int rs[NWT];
  auto load = [&](int c0) {
#pragma unroll
    for (int u = 0; u < NXT; ++u) {
      const int e = tid + u * 256;
      float v = 0.f;
      if (e < NX) {
        const int ci = e / (HR * WP), rem = e - ci * (HR * WP), hr = rem / WP, wc = rem - hr * WP;
        const int ih = oh0 - 1 + hr, iw = wc - 1;
        if ((unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)WW)
          v = IN[(int64_t)(c0 + ci) * HW + ih * WW + iw];
      }
      rx[u] = v;
    }
#pragma unroll
    for (int u = 0; u < NWT; ++u) {
      // e runs in memory order of the filter (tap fastest), so a wave's
      // loads are contiguous; the slot keeps the [tap][ci][co] LDS order
      const int e = tid + u * 256;
      float v = 0.f;
      int slot = 0;
      if (e < NW) {
        if (!FLIP) {  // filter [out = co0+co][in = c0+ci][tap]
          const int co = e / (CC * 9), rem = e - co * (CC * 9), ci = rem / 9, tap = rem - ci * 9;
          v = Wt[((int64_t)(co0 + co) * a.Cin + c0 + ci) * 9 + tap];
          slot = (tap * CC + ci) * BN + (co ^ ((ci & 1) ? SWZ : 0));
        } else {      // original filter [its out = c0+ci][its in = co0+co][8 - tap]
          const int ci = e / (BN * 9), rem = e - ci * (BN * 9), co = rem / 9, t = rem - co * 9;
          v = Wt[((int64_t)(c0 + ci) * a.Cout + co0 + co) * 9 + t];
          slot = ((8 - t) * CC + ci) * BN + (co ^ ((ci & 1) ? SWZ : 0));
        }
      }
      rw[u] = v;
      rs[u] = slot;
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int u = 0; u < NXT; ++u) {
      const int e = tid + u * 256;
      if (e < NX) {
        const int ci = e / (HR * WP), rem = e - ci * (HR * WP);
        xs[buf][ci * CS + rem] = rx[u];
      }
    }
#pragma unroll
    for (int u = 0; u < NWT; ++u)
      if (tid + u * 256 < NW) ws[buf][rs[u]] = rw[u];
  };

  // lane bases: pixel of each of this wave's 16-pixel blocks, and column
  int xbase[TM];
#pragma unroll
  for (int t = 0; t < TM; ++t) {
    const int m = (wave * TM + t) * 16 + (lane & 15);
    const int ohl = m / WW, ow = m - ohl * WW;
    xbase[t] = kq * CS + ohl * WP + ow;
  }
  const int wbase = kq * BN + (lane & 15);
  const int wswz = (kq & 1) ? SWZ : 0;

  v4f acc[TM][TN];
#pragma unroll
  for (int x = 0; x < TM; ++x)
#pragma unroll
    for (int y = 0; y < TN; ++y) acc[x][y] = v4f{0.f, 0.f, 0.f, 0.f};

  load(0);
  store(0);
  __syncthreads();
  for (int c = 0; c < nchunk; ++c) {
    const int cur = c & 1;
    if (c + 1 < nchunk) load((c + 1) * CC);
    const float* X = xs[cur];
    const float* Wl = ws[cur];
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) {
      const int r = tap / 3, s = tap - r * 3;
#pragma unroll
      for (int cg = 0; cg < CC / 4; ++cg) {
        float av[TM], bv[TN];
#pragma unroll
        for (int t = 0; t < TM; ++t) av[t] = X[xbase[t] + cg * 4 * CS + r * WP + s];
#pragma unroll
        for (int u = 0; u < TN; ++u) bv[u] = Wl[wbase + (tap * CC + cg * 4) * BN + ((u * 16) ^ wswz)];
#pragma unroll
        for (int t = 0; t < TM; ++t)
#pragma unroll
          for (int u = 0; u < TN; ++u) acc[t][u] = mfma4(av[t], bv[u], acc[t][u]);
      }
    }
    if (c + 1 < nchunk) store(cur ^ 1);
    __syncthreads();
  }

  // epilogue: acc[t][u][i] is pixel (wave*TM + t)*16 + 4*kq + i, channel
  // co0 + u*16 + (lane & 15) of this tile -- four consecutive pixels of one
  // channel per lane, so every operand moves as one 16-byte access
  float* OUT = a.out + (int64_t)n_img * a.Cout * HW;
  double s1[TN], s2[TN];
#pragma unroll
  for (int u = 0; u < TN; ++u) s1[u] = s2[u] = 0.0;
#pragma unroll
  for (int u = 0; u < TN; ++u) {
    const int co = co0 + u * 16 + (lane & 15);
    float bv = 0.f, bm = 0.f, bi = 0.f;
    if (!FLIP && a.bias) bv = a.bias[(int64_t)j * a.pstride + co];
    if (FLIP && a.bn_part) {
      bm = a.bn_mean[j * a.Cout + co];
      bi = a.bn_istd[j * a.Cout + co];
    }
#pragma unroll
    for (int t = 0; t < TM; ++t) {
      const int p0 = oh0 * WW + (wave * TM + t) * 16 + 4 * kq;  // first pixel in the plane
      const int64_t idx = (int64_t)co * HW + p0;
      v4f v = acc[t][u];
      if (!FLIP) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float e = v[i] + bv;
          if (a.relu) e = e > 0.f ? e : 0.f;
          v[i] = e;
          s1[u] += (double)e;
          s2[u] += (double)e * e;
        }
        *reinterpret_cast<v4f*>(OUT + idx) = v;
      } else {
        const int64_t gidx = (int64_t)n_img * a.Cout * HW + idx;
        if (a.accumulate) v += *reinterpret_cast<const v4f*>(OUT + idx);
        if (a.add_mode == ADD_SAME) {
          v += *reinterpret_cast<const v4f*>(a.add + gidx);
        } else if (a.add_mode == ADD_SUBSAMPLE) {
          const int st = a.add_st;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int p = p0 + i, ih = p / WW, iw = p - ih * WW;
            if (ih % st == 0 && iw % st == 0)
              v[i] += a.add[(((int64_t)n_img * a.add_C + co) * (H / st) + ih / st) * (WW / st) +
                            iw / st];
          }
        }
        if (a.mask) {
          const v4f m = *reinterpret_cast<const v4f*>(a.mask + gidx);
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (!(m[i] > 0.f)) v[i] = 0.f;
        }
        *reinterpret_cast<v4f*>(OUT + idx) = v;
        if (a.bn_part) {
          const v4f xv = *reinterpret_cast<const v4f*>(a.bn_x + gidx);
          v4f yv = v4f{1.f, 1.f, 1.f, 1.f};
          if (a.bn_y) yv = *reinterpret_cast<const v4f*>(a.bn_y + gidx);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float d = (yv[i] > 0.f) ? v[i] : 0.f;
            const float xh = (xv[i] - bm) * bi;
            s1[u] += (double)d;
            s2[u] += (double)d * xh;
          }
        }
      }
    }
  }
  double* part = FLIP ? a.bn_part : a.stats;
  if (!part) return;
  // per-channel partial sums of the tile: lanes of a column by xor
  // butterfly, then the four waves in order
  __shared__ double red[4][BN][2];
#pragma unroll
  for (int u = 0; u < TN; ++u) {
    double x = s1[u], y = s2[u];
    x += shfl_xor_d(x, 16);
    y += shfl_xor_d(y, 16);
    x += shfl_xor_d(x, 32);
    y += shfl_xor_d(y, 32);
    if (lane < 16) {
      red[wave][u * 16 + lane][0] = x;
      red[wave][u * 16 + lane][1] = y;
    }
  }
  __syncthreads();
  if (tid < BN) {
    const double x = ((red[0][tid][0] + red[1][tid][0]) + red[2][tid][0]) + red[3][tid][0];
    const double y = ((red[0][tid][1] + red[1][tid][1]) + red[2][tid][1]) + red[3][tid][1];
    double* o = part + (((int64_t)j * a.Cout + co0 + tid) * gridDim.x + blockIdx.x) * 2;
    o[0] = x;
    o[1] = y;
  }
}

// Weight gradient of the same convolutions:
//   dW[co][ci][r][s] = sum over the replica's images n and pixels p of
//                      dY[n][co][p] * X[n][ci][p + (r - 1, s - 1)].
// A workgroup owns one 16 x 16 block of (co, ci) and all nine taps, and a
// run of "units" (TH full rows of one image).  Per unit it stages dY
// [16][TH*WW] and the X rows with their halo [16][TH+2][WW+2] in LDS once;
// every tap then reads X at a constant offset.  MFMA: rows = co (A = dY),
// columns = ci (B = X), contraction = 4 consecutive pixels of one row.  The
// four waves take interleaved 4-pixel steps and their partial sums are
// added in wave order; the result goes to dw (one split) or to the split's
// slot of `partial` for the fixed-order split reduction.
struct WgradArgs {
  int k, b, H;
  int Ci, Co;
  const float* x;   // [k*b][Ci][H][W]
  const float* dy;  // [k*b][Co][H][W]
  float* dw;        // replica 0 gradient [Co][Ci][3][3] (splits == 1)
  int64_t pstride;
  float* partial;   // [k][splits][Co][Ci*9] (splits > 1)
  int splits, per;  // units of a replica: b * H / TH, `per` of them per split
};

// LDS row stride with stride % 64 == 34: the 16 channels x 4 pixels a
// 64-lane read touches fall on (nearly) distinct banks.
constexpr int pad34(int n) { return n + ((34 - n % 64) + 64) % 64; }

template <int WW, int TH>
__global__ __launch_bounds__(256) void conv3x3_wgrad_k(WgradArgs a) {
  constexpr int WP = WW + 2, HR = TH + 2;
  constexpr int SA = pad34(TH * WW);      // dY tile channel stride
  constexpr int SB = pad34(HR * WP);      // X tile channel stride
  constexpr int NQ = TH * WW / 4;         // 4-pixel steps per unit
  constexpr int QW = NQ / 4;              // per wave
  constexpr int NA4 = 16 * TH * WW / 4;   // dY float4s per unit
  constexpr int NA4T = (NA4 + 255) / 256;
  constexpr int NX = 16 * HR * WP;        // X elements per unit
  constexpr int NXT = (NX + 255) / 256;
  constexpr int RED = 4 * 16 * 144;       // cross-wave reduction buffer
  constexpr int TILE = 16 * SA + 16 * SB;
  static_assert(NQ % 4 == 0, "unit must split evenly over the waves");
  __shared__ __attribute__((aligned(16))) float lds[TILE > RED ? TILE : RED];
  float* As = lds;
  float* Bs = lds + 16 * SA;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, kq = lane >> 4, l16 = lane & 15;
  const int nci = a.Ci / 16;
  const int co0 = (blockIdx.x / nci) * 16, ci0 = (blockIdx.x % nci) * 16;
  const int split = blockIdx.y, j = blockIdx.z;
  const int H = a.H, HW = H * WW, tiles_img = H / TH;
  const int units = a.b * tiles_img;
  const int u0 = split * a.per, u1 = min(units, u0 + a.per);

  v4f acc[9];
#pragma unroll
  for (int t = 0; t < 9; ++t) acc[t] = v4f{0.f, 0.f, 0.f, 0.f};

  for (int u = u0; u < u1; ++u) {
    const int img = u / tiles_img, h0 = (u - img * tiles_img) * TH;
    const int n = j * a.b + img;
    const float* DY = a.dy + ((int64_t)n * a.Co + co0) * HW + h0 * WW;
    const float* X = a.x + ((int64_t)n * a.Ci + ci0) * HW;
    v4f ra[NA4T];
    float rx[NXT];
#pragma unroll
    for (int i = 0; i < NA4T; ++i) {
      const int e = tid + i * 256;
      if (e < NA4) {
        const int c = e / (TH * WW / 4), q = e - c * (TH * WW / 4);
        ra[i] = *reinterpret_cast<const v4f*>(DY + (int64_t)c * HW + q * 4);
      }
    }
#pragma unroll
    for (int i = 0; i < NXT; ++i) {
      const int e = tid + i * 256;
      float v = 0.f;
      if (e < NX) {
        const int c = e / (HR * WP), rem = e - c * (HR * WP), hr = rem / WP, wc = rem - hr * WP;
        const int ih = h0 - 1 + hr, iw = wc - 1;
        if ((unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)WW)
          v = X[(int64_t)c * HW + ih * WW + iw];
      }
      rx[i] = v;
    }
    __syncthreads();  // the previous unit's reads of the tiles are done
#pragma unroll
    for (int i = 0; i < NA4T; ++i) {
      const int e = tid + i * 256;
      if (e < NA4) {
        const int c = e / (TH * WW / 4), q = e - c * (TH * WW / 4);
        float* d = As + c * SA + q * 4;
        d[0] = ra[i][0];
        d[1] = ra[i][1];
        d[2] = ra[i][2];
        d[3] = ra[i][3];
      }
    }
#pragma unroll
    for (int i = 0; i < NXT; ++i) {
      const int e = tid + i * 256;
      if (e < NX) {
        const int c = e / (HR * WP), rem = e - c * (HR * WP);
        Bs[c * SB + rem] = rx[i];
      }
    }
    __syncthreads();
#pragma unroll 2
    for (int i = 0; i < QW; ++i) {
      const int q = wave + 4 * i;
      const int h = q / (WW / 4), w = (q - h * (WW / 4)) * 4;
      const float av = As[l16 * SA + h * WW + w + kq];
      const float* xb = Bs + l16 * SB + h * WP + w + kq;
      float bv[9];
#pragma unroll
      for (int t = 0; t < 9; ++t) bv[t] = xb[(t / 3) * WP + (t % 3)];
#pragma unroll
      for (int t = 0; t < 9; ++t) acc[t] = mfma4(av, bv[t], acc[t]);
    }
  }

  // acc[t][r]: co = co0 + 4*kq + r, ci = ci0 + l16, tap t.  Waves in order.
  __syncthreads();
#pragma unroll
  for (int t = 0; t < 9; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) lds[(wave * 16 + 4 * kq + r) * 144 + l16 * 9 + t] = acc[t][r];
  __syncthreads();
  const int64_t wn = (int64_t)a.Co * a.Ci * 9;
  float* out = a.splits == 1 ? a.dw + (int64_t)j * a.pstride
                             : a.partial + (int64_t)(j * a.splits + split) * wn;
  for (int e = tid; e < 16 * 144; e += 256) {
    const int c = e / 144, rem = e - c * 144;
    const float v = ((lds[e] + lds[2304 + e]) + lds[4608 + e]) + lds[6912 + e];
    out[(int64_t)(co0 + c) * a.Ci * 9 + ci0 * 9 + rem] = v;
  }
}

template <int WW, int TH>
hipError_t launch_wgrad(const WgradArgs& a, hipStream_t s, const char** name) {
  dim3 grid((unsigned)((a.Co / 16) * (a.Ci / 16)), (unsigned)a.splits, (unsigned)a.k);
  klaunch(conv3x3_wgrad_k<WW, TH>, grid, dim3(256), 0, s, a);
  if (name) {
    static const std::string n =
        std::string("conv3x3_wgrad_k<") + std::to_string(WW) + ", " + std::to_string(TH) + ">";
    *name = n.c_str();
  }
  return hipGetLastError();
}

template <int WW, int TH, int BN, int CC, bool FLIP>
const char* direct_name() {
  static const std::string n = std::string("conv3x3_k<") + std::to_string(WW) + ", " +
                               std::to_string(TH) + ", " + std::to_string(BN) + ", " +
                               std::to_string(CC) + ", " + (FLIP ? "true" : "false") + ">";
  return n.c_str();
}

template <int WW, int TH, int BN, int CC, bool FLIP>
hipError_t launch(const DirectArgs& a, hipStream_t s, const char** name) {
  dim3 grid((unsigned)(a.b * (a.H / TH)), (unsigned)(a.Cout / BN), (unsigned)a.k);
  klaunch((conv3x3_k<WW, TH, BN, CC, FLIP>), grid, dim3(256), 0, s, a);
  if (name) *name = direct_name<WW, TH, BN, CC, FLIP>();
  return hipGetLastError();
}

// Built for square images of width 8, 16 or 32 and channel counts that
// are multiples of 16.  Tile choice: TH output rows (a multiple of 64
// pixels) and BN output channels; the largest tile that still gives every
// CU two workgroups over all replicas, else the smallest.
struct DirectTile {
  int th, bn;
};

constexpr int64_t DIRECT_MIN_WGS = 512;

bool direct_ok(int H, int W, int Cin, int Cout, int R, int st, int pad) {
  if (R != 3 || st != 1 || pad != 1 || H != W) return false;
  if (W != 8 && W != 16 && W != 32) return false;
  return Cin % 16 == 0 && Cout % 16 == 0;
}

DirectTile direct_pick(int k, int b, int W, int Cout) {
  const int th_max = W == 32 ? 4 : 8, th_min = W == 32 ? 2 : (W == 16 ? 4 : 8);
  auto wgs = [&](int th, int bn) { return (int64_t)k * b * (W / th) * (Cout / bn); };
  const int bn_max = Cout % 32 == 0 ? 32 : 16;
  if (wgs(th_max, bn_max) >= DIRECT_MIN_WGS) return {th_max, bn_max};
  if (wgs(th_min, bn_max) >= DIRECT_MIN_WGS) return {th_min, bn_max};
  return {th_min, 16};
}

template <bool FLIP, int WW>
hipError_t dispatch_w(const DirectArgs& a, DirectTile t, hipStream_t s, const char** name) {
  constexpr int TH1 = WW == 32 ? 4 : 8, TH2 = WW == 32 ? 2 : (WW == 16 ? 4 : 8);
  if (t.th == TH1) {
    if (t.bn == 32) return launch<WW, TH1, 32, 16, FLIP>(a, s, name);
    return launch<WW, TH1, 16, 16, FLIP>(a, s, name);
  }
  if (t.bn == 32) return launch<WW, TH2, 32, 16, FLIP>(a, s, name);
  return launch<WW, TH2, 16, 16, FLIP>(a, s, name);
}

template <bool FLIP>
hipError_t dispatch(const DirectArgs& a, int W, hipStream_t s, const char** name) {
  const DirectTile t = direct_pick(a.k, a.b, W, a.Cout);
  if (W == 32) return dispatch_w<FLIP, 32>(a, t, s, name);
  if (W == 16) return dispatch_w<FLIP, 16>(a, t, s, name);
  return dispatch_w<FLIP, 8>(a, t, s, name);
}

// Weight gradient: units of 8 rows; the split gives every CU two
// workgroups over all replicas and channel blocks where the units allow.
constexpr int WG_TH = 8;

void wgrad_split(const ConvGeom& g, int* splits, int* per) {
  const int units = g.b * (g.H / WG_TH);
  const int64_t blocks = (int64_t)g.k * (g.Co / 16) * (g.Ci / 16);
  int sp = (int)std::max<int64_t>(1, std::min<int64_t>(units, (DIRECT_MIN_WGS + blocks - 1) / blocks));
  const int pr = (units + sp - 1) / sp;
  *per = pr;
  *splits = (units + pr - 1) / pr;
}

}  // namespace

bool conv_direct_wgrad_ok(const ConvGeom& g) {
  return direct_ok(g.H, g.W, g.Ci, g.Co, g.R, g.st, g.pad);
}

int conv_direct_wgrad_splits(const ConvGeom& g) {
  int sp = 1, per = 1;
  wgrad_split(g, &sp, &per);
  return sp;
}

hipError_t conv_direct_wgrad(const ConvBwdWeightArgs& w, hipStream_t s, const char** name) {
  WgradArgs a{};
  a.k = w.g.k; a.b = w.g.b; a.H = w.g.H;
  a.Ci = w.g.Ci; a.Co = w.g.Co;
  a.x = w.x; a.dy = w.dy; a.dw = w.dw; a.pstride = w.pstride; a.partial = w.partial;
  wgrad_split(w.g, &a.splits, &a.per);
  if (w.splits != a.splits) return hipErrorInvalidValue;  // scratch sized for another split
  if (w.g.W == 32) return launch_wgrad<32, WG_TH>(a, s, name);
  if (w.g.W == 16) return launch_wgrad<16, WG_TH>(a, s, name);
  return launch_wgrad<8, WG_TH>(a, s, name);
}

bool conv_direct_fwd_ok(const ConvGeom& g) {
  return direct_ok(g.H, g.W, g.Ci, g.Co, g.R, g.st, g.pad);
}

bool conv_direct_bwd_data_ok(const ConvGeom& g) {
  return direct_ok(g.H, g.W, g.Co, g.Ci, g.R, g.st, g.pad);
}

int conv_direct_fwd_tiles(const ConvGeom& g) {
  return g.b * (g.H / direct_pick(g.k, g.b, g.W, g.Co).th);
}

int conv_direct_bwd_data_tiles(const ConvGeom& g) {
  return g.b * (g.H / direct_pick(g.k, g.b, g.W, g.Ci).th);
}

hipError_t conv_direct_fwd(const ConvFwdArgs& f, hipStream_t s, const char** name) {
  DirectArgs a{};
  a.k = f.g.k; a.b = f.g.b; a.H = f.g.H;
  a.Cin = f.g.Ci; a.Cout = f.g.Co;
  a.in = f.x; a.w = f.w; a.pstride = f.pstride; a.out = f.y;
  a.bias = f.bias; a.relu = f.relu; a.stats = f.stats;
  a.add_mode = ADD_NONE;
  return dispatch<false>(a, f.g.W, s, name);
}

hipError_t conv_direct_bwd_data(const ConvBwdDataArgs& d, hipStream_t s, const char** name) {
  DirectArgs a{};
  a.k = d.g.k; a.b = d.g.b; a.H = d.g.H;
  a.Cin = d.g.Co; a.Cout = d.g.Ci;
  a.in = d.dy; a.w = d.w; a.pstride = d.pstride; a.out = d.dx;
  a.accumulate = d.accumulate; a.mask = d.mask;
  a.add = d.add; a.add_mode = d.add_mode; a.add_C = d.add_C; a.add_st = d.add_st;
  a.bn_part = d.bn_part; a.bn_x = d.bn_x; a.bn_y = d.bn_y;
  a.bn_mean = d.bn_mean; a.bn_istd = d.bn_istd;
  return dispatch<true>(a, d.g.W, s, name);
}

}  // namespace cbk
