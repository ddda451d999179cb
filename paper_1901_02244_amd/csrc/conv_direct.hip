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
// Grid: as many workgroups as fit on the chip at once; each takes every G-th
// tile (replica, output-channel tile, TH rows of one image) and prefetches
// the next tile's inputs while it computes.  Epilogues match the implicit
// GEMM's: bias, ReLU and the batch-norm partial sums of the forward;
// accumulate, residual add, ReLU mask and the batch-norm backward partial
// sums of the data gradient.
#include "kernels.hpp"

#include <algorithm>
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
  const float* bn_gamma;  // RC: replica 0 gamma [Cout], beta at + Cout
  int rc_mask;            // RC: the decision also zeroes dX (the mask's role)
};

// RC (data gradient only): the batch norm has a ReLU and no residual input,
// so the epilogue takes that ReLU's decision as bn_affine of bn_x, which it
// reads anyway, instead of reading the norm's output (bn_y's role, for the
// partial sums) or, when that output is this layer's input, the mask
// (rc_mask: the decision also zeroes dX).
// ST (forward only): the convolution's stride.  WW and a.H are the output's
// width and height; the input is ST times as wide and high, and its tile
// spans (TH - 1) ST + 3 rows of (WW - 1) ST + 3 pixels.
template <int WW, int TH, int BN, int CC, bool FLIP, bool RC, int ST>
__global__ __launch_bounds__(256) void conv3x3_k(DirectArgs a) {
  static_assert(FLIP || !RC, "the mask recompute belongs to the data gradient");
  static_assert(ST == 1 || (ST == 2 && !FLIP), "stride 2 is a forward tile");
  constexpr int WI = WW * ST;             // input width
  constexpr int WP = (WW - 1) * ST + 3, HR = (TH - 1) * ST + 3;
  constexpr int NPIX = HR * WP;           // pixels of the input tile (with border)
  constexpr int M = TH * WW;              // output pixels per tile
  constexpr int TM = M / 64;              // 16-pixel blocks per wave (waves split M)
  constexpr int TN = BN / 16;
  constexpr int C4 = CC / 4;              // channel quads per chunk
  // LDS tiles hold four consecutive channels of a pixel (or of a filter
  // row and tap) as one 16-byte quad, so that one ds_read_b128 gives a lane
  // the operands of four MFMAs.  Within an MFMA the lane group kq = lane / 16
  // takes channel 16g + 4kq + q of the quad read for MFMA (g, q).
  // Input tile: [pixel][CC channels], pixel stride PS = CC + 4 floats (the
  // padding puts the 16 pixels of a read, and of a store, on distinct banks).
  // Filter tile: [row][tap][CC channels], row stride WS = 9 CC + 4; a row
  // is an output channel of the forward, an output channel of the data
  // gradient (input channel of the filter) when flipped; the flipped
  // filter's taps are read in reverse (8 - tap).
  constexpr int PS = CC + 4;
  constexpr int WS = 9 * CC + 4;
  constexpr int NX = C4 * NPIX;           // input quads per chunk
  constexpr int NXT = (NX + 255) / 256;
  constexpr int NW = BN * 9 * C4;         // filter quads per chunk
  constexpr int NWT = (NW + 255) / 256;
  static_assert(TM >= 1 && M % 64 == 0, "tile must cover whole 64-pixel wave strips");
  static_assert(CC % 16 == 0, "a chunk is whole 16-channel MFMA groups");
  // One LDS copy of each tile: the next chunk waits in registers until
  // every wave is done with this one, which keeps the footprint small
  // enough for four or five workgroups per CU.
  __shared__ __attribute__((aligned(16))) float xs[NPIX * PS];
  __shared__ __attribute__((aligned(16))) float ws[BN * WS];
  __shared__ double red[4][BN][2];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, kq = lane >> 4;
  const int H = a.H, HW = H * WW;         // output plane
  const int HI = H * ST, HWI = HI * WI;   // input plane
  const int tiles_img = H / TH;
  const int rows_rep = a.b * tiles_img;            // row tiles of one replica
  const int per_rep = rows_rep * (a.Cout / BN);    // tiles of one replica
  const int T = a.k * per_rep;
  const int nchunk = a.Cin / CC;

  // Tile t: replica, row tile (image-major), then output-channel tile, so
  // that the tiles reading one input tile are numbered together and, with
  // the XCD-major numbering below, fetch it into one XCD's L2.
  struct Tile {
    int j, co0, rt, img, oh0;
  };
  auto decode = [&](int t) {
    Tile d;
    d.j = t / per_rep;
    const int r = t - d.j * per_rep;
    d.rt = r / (a.Cout / BN);
    const int ct = r - d.rt * (a.Cout / BN);
    d.co0 = ct * BN;
    d.img = d.rt / tiles_img;
    d.oh0 = (d.rt - d.img * tiles_img) * TH;
    return d;
  };

  v4f rx[NXT], rw[NWT];
  auto load = [&](const Tile& d, int c0) {
    const auto src = buf_rsrc(a.in + ((int64_t)(d.j * a.b + d.img) * a.Cin) * HWI,
                              (uint32_t)(a.Cin * HWI * 4));
    const auto wsrc = buf_rsrc(a.w + (int64_t)d.j * a.pstride, (uint32_t)(a.Cin * a.Cout * 36));
#pragma unroll
    for (int u = 0; u < NXT; ++u) {
      // quad e: channels c0 + 4 c4 .. +3 of tile pixel pix; consecutive
      // lanes take consecutive pixels, so each of the four reads is
      // coalesced along the image row
      const int e = tid + u * 256;
      const int c4 = e / NPIX, pix = e - c4 * NPIX, hr = pix / WP, wc = pix - hr * WP;
      const int ih = d.oh0 * ST - 1 + hr, iw = wc - 1;
      const bool ok = (NX % 256 == 0 || e < NX) && (unsigned)ih < (unsigned)HI &&
                      (unsigned)iw < (unsigned)WI;
      const uint32_t o = (uint32_t)(((c0 + 4 * c4) * HWI + ih * WI + iw) * 4);
#pragma unroll
      for (int q = 0; q < 4; ++q) rx[u][q] = buf_ld(src, ok ? o + (uint32_t)(q * HWI * 4) : OUTSIDE);
    }
#pragma unroll
    for (int u = 0; u < NWT; ++u) {
      // quad e: row, tap, four consecutive channels of the chunk.  Forward:
      // filter [co0 + row][c0 + 4 c4 + q][tap]; flipped: filter
      // [c0 + 4 c4 + q][co0 + row][tap], enumerated with row and tap
      // fastest so that the reads follow memory order.
      const int e = tid + u * 256;
      int row, tap, c4;
      if (FLIP) {
        c4 = e / (BN * 9);
        const int rem = e - c4 * (BN * 9);
        row = rem / 9;
        tap = rem - row * 9;
      } else {
        row = e / (9 * C4);
        const int rem = e - row * (9 * C4);
        tap = rem / C4;
        c4 = rem - tap * C4;
      }
      const bool ok = NW % 256 == 0 || e < NW;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int el = FLIP ? ((c0 + 4 * c4 + q) * a.Cout + d.co0 + row) * 9 + tap
                            : ((d.co0 + row) * a.Cin + c0 + 4 * c4 + q) * 9 + tap;
        rw[u][q] = buf_ld(wsrc, ok ? (uint32_t)(el * 4) : OUTSIDE);
      }
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int u = 0; u < NXT; ++u) {
      const int e = tid + u * 256;
      if (NX % 256 == 0 || e < NX) {
        const int c4 = e / NPIX, pix = e - c4 * NPIX;
        *reinterpret_cast<v4f*>(&xs[pix * PS + 4 * c4]) = rx[u];
      }
    }
#pragma unroll
    for (int u = 0; u < NWT; ++u) {
      const int e = tid + u * 256;
      if (NW % 256 == 0 || e < NW) {
        int row, tap, c4;
        if (FLIP) {
          c4 = e / (BN * 9);
          const int rem = e - c4 * (BN * 9);
          row = rem / 9;
          tap = rem - row * 9;
        } else {
          row = e / (9 * C4);
          const int rem = e - row * (9 * C4);
          tap = rem / C4;
          c4 = rem - tap * C4;
        }
        *reinterpret_cast<v4f*>(&ws[row * WS + tap * CC + 4 * c4]) = rw[u];
      }
    }
  };

  // lane bases: LDS quad of each of this wave's 16-pixel blocks (tap 0,
  // channel group 0), and of the lane's filter row
  int xbase[TM];
#pragma unroll
  for (int t = 0; t < TM; ++t) {
    const int m = (wave * TM + t) * 16 + (lane & 15);
    const int ohl = m / WW, ow = m - ohl * WW;
    xbase[t] = (ohl * ST * WP + ow * ST) * PS + 4 * kq;
  }
  const int wbase = (lane & 15) * WS + 4 * kq;

  // Epilogue operands of the data gradient (ReLU mask, the next batch
  // norm's x and y), four consecutive pixels of one channel per lane and
  // block, are loaded before the tile's last chunk of MFMAs, so their
  // latency overlaps that chunk.
  v4f e_mask[TM][TN], e_x[TM][TN], e_y[TM][TN];
  auto gofs = [&](const Tile& d, int t, int u) {  // (plane offset, first pixel)
    const int co = d.co0 + u * 16 + (lane & 15);
    const int p0 = d.oh0 * WW + (wave * TM + t) * 16 + 4 * kq;
    return (int64_t)((d.j * a.b + d.img) * a.Cout + co) * HW + p0;
  };
  auto prefetch_epilogue = [&](const Tile& d, v4f (&m)[TM][TN], v4f (&x)[TM][TN],
                               v4f (&y)[TM][TN]) {
    if (!FLIP) return;
#pragma unroll
    for (int t = 0; t < TM; ++t)
#pragma unroll
      for (int u = 0; u < TN; ++u) {
        const int64_t g = gofs(d, t, u);
        if (a.mask) m[t][u] = *reinterpret_cast<const v4f*>(a.mask + g);
        if (a.bn_part) {
          x[t][u] = *reinterpret_cast<const v4f*>(a.bn_x + g);
          if (!RC && a.bn_y) y[t][u] = *reinterpret_cast<const v4f*>(a.bn_y + g);
        }
      }
  };

  v4f acc[TM][TN];
  auto epilogue = [&](const Tile& d) {
    // acc[t][u][i] is pixel (wave*TM + t)*16 + 4*kq + i, channel
    // co0 + u*16 + (lane & 15) of the tile
    double s1[TN], s2[TN];
#pragma unroll
    for (int u = 0; u < TN; ++u) s1[u] = s2[u] = 0.0;
#pragma unroll
    for (int u = 0; u < TN; ++u) {
      const int co = d.co0 + u * 16 + (lane & 15);
      float bv = 0.f, bm = 0.f, bi = 0.f;
      if (!FLIP && a.bias) bv = a.bias[(int64_t)d.j * a.pstride + co];
      if (FLIP && a.bn_part) {
        bm = a.bn_mean[d.j * a.Cout + co];
        bi = a.bn_istd[d.j * a.Cout + co];
      }
      float ga = 0.f, be = 0.f;
      if (RC) {
        ga = a.bn_gamma[(int64_t)d.j * a.pstride + co];
        be = a.bn_gamma[(int64_t)d.j * a.pstride + a.Cout + co];
      }
#pragma unroll
      for (int t = 0; t < TM; ++t) {
        const int64_t g = gofs(d, t, u);
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
          *reinterpret_cast<v4f*>(a.out + g) = v;
        } else {
          if (a.accumulate) v += *reinterpret_cast<const v4f*>(a.out + g);
          if (a.add_mode == ADD_SAME) {
            v += *reinterpret_cast<const v4f*>(a.add + g);
          } else if (a.add_mode == ADD_SUBSAMPLE) {
            const int st = a.add_st;
            const int p0 = d.oh0 * WW + (wave * TM + t) * 16 + 4 * kq;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int p = p0 + i, ih = p / WW, iw = p - ih * WW;
              if (ih % st == 0 && iw % st == 0)
                v[i] += a.add[(((int64_t)(d.j * a.b + d.img) * a.add_C + co) * ((H + st - 1) / st) +
                               ih / st) * ((WW + st - 1) / st) + iw / st];
            }
          }
          bool r[4];
          if (RC)
#pragma unroll
            for (int i = 0; i < 4; ++i) r[i] = bn_affine(e_x[t][u][i], bm, bi, ga, be) > 0.f;
          if (RC && a.rc_mask) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (!r[i]) v[i] = 0.f;
          } else if (a.mask) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (!(e_mask[t][u][i] > 0.f)) v[i] = 0.f;
          }
          *reinterpret_cast<v4f*>(a.out + g) = v;
          if (a.bn_part) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const bool keep = RC ? r[i] : (!a.bn_y || e_y[t][u][i] > 0.f);
              const float dd = keep ? v[i] : 0.f;
              const float xh = (e_x[t][u][i] - bm) * bi;
              s1[u] += (double)dd;
              s2[u] += (double)dd * xh;
            }
          }
        }
      }
    }
    double* part = FLIP ? a.bn_part : a.stats;
    if (!part) return;
    // per-channel partial sums of the tile: lanes of a column by xor
    // butterfly, then the four waves in order.  (Every chunk ends with a
    // barrier, so the previous tile's reads of red are done.)
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
      double* o = part + (((int64_t)d.j * a.Cout + d.co0 + tid) * rows_rep + d.rt) * 2;
      o[0] = x;
      o[1] = y;
    }
  };

  // Workgroup w takes tiles w, w + G, w + 2G, ...  Every (tile, chunk) item
  // prefetches the next item's inputs into registers before its MFMAs.
  const int G = gridDim.x;
  int t = xcd_major(blockIdx.x, G);
  Tile d = decode(t);
  load(d, 0);
  store();
  __syncthreads();
  while (true) {
#pragma unroll
    for (int x = 0; x < TM; ++x)
#pragma unroll
      for (int y = 0; y < TN; ++y) acc[x][y] = v4f{0.f, 0.f, 0.f, 0.f};
    const bool more = t + G < T;
    const Tile dn = more ? decode(t + G) : d;
    for (int c = 0; c < nchunk; ++c) {
      const bool last = c + 1 == nchunk;
      const bool has_next = !last || more;
      if (has_next) load(last ? dn : d, last ? 0 : (c + 1) * CC);
      if (last) prefetch_epilogue(d, e_mask, e_x, e_y);
      const float* X = xs;
      const float* Wl = ws;
#pragma unroll
      for (int tap = 0; tap < 9; ++tap) {
        const int r = tap / 3, s = tap - r * 3;
        const int tw = FLIP ? 8 - tap : tap;
#pragma unroll
        for (int g = 0; g < CC / 16; ++g) {
          v4f av[TM], bv[TN];
#pragma unroll
          for (int x = 0; x < TM; ++x)
            av[x] = *reinterpret_cast<const v4f*>(&X[xbase[x] + (r * WP + s) * PS + 16 * g]);
#pragma unroll
          for (int u = 0; u < TN; ++u)
            bv[u] = *reinterpret_cast<const v4f*>(&Wl[wbase + u * 16 * WS + tw * CC + 16 * g]);
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int x = 0; x < TM; ++x)
#pragma unroll
              for (int u = 0; u < TN; ++u) acc[x][u] = mfma4(av[x][q], bv[u][q], acc[x][u]);
        }
      }
      if (has_next) {
        __syncthreads();
        store();
      }
      __syncthreads();
    }
    epilogue(d);
    if (!more) break;
    t += G;
    d = dn;
  }
}

// Data gradient of a 3x3, stride 2, pad 1 convolution, by output parity.
// dX[ci][ih][iw] = sum over co and the taps (r, s) with ih + 1 - r and
// iw + 1 - s even of W[co][ci][r][s] dY[co][(ih + 1 - r) / 2][(iw + 1 - s) / 2].
// Split dX by (ih % 2, iw % 2) = (ph, pw): each class is a stride-1
// convolution on the dY grid, class pixel (m, n) = dX pixel (2m+ph, 2n+pw),
// over the taps r in {1} (ph = 0) or {0, 2} (ph = 1), likewise s, reading dY
// at (m + (ph + 1 - r) / 2, n + (pw + 1 - s) / 2) -- 9 taps over the four
// classes instead of the 4 x 9 of a zero-filled implicit GEMM.  A
// workgroup computes all four classes of THO dY rows (2*THO dX rows) for BN
// dX channels from one dY tile in LDS (rows m0 .. m0+THO, columns 0 .. WO,
// zero beyond the image).  MFMA rows are 16 consecutive class pixels, so
// a lane holds the pw = 0 and pw = 1 values of the same four positions:
// 8 consecutive dX pixels, moved as two float4s in the epilogue.
template <int WO, int THO, int BN, int CC>
__global__ __launch_bounds__(256) void conv3x3s2_dgrad_k(DirectArgs a) {
  constexpr int WPo = WO + 1, HRo = THO + 1;
  constexpr int CS = pad_cs(HRo * WPo);
  constexpr int MC = THO * WO;            // pixels of one class per tile
  constexpr int TM = MC / 64;             // 16-pixel blocks per wave and class
  constexpr int TN = BN / 16;
  constexpr int WS = BN == 16 ? 144 : 304;  // filter rows: contraction channel
  constexpr int WRUN = BN * 9;
  constexpr int NX = CC * HRo * WPo, NXT = (NX + 255) / 256;
  constexpr int NW = CC * WRUN, NWT = (NW + 255) / 256;
  static_assert(TM >= 1 && MC % 64 == 0, "class tile must cover whole 64-pixel wave strips");
  __shared__ __attribute__((aligned(16))) float xs[2][CC * CS];
  __shared__ __attribute__((aligned(16))) float ws[2][CC * WS];
  __shared__ double red[4][BN][2];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, kq = lane >> 4;
  const int l16 = lane & 15;
  const int HO = a.H / 2, W = 2 * WO, HW = a.H * W, HWo = HO * WO;
  const int tiles_img = HO / THO;
  const int rows_rep = a.b * tiles_img;
  const int per_rep = rows_rep * (a.Cout / BN);
  const int T = a.k * per_rep;
  const int nchunk = a.Cin / CC;

  struct Tile {
    int j, co0, rt, img, m0;
  };
  auto decode = [&](int t) {
    Tile d;
    d.j = t / per_rep;
    const int r = t - d.j * per_rep;
    d.rt = r / (a.Cout / BN);
    const int ct = r - d.rt * (a.Cout / BN);
    d.co0 = ct * BN;  // first dX channel of the tile
    d.img = d.rt / tiles_img;
    d.m0 = (d.rt - d.img * tiles_img) * THO;
    return d;
  };

  float rx[NXT], rw[NWT];
  auto load = [&](const Tile& d, int c0) {
    const auto src = buf_rsrc(a.in + ((int64_t)(d.j * a.b + d.img) * a.Cin) * HWo,
                              (uint32_t)(a.Cin * HWo * 4));
    const auto wsrc = buf_rsrc(a.w + (int64_t)d.j * a.pstride, (uint32_t)(a.Cin * a.Cout * 36));
#pragma unroll
    for (int u = 0; u < NXT; ++u) {
      const int e = tid + u * 256;
      const int c = e / (HRo * WPo), rem = e - c * (HRo * WPo), hr = rem / WPo, wc = rem - hr * WPo;
      const int m = d.m0 + hr;
      const bool ok = (NX % 256 == 0 || e < NX) && m < HO && wc < WO;
      rx[u] = buf_ld(src, ok ? (uint32_t)(((c0 + c) * HWo + m * WO + wc) * 4) : OUTSIDE);
    }
#pragma unroll
    for (int u = 0; u < NWT; ++u) {
      // the filter [co][ci][tap] of the convolution: rows co = c0 + row (the
      // contraction), runs over ci in the tile and the taps
      const int e = tid + u * 256;
      const int row = e / WRUN, rem = e - row * WRUN;
      const int el = ((c0 + row) * a.Cout + d.co0) * 9 + rem;
      rw[u] = buf_ld(wsrc, (NW % 256 == 0 || e < NW) ? (uint32_t)(el * 4) : OUTSIDE);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int u = 0; u < NXT; ++u) {
      const int e = tid + u * 256;
      if (e < NX) {
        const int c = e / (HRo * WPo);
        xs[buf][c * CS + e - c * (HRo * WPo)] = rx[u];
      }
    }
#pragma unroll
    for (int u = 0; u < NWT; ++u) {
      const int e = tid + u * 256;
      if (e < NW) {
        const int row = e / WRUN;
        ws[buf][row * WS + e - row * WRUN] = rw[u];
      }
    }
  };

  // lane pixel of each 16-pixel class block: (mloc, n)
  int xbase[TM];
#pragma unroll
  for (int t = 0; t < TM; ++t) {
    const int m = (wave * TM + t) * 16 + l16;
    const int ml = m / WO, n = m - ml * WO;
    xbase[t] = kq * CS + ml * WPo + n;
  }
  const int wbase = kq * WS + l16 * 9;

  // acc[ph][pw][t][u]
  v4f acc[2][2][TM][TN];

  auto epilogue = [&](const Tile& d) {
    const int n_img = d.j * a.b + d.img;
    double s1[TN], s2[TN];
#pragma unroll
    for (int u = 0; u < TN; ++u) s1[u] = s2[u] = 0.0;
#pragma unroll
    for (int u = 0; u < TN; ++u) {
      const int ci = d.co0 + u * 16 + l16;
      float bm = 0.f, bi = 0.f;
      if (a.bn_part) {
        bm = a.bn_mean[d.j * a.Cout + ci];
        bi = a.bn_istd[d.j * a.Cout + ci];
      }
#pragma unroll
      for (int t = 0; t < TM; ++t) {
        const int mp = (wave * TM + t) * 16 + 4 * kq;  // first of the lane's 4 class pixels
        const int ml = mp / WO, n = mp - ml * WO;
#pragma unroll
        for (int ph = 0; ph < 2; ++ph) {
          const int ih = 2 * (d.m0 + ml) + ph;
          const int64_t idx = ((int64_t)n_img * a.Cout + ci) * HW + ih * W + 2 * n;
          // dX pixels 2n .. 2n+7 of row ih: even columns from class pw = 0
          v4f lo, hi;
          lo[0] = acc[ph][0][t][u][0]; lo[1] = acc[ph][1][t][u][0];
          lo[2] = acc[ph][0][t][u][1]; lo[3] = acc[ph][1][t][u][1];
          hi[0] = acc[ph][0][t][u][2]; hi[1] = acc[ph][1][t][u][2];
          hi[2] = acc[ph][0][t][u][3]; hi[3] = acc[ph][1][t][u][3];
          if (a.accumulate) {
            lo += *reinterpret_cast<const v4f*>(a.out + idx);
            hi += *reinterpret_cast<const v4f*>(a.out + idx + 4);
          }
          if (a.add_mode == ADD_SAME) {
            lo += *reinterpret_cast<const v4f*>(a.add + idx);
            hi += *reinterpret_cast<const v4f*>(a.add + idx + 4);
          } else if (a.add_mode == ADD_SUBSAMPLE && a.add_st == 2 && ph == 0) {
            // even rows and columns take src[n][ci][ih/2][iw/2]: the four
            // class positions (m, n .. n+3)
            const v4f sv = *reinterpret_cast<const v4f*>(
                a.add + (((int64_t)n_img * a.add_C + ci) * HO + d.m0 + ml) * WO + n);
            lo[0] += sv[0]; lo[2] += sv[1]; hi[0] += sv[2]; hi[2] += sv[3];
          }
          if (a.mask) {
            const v4f m0 = *reinterpret_cast<const v4f*>(a.mask + idx);
            const v4f m1 = *reinterpret_cast<const v4f*>(a.mask + idx + 4);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              if (!(m0[i] > 0.f)) lo[i] = 0.f;
              if (!(m1[i] > 0.f)) hi[i] = 0.f;
            }
          }
          *reinterpret_cast<v4f*>(a.out + idx) = lo;
          *reinterpret_cast<v4f*>(a.out + idx + 4) = hi;
          if (a.bn_part) {
            const v4f x0 = *reinterpret_cast<const v4f*>(a.bn_x + idx);
            const v4f x1 = *reinterpret_cast<const v4f*>(a.bn_x + idx + 4);
            v4f y0 = v4f{1.f, 1.f, 1.f, 1.f}, y1 = y0;
            if (a.bn_y) {
              y0 = *reinterpret_cast<const v4f*>(a.bn_y + idx);
              y1 = *reinterpret_cast<const v4f*>(a.bn_y + idx + 4);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float d0 = y0[i] > 0.f ? lo[i] : 0.f;
              s1[u] += (double)d0;
              s2[u] += (double)d0 * ((x0[i] - bm) * bi);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float d1 = y1[i] > 0.f ? hi[i] : 0.f;
              s1[u] += (double)d1;
              s2[u] += (double)d1 * ((x1[i] - bm) * bi);
            }
          }
        }
      }
    }
    if (!a.bn_part) return;
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
      double* o = a.bn_part + (((int64_t)d.j * a.Cout + d.co0 + tid) * rows_rep + d.rt) * 2;
      o[0] = x;
      o[1] = y;
    }
  };

  const int G = gridDim.x;
  int t = xcd_major(blockIdx.x, G);
  Tile d = decode(t);
  load(d, 0);
  store(0);
  __syncthreads();
  int cur = 0;
  while (true) {
#pragma unroll
    for (int ph = 0; ph < 2; ++ph)
#pragma unroll
      for (int pw = 0; pw < 2; ++pw)
#pragma unroll
        for (int x = 0; x < TM; ++x)
#pragma unroll
          for (int y = 0; y < TN; ++y) acc[ph][pw][x][y] = v4f{0.f, 0.f, 0.f, 0.f};
    const bool more = t + G < T;
    const Tile dn = more ? decode(t + G) : d;
    for (int c = 0; c < nchunk; ++c) {
      const bool last = c + 1 == nchunk;
      if (!last || more) load(last ? dn : d, last ? 0 : (c + 1) * CC);
      const float* X = xs[cur];
      const float* Wl = ws[cur];
#pragma unroll
      for (int ph = 0; ph < 2; ++ph)
#pragma unroll
        for (int pw = 0; pw < 2; ++pw)
#pragma unroll
          for (int ir = 0; ir < 1 + ph; ++ir)
#pragma unroll
            for (int is = 0; is < 1 + pw; ++is) {
              // taps of the class: r = 1 (ph = 0) or r in {0, 2} (ph = 1)
              const int r = ph ? 2 * ir : 1, s = pw ? 2 * is : 1;
              const int dr = (ph + 1 - r) / 2, ds = (pw + 1 - s) / 2;
              const int tap = r * 3 + s;
#pragma unroll
              for (int cg = 0; cg < CC / 4; ++cg) {
                float av[TM], bv[TN];
#pragma unroll
                for (int x = 0; x < TM; ++x) av[x] = X[xbase[x] + cg * 4 * CS + dr * WPo + ds];
#pragma unroll
                for (int u = 0; u < TN; ++u) bv[u] = Wl[wbase + cg * 4 * WS + u * 144 + tap];
#pragma unroll
                for (int x = 0; x < TM; ++x)
#pragma unroll
                  for (int u = 0; u < TN; ++u)
                    acc[ph][pw][x][u] = mfma4(av[x], bv[u], acc[ph][pw][x][u]);
              }
            }
      if (!last || more) store(cur ^ 1);
      __syncthreads();
      cur ^= 1;
    }
    epilogue(d);
    if (!more) break;
    t += G;
    d = dn;
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
  int k, b, H;      // H: the height of dY
  int Ci, Co;
  const float* x;   // [k*b][Ci][H*ST][W*ST]
  const float* dy;  // [k*b][Co][H][W]
  float* dw;        // replica 0 gradient [Co][Ci][3][3] (splits == 1)
  int64_t pstride;
  float* partial;   // [k][splits][Co][Ci*9] (splits > 1)
  int splits, per;  // units of a replica: b * H / TH, `per` of them per split
};

// LDS row stride with stride % 64 == 34: the 16 channels x 4 pixels a
// 64-lane read touches fall on (nearly) distinct banks.
constexpr int pad34(int n) { return n + ((34 - n % 64) + 64) % 64; }

// ST: the convolution's stride.  WW is dY's width; the X tile of a unit
// spans (TH - 1) ST + 3 rows of (WW - 1) ST + 3 pixels.
template <int WW, int TH, int ST>
__global__ __launch_bounds__(256) void conv3x3_wgrad_k(WgradArgs a) {
  constexpr int WI = WW * ST;             // X width
  constexpr int WP = (WW - 1) * ST + 3, HR = (TH - 1) * ST + 3;
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
  // The (co, ci) blocks of one replica and split read the same X and dY
  // rows.  Workgroups reach the XCDs in turn, so the grid is renumbered
  // XCD-major: such blocks share one XCD's L2 instead of fetching the rows
  // into several.
  const int gx = gridDim.x, gy = gridDim.y;
  const int lin = xcd_major(blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z), gx * gy * gridDim.z);
  const int bx = lin % gx, rest = lin / gx;
  const int co0 = (bx / nci) * 16, ci0 = (bx % nci) * 16;
  const int split = rest % gy, j = rest / gy;
  const int H = a.H, HW = H * WW, tiles_img = H / TH;
  const int HI = H * ST, HWI = HI * WI;
  const int units = a.b * tiles_img;
  const int u0 = split * a.per, u1 = min(units, u0 + a.per);

  v4f acc[9];
#pragma unroll
  for (int t = 0; t < 9; ++t) acc[t] = v4f{0.f, 0.f, 0.f, 0.f};

  // Unit u's tiles go to registers while the unit before it computes.
  v4f ra[NA4T];
  float rx[NXT];
  auto load = [&](int u) {
    const int img = u / tiles_img, h0 = (u - img * tiles_img) * TH;
    const int n = j * a.b + img;
    const float* DY = a.dy + ((int64_t)n * a.Co + co0) * HW + h0 * WW;
    const float* X = a.x + ((int64_t)n * a.Ci + ci0) * HWI;
#pragma unroll
    for (int i = 0; i < NA4T; ++i) {
      const int e = tid + i * 256;
      if (e < NA4) {
        const int c = e / (TH * WW / 4), q = e - c * (TH * WW / 4);
        ra[i] = *reinterpret_cast<const v4f*>(DY + (int64_t)c * HW + q * 4);
      }
    }
    const auto xsrc = buf_rsrc(X, (uint32_t)(16 * HWI * 4));
#pragma unroll
    for (int i = 0; i < NXT; ++i) {
      const int e = tid + i * 256;
      const int c = e / (HR * WP), rem = e - c * (HR * WP), hr = rem / WP, wc = rem - hr * WP;
      const int ih = h0 * ST - 1 + hr, iw = wc - 1;
      const bool ok = (NX % 256 == 0 || e < NX) && (unsigned)ih < (unsigned)HI &&
                      (unsigned)iw < (unsigned)WI;
      rx[i] = buf_ld(xsrc, ok ? (uint32_t)((c * HWI + ih * WI + iw) * 4) : OUTSIDE);
    }
  };
  auto store = [&]() {
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
  };

  if (u0 < u1) load(u0);
  for (int u = u0; u < u1; ++u) {
    __syncthreads();  // the previous unit's reads of the tiles are done
    store();
    __syncthreads();
    if (u + 1 < u1) load(u + 1);
#pragma unroll 2
    for (int i = 0; i < QW; ++i) {
      const int q = wave + 4 * i;
      const int h = q / (WW / 4), w = (q - h * (WW / 4)) * 4;
      const float av = As[l16 * SA + h * WW + w + kq];
      const float* xb = Bs + l16 * SB + (h * WP + w + kq) * ST;
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

template <int WW, int TH, int ST>
hipError_t launch_wgrad(const WgradArgs& a, hipStream_t s, const char** name) {
  dim3 grid((unsigned)((a.Co / 16) * (a.Ci / 16)), (unsigned)a.splits, (unsigned)a.k);
  klaunch(conv3x3_wgrad_k<WW, TH, ST>, grid, dim3(256), 0, s, a);
  if (name) {
    static const std::string n = std::string("conv3x3_wgrad_k<") + std::to_string(WW) + ", " +
                                 std::to_string(TH) + ", " + std::to_string(ST) + ">";
    *name = n.c_str();
  }
  return hipGetLastError();
}

template <int WO, int THO, int BN, int CC>
hipError_t launch_s2(const DirectArgs& a, hipStream_t s, const char** name) {
  static int resident = 0;
  if (!resident) {
    int per_cu = 0, cus = 0, dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, conv3x3s2_dgrad_k<WO, THO, BN, CC>,
                                                     256, 0) != hipSuccess)
      return hipErrorInvalidValue;
    resident = std::max(1, per_cu) * std::max(1, cus);
  }
  const int64_t T = (int64_t)a.k * a.b * (a.H / 2 / THO) * (a.Cout / BN);
  const int64_t per = (T + resident - 1) / resident;
  const int64_t G = (T + per - 1) / per;
  klaunch(conv3x3s2_dgrad_k<WO, THO, BN, CC>, dim3((unsigned)G), dim3(256), 0, s, a);
  if (name) {
    static const std::string n = std::string("conv3x3s2_dgrad_k<") + std::to_string(WO) + ", " +
                                 std::to_string(THO) + ", " + std::to_string(BN) + ", " +
                                 std::to_string(CC) + ">";
    *name = n.c_str();
  }
  return hipGetLastError();
}

template <int WW, int TH, int BN, int CC, bool FLIP, bool RC, int ST>
const char* direct_name() {
  static const std::string n = std::string("conv3x3_k<") + std::to_string(WW) + ", " +
                               std::to_string(TH) + ", " + std::to_string(BN) + ", " +
                               std::to_string(CC) + ", " + (FLIP ? "true" : "false") + ", " +
                               (RC ? "true" : "false") + ", " + std::to_string(ST) + ">";
  return n.c_str();
}

template <int WW, int TH, int BN, int CC, bool FLIP, bool RC, int ST>
hipError_t launch(const DirectArgs& a, hipStream_t s, const char** name) {
  // as many workgroups as are resident at once, each taking an equal share
  // of the tiles (the last share may be one short)
  static int resident = 0;
  if (!resident) {
    int per_cu = 0, cus = 0, dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &per_cu, conv3x3_k<WW, TH, BN, CC, FLIP, RC, ST>, 256, 0) != hipSuccess)
      return hipErrorInvalidValue;
    resident = std::max(1, per_cu) * std::max(1, cus);
  }
  const int64_t T = (int64_t)a.k * a.b * (a.H / TH) * (a.Cout / BN);
  const int64_t per = (T + resident - 1) / resident;
  const int64_t G = (T + per - 1) / per;
  klaunch(conv3x3_k<WW, TH, BN, CC, FLIP, RC, ST>, dim3((unsigned)G), dim3(256), 0, s, a);
  if (name) *name = direct_name<WW, TH, BN, CC, FLIP, RC, ST>();
  return hipGetLastError();
}

// Built for square images of width 8, 16 or 32 and channel counts that
// are multiples of 16.  Tile choice: 16 output channels and TH output rows
// (a multiple of 64 pixels), the taller TH if it still gives every CU two
// workgroups over all replicas.  32-channel tiles measured slower: at
// width 16, k=4 b=32, 4 rows x 32 channels took 10.1 us per forward launch
// and 8 rows x 16 channels 9.4 us (+0.7% per step).
struct DirectTile {
  int th, bn;
};

constexpr int64_t DIRECT_MIN_WGS = 512;

bool direct_ok(int H, int W, int Cin, int Cout, int R, int st, int pad) {
  if (R != 3 || st != 1 || pad != 1 || H != W) return false;
  if (W != 8 && W != 16 && W != 32) return false;
  return Cin % 16 == 0 && Cout % 16 == 0;
}

// The forward at width 32 takes 8 rows (4 if that leaves too few
// workgroups): it runs alone, and the taller tile is faster (11.1 -> 10.8 us
// at k=4 b=32, +0.2% per step).  The data gradient keeps 4 (or 2): it shares
// the chip with the weight gradients, and 8 rows there made the step 0.4%
// slower although each launch was faster.
DirectTile direct_pick(int k, int b, int W, int Cout, bool flip) {
  const int th_max = (W == 32 && flip) ? 4 : 8;
  const int th_min = W == 32 ? (flip ? 2 : 4) : (W == 16 ? 4 : 8);
  const int64_t wgs = (int64_t)k * b * (W / th_max) * (Cout / 16);
  return {wgs >= DIRECT_MIN_WGS ? th_max : th_min, 16};
}

template <bool FLIP, bool RC, int ST, int WW>
hipError_t dispatch_w(const DirectArgs& a, DirectTile t, hipStream_t s, const char** name) {
  constexpr int TH1 = (WW == 32 && FLIP) ? 4 : 8;
  constexpr int TH2 = WW == 32 ? (FLIP ? 2 : 4) : (WW == 16 ? 4 : 8);
  if (t.bn != 16) return hipErrorInvalidValue;
  if (t.th == TH1) return launch<WW, TH1, 16, 16, FLIP, RC, ST>(a, s, name);
  return launch<WW, TH2, 16, 16, FLIP, RC, ST>(a, s, name);
}

// W: the output width
template <bool FLIP, bool RC, int ST = 1>
hipError_t dispatch(const DirectArgs& a, int W, hipStream_t s, const char** name) {
  const DirectTile t = direct_pick(a.k, a.b, W, a.Cout, FLIP);
  if constexpr (ST == 1)
    if (W == 32) return dispatch_w<FLIP, RC, ST, 32>(a, t, s, name);
  if (W == 16) return dispatch_w<FLIP, RC, ST, 16>(a, t, s, name);
  return dispatch_w<FLIP, RC, ST, 8>(a, t, s, name);
}

// Weight gradient: units of 4 or 8 rows (below), so that a workgroup
// has several units to pipeline; the split gives every CU two workgroups
// over all replicas and channel blocks where the units allow.  With at
// most 128 images per step it gives one per CU: the weight gradients run
// beside the data-gradient chain, whose kernels are then small, and leave
// it the other slots (ResNet-32 k=4 b=32 +0.5%, k=2..8 at b=16 +0.5-3%,
// one replica of 128 +3.4%; at k=16 and 32, b=16, one per CU lost 1-2%).
// The 32x32 layers keep two per CU (k=4 b=32 +0.5%; two per CU for the
// 16x16 or the 8x8 layers instead measured -0.1% and -0.6%).
// At width 16, 8-row units (stride 1; 11.4 us per ResNet-32 k=4 b=32 launch
// against 13.3 us with 4 rows, +0.4% per step) but 4-row units for the
// stride-2 layer (10.3 us against 11.9 us with 8 rows).
constexpr int WG_TH32 = 4, WG_TH16 = 8, WG_TH16_S2 = 4, WG_TH8 = 8;
int wgrad_th(int W, int st) {
  return W == 32 ? WG_TH32 : W == 16 ? (st == 2 ? WG_TH16_S2 : WG_TH16) : WG_TH8;
}

void wgrad_split(const ConvGeom& g, int* splits, int* per) {
  const int units = g.b * (g.Ho / wgrad_th(g.Wo, g.st));
  const int64_t blocks = (int64_t)g.k * (g.Co / 16) * (g.Ci / 16);
  const int64_t wgs =
      ((int64_t)g.k * g.b <= 128 && g.Wo != 32) ? DIRECT_MIN_WGS / 2 : DIRECT_MIN_WGS;
  int sp = (int)std::max<int64_t>(1, std::min<int64_t>(units, (wgs + blocks - 1) / blocks));
  const int pr = (units + sp - 1) / sp;
  *per = pr;
  *splits = (units + pr - 1) / pr;
}

}  // namespace

// Stride-2 data gradient: dY widths 8 and 16 (dX 16 and 32), channel
// counts multiples of 16; THO dY rows per tile (64 class pixels).
int s2_tho(int WO) { return WO == 16 ? 4 : 8; }

bool conv_s2_dgrad_ok(const ConvGeom& g) {
  return g.R == 3 && g.S == 3 && g.st == 2 && g.pad == 1 && g.H == g.W && g.H % 2 == 0 &&
         (g.W == 16 || g.W == 32) && g.Ho == g.H / 2 && g.Ci % 16 == 0 && g.Co % 16 == 0;
}

int conv_s2_dgrad_tiles(const ConvGeom& g) { return g.b * (g.Ho / s2_tho(g.Wo)); }

hipError_t conv_s2_dgrad(const ConvBwdDataArgs& d, hipStream_t s, const char** name) {
  DirectArgs a{};
  a.k = d.g.k; a.b = d.g.b; a.H = d.g.H;
  a.Cin = d.g.Co; a.Cout = d.g.Ci;
  a.in = d.dy; a.w = d.w; a.pstride = d.pstride; a.out = d.dx;
  a.accumulate = d.accumulate; a.mask = d.mask;
  a.add = d.add; a.add_mode = d.add_mode; a.add_C = d.add_C; a.add_st = d.add_st;
  a.bn_part = d.bn_part; a.bn_x = d.bn_x; a.bn_y = d.bn_y;
  a.bn_mean = d.bn_mean; a.bn_istd = d.bn_istd;
  if (a.add_mode == ADD_SUBSAMPLE && a.add_st != 2) return hipErrorInvalidValue;
  if (d.g.Wo == 16) return launch_s2<16, 4, 16, 16>(a, s, name);
  return launch_s2<8, 8, 16, 16>(a, s, name);
}

// Stride 2 (forward and weight gradient): square inputs of width 16 or 32
// (outputs 8 or 16).
bool direct_s2_ok(const ConvGeom& g) {
  return g.R == 3 && g.S == 3 && g.st == 2 && g.pad == 1 && g.H == g.W && g.H % 2 == 0 &&
         (g.W == 16 || g.W == 32) && g.Ho == g.H / 2 && g.Wo == g.W / 2 && g.Ci % 16 == 0 &&
         g.Co % 16 == 0;
}

bool conv_direct_wgrad_ok(const ConvGeom& g) {
  return direct_ok(g.H, g.W, g.Ci, g.Co, g.R, g.st, g.pad) || direct_s2_ok(g);
}

int conv_direct_wgrad_splits(const ConvGeom& g) {
  int sp = 1, per = 1;
  wgrad_split(g, &sp, &per);
  return sp;
}

hipError_t conv_direct_wgrad(const ConvBwdWeightArgs& w, hipStream_t s, const char** name) {
  WgradArgs a{};
  a.k = w.g.k; a.b = w.g.b; a.H = w.g.Ho;
  a.Ci = w.g.Ci; a.Co = w.g.Co;
  a.x = w.x; a.dy = w.dy; a.dw = w.dw; a.pstride = w.pstride; a.partial = w.partial;
  wgrad_split(w.g, &a.splits, &a.per);
  if (w.splits != a.splits) return hipErrorInvalidValue;  // scratch sized for another split
  if (w.g.st == 2) {
    if (w.g.Wo == 16) return launch_wgrad<16, WG_TH16_S2, 2>(a, s, name);
    return launch_wgrad<8, WG_TH8, 2>(a, s, name);
  }
  if (w.g.W == 32) return launch_wgrad<32, WG_TH32, 1>(a, s, name);
  if (w.g.W == 16) return launch_wgrad<16, WG_TH16, 1>(a, s, name);
  return launch_wgrad<8, WG_TH8, 1>(a, s, name);
}


bool conv_direct_fwd_ok(const ConvGeom& g) {
  return direct_ok(g.H, g.W, g.Ci, g.Co, g.R, g.st, g.pad) || direct_s2_ok(g);
}

bool conv_direct_bwd_data_ok(const ConvGeom& g) {
  return direct_ok(g.H, g.W, g.Co, g.Ci, g.R, g.st, g.pad);
}

int conv_direct_fwd_tiles(const ConvGeom& g) {
  return g.b * (g.Ho / direct_pick(g.k, g.b, g.Wo, g.Co, false).th);
}

int conv_direct_bwd_data_tiles(const ConvGeom& g) {
  return g.b * (g.H / direct_pick(g.k, g.b, g.W, g.Ci, true).th);
}

hipError_t conv_direct_fwd(const ConvFwdArgs& f, hipStream_t s, const char** name) {
  DirectArgs a{};
  a.k = f.g.k; a.b = f.g.b; a.H = f.g.Ho;
  a.Cin = f.g.Ci; a.Cout = f.g.Co;
  a.in = f.x; a.w = f.w; a.pstride = f.pstride; a.out = f.y;
  a.bias = f.bias; a.relu = f.relu; a.stats = f.stats;
  a.add_mode = ADD_NONE;
  if (f.g.st == 2) return dispatch<false, false, 2>(a, f.g.Wo, s, name);
  return dispatch<false, false>(a, f.g.W, s, name);
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
  if (d.bn_gamma && d.bn_part && d.bn_x && (d.bn_y || (d.mask_from_bn && d.mask))) {
    a.bn_gamma = d.bn_gamma;
    a.rc_mask = !d.bn_y;
    if (a.rc_mask) a.mask = nullptr;
    a.bn_y = nullptr;
    return dispatch<true, true>(a, d.g.W, s, name);
  }
  return dispatch<true, false>(a, d.g.W, s, name);
}

}  // namespace cbk
