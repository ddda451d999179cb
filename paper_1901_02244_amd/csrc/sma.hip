// sma.hip -- the synchronisation of Algorithm 1 (Sec. 3.2) as one fused,
// HBM-streaming pass over all k replicas.
//
// For every parameter e, with the replica values from before the update:
//   c_j  = alpha (w_j - z)                         (correction)
//   w_j <- w_j - lr g_j - c_j [+ mu_L (w_j - w_j_prev)]
//   z   <- z + sum_j c_j + mu (z - z_prev),  z_prev <- old z
// The corrections are never written to memory.  Traffic per iteration is
// 4P(3k+4) bytes: read w_j, g_j, z, z_prev; write w_j, z, z_prev.
//
// Work decomposition: a wave covers 64/R float4 columns; the R lane groups
// of a wave take replicas j = r, r+R, r+2R, ... of the same columns, and
// their partial correction sums are combined with an xor butterfly across
// the lane groups (a fixed sequence of commutative adds, so every lane ends
// with the same bits and the result is reproducible).  R = 1 for large P
// (each lane streams all k replicas of its column; sma_cols_k below for the
// largest P); larger R keeps enough waves in flight when P is small.
#include "kernels.hpp"

namespace cbk {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

inline unsigned cdiv(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }

template <bool NT>
__device__ __forceinline__ v4f ld(const v4f* p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}
template <bool NT>
__device__ __forceinline__ void st(v4f* p, v4f v) {
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

template <int R, bool CORRECT, bool LMOM, bool NT>
__global__ __launch_bounds__(256) void sma_k(SMAArgs a) {
  constexpr int C = 64 / R;  // float4 columns per wave
  constexpr int U = 2;       // replicas loaded before any is updated
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane / C, col = lane - r * C;
  const int64_t e = ((int64_t)blockIdx.x * 4 + wave) * C + col;
  const bool ok = e < a.P4;

  v4f* __restrict__ W = reinterpret_cast<v4f*>(a.W);
  const v4f* __restrict__ G = reinterpret_cast<const v4f*>(a.G);
  v4f* __restrict__ Wp = reinterpret_cast<v4f*>(a.Wprev);
  v4f z = {0.f, 0.f, 0.f, 0.f};
  if (CORRECT && ok) z = reinterpret_cast<const v4f*>(a.z)[e];
  v4f S = {0.f, 0.f, 0.f, 0.f};
  const float al = a.alpha, lr = a.lr, ml = a.mu_l;

  if (ok) {
    int j = r;
    for (; j + (U - 1) * R < a.k; j += U * R) {
      v4f w[U], g[U], wp[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        w[u] = ld<NT>(W + (j + u * R) * a.wstride4 + e);
        g[u] = ld<NT>(G + (j + u * R) * a.gstride4 + e);
        if (LMOM) wp[u] = ld<NT>(Wp + (j + u * R) * a.wstride4 + e);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        v4f c = {0.f, 0.f, 0.f, 0.f};
        if (CORRECT) c = al * (w[u] - z);
        v4f wn = w[u] - lr * g[u] - c;
        if (LMOM) {
          wn += ml * (w[u] - wp[u]);
          st<NT>(Wp + (j + u * R) * a.wstride4 + e, w[u]);
        }
        st<NT>(W + (j + u * R) * a.wstride4 + e, wn);
        S += c;
      }
    }
    for (; j < a.k; j += R) {
      const v4f w = ld<NT>(W + j * a.wstride4 + e);
      const v4f g = ld<NT>(G + j * a.gstride4 + e);
      v4f c = {0.f, 0.f, 0.f, 0.f};
      if (CORRECT) c = al * (w - z);
      v4f wn = w - lr * g - c;
      if (LMOM) {
        const v4f wp = ld<NT>(Wp + j * a.wstride4 + e);
        wn += ml * (w - wp);
        st<NT>(Wp + j * a.wstride4 + e, w);
      }
      st<NT>(W + j * a.wstride4 + e, wn);
      S += c;
    }
  }
  if (!CORRECT) return;
  // combine the R lane groups' partial sums (all lanes take part)
#pragma unroll
  for (int o = C; o < 64; o <<= 1) {
    S.x += __shfl_xor(S.x, o, 64);
    S.y += __shfl_xor(S.y, o, 64);
    S.z += __shfl_xor(S.z, o, 64);
    S.w += __shfl_xor(S.w, o, 64);
  }
  if (r == 0 && ok) {
    v4f* Z = reinterpret_cast<v4f*>(a.z);
    v4f* Zp = reinterpret_cast<v4f*>(a.zp);
    const v4f zp = Zp[e];
    Z[e] = z + S + a.mu * (z - zp);
    Zp[e] = z;
  }
}

template <int R>
hipError_t launch_r(const SMAArgs& a, bool nt, hipStream_t s) {
  constexpr int C = 64 / R;
  dim3 grid(cdiv(a.P4, 4 * C)), block(256);
  const bool lm = a.Wprev != nullptr;
#define CB_SMA_LAUNCH(CORR, LM, NTV) \
  klaunch((sma_k<R, CORR, LM, NTV>), grid, block, 0, s, a)
  if (a.correct) {
    if (lm) {
      if (nt) CB_SMA_LAUNCH(true, true, true); else CB_SMA_LAUNCH(true, true, false);
    } else {
      if (nt) CB_SMA_LAUNCH(true, false, true); else CB_SMA_LAUNCH(true, false, false);
    }
  } else {
    if (lm) {
      if (nt) CB_SMA_LAUNCH(false, true, true); else CB_SMA_LAUNCH(false, true, false);
    } else {
      if (nt) CB_SMA_LAUNCH(false, false, true); else CB_SMA_LAUNCH(false, false, false);
    }
  }
#undef CB_SMA_LAUNCH
  return hipGetLastError();
}

// The largest P: each lane takes CPL float4 columns, C apart, one replica
// at a time (used with R = 1, CPL = 16).  A wave then streams 16 KB
// contiguous per replica array instead of 1 KB, the loads in flight fill the
// register file (one wave per SIMD), and the long contiguous runs keep HBM
// pages open (25.6M x 32: 2.01 -> 1.83 ms).  The same arithmetic per
// element as sma_k; a separate kernel because folding the two into one
// template changed the register allocation, and the timing, of sma_k's
// small-P forms.
template <int R, bool CORRECT, bool LMOM, bool NT, int CPL>
__global__ __launch_bounds__(256) void sma_cols_k(SMAArgs a) {
  constexpr int C = 64 / R;  // float4 columns per wave and pass
  constexpr int U = CPL > 1 ? 1 : 2;  // replicas loaded before any is updated
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane / C, col = lane - r * C;
  const int64_t e0 = ((int64_t)blockIdx.x * 4 + wave) * C * CPL + col;

  v4f* __restrict__ W = reinterpret_cast<v4f*>(a.W);
  const v4f* __restrict__ G = reinterpret_cast<const v4f*>(a.G);
  v4f* __restrict__ Wp = reinterpret_cast<v4f*>(a.Wprev);
  const float al = a.alpha, lr = a.lr, ml = a.mu_l;
  v4f z[CPL], S[CPL];
  bool ok[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    ok[c] = e0 + c * C < a.P4;
    z[c] = v4f{0.f, 0.f, 0.f, 0.f};
    S[c] = v4f{0.f, 0.f, 0.f, 0.f};
    if (CORRECT && ok[c]) z[c] = reinterpret_cast<const v4f*>(a.z)[e0 + c * C];
  }
  int j = r;
  for (; j + (U - 1) * R < a.k; j += U * R) {
    v4f w[U][CPL], g[U][CPL], wp[U][CPL];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        if (!ok[c]) continue;
        const int64_t e = e0 + c * C;
        w[u][c] = ld<NT>(W + (j + u * R) * a.wstride4 + e);
        g[u][c] = ld<NT>(G + (j + u * R) * a.gstride4 + e);
        if (LMOM) wp[u][c] = ld<NT>(Wp + (j + u * R) * a.wstride4 + e);
      }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        if (!ok[c]) continue;
        const int64_t e = e0 + c * C;
        v4f cc = {0.f, 0.f, 0.f, 0.f};
        if (CORRECT) cc = al * (w[u][c] - z[c]);
        v4f wn = w[u][c] - lr * g[u][c] - cc;
        if (LMOM) {
          wn += ml * (w[u][c] - wp[u][c]);
          st<NT>(Wp + (j + u * R) * a.wstride4 + e, w[u][c]);
        }
        st<NT>(W + (j + u * R) * a.wstride4 + e, wn);
        S[c] += cc;
      }
  }
  for (; j < a.k; j += R)
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      if (!ok[c]) continue;
      const int64_t e = e0 + c * C;
      const v4f w = ld<NT>(W + j * a.wstride4 + e);
      const v4f g = ld<NT>(G + j * a.gstride4 + e);
      v4f cc = {0.f, 0.f, 0.f, 0.f};
      if (CORRECT) cc = al * (w - z[c]);
      v4f wn = w - lr * g - cc;
      if (LMOM) {
        const v4f wp = ld<NT>(Wp + j * a.wstride4 + e);
        wn += ml * (w - wp);
        st<NT>(Wp + j * a.wstride4 + e, w);
      }
      st<NT>(W + j * a.wstride4 + e, wn);
      S[c] += cc;
    }
  if (!CORRECT) return;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
#pragma unroll
    for (int o = C; o < 64; o <<= 1) {
      S[c].x += __shfl_xor(S[c].x, o, 64);
      S[c].y += __shfl_xor(S[c].y, o, 64);
      S[c].z += __shfl_xor(S[c].z, o, 64);
      S[c].w += __shfl_xor(S[c].w, o, 64);
    }
    if (r == 0 && ok[c]) {
      const int64_t e = e0 + c * C;
      v4f* Z = reinterpret_cast<v4f*>(a.z);
      v4f* Zp = reinterpret_cast<v4f*>(a.zp);
      const v4f zp = Zp[e];
      Z[e] = z[c] + S[c] + a.mu * (z[c] - zp);
      Zp[e] = z[c];
    }
  }
}

hipError_t launch_cols(const SMAArgs& a, bool nt, hipStream_t s) {
  constexpr int CPL = 16;
  dim3 grid(cdiv(a.P4, 4 * 64 * CPL)), block(256);
  const bool lm = a.Wprev != nullptr;
#define CB_SMA_LAUNCH(CORR, LM, NTV) klaunch((sma_cols_k<1, CORR, LM, NTV, CPL>), grid, block, 0, s, a)
  if (a.correct) {
    if (lm) {
      if (nt) CB_SMA_LAUNCH(true, true, true); else CB_SMA_LAUNCH(true, true, false);
    } else {
      if (nt) CB_SMA_LAUNCH(true, false, true); else CB_SMA_LAUNCH(true, false, false);
    }
  } else {
    if (lm) {
      if (nt) CB_SMA_LAUNCH(false, true, true); else CB_SMA_LAUNCH(false, true, false);
    } else {
      if (nt) CB_SMA_LAUNCH(false, false, true); else CB_SMA_LAUNCH(false, false, false);
    }
  }
#undef CB_SMA_LAUNCH
  return hipGetLastError();
}

__global__ void nonfinite_k(const float* z, int64_t n, int* flag) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n && !isfinite(z[i])) flag[0] = 1;
}

__global__ void zero_ints_k(int* p, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0;
}

}  // namespace

hipError_t sma_step(const SMAArgs& a, hipStream_t s, const char** name) {
  if (a.P4 <= 0 || a.k <= 0) return hipSuccess;
  // Lane groups per wave: enough waves to cover the chip, never more
  // groups than replicas.
  int R = 1;
  while (R < 16 && 2 * R <= a.k && a.P4 * R < (int64_t)256 * 2048) R *= 2;
  // Stream past the caches when the replicas cannot stay resident anyway.
  const bool nt = (int64_t)a.k * a.P4 * 16 > ((int64_t)256 << 20);
  // 16 columns per lane from 16 replicas (ResNet-50's P: 0.99 -> 0.95 ms at
  // k = 16, 2.03 -> 1.85 ms at 32; level at 12, slower below), once there
  // are enough columns for one such wave on every SIMD of the chip (256
  // CUs x 4)
  if (R == 1 && a.k >= 16 && a.P4 >= (int64_t)256 * 4 * 64 * 16) {
    if (name) *name = a.correct ? "sma_cols_k" : "sma_cols_k<local step>";
    return launch_cols(a, nt, s);
  }
  switch (R) {
    case 1: return launch_r<1>(a, nt, s);
    case 2: return launch_r<2>(a, nt, s);
    case 4: return launch_r<4>(a, nt, s);
    case 8: return launch_r<8>(a, nt, s);
    default: return launch_r<16>(a, nt, s);
  }
}

hipError_t nonfinite_scan(const float* z, int64_t n, int* flag, hipStream_t s) {
  klaunch(nonfinite_k, dim3(cdiv(n, 256)), dim3(256), 0, s, z, n, flag);
  return hipGetLastError();
}

hipError_t zero_ints(int* p, int n, hipStream_t s) {
  klaunch(zero_ints_k, dim3(cdiv(n, 256)), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace cbk
