// eql_gconv.h -- the rotation-equivariant group convolution on a square grid
// (rotations by 360/T degrees, T in {1, 2, 4}, acting on the image plane and
// on the group axis of the features) on the C_T kernels: patch gather, its
// adjoint, and the weight permutation both ways.
//
// Sec. 5 names equivariant convolutions as the next operators for the
// method.  The group convolution
//   out[n,o,r] = sum_{d in window} sum_s sum_c psi[R^-r d][(s - r) mod T][o][c] f[n + d, c, s] + b[o]
// (n a pixel, d an offset of the k x k window, R the rotation of offsets)
// splits the window into rotation orbits {R^j d0 : j = 0..T-1} (base point d0
// in a fundamental domain) and the centre.  With u = s - j (mod T), an orbit's
// contribution is
//   sum_{c,u} sum_j Phi[o, (c,u), j - r] X[n, (c,u), j],
//   X[n, (c,u), j] = f[n + R^j d0, c, (u + j) mod T],
//   Phi[o, (c,u), l] = psi[R^l d0][(u + l) mod T][o][c],
// a circular correlation along j -- so the whole convolution is ONE C_T layer
// with k*k*Cin input channels (orbit blocks of Cin*T channels, then the
// centre block of Cin channels with X[n, c, s] = f[n, c, s]) whose weight, in
// the convolution lag m of the C_T kernels, is w[m][o][c'] = Phi[o][c'][-m].
// The rDFT path and its T/2 saving apply to it unchanged.
//
// Channel c' of the gathered rows: orbit O, input channel c, sheared group
// index u -> O*Cin*T + c*T + u; centre channel c -> n_orb*Cin*T + c.
// Orbit base points, in order: T = 4 {a > 0, b >= 0}; T = 2 {a > 0} then
// {a = 0, b > 0}; T = 1 every offset but the centre, row-major; each set
// row-major over (a, b) with a the row offset.  R(a, b) = (-b, a) for T = 4,
// (-a, -b) for T = 2.
//
// Layouts: f, df [N = B*H*W pixels, Cin, T]; X, dX [N, k*k*Cin, T];
// psi, dpsi [k, k, T, Cout, Cin] at (a + k/2, b + k/2, lag); w, dw
// [T, Cout, k*k*Cin].  Every kernel gathers (each output element written
// once, no atomics).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace eqk {

struct GconvDims {
  int T, k, h, Cin, n_orb, Cin2;  // n_orb orbits of T offsets; Cin2 = k*k*Cin
};

__host__ __device__ inline GconvDims gconv_dims(int T, int k, int Cin) {
  GconvDims d;
  d.T = T;
  d.k = k;
  d.h = k / 2;
  d.Cin = Cin;
  d.n_orb = (k * k - 1) / T;
  d.Cin2 = k * k * Cin;
  return d;
}

// offset (a, b) turned by R^n (n any integer)
__device__ __forceinline__ void gconv_rot(int n, int T, int& a, int& b) {
  const int q = T == 4 ? 1 : (T == 2 ? 2 : 0);
  const int turns = (((n % T) + T) % T) * q;
  for (int i = 0; i < turns; ++i) {
    const int na = -b, nb = a;
    a = na;
    b = nb;
  }
}

// base point of orbit O
__device__ __forceinline__ void gconv_base(const GconvDims& d, int O, int& a, int& b) {
  if (d.T == 4) {
    a = 1 + O / (d.h + 1);
    b = O % (d.h + 1);
  } else if (d.T == 2) {
    const int w = 2 * d.h + 1;
    if (O < d.h * w) {
      a = 1 + O / w;
      b = -d.h + O % w;
    } else {
      a = 0;
      b = 1 + (O - d.h * w);
    }
  } else {
    const int idx = O < (d.k * d.k - 1) / 2 ? O : O + 1;
    a = idx / d.k - d.h;
    b = idx % d.k - d.h;
  }
}

// for an offset (a, b) != (0, 0): its orbit O and the turn l with R^l base = (a, b)
__device__ __forceinline__ void gconv_orbit_of(const GconvDims& d, int a, int b, int& O, int& l) {
  O = 0;
  l = 0;
  for (int t = 0; t < d.T; ++t) {
    int x = a, y = b;
    gconv_rot(-t, d.T, x, y);  // candidate base point R^-t (a, b)
    bool in_domain;
    int o;
    if (d.T == 4) {
      in_domain = x > 0 && y >= 0;
      o = (x - 1) * (d.h + 1) + y;
    } else if (d.T == 2) {
      const int w = 2 * d.h + 1;
      in_domain = x > 0 || (x == 0 && y > 0);
      o = x > 0 ? (x - 1) * w + (y + d.h) : d.h * w + (y - 1);
    } else {
      in_domain = true;
      const int idx = (x + d.h) * d.k + (y + d.h);
      o = idx < (d.k * d.k - 1) / 2 ? idx : idx - 1;
    }
    if (in_domain) {
      O = o;
      l = t;
      return;
    }
  }
}

// Gather and scatter run one wave per output pixel, T and k fixed at compile
// time: the channel split (c, u) = (q / T, q % T) is shifts, the orbit loops
// unroll and their offsets fold to constants; the pixel is wave-uniform.  Blocks are ordered so that
// each XCD (blocks dealt round-robin over the 8 of them) takes one contiguous
// run of pixels: neighbouring pixels, which read the same halo rows, then
// share that XCD's L2.
constexpr int kGconvWaves = 4;  // waves (pixels) per 256-thread block

__device__ __forceinline__ int64_t gconv_xcd_block(int64_t bid, int64_t G) {
  const int64_t q = G / 8, r = G % 8, xcd = bid % 8, idx = bid / 8;
  return xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
}

template <typename E, int T>
struct alignas(sizeof(E) * T) GconvVec {
  E v[T];
};

// X[p][c'][j] for one pixel p per wave: orbit blocks X[p][O*Cin*T + c*T + u][j]
// = f[p + R^j d0_O][c][(u + j) mod T] (zero outside the image), one vector of
// T entries per lane and channel; then the centre block, a copy of f[p].  VEC:
// X is aligned to T elements, so each lane stores its T entries at once.
template <typename E, int T, int K, bool VEC>
__device__ __forceinline__ void gconv_gather_pixel(const E* __restrict__ f, E* __restrict__ X, int64_t p, int H,
                                                   int W, int Cin, const GconvDims& d) {
  const int lane = threadIdx.x & 63;
  const int CT = Cin * T;
  const int x = (int)(p % W);
  const int64_t ny = p / W;
  const int y = (int)(ny % H);
  const int64_t img = (ny / H) * H * W;  // first pixel of p's image
  E* const row = X + p * d.Cin2 * T;
#pragma unroll
  for (int O = 0; O < (K * K - 1) / T; ++O) {
    int a0, b0;
    gconv_base(d, O, a0, b0);
    int64_t src[T];
    bool ok[T];
#pragma unroll
    for (int j = 0; j < T; ++j) {
      int a = a0, b = b0;
      gconv_rot(j, T, a, b);
      const int yy = y + a, xx = x + b;
      ok[j] = yy >= 0 && yy < H && xx >= 0 && xx < W;
      src[j] = ok[j] ? (img + (int64_t)yy * W + xx) * CT : 0;
    }
    E* const dst = row + (int64_t)O * CT * T;
    for (int q = lane; q < CT; q += 64) {
      const int c = q / T, u = q % T;
      GconvVec<E, T> v;
#pragma unroll
      for (int j = 0; j < T; ++j) v.v[j] = ok[j] ? f[src[j] + c * T + (u + j) % T] : (E)0.0f;
      if constexpr (VEC) {
        *reinterpret_cast<GconvVec<E, T>*>(dst + (int64_t)q * T) = v;
      } else {
#pragma unroll
        for (int j = 0; j < T; ++j) dst[(int64_t)q * T + j] = v.v[j];
      }
    }
  }
  const E* const fs = f + p * CT;
  E* const dc = row + (int64_t)d.n_orb * CT * T;
  for (int q = lane; q < CT; q += 64) dc[q] = fs[q];
}

// pixel groups of kGconvWaves pixels, one per block, block-strided when the
// grid is capped
template <typename E, int T, int K, bool VEC>
__global__ __launch_bounds__(256) void eql_gconv_gather_kernel(const E* __restrict__ f, E* __restrict__ X,
                                                               int64_t n_pix, int H, int W, int Cin) {
  const GconvDims d = gconv_dims(T, K, Cin);
  for (int64_t g = gconv_xcd_block(blockIdx.x, gridDim.x); g * kGconvWaves < n_pix; g += gridDim.x) {
    const int64_t p = g * kGconvWaves + (threadIdx.x >> 6);
    if (p < n_pix) gconv_gather_pixel<E, T, K, VEC>(f, X, p, H, W, Cin, d);
  }
}

// df[p][c][s] = sum of the entries of dX that the gather filled from
// f[p][c][s] (its adjoint): the centre entry, then for each orbit O and turn j
// the entry of the pixel p - R^j d0_O at channel (O, c, (s - j) mod T), group
// index j; summed in fp32 in that fixed order.  One wave per pixel p.  Every
// load is issued (an entry outside the image reads p's own row and adds
// zero), so the loads of all orbits are in flight together.
template <typename E, int T, int K>
__device__ __forceinline__ void gconv_scatter_pixel(const E* __restrict__ dX, E* __restrict__ df, int64_t p,
                                                    int H, int W, int Cin, const GconvDims& d) {
  const int lane = threadIdx.x & 63;
  const int CT = Cin * T;
  const int64_t rowlen = (int64_t)d.Cin2 * T;
  const int x = (int)(p % W);
  const int64_t ny = p / W;
  const int y = (int)(ny % H);
  const int64_t img = (ny / H) * H * W;
  for (int q = lane; q < CT; q += 64) {
    const int c = q / T, s = q % T;
    float acc = (float)dX[p * rowlen + (int64_t)d.n_orb * CT * T + q];  // centre
#pragma unroll
    for (int O = 0; O < (K * K - 1) / T; ++O) {
      int a0, b0;
      gconv_base(d, O, a0, b0);
#pragma unroll
      for (int j = 0; j < T; ++j) {
        int a = a0, b = b0;
        gconv_rot(j, T, a, b);
        const int ys = y - a, xs = x - b;  // the pixel whose row read p at this entry
        const bool ok = ys >= 0 && ys < H && xs >= 0 && xs < W;
        const int64_t ps = ok ? img + (int64_t)ys * W + xs : p;
        const int u = (s - j + T) % T;
        const float v = (float)dX[ps * rowlen + (int64_t)O * CT * T + (c * T + u) * T + j];
        acc += ok ? v : 0.0f;
      }
    }
    df[p * CT + q] = (E)acc;
  }
}

template <typename E, int T, int K>
__global__ __launch_bounds__(256) void eql_gconv_scatter_kernel(const E* __restrict__ dX, E* __restrict__ df,
                                                                int64_t n_pix, int H, int W, int Cin) {
  const GconvDims d = gconv_dims(T, K, Cin);
  for (int64_t g = gconv_xcd_block(blockIdx.x, gridDim.x); g * kGconvWaves < n_pix; g += gridDim.x) {
    const int64_t p = g * kGconvWaves + (threadIdx.x >> 6);
    if (p < n_pix) gconv_scatter_pixel<E, T, K>(dX, df, p, H, W, Cin, d);
  }
}

// w[m][o][c'] from psi
template <typename E, bool ADJ = false>
__global__ __launch_bounds__(256) void eql_gconv_pack_kernel(const E* __restrict__ psi, E* __restrict__ w,
                                                             int T, int Cin, int Cout, int k) {
  // ADJ: the weight of the adjoint convolution (the input gradient as a group
  // convolution of the output gradient), psi'[d][l][c][o] = psi[-R^-l d][-l
  // mod T][o][c], packed as a layer with k*k*Cout inputs and Cin outputs:
  // w'[T, Cin, k*k*Cout].  Here Ci / Co name that layer's channel counts.
  const int Ci = ADJ ? Cout : Cin, Co = ADJ ? Cin : Cout;
  const GconvDims d = gconv_dims(T, k, Ci);
  const int64_t total = (int64_t)T * Co * d.Cin2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int ob = d.n_orb * Ci * T;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int cc = (int)(i % d.Cin2);
    const int64_t r = i / d.Cin2;
    const int o = (int)(r % Co);
    const int m = (int)(r / Co);
    const int l = (T - m) % T;
    int a = 0, b = 0, c, sp;
    if (cc < ob) {
      const int O = cc / (Ci * T);
      const int rem = cc - O * Ci * T;
      c = rem / T;
      const int u = rem - c * T;
      gconv_base(d, O, a, b);
      gconv_rot(l, T, a, b);
      sp = (u + l) % T;
    } else {
      c = cc - ob;
      sp = l;
    }
    if constexpr (ADJ) {
      // psi'[(a,b)][sp][o][c] = psi[-R^-sp (a,b)][-sp mod T][c][o]
      gconv_rot(-sp, T, a, b);
      w[i] = psi[((((int64_t)(d.h - a) * k + (d.h - b)) * T + (T - sp) % T) * Cout + c) * Cin + o];
    } else {
      w[i] = psi[((((int64_t)(a + d.h) * k + (b + d.h)) * T + sp) * Cout + o) * Cin + c];
    }
  }
}

// dpsi[(a,b)][sp][o][c] from dw (the inverse permutation)
template <typename E>
__global__ __launch_bounds__(256) void eql_gconv_unpack_kernel(const E* __restrict__ dw, E* __restrict__ dpsi,
                                                               int T, int Cin, int Cout, int k) {
  const GconvDims d = gconv_dims(T, k, Cin);
  const int64_t total = (int64_t)k * k * T * Cout * Cin;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int ob = d.n_orb * Cin * T;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int c = (int)(i % Cin);
    int64_t r = i / Cin;
    const int o = (int)(r % Cout);
    r /= Cout;
    const int sp = (int)(r % T);
    r /= T;
    const int b = (int)(r % k) - d.h;
    const int a = (int)(r / k) - d.h;
    int m, cc;
    if (a == 0 && b == 0) {
      m = (T - sp) % T;
      cc = ob + c;
    } else {
      int O, l;
      gconv_orbit_of(d, a, b, O, l);
      m = (T - l) % T;
      const int u = ((sp - l) % T + T) % T;
      cc = O * Cin * T + c * T + u;
    }
    dpsi[i] = dw[((int64_t)m * Cout + o) * d.Cin2 + cc];
  }
}

}  // namespace eqk
