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
// [T, Cout, k*k*Cin].  Every kernel is a grid-stride gather (each output
// element written once, no atomics).
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

// X[n][c'][j] from f (zero outside the image)
template <typename E>
__global__ __launch_bounds__(256) void eql_gconv_gather_kernel(const E* __restrict__ f, E* __restrict__ X,
                                                               int64_t B, int H, int W, int T, int Cin,
                                                               int k) {
  const GconvDims d = gconv_dims(T, k, Cin);
  const int64_t total = B * H * W * d.Cin2 * T;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int j = (int)(i % T);
    const int64_t r = i / T;
    const int cc = (int)(r % d.Cin2);
    const int64_t n = r / d.Cin2;
    const int x = (int)(n % W);
    const int y = (int)((n / W) % H);
    const int64_t bimg = n / ((int64_t)W * H);
    int a = 0, b = 0, c, s;
    const int ob = d.n_orb * Cin * T;
    if (cc < ob) {
      const int O = cc / (Cin * T);
      const int rem = cc - O * Cin * T;
      c = rem / T;
      const int u = rem - c * T;
      gconv_base(d, O, a, b);
      gconv_rot(j, T, a, b);
      s = (u + j) % T;
    } else {
      c = cc - ob;
      s = j;
    }
    const int yy = y + a, xx = x + b;
    E v = (E)0.0f;
    if (yy >= 0 && yy < H && xx >= 0 && xx < W)
      v = f[(((bimg * H + yy) * W + xx) * Cin + c) * T + s];
    X[i] = v;
  }
}

// df[n][c][s] = sum over the entries of X that read f[n][c][s] of dX (the
// adjoint of the gather), summed in fp32 in a fixed order
template <typename E>
__global__ __launch_bounds__(256) void eql_gconv_scatter_kernel(const E* __restrict__ dX, E* __restrict__ df,
                                                                int64_t B, int H, int W, int T, int Cin,
                                                                int k) {
  const GconvDims d = gconv_dims(T, k, Cin);
  const int64_t total = B * H * W * Cin * T;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int ob = d.n_orb * Cin * T;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int s = (int)(i % T);
    const int64_t r = i / T;
    const int c = (int)(r % Cin);
    const int64_t n = r / Cin;
    const int x = (int)(n % W);
    const int y = (int)((n / W) % H);
    const int64_t bimg = n / ((int64_t)W * H);
    float acc = (float)dX[(n * d.Cin2 + ob + c) * T + s];  // centre
    for (int O = 0; O < d.n_orb; ++O) {
      for (int j = 0; j < T; ++j) {
        int a, b;
        gconv_base(d, O, a, b);
        gconv_rot(j, T, a, b);
        const int ys = y - a, xs = x - b;  // the pixel whose row read (y, x) at this entry
        if (ys < 0 || ys >= H || xs < 0 || xs >= W) continue;
        const int u = ((s - j) % T + T) % T;
        const int64_t ns = (bimg * H + ys) * W + xs;
        acc += (float)dX[(ns * d.Cin2 + O * Cin * T + c * T + u) * T + j];
      }
    }
    df[i] = (E)acc;
  }
}

// w[m][o][c'] from psi
template <typename E>
__global__ __launch_bounds__(256) void eql_gconv_pack_kernel(const E* __restrict__ psi, E* __restrict__ w,
                                                             int T, int Cin, int Cout, int k) {
  const GconvDims d = gconv_dims(T, k, Cin);
  const int64_t total = (int64_t)T * Cout * d.Cin2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int ob = d.n_orb * Cin * T;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int cc = (int)(i % d.Cin2);
    const int64_t r = i / d.Cin2;
    const int o = (int)(r % Cout);
    const int m = (int)(r / Cout);
    const int l = (T - m) % T;
    int a = 0, b = 0, c, sp;
    if (cc < ob) {
      const int O = cc / (Cin * T);
      const int rem = cc - O * Cin * T;
      c = rem / T;
      const int u = rem - c * T;
      gconv_base(d, O, a, b);
      gconv_rot(l, T, a, b);
      sp = (u + l) % T;
    } else {
      c = cc - ob;
      sp = l;
    }
    w[i] = psi[((((int64_t)(a + d.h) * k + (b + d.h)) * T + sp) * Cout + o) * Cin + c];
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
