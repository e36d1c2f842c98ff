// eql_dihedral.h -- the equivariant linear layer over the dihedral group D_T
// (rotations and reflections of a regular T-gon) on the C_T kernels: weight
// expansion and gradient folding.
//
// The C_T layer shares one weight block per group element (Sec. 3.1,
// Eq. 1-2); Sec. 5 names reflection groups as the next groups to cover.  Over
// D_T, with elements (t, m) = r^t s^m stored at m*T + t, the same rule reads
//   y[n,o,g] = sum_h sum_c W[h^-1 g][o][c] x[n,c,h] + b[o].
// Split by the reflection bits m_g of g and m_h of h, with j = t_g - t_h:
//   h^-1 g = ( j, m_g)          for m_h = 0,
//   h^-1 g = (-j, 1 xor m_g)    for m_h = 1,
// four circular convolutions along the rotation axis.  With the channels
// (c, m_h) -> 2c + m_h and (o, m_g) -> 2o + m_g -- the memory order of
// x [N, Cin, 2T] read as [N, 2Cin, T] -- this is the C_T layer with
// 2 Cin -> 2 Cout channels, the weight
//   w2[j][2o + m_g][2c + m_h] = W[(m_g xor m_h) T + ((-1)^m_h j mod T)][o][c]
// and the bias b2[2o + m_g] = b[o].  So every step of the rDFT path (and its
// T/2 saving) applies unchanged; the gradients with respect to W and b fold
// back from those of w2 and b2:
//   dW[q T + l][o][c] = sum_{m_g} dw2[(-1)^m_h l mod T][2o + m_g][2c + m_h],
//                       m_h = q xor m_g,
//   db[o] = db2[2o] + db2[2o + 1]
// (each W entry appears in w2 at exactly these two places).  Both kernels are
// weight-sized gathers; the fold sums in fp32 and rounds once.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace eqk {

template <typename E>
__global__ __launch_bounds__(256) void eql_dihedral_expand_kernel(const E* __restrict__ W,
                                                                  const E* __restrict__ b,
                                                                  E* __restrict__ w2,
                                                                  E* __restrict__ b2, int T, int Cin,
                                                                  int Cout) {
  const int C2 = 2 * Cin, O2 = 2 * Cout;
  const int64_t total = (int64_t)T * O2 * C2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int cc = (int)(i % C2);
    const int64_t r = i / C2;
    const int oo = (int)(r % O2);
    const int j = (int)(r / O2);
    const int c = cc >> 1, mh = cc & 1, o = oo >> 1, mg = oo & 1;
    const int l = mh ? (T - j) % T : j;
    w2[i] = W[((int64_t)((mg ^ mh) * T + l) * Cout + o) * Cin + c];
  }
  if (b2 != nullptr && blockIdx.x == 0)
    for (int oo = threadIdx.x; oo < O2; oo += blockDim.x) b2[oo] = b[oo >> 1];
}

template <typename E>
__global__ __launch_bounds__(256) void eql_dihedral_fold_kernel(const E* __restrict__ dw2,
                                                                const E* __restrict__ db2,
                                                                E* __restrict__ dW,
                                                                E* __restrict__ db, int T, int Cin,
                                                                int Cout) {
  const int C2 = 2 * Cin, O2 = 2 * Cout;
  const int64_t total = (int64_t)2 * T * Cout * Cin;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int c = (int)(i % Cin);
    const int64_t r = i / Cin;
    const int o = (int)(r % Cout);
    const int u = (int)(r / Cout);
    const int q = u / T, l = u - (u / T) * T;
    float s = 0.0f;
#pragma unroll
    for (int mg = 0; mg < 2; ++mg) {
      const int mh = q ^ mg;
      const int j = mh ? (T - l) % T : l;
      s += (float)dw2[((int64_t)j * O2 + 2 * o + mg) * C2 + 2 * c + mh];
    }
    dW[i] = (E)s;
  }
  if (db != nullptr && blockIdx.x == 0)
    for (int o = threadIdx.x; o < Cout; o += blockDim.x)
      db[o] = (E)((float)db2[2 * o] + (float)db2[2 * o + 1]);
}

}  // namespace eqk
