// eql_kernels.h -- gfx950 kernel templates of the C_T equivariant linear layer.
//
//   eql_wspec_kernel        weight spectrum (Alg. 1 step 1 applied to the shared
//                           parameters, Sec. 3.2.1 Eq. 4), stored as T real planes
//   (eql_gemm_kernel, the forward and input-gradient kernel, is in eql_gemm.h)
//   (the weight-gradient kernels are in eql_wgrad.h)
//
// Layout conventions (row-major): x[N,Cin,T], y[N,Cout,T], w[T,Cout,Cin].
#pragma once
#include "eql_common.h"

namespace eqk {

// ---------------------------------------------------------------------------
// Weight spectrum.  For every (o, c): the T lags w[0..T-1, o, c] are transformed
// by the same real DFT as the activations, giving What_k[o, c] in plane form.
// Two zero-padded copies are written:
//   forward  layout  F[p][o][c], dims [T][CoF][CiF]     (operand of the forward)
//   backward layout  B[p][c][o], dims [T][CinB][CoutB]  (operand of the input gradient)
// A workgroup of 256 threads owns a 16 x 16 tile of (o, c), one element per
// thread (small tiles give many workgroups, hence many loads in flight, for
// this small, latency-bound kernel): it reads w along c, writes F along c, and
// writes B along o from a transposed copy in LDS.  Every extent is a multiple
// of 32; tiles cover the larger of the two layouts' extents, and entries past
// Cout or Cin are zero.
template <int T, bool F16>
__global__ __launch_bounds__(256) void eql_wspec_kernel(const void* __restrict__ w,
                                                        void* __restrict__ wspec, int Cin, int Cout,
                                                        int CoF, int CiF, int CinB, int CoutB) {
  using E = typename Elem<F16>::T;
  __shared__ E tile[T][16][17];  // [p][c][o]
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int o0 = blockIdx.x * 16, c0 = blockIdx.y * 16;
  const E* wp = reinterpret_cast<const E*>(w);
  E* F = reinterpret_cast<E*>(wspec);
  E* Bl = F + (int64_t)T * CoF * CiF;
  {
    const int o = o0 + ty, c = c0 + tx;
    const bool ok = o < Cout && c < Cin;
    float v[T], P[T];
#pragma unroll
    for (int j = 0; j < T; ++j) v[j] = ok ? (float)wp[((int64_t)j * Cout + o) * Cin + c] : 0.0f;
    rdft<T>(v, P);
#pragma unroll
    for (int p = 0; p < T; ++p) {
      const E e = (E)P[p];
      tile[p][tx][ty] = e;
      if (o < CoF && c < CiF) F[((int64_t)p * CoF + o) * CiF + c] = e;
    }
  }
  __syncthreads();
  const int c = c0 + ty, o = o0 + tx;
  if (c < CinB && o < CoutB) {
#pragma unroll
    for (int p = 0; p < T; ++p) Bl[((int64_t)p * CinB + c) * CoutB + o] = tile[p][ty][tx];
  }
}

}  // namespace eqk
