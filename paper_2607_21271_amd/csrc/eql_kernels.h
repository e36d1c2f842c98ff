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
//   forward  layout  F[p][o][c], dims [T][CoF][CiF]     (A operand of the forward)
//   backward layout  B[p][c][o], dims [T][CinB][CoutB]  (A operand of the input gradient)
// Threads [0, CoF*CiF) fill F with c fastest; the next CinB*CoutB threads fill
// B with o fastest, so both sets of stores are coalesced.
template <int T, bool F16>
__global__ __launch_bounds__(256) void eql_wspec_kernel(const void* __restrict__ w,
                                                        void* __restrict__ wspec, int Cin, int Cout,
                                                        int CoF, int CiF, int CinB, int CoutB) {
  using E = typename Elem<F16>::T;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t nF = (int64_t)CoF * CiF;
  const int64_t nB = (int64_t)CinB * CoutB;
  int o, c;
  bool toF;
  if (idx < nF) {
    o = (int)(idx / CiF);
    c = (int)(idx - (int64_t)o * CiF);
    toF = true;
  } else if (idx < nF + nB) {
    const int64_t j = idx - nF;
    c = (int)(j / CoutB);
    o = (int)(j - (int64_t)c * CoutB);
    toF = false;
  } else {
    return;
  }
  float v[T];
  const E* wp = reinterpret_cast<const E*>(w);
  const bool ok = o < Cout && c < Cin;
#pragma unroll
  for (int j = 0; j < T; ++j) v[j] = ok ? (float)wp[((int64_t)j * Cout + o) * Cin + c] : 0.0f;
  float P[T];
  rdft<T>(v, P);
  E* F = reinterpret_cast<E*>(wspec);
  if (toF) {
#pragma unroll
    for (int p = 0; p < T; ++p) F[((int64_t)p * CoF + o) * CiF + c] = (E)P[p];
  } else {
    E* Bl = F + (int64_t)T * CoF * CiF;
#pragma unroll
    for (int p = 0; p < T; ++p) Bl[((int64_t)p * CinB + c) * CoutB + o] = (E)P[p];
  }
}

}  // namespace eqk
