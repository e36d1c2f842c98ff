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
// A workgroup of 256 threads owns a tile of kWsC = 64 input channels x WO
// output channels (WO = 256 * VEC / 64: 32 for 16-bit elements, 16 for fp32).  Thread
// (o, chunk) loads VEC = 16 / EB consecutive input channels of one output
// channel at every lag, all T loads in flight at once (one memory round
// trip), transforms them in fp32, rounds once, writes the VEC entries of F as
// one 16-byte run per plane and stages them in LDS; the tile is then written
// to B from LDS, VEC consecutive output channels (16 bytes) per thread and
// plane.  Every extent is a multiple of 32; tiles cover the larger of the two
// layouts' extents, and entries past Cout or Cin are zero.  Inputs whose base
// or row stride is not a multiple of 16 bytes are read element by element.
constexpr int kWsC = 64;
template <int T, int DT>
__global__ __launch_bounds__(256) void eql_wspec_kernel(const void* __restrict__ w,
                                                        void* __restrict__ wspec, int Cin, int Cout,
                                                        int CoF, int CiF, int CinB, int CoutB) {
  using E = typename Elem<DT>::T;
  constexpr int EB = Elem<DT>::bytes;
  constexpr int VEC = 16 / EB;             // channels per 16-byte run
  constexpr int CPR = kWsC / VEC;          // threads per output channel of the tile
  constexpr int WO = 256 / CPR;            // output channels per tile
  __shared__ __attribute__((aligned(16))) E tile[T][kWsC][WO];  // [p][c][o]
  const int tid = threadIdx.x;
  const int o0 = blockIdx.x * WO, c0 = blockIdx.y * kWsC;
  const E* wp = reinterpret_cast<const E*>(w);
  E* F = reinterpret_cast<E*>(wspec);
  E* Bl = F + (int64_t)T * CoF * CiF;
  {
    const int ol = tid / CPR, cl = (tid - ol * CPR) * VEC;
    const int o = o0 + ol, c = c0 + cl;
    float v[T][VEC];
    const bool vec_ok = Cin % VEC == 0 && (reinterpret_cast<uintptr_t>(w) & 15) == 0;
    if (vec_ok && o < Cout && c + VEC <= Cin) {
      u32x4 raw[T];
#pragma unroll
      for (int j = 0; j < T; ++j)
        raw[j] = *reinterpret_cast<const u32x4*>(wp + ((int64_t)j * Cout + o) * Cin + c);
#pragma unroll
      for (int j = 0; j < T; ++j) {
        E e[VEC];
        __builtin_memcpy(e, &raw[j], 16);
#pragma unroll
        for (int q = 0; q < VEC; ++q) v[j][q] = (float)e[q];
      }
    } else {
#pragma unroll
      for (int j = 0; j < T; ++j)
#pragma unroll
        for (int q = 0; q < VEC; ++q)
          v[j][q] = (o < Cout && c + q < Cin) ? (float)wp[((int64_t)j * Cout + o) * Cin + c + q] : 0.0f;
    }
    E P[T][VEC];
#pragma unroll
    for (int q = 0; q < VEC; ++q) {
      float u[T], U[T];
#pragma unroll
      for (int j = 0; j < T; ++j) u[j] = v[j][q];
      rdft<T>(u, U);
#pragma unroll
      for (int p = 0; p < T; ++p) P[p][q] = (E)U[p];
    }
#pragma unroll
    for (int p = 0; p < T; ++p) {
      if (o < CoF && c < CiF) {
        u32x4 run;
        __builtin_memcpy(&run, P[p], 16);
        *reinterpret_cast<u32x4*>(F + ((int64_t)p * CoF + o) * CiF + c) = run;
      }
#pragma unroll
      for (int q = 0; q < VEC; ++q) tile[p][cl + q][ol] = P[p][q];
    }
  }
  __syncthreads();
  {
    // thread (c, o-run): VEC consecutive output channels of input channel c
    constexpr int RPC = WO / VEC;          // runs per input channel
    const int cl = tid / RPC, ol = (tid - cl * RPC) * VEC;
    const int c = c0 + cl, o = o0 + ol;
    if (cl < kWsC && c < CinB && o < CoutB) {
#pragma unroll
      for (int p = 0; p < T; ++p)
        *reinterpret_cast<u32x4*>(Bl + ((int64_t)p * CinB + c) * CoutB + o) =
            *reinterpret_cast<const u32x4*>(&tile[p][cl][ol]);
    }
  }
}

}  // namespace eqk
