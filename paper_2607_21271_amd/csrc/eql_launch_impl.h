// eql_launch_impl.h -- tile choice and launches for one element type.  Included
// by exactly one instantiation unit per dtype (EQK_F16 = 0 or 1).
#pragma once
#include "eql_kernels.h"
#include "eql_launch.h"

namespace eqk {

template <int T, bool F16>
hipError_t wspec_t(const void* w, void* wspec, int Cin, int Cout, hipStream_t s) {
  const WspecDims d = wspec_dims(Cin, Cout);
  const int64_t OD = d.CoF > d.CoutB ? d.CoF : d.CoutB;
  const int64_t CD = d.CiF > d.CinB ? d.CiF : d.CinB;
  const int64_t total = OD * CD;
  const unsigned blocks = (unsigned)((total + 255) / 256);
  hipLaunchKernelGGL((eql_wspec_kernel<T, F16>), dim3(blocks), dim3(256), 0, s, w, wspec, Cin,
                     Cout, d.CoF, d.CiF, d.CinB, d.CoutB);
  return hipGetLastError();
}

template <int T, bool F16, bool BWD, int BM, int WO>
hipError_t gemm_variant(const GemmArgs& a) {
  constexpr int BO = 4 * WO;
  const int64_t n_rt = (a.N + BM - 1) / BM;
  const int n_ot = (a.Co + BO - 1) / BO;
  const int64_t n_tiles = n_rt * n_ot;
  const int64_t grid = (n_tiles + 7) / 8 * 8;
  hipLaunchKernelGGL((eql_gemm_kernel<T, F16, BWD, BM, WO>), dim3((unsigned)grid), dim3(256), 0,
                     a.stream, a.in, a.wsp, a.bias, a.out, a.N, a.Ci, a.Co, a.Ci_pad, a.Co_pad,
                     n_ot, (int)n_tiles);
  return hipGetLastError();
}

// Accumulators per lane are T * (WO/16) * (BM/16) * 4 floats; the variants keep
// that at or below 128 so they stay resident beside the operand fragments.
template <int T, bool F16, bool BWD>
hipError_t gemm_t(const GemmArgs& a) {
  if constexpr (T <= 8) {
    if (a.Co > 64) return gemm_variant<T, F16, BWD, 32, 32>(a);
    return gemm_variant<T, F16, BWD, 64, 16>(a);
  } else {
    return gemm_variant<T, F16, BWD, 32, 16>(a);
  }
}

template <int T, bool F16, int BC, int BO>
hipError_t wgrad_variant(const WgradArgs& a, const WgradPlan& p) {
  const int per = p.n_ct * p.n_ot;
  if (p.S > 0) {
    const int64_t n_tiles = (int64_t)p.S * per;
    const int64_t grid = (n_tiles + 7) / 8 * 8;
    hipLaunchKernelGGL((eql_wgrad_kernel<T, F16, BC, BO>), dim3((unsigned)grid), dim3(256), 0,
                       a.stream, a.x, a.dy, a.part, a.db ? a.dbpart : nullptr, a.N, a.Cin, a.Cout,
                       p.rows_per_split, p.n_ct, p.n_ot, (int)n_tiles, p.Cin_pad, p.Cout_pad);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t total = (int64_t)a.Cout * a.Cin + a.Cout;
  hipLaunchKernelGGL((eql_wgrad_reduce_kernel<T, F16>), dim3((unsigned)((total + 255) / 256)),
                     dim3(256), 0, a.stream, a.part, a.dbpart, a.dw, a.db, p.S, a.Cin, a.Cout,
                     p.Cin_pad, p.Cout_pad);
  return hipGetLastError();
}

template <int T, bool F16>
hipError_t wgrad_t(const WgradArgs& a, const WgradPlan& p) {
  // The plan picks 64 x 64 tiles for T <= 8 and 32 x 32 above (see wgrad_plan).
  if constexpr (T <= 8) {
    if (p.BC != 64) return hipErrorInvalidValue;
    return wgrad_variant<T, F16, 64, 64>(a, p);
  } else {
    if (p.BC != 32) return hipErrorInvalidValue;
    return wgrad_variant<T, F16, 32, 32>(a, p);
  }
}

#define EQK_T_SWITCH(T_, CALL)       \
  switch (T_) {                      \
    case 1: return CALL(1);          \
    case 2: return CALL(2);          \
    case 3: return CALL(3);          \
    case 4: return CALL(4);          \
    case 5: return CALL(5);          \
    case 6: return CALL(6);          \
    case 7: return CALL(7);          \
    case 8: return CALL(8);          \
    case 9: return CALL(9);          \
    case 10: return CALL(10);        \
    case 11: return CALL(11);        \
    case 12: return CALL(12);        \
    case 13: return CALL(13);        \
    case 14: return CALL(14);        \
    case 15: return CALL(15);        \
    case 16: return CALL(16);        \
    default: return hipErrorInvalidValue; \
  }

}  // namespace eqk
