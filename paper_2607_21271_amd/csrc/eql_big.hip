// eql_big.hip -- instantiations and launches of the large-tile kernels: the
// forward / input gradient (eql_gemm_big.h) and the weight gradient
// (eql_wgrad_big.h).  Built without the flag that keeps MFMA accumulators in
// the general registers: these kernels' accumulators (T * 64 per lane) live
// in the accumulation registers.
#include "eql_gemm_big.h"
#include "eql_launch.h"
#include "eql_wgrad_big.h"

namespace eqk {
namespace {

template <int T, int DT, bool BWD, bool GAUSS = false>
hipError_t big_t(const BigArgs& a) {
  auto k = eql_gemm_big_kernel<T, DT, BWD, GAUSS>;
  const int lds = big_lds_bytes(T, GAUSS);
  hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  const int64_t n_rt = (a.N + kBigBM - 1) / kBigBM;
  const int bn = big_bn(GAUSS);
  const int n_ct = (a.Co + bn - 1) / bn;
  if (n_rt * n_ct >= ((int64_t)1 << 31) || a.w_rows < a.Co || a.w_pitch < a.Ci) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k, dim3((unsigned)(n_rt * n_ct)), dim3(kBigThreads), lds, a.stream, a.in, a.wsp, a.bias,
                     a.out, a.N, a.Ci, a.Co, a.w_rows, a.w_pitch, (int)n_rt, n_ct);
  return hipGetLastError();
}

template <int DT>
hipError_t big_dt(int T, bool bwd, const BigArgs& a) {
  if (T == 2) return bwd ? big_t<2, DT, true>(a) : big_t<2, DT, false>(a);
  if constexpr (DT == kF32) {
    if (T == 4 && big_gauss(T, DT))
      return bwd ? big_t<4, DT, true, true>(a) : big_t<4, DT, false, true>(a);
  }
  if (T == 4) return bwd ? big_t<4, DT, true>(a) : big_t<4, DT, false>(a);
  return hipErrorInvalidValue;
}

template <int T, int DT, bool GAUSS = false>
hipError_t wgrad_big_t(const WgradArgs& a, const WgradPlan& p) {
  const int bo = wgrad_big_bo(GAUSS);
  const int kr = kWbRB / (DT == kF32 ? 4 : 2);
  if (p.kind != 2 || p.BC != kWbBC || p.BO != bo || p.KR != kr || p.rows_per_split % kWbKR != 0 ||
      p.Cin_pad % kWbBC != 0 || p.Cout_pad % bo != 0 || p.N_pad % 64 != 0 || !a.xs || !a.ds)
    return hipErrorInvalidValue;
  const int64_t n_rb = p.N_pad / 64;  // pre-pass blocks: 64 rows x 32 channels
  const int ncb_x = p.Cin_pad / 32, ncb_d = p.Cout_pad / 32;
  hipLaunchKernelGGL((eql_spec_rows_kernel<T, DT>), dim3((unsigned)(n_rb * ncb_x)), dim3(256), 0, a.stream, a.x,
                     a.xs, a.N, a.Cin, p.Cin_pad, p.N_pad, ncb_x);
  hipLaunchKernelGGL((eql_spec_rows_kernel<T, DT>), dim3((unsigned)(n_rb * ncb_d)), dim3(256), 0, a.stream, a.dy,
                     a.ds, a.N, a.Cout, p.Cout_pad, p.N_pad, ncb_d);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  auto k = eql_wgrad_big_kernel<T, DT, GAUSS>;
  const int lds = wgrad_big_lds_bytes(T, GAUSS);
  e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  const int64_t G = (int64_t)p.S * p.n_ct * p.n_ot;
  hipLaunchKernelGGL(k, dim3((unsigned)G), dim3(kBigThreads), lds, a.stream, a.xs, a.ds, a.part,
                     a.db ? a.dbpart : nullptr, p.N_pad, p.Cin_pad, p.Cout_pad, p.n_ct, p.n_ot, p.S,
                     p.rows_per_split);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_wgrad_big(int dt, int T, const WgradArgs& a, const WgradPlan& p) {
  if (!wgrad_big_fits(a.N, T, a.Cin, a.Cout, dt)) return hipErrorInvalidValue;
  if (dt == kF16) return T == 2 ? wgrad_big_t<2, kF16>(a, p) : T == 4 ? wgrad_big_t<4, kF16>(a, p) : hipErrorInvalidValue;
  if (dt == kBF16) return T == 2 ? wgrad_big_t<2, kBF16>(a, p) : T == 4 ? wgrad_big_t<4, kBF16>(a, p) : hipErrorInvalidValue;
  if (dt == kF32) {
    if (T == 2) return wgrad_big_t<2, kF32>(a, p);
    // the plan's o-tile names the form (96: three products)
    if (T == 4) return p.BO == wgrad_big_bo(true) ? wgrad_big_t<4, kF32, true>(a, p) : wgrad_big_t<4, kF32>(a, p);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm_big(int dt, int T, bool bwd, const BigArgs& a) {
  if (!gemm_big_fits(T, a.Ci, a.Co, dt)) return hipErrorInvalidValue;
  if (dt == kF16) return big_dt<kF16>(T, bwd, a);
  if (dt == kBF16) return big_dt<kBF16>(T, bwd, a);
  if (dt == kF32) return big_dt<kF32>(T, bwd, a);
  return hipErrorInvalidValue;
}

}  // namespace eqk
