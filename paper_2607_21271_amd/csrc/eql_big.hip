// eql_big.hip -- instantiations and launch of the large-tile forward /
// input-gradient kernel (eql_gemm_big.h).  Built without the flag that keeps
// MFMA accumulators in the general registers: this kernel's accumulators
// (T * 64 per lane) live in the accumulation registers.
#include "eql_gemm_big.h"
#include "eql_launch.h"

namespace eqk {
namespace {

template <int T, int DT, bool BWD>
hipError_t big_t(const BigArgs& a) {
  auto k = eql_gemm_big_kernel<T, DT, BWD>;
  const int lds = big_lds_bytes(T);
  hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  const int64_t n_rt = (a.N + kBigBM - 1) / kBigBM;
  const int n_ct = (a.Co + kBigBN - 1) / kBigBN;
  if (n_rt * n_ct >= ((int64_t)1 << 31) || a.w_rows < a.Co || a.w_pitch < a.Ci) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k, dim3((unsigned)(n_rt * n_ct)), dim3(kBigThreads), lds, a.stream, a.in, a.wsp, a.bias,
                     a.out, a.N, a.Ci, a.Co, a.w_rows, a.w_pitch, (int)n_rt, n_ct);
  return hipGetLastError();
}

template <int DT>
hipError_t big_dt(int T, bool bwd, const BigArgs& a) {
  if (T == 2) return bwd ? big_t<2, DT, true>(a) : big_t<2, DT, false>(a);
  if (T == 4) return bwd ? big_t<4, DT, true>(a) : big_t<4, DT, false>(a);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm_big(int dt, int T, bool bwd, const BigArgs& a) {
  if (!gemm_big_fits(T, a.Ci, a.Co, dt != kF32)) return hipErrorInvalidValue;
  if (dt == kF16) return big_dt<kF16>(T, bwd, a);
  if (dt == kBF16) return big_dt<kBF16>(T, bwd, a);
  return hipErrorInvalidValue;
}

}  // namespace eqk
