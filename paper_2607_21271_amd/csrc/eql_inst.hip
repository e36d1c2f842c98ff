// eql_inst.hip -- kernel instantiations and launches for one group order and
// element type.  Compiled once per (T, dtype) with -DEQK_T=<1..16> and
// -DEQK_F16=<0|1>, so the instantiations build in parallel.
#include "eql_launch_impl.h"

#if !defined(EQK_T) || !defined(EQK_F16)
#error "compile with -DEQK_T=<1..16> -DEQK_F16=<0|1>"
#endif

namespace eqk {

template <int T, bool F16>
hipError_t Inst<T, F16>::wspec(const void* w, void* wspec, int Cin, int Cout, hipStream_t s) {
  return wspec_t<T, F16>(w, wspec, Cin, Cout, s);
}

template <int T, bool F16>
hipError_t Inst<T, F16>::gemm(bool bwd, const GemmArgs& a) {
  return bwd ? gemm_t<T, F16, true>(a) : gemm_t<T, F16, false>(a);
}

template <int T, bool F16>
hipError_t Inst<T, F16>::wgrad(const WgradArgs& a, const WgradPlan& p) {
  return wgrad_t<T, F16>(a, p);
}

template <int T, bool F16>
hipError_t Inst<T, F16>::bwd_fused(const FusedArgs& a, const FusedPlan& p) {
  return fused_t<T, F16>(a, p);
}

template struct Inst<EQK_T, (EQK_F16 != 0)>;

}  // namespace eqk
