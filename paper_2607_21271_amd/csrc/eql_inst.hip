// eql_inst.hip -- kernel instantiations and launches for one group order and
// element type.  Compiled once per (T, dtype) with -DEQK_T=<1..16> and
// -DEQK_DT=<0|1|2> (fp32, fp16, bf16), so the instantiations build in parallel.
#include "eql_launch_impl.h"

#if !defined(EQK_T) || !defined(EQK_DT)
#error "compile with -DEQK_T=<1..16> -DEQK_DT=<0|1|2>"
#endif

namespace eqk {

template <int T, int DT>
hipError_t Inst<T, DT>::wspec(const void* w, void* wspec, int Cin, int Cout, hipStream_t s) {
  return wspec_t<T, DT>(w, wspec, Cin, Cout, s);
}

template <int T, int DT>
hipError_t Inst<T, DT>::gemm(bool bwd, const GemmArgs& a) {
  return bwd ? gemm_t<T, DT, true>(a) : gemm_t<T, DT, false>(a);
}

template <int T, int DT>
hipError_t Inst<T, DT>::gemm_gather(const GemmArgs& a) {
  return gemm_gather_t<T, DT>(a);
}

template <int T, int DT>
hipError_t Inst<T, DT>::wgrad(const WgradArgs& a, const WgradPlan& p) {
  return wgrad_t<T, DT>(a, p);
}

template <int T, int DT>
hipError_t Inst<T, DT>::bwd_fused(const FusedArgs& a, const FusedPlan& p) {
  return fused_t<T, DT>(a, p);
}

template struct Inst<EQK_T, EQK_DT>;

}  // namespace eqk
