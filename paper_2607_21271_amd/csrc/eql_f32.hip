// eql_f32.hip -- f32 instantiations of the weight-spectrum, spectral-GEMM and
// weight-gradient kernels for T = 1..16.
#include "eql_launch_impl.h"

namespace eqk {

hipError_t launch_wspec_f32(int T, const void* w, void* wspec, int Cin, int Cout, hipStream_t s) {
#define EQK_CALL(t) wspec_t<t, false>(w, wspec, Cin, Cout, s)
  EQK_T_SWITCH(T, EQK_CALL)
#undef EQK_CALL
}

hipError_t launch_gemm_f32(int T, bool bwd, const GemmArgs& a) {
  if (bwd) {
#define EQK_CALL(t) gemm_t<t, false, true>(a)
    EQK_T_SWITCH(T, EQK_CALL)
#undef EQK_CALL
  }
#define EQK_CALL(t) gemm_t<t, false, false>(a)
  EQK_T_SWITCH(T, EQK_CALL)
#undef EQK_CALL
}

hipError_t launch_wgrad_f32(int T, const WgradArgs& a, const WgradPlan& p) {
#define EQK_CALL(t) wgrad_t<t, false>(a, p)
  EQK_T_SWITCH(T, EQK_CALL)
#undef EQK_CALL
}

}  // namespace eqk
