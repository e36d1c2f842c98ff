// eql_dispatch.cpp -- run-time dispatch over the group order T (1..16) and the
// element type to the per-(T, dtype) launch objects of eql_inst.hip.
#include "eql_launch.h"

namespace eqk {
namespace {

template <int DT, typename F>
hipError_t by_t(int T, F&& f) {
  switch (T) {
#define EQK_CASE(t) \
  case t: return f(Inst<t, DT>{});
    EQK_CASE(1) EQK_CASE(2) EQK_CASE(3) EQK_CASE(4) EQK_CASE(5) EQK_CASE(6) EQK_CASE(7)
    EQK_CASE(8) EQK_CASE(9) EQK_CASE(10) EQK_CASE(11) EQK_CASE(12) EQK_CASE(13) EQK_CASE(14)
    EQK_CASE(15) EQK_CASE(16)
#undef EQK_CASE
    default: return hipErrorInvalidValue;
  }
}

template <typename F>
hipError_t by_type(int dt, int T, F&& f) {
  if (dt == kF16) return by_t<kF16>(T, f);
  if (dt == kBF16) return by_t<kBF16>(T, f);
  if (dt == kF32) return by_t<kF32>(T, f);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_wspec(int dt, int T, const void* w, void* wspec, int Cin, int Cout, hipStream_t s) {
  return by_type(dt, T, [&](auto inst) { return decltype(inst)::wspec(w, wspec, Cin, Cout, s); });
}

hipError_t launch_gemm(int dt, int T, bool bwd, const GemmArgs& a) {
  return by_type(dt, T, [&](auto inst) { return decltype(inst)::gemm(bwd, a); });
}

hipError_t launch_gemm_gather(int dt, int T, const GemmArgs& a) {
  return by_type(dt, T, [&](auto inst) { return decltype(inst)::gemm_gather(a); });
}

hipError_t launch_wgrad(int dt, int T, const WgradArgs& a, const WgradPlan& p) {
  return by_type(dt, T, [&](auto inst) { return decltype(inst)::wgrad(a, p); });
}

hipError_t launch_bwd_fused(int dt, int T, const FusedArgs& a, const FusedPlan& p) {
  return by_type(dt, T, [&](auto inst) { return decltype(inst)::bwd_fused(a, p); });
}

}  // namespace eqk
