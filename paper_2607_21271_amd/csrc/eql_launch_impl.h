// eql_launch_impl.h -- tile choice and launches for one group order and element
// type.  Included only by eql_inst.hip, which is compiled once per (T, dtype).
#pragma once
#include <mutex>

#include "eql_gemm.h"
#include "eql_kernels.h"
#include "eql_wgrad.h"
#include "eql_wgrad_rd.h"
#include "eql_bwd_fused.h"
#include "eql_launch.h"

namespace eqk {

template <int T, int DT>
hipError_t wspec_t(const void* w, void* wspec, int Cin, int Cout, hipStream_t s) {
  const WspecDims d = wspec_dims(T, Cin, Cout, DT != kF32);
  const int omax = d.CoF > d.CoutB ? d.CoF : d.CoutB;  // tiles cover both layouts
  const int cmax = d.CiF > d.CinB ? d.CiF : d.CinB;
  constexpr int WO = 256 * (DT != kF32 ? 8 : 4) / kWsC;  // output channels per tile (eql_wspec_kernel)
  hipLaunchKernelGGL((eql_wspec_kernel<T, DT>),
                     dim3((unsigned)((omax + WO - 1) / WO), (unsigned)((cmax + kWsC - 1) / kWsC)),
                     dim3(256), 0, s, w, wspec, Cin, Cout, d.CoF, d.CiF, d.CinB, d.CoutB);
  return hipGetLastError();
}

// Resident workgroups per CU of one kernel at a given dynamic LDS size,
// cached per (device, kernel, LDS).  The cache is shared by every host thread:
// lookups and inserts hold one mutex (an entry never changes once written).
inline int occupancy(const void* kernel, int threads, int lds) {
  struct Entry { const void* k; int dev, lds, occ; };
  static std::mutex mu;
  static Entry cache[512];
  static int n_cache = 0;
  int dev = 0;
  (void)hipGetDevice(&dev);
  {
    std::lock_guard<std::mutex> lock(mu);
    for (int i = 0; i < n_cache; ++i)
      if (cache[i].k == kernel && cache[i].dev == dev && cache[i].lds == lds) return cache[i].occ;
  }
  int occ = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, threads, lds) != hipSuccess || occ <= 0) {
    (void)hipGetLastError();
    occ = 1;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (n_cache < 512) cache[n_cache++] = Entry{kernel, dev, lds, occ};
  return occ;
}

// Persistent grid: one workgroup per resident slot (CUs x occupancy), and no
// workgroup with fewer than 32 rows.
inline int persistent_grid(const void* kernel, int threads, int lds, int64_t N, int64_t row_bytes) {
  const int64_t slots = (int64_t)device_cu_count() * occupancy(kernel, threads, lds);
  const int64_t by_rows = (N + 31) / 32;
  int64_t g = slots < by_rows ? slots : by_rows;
  if (g < 1) g = 1;
  // each workgroup addresses its rows (plus one round of slack) with 31-bit offsets
  while ((N / g + 65) * row_bytes >= ((int64_t)1 << 31)) g *= 2;
  return (int)g;
}

template <int T, int DT, bool BWD, int OT, int MODE, int NKR, bool NARROW = false, bool GATHER = false>
hipError_t gemm_variant(const GemmArgs& a) {
  static_assert(GemmShape<T, DT>::WV == gemm_wide_load_c(T, DT != kF32), "host and kernel load widths");
  auto k = eql_gemm_kernel<T, DT, BWD, OT, MODE, NKR, NARROW, GATHER>;
  const int lds = a.plan.lds_bytes;
  if (lds != gemm_lds_c(T, DT != kF32, OT, gemm_wblocks(MODE, a.plan.n_oc, a.plan.n_ks)) || lds > kLdsBytes ||
      (MODE == kRes && a.plan.n_ks != NKR))
    return hipErrorInvalidValue;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
  }
  // input and output rows are addressed with 31-bit offsets per workgroup
  const int grid = persistent_grid((const void*)k, kGemmThreads, lds, a.N,
                                   (int64_t)(a.Ci > a.Co ? a.Ci : a.Co) * T * (DT != kF32 ? 2 : 4));
  hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(kGemmThreads), lds, a.stream, a.in, a.wsp, a.bias, a.out,
                     a.N, a.Ci, a.Co, a.Ci_pad, a.plan.Co_pad, a.plan.n_oc, a.plan.n_ks, a.geo);
  return hipGetLastError();
}

template <int T, int DT, bool BWD, int MODE, bool GATHER = false>
hipError_t gemm_ot(const GemmArgs& a) {
  hipError_t r = hipErrorInvalidValue;
  static_for<8>([&](auto oi) {
    constexpr int OT = decltype(oi)::value + 1;
    if constexpr (gemm_ot_inst(T, DT != kF32, OT)) {
      if (a.plan.OT == OT) r = gemm_variant<T, DT, BWD, OT, MODE, 0, false, GATHER>(a);
    }
  });
  return r;
}

// Forward with the implicit patch gather (group convolution, T in {1, 2,
// 4}): the plan's mode is streamed or resident weights, never narrow loads.
template <int T, int DT>
hipError_t gemm_gather_t(const GemmArgs& a) {
  if constexpr (T == 1 || T == 2 || T == 4) {
    const GemmPlan& p = a.plan;
    if (p.narrow) return hipErrorInvalidValue;
    if (p.mode == kStat) return gemm_ot<T, DT, false, kStat, true>(a);
    if (p.mode == kStream) return gemm_ot<T, DT, false, kStream, true>(a);
  }
  return hipErrorInvalidValue;
}

template <int T, int DT, bool BWD>
hipError_t gemm_t(const GemmArgs& a) {
  constexpr int OTR = gemm_otmax_c(T, DT != kF32) / 2 < 1 ? 1 : gemm_otmax_c(T, DT != kF32) / 2;
  constexpr bool kResOk = T <= 8 && GemmShape<T, DT>::FB <= 16;
  const GemmPlan& p = a.plan;
  if (p.narrow) {
    if (p.OT != 1 || p.mode != kStream) return hipErrorInvalidValue;
    return gemm_variant<T, DT, BWD, 1, kStream, 0, true>(a);
  }
  if (((int64_t)a.Ci * T * (DT != kF32 ? 2 : 4)) % GemmShape<T, DT>::WV != 0) return hipErrorInvalidValue;
  if (p.mode == kRes) {
    if constexpr (kResOk) {
      if (p.OT != OTR) return hipErrorInvalidValue;
      if (p.n_ks == 1) return gemm_variant<T, DT, BWD, OTR, kRes, 1>(a);
      if (p.n_ks == 2) return gemm_variant<T, DT, BWD, OTR, kRes, 2>(a);
      if (p.n_ks == 3) return gemm_variant<T, DT, BWD, OTR, kRes, 3>(a);
    }
    return hipErrorInvalidValue;
  }
  if (p.mode == kStat) return gemm_ot<T, DT, BWD, kStat>(a);
  if (p.mode == kStream) return gemm_ot<T, DT, BWD, kStream>(a);
  return hipErrorInvalidValue;
}

// The split-partial reduction (both weight-gradient kernels write the same
// partial layout).
template <int T, int DT>
hipError_t wgrad_reduce(const WgradArgs& a, const WgradPlan& p);

template <int T, int DT, int CT, int OT>
hipError_t wgrad_rd_variant(const WgradArgs& a, const WgradPlan& p) {
  if (p.S > 0) {
    constexpr int NW = kRdWaves;
    const int lds = (NW - 1) * rd_wave_acc_bytes<T, CT, OT>() + NW * OT * 16 * 4;
    auto k = eql_wgrad_rd_kernel<T, DT, CT, OT, NW>;
    if (lds > kLdsBytes) return hipErrorInvalidValue;
    if (lds > 64 * 1024) {
      hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
      if (e != hipSuccess) return e;
    }
    const int64_t G = (int64_t)p.S * p.n_ct * p.n_ot;
    const int64_t blocks = (G + 7) / 8 * 8;  // whole groups of 8 (one per XCD)
    hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(64 * NW), lds, a.stream, a.x, a.dy, a.part,
                       a.db ? a.dbpart : nullptr, a.N, a.Cin, a.Cout, p.rows_per_split, p.n_ct,
                       p.n_ot, p.S, p.Cin_pad, p.Cout_pad);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return wgrad_reduce<T, DT>(a, p);
}

template <int T, int DT, int WGC, int CT, int OTW>
hipError_t wgrad_variant(const WgradArgs& a, const WgradPlan& p) {
  if (p.S > 0) {
    // whole groups of 8 splits (see the tile order in eql_wgrad_kernel)
    const int64_t n_blocks = (int64_t)(p.S + 7) / 8 * 8 * p.n_ct * p.n_ot;
    hipLaunchKernelGGL((eql_wgrad_kernel<T, DT, WGC, 8 / WGC, CT, OTW>), dim3((unsigned)n_blocks),
                       dim3(512), 0, a.stream, a.x, a.dy, a.part, a.db ? a.dbpart : nullptr, a.N,
                       a.Cin, a.Cout, p.rows_per_split, p.n_ct, p.n_ot, p.S, p.Cin_pad,
                       p.Cout_pad);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return wgrad_reduce<T, DT>(a, p);
}

template <int T, int DT>
hipError_t wgrad_reduce(const WgradArgs& a, const WgradPlan& p) {
  // threads, items per workgroup and split groups of eql_wgrad_reduce_kernel
  const int64_t items = (int64_t)(p.Cin_pad / 4) * p.Cout_pad;
  int nthr = 0, ipw = 0, G = 0;
  wgrad_reduce_shape(T, p.S, items, nthr, ipw, G);
  const int NS = nthr / G;
  const unsigned blocks =
      (unsigned)((items + ipw - 1) / ipw + (a.db ? (a.Cout + NS - 1) / NS : 0));
  if (nthr == 256)
    hipLaunchKernelGGL((eql_wgrad_reduce_kernel<T, DT, 256>), dim3(blocks), dim3(256), 0, a.stream,
                       a.part, a.dbpart, a.dw, a.db, p.S, a.Cin, a.Cout, p.Cin_pad, p.Cout_pad, ipw, G);
  else
    hipLaunchKernelGGL((eql_wgrad_reduce_kernel<T, DT, 1024>), dim3(blocks), dim3(1024), 0, a.stream,
                       a.part, a.dbpart, a.dw, a.db, p.S, a.Cin, a.Cout, p.Cin_pad, p.Cout_pad, ipw, G);
  return hipGetLastError();
}

// Single-pass backward: the fused kernel (one workgroup per row split), then
// the split-partial reduction of the weight gradient.
template <int T, int DT, int WGC, int CT, int OTW>
hipError_t fused_variant(const FusedArgs& f, const FusedPlan& p) {
  constexpr int BC = WGC * 16 * CT, BO = (8 / WGC) * 16 * OTW;
  constexpr int KR = DT != kF32 ? 32 : 16;
  if (p.BC != BC || p.BO != BO || p.KR != KR || p.nks * KR > BO || p.C16 > BC ||
      p.lds != fused_lds_bytes(T, BC, BO, KR, p.nks, p.C16, p.dbuf != 0) || p.lds > kLdsBytes)
    return hipErrorInvalidValue;
  WgradArgs a{};
  a.x = f.x;
  a.dy = f.dy;
  a.dw = f.dw;
  a.db = f.db;
  a.part = f.part;
  a.dbpart = f.dbpart;
  a.N = f.N;
  a.Cin = f.Cin;
  a.Cout = f.Cout;
  a.stream = f.stream;
  WgradPlan wp{};
  wp.S = p.S;
  wp.Cin_pad = BC;
  wp.Cout_pad = BO;
  if (p.S > 0) {
    auto k = eql_bwd_fused_kernel<T, DT, WGC, CT, OTW>;
    if (p.lds > 64 * 1024) {
      hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, p.lds);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k, dim3((unsigned)p.S), dim3(512), p.lds, f.stream, f.x, f.dy, f.wsp, f.dx, f.part,
                       f.db ? f.dbpart : nullptr, f.N, f.Cin, f.Cout, p.rows_per_split, p.S, f.CinB,
                       f.CoutB, p.nks, p.dbuf);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return wgrad_reduce<T, DT>(a, wp);
}

template <int T, int DT>
hipError_t fused_t(const FusedArgs& f, const FusedPlan& p) {
  // the variants of fused_plan that fit the registers (fused_variant_ok)
#define EQK_FU(W_, C_, O_)                                                  \
  if constexpr (DT != kBF16 && fused_variant_ok(T, DT == kF16, W_, C_, O_)) { \
    if (p.wgc == (W_) && p.ct == (C_) && p.otw == (O_))                    \
      return fused_variant<T, DT, W_, C_, O_>(f, p);                       \
  }
  EQK_FU(2, 1, 1)
  EQK_FU(4, 1, 1)
  EQK_FU(2, 1, 2)
  EQK_FU(2, 2, 1)
  EQK_FU(2, 1, 3)
#undef EQK_FU
  return hipErrorInvalidValue;
}

template <int T, int DT>
hipError_t wgrad_t(const WgradArgs& a, const WgradPlan& p) {
  // large-tile plan: its pre-passes and product kernel ran (launch_wgrad_big)
  if (p.kind == 2) return wgrad_reduce<T, DT>(a, p);
  if (p.kind == 1) {
#define EQK_RD(C_, O_)                                             \
  if constexpr (rd_fits(T, C_, O_)) {                              \
    if (p.ct == (C_) && p.otw == (O_)) return wgrad_rd_variant<T, DT, C_, O_>(a, p); \
  }
    EQK_RD(1, 1)
    EQK_RD(1, 2)
    EQK_RD(2, 1)
    EQK_RD(2, 2)
    EQK_RD(2, 4)
    EQK_RD(4, 2)
#undef EQK_RD
    return hipErrorInvalidValue;
  }
  // the variants of wgrad_plan whose accumulators fit (CT * OTW * T * 4 <= 96)
#define EQK_WG(W_, C_, O_)                                                                    \
  if constexpr ((C_) * (O_) * T * 4 <= 96 &&                                                 \
                T * ((W_) * 16 * (C_) + (8 / (W_)) * 16 * (O_)) * 64 <= 160 * 1024 - 4096) {   \
    if (p.wgc == (W_) && p.ct == (C_) && p.otw == (O_))                                      \
      return wgrad_variant<T, DT, W_, C_, O_>(a, p);                                         \
  }
  EQK_WG(2, 1, 1)
  EQK_WG(2, 2, 1)
  EQK_WG(2, 3, 1)
  EQK_WG(2, 1, 2)
  EQK_WG(2, 1, 3)
  EQK_WG(4, 1, 1)
  EQK_WG(4, 1, 2)
  EQK_WG(4, 1, 3)
#undef EQK_WG
  return hipErrorInvalidValue;
}

}  // namespace eqk
