// eql_launch.h -- internal launch interface between the C-ABI layer and the
// per-dtype kernel instantiation units.  Host code only.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace eqk {

inline int round_up(int v, int m) { return (v + m - 1) / m * m; }

// Plan of the forward / input-gradient kernel for one direction (Ci -> Co).
// Mirrors eql_gemm_kernel in eql_gemm.h: KW contraction channels per lane and
// step; each wave of a pair computes OT output tiles of 16, so an o-chunk is
// 32*OT channels.  Accumulators per lane (T*OT*4 floats) stay at or below 96
// so two waves fit on each SIMD; the resident-spectrum variant uses half.
struct GemmPlan {
  int kw, kstep;   // channels per lane group and per step
  int n_ks;        // contraction steps
  int OT, OC;      // o-tiles per wave, channels per chunk
  int n_oc;        // o-chunks
  bool res;        // spectrum resident across o-chunks
  int Co_pad;      // padded weight rows (n_oc * OC)
};
inline int gemm_kw(int T, bool f16) {
  const int fit = 128 / (T * (f16 ? 2 : 4));
  if (f16) return fit >= 8 ? 8 : 4;
  return fit >= 8 ? 8 : fit >= 4 ? 4 : fit >= 2 ? 2 : 1;
}
// o-tiles per wave: at most 96 accumulator floats per lane (T*OT*4), and the
// two weight buffers plus the spectrum buffer within 160 KB of LDS.
constexpr int gemm_otmax_c(int T, int kw, int eb) {
  const int rb = 4 * kw * eb;
  const int by_acc = 24 / T > 8 ? 8 : (24 / T < 1 ? 1 : 24 / T);
  const int by_lds = 163840 / (64 * T * rb) - 1;
  return by_acc < by_lds ? by_acc : (by_lds < 1 ? 1 : by_lds);
}
inline int gemm_otmax(int T, bool f16) { return gemm_otmax_c(T, gemm_kw(T, f16), f16 ? 2 : 4); }
inline int gemm_otres(int T, bool f16) {
  return gemm_otmax(T, f16) / 2 < 1 ? 1 : gemm_otmax(T, f16) / 2;
}
inline GemmPlan gemm_plan(int T, int Ci, int Co, bool f16) {
  GemmPlan p{};
  p.kw = gemm_kw(T, f16);
  p.kstep = 4 * p.kw;
  p.n_ks = (Ci + p.kstep - 1) / p.kstep;
  const int per_wave = ((Co + 15) / 16 + 1) / 2;  // o-tiles per wave for one chunk
  const int otmax = gemm_otmax(T, f16);
  if (per_wave <= otmax) {
    p.OT = per_wave <= 1 ? 1 : per_wave <= 2 ? 2 : (per_wave <= 4 && otmax >= 4) ? 4 : otmax;
    if (p.OT > otmax) p.OT = otmax;
    p.n_oc = 1;
    p.res = false;
  } else if (T <= 8 && p.n_ks <= 3 && p.kw * (f16 ? 2 : 4) <= 16) {
    p.OT = gemm_otres(T, f16);
    p.n_oc = (Co + 32 * p.OT - 1) / (32 * p.OT);
    p.res = true;
  } else {
    p.OT = otmax;
    p.n_oc = (Co + 32 * otmax - 1) / (32 * otmax);
    p.res = false;
  }
  p.OC = 32 * p.OT;
  p.Co_pad = p.n_oc * p.OC;
  return p;
}

// Padded extents of the weight spectrum: rows to the o-chunks of the pass that
// reads the layout, columns to 32 (a multiple of every contraction step).
constexpr int kColPad = 32;
struct WspecDims {
  int CoF, CiF, CinB, CoutB;
};
inline WspecDims wspec_dims(int T, int Cin, int Cout, bool f16) {
  return {gemm_plan(T, Cin, Cout, f16).Co_pad, round_up(Cin, kColPad),
          gemm_plan(T, Cout, Cin, f16).Co_pad, round_up(Cout, kColPad)};
}

// Compute units of the current device (cached); 256 if unknown.
int device_cu_count();

// Plan of the split-row weight gradient: workgroup tile (a WGC x WGO wave grid
// of CT x OTW tiles of 16 channels per wave), split count and the padded
// partial extents.  Depends only on the problem, not on the device, so results
// are reproducible across devices of the same model.
struct WgradPlan {
  int wgc, ct, otw; // variant: wave grid rows (WGO = 8 / wgc), tiles per wave
  int BC, BO;       // channel tile of one workgroup
  int KR;           // rows per chunk
  int n_ct, n_ot;   // channel tiles
  int S;            // splits
  int64_t rows_per_split;
  int Cin_pad, Cout_pad;
  size_t part_bytes, dbpart_bytes;
};
WgradPlan wgrad_plan(int64_t N, int T, int Cin, int Cout, bool f16);

struct GemmArgs {
  const void* in;
  const void* wsp;   // plane block of the layout this pass reads
  const void* bias;  // forward only; may be null
  void* out;
  int64_t N;
  int Ci, Co, Ci_pad;
  GemmPlan plan;
  hipStream_t stream;
};

struct WgradArgs {
  const void* x;
  const void* dy;
  void* dw;
  void* db;          // may be null
  float* part;
  float* dbpart;
  int64_t N;
  int Cin, Cout;
  hipStream_t stream;
};

hipError_t launch_wspec_f32(int T, const void* w, void* wspec, int Cin, int Cout, hipStream_t s);
hipError_t launch_wspec_f16(int T, const void* w, void* wspec, int Cin, int Cout, hipStream_t s);
hipError_t launch_gemm_f32(int T, bool bwd, const GemmArgs& a);
hipError_t launch_gemm_f16(int T, bool bwd, const GemmArgs& a);
hipError_t launch_wgrad_f32(int T, const WgradArgs& a, const WgradPlan& p);
hipError_t launch_wgrad_f16(int T, const WgradArgs& a, const WgradPlan& p);

}  // namespace eqk
