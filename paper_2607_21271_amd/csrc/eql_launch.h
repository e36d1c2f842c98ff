// eql_launch.h -- internal launch interface between the C-ABI layer and the
// per-dtype kernel instantiation units.  Host code only.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace eqk {

// Padded extents of the weight spectrum (see eql_wspec_kernel): rows are padded
// to the largest output-channel tile, columns to the contraction chunk.
constexpr int kRowPad = 128;
constexpr int kColPad = 32;
inline int round_up(int v, int m) { return (v + m - 1) / m * m; }

struct WspecDims {
  int CoF, CiF, CinB, CoutB;
};
inline WspecDims wspec_dims(int Cin, int Cout) {
  return {round_up(Cout, kRowPad), round_up(Cin, kColPad), round_up(Cin, kRowPad),
          round_up(Cout, kColPad)};
}

// Plan of the split-row weight gradient: tile sizes, split count and the
// padded partial extents.  Depends only on the problem, not on the device,
// so results are reproducible across devices of the same model.
struct WgradPlan {
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
  int Ci, Co, Ci_pad, Co_pad;
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
