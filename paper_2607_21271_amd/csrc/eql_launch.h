// eql_launch.h -- internal launch interface between the C-ABI layer and the
// per-dtype kernel instantiation units.  Host code only.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>

#include "eql_config.h"

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
  int mode;        // GemmMode: 0 streamed weights, 1 + resident spectrum, 2 resident weights
  bool narrow;     // row stride not a multiple of the wide load: element loads, OT = 1, mode 0
  int Co_pad;      // padded weight rows (n_oc * OC)
  int lds_bytes;   // dynamic LDS of one workgroup
};
constexpr int kLdsBytes = 160 * 1024;
// w16: 16-bit elements (fp16 or bf16), which share every shape and layout.
constexpr int gemm_kw_c(int T, bool w16) {
  const int fit = 128 / (T * (w16 ? 2 : 4));
  if (w16) return fit >= 8 ? 8 : 4;
  return fit >= 8 ? 8 : fit >= 4 ? 4 : fit >= 2 ? 2 : 1;
}
inline int gemm_kw(int T, bool w16) { return gemm_kw_c(T, w16); }
constexpr int gemm_rb_c(int T, bool w16) { return 4 * gemm_kw_c(T, w16) * (w16 ? 2 : 4); }
// LDS of one workgroup with n_wblocks weight blocks: two spectrum buffers of
// 16*pairs*T rows and the blocks of 32*OT*T rows, each row RB bytes.
constexpr int gemm_lds_c(int T, bool w16, int OT, int n_wblocks) {
  return (2 * kGemmRoundRows * T + n_wblocks * 32 * OT * T) * gemm_rb_c(T, w16);
}
// o-tiles per wave: at most 96 accumulator floats per lane (T*OT*4), and two
// weight blocks plus the spectrum buffers within the LDS.
constexpr int gemm_otmax_c(int T, bool w16) {
  const int by_acc = 24 / T > 8 ? 8 : (24 / T < 1 ? 1 : 24 / T);
  int by_lds = 1;
  while (by_lds < 8 && gemm_lds_c(T, w16, by_lds + 1, 2) <= kLdsBytes) ++by_lds;
  return by_acc < by_lds ? by_acc : by_lds;
}
inline int gemm_otmax(int T, bool w16) { return gemm_otmax_c(T, w16); }
inline int gemm_otres(int T, bool w16) {
  return gemm_otmax(T, w16) / 2 < 1 ? 1 : gemm_otmax(T, w16) / 2;
}
// o-tile counts that have a kernel instantiation: 1, 2, 3, 4, 6, 8 up to the maximum.
constexpr bool gemm_ot_inst(int T, bool w16, int OT) {
  return OT >= 1 && OT <= gemm_otmax_c(T, w16) && (OT <= 4 || OT == 6 || OT == 8);
}
inline int gemm_ot_round(int T, bool w16, int want) {
  for (int ot = want; ot <= gemm_otmax(T, w16); ++ot)
    if (gemm_ot_inst(T, w16, ot)) return ot;
  return gemm_otmax(T, w16);
}
// Widest activation load of one lane's run (KW/2 channels x T elements); the
// row stride Ci*T*EB must be a multiple of it (eql_gemm.h GemmShape::WV).
constexpr int gemm_wide_load_c(int T, bool w16) {
  const int nbh = gemm_kw_c(T, w16) / 2 * T * (w16 ? 2 : 4);
  return nbh % 16 == 0 ? 16 : nbh % 8 == 0 ? 8 : 4;
}
// Weight blocks held in LDS: two streamed blocks, two regions of n_ks blocks
// (resident spectrum), or every block (resident weights).
constexpr int gemm_wblocks(int mode, int n_oc, int n_ks) {
  return mode == 2 ? n_oc * n_ks : mode == 1 ? 2 * n_ks : 2;
}
// EQL_GEMM_MODE=0/1/2 forces a weight mode where it is valid (tests, A/B timing).
int gemm_forced_mode();
inline GemmPlan gemm_plan(int T, int Ci, int Co, bool w16) {
  GemmPlan p{};
  p.kw = gemm_kw(T, w16);
  p.kstep = 4 * p.kw;
  p.n_ks = (Ci + p.kstep - 1) / p.kstep;
  const int per_wave = ((Co + 15) / 16 + 1) / 2;  // o-tiles per wave for one chunk
  const int otmax = gemm_otmax(T, w16);
  // resident spectrum: two LDS regions of n_ks weight blocks each
  const bool res_ok = T <= 8 && p.n_ks <= 3 && p.kw * (w16 ? 2 : 4) <= 16 &&
                      gemm_lds_c(T, w16, gemm_otres(T, w16), 2 * p.n_ks) <= kLdsBytes;
  if (per_wave <= otmax) {
    p.OT = gemm_ot_round(T, w16, per_wave);
    p.n_oc = 1;
    p.mode = 0;
  } else if (res_ok) {
    p.OT = gemm_otres(T, w16);
    p.n_oc = (Co + 32 * p.OT - 1) / (32 * p.OT);
    p.mode = 1;
  } else {
    p.OT = otmax;
    p.n_oc = (Co + 32 * otmax - 1) / (32 * otmax);
    p.mode = 0;
  }
  // every weight block resident when they all fit
  if (gemm_lds_c(T, w16, p.OT, p.n_oc * p.n_ks) <= kLdsBytes) p.mode = 2;
  const int forced = gemm_forced_mode();
  if (forced == 0 || (forced == 1 && res_ok && p.OT == gemm_otres(T, w16))) p.mode = forced;
  p.narrow = ((int64_t)Ci * T * (w16 ? 2 : 4)) % gemm_wide_load_c(T, w16) != 0;
  if (p.narrow) {
    p.OT = 1;
    p.n_oc = (Co + 31) / 32;
    p.mode = 0;
  }
  p.OC = 32 * p.OT;
  p.Co_pad = p.n_oc * p.OC;
  p.lds_bytes = gemm_lds_c(T, w16, p.OT, gemm_wblocks(p.mode, p.n_oc, p.n_ks));
  return p;
}

// Row-count adjustment at launch: resident weights pay for loading every block
// up front, which only amortises when a workgroup runs several 64-row rounds;
// with at most one round per CU the streamed mode overlaps that load with the
// MFMAs.  Changes only the mode (never OT or the chunking), so the weight
// spectrum layout is the same either way.
inline void gemm_plan_rows(GemmPlan& p, int64_t N, int T, bool w16, int cus) {
  if (p.mode == 2 && gemm_forced_mode() < 0 && N < (int64_t)2 * 64 * cus) {
    p.mode = 0;
    p.lds_bytes = gemm_lds_c(T, w16, p.OT, gemm_wblocks(0, p.n_oc, p.n_ks));
  }
}

// Padded extents of the weight spectrum: rows to the o-chunks of the pass that
// reads the layout, columns to 32 (a multiple of every contraction step).
constexpr int kColPad = 32;
struct WspecDims {
  int CoF, CiF, CinB, CoutB;
};
inline WspecDims wspec_dims(int T, int Cin, int Cout, bool w16) {
  return {gemm_plan(T, Cin, Cout, w16).Co_pad, round_up(Cin, kColPad),
          gemm_plan(T, Cout, Cin, w16).Co_pad, round_up(Cout, kColPad)};
}

// Compute units of the current device (cached); 256 if unknown.
int device_cu_count();

// Plan of the split-row weight gradient: kernel, workgroup tile, split count
// and the padded partial extents.  kind 0: eql_wgrad_kernel (operands staged
// in LDS, a WGC x WGO wave grid of CT x OTW blocks of 16 x 16 channels per
// wave); kind 1: eql_wgrad_rd_kernel (register-direct operands, kRdWaves
// waves on one tile of CT x OTW blocks).  Depends only on the problem, not on
// the device, so results are reproducible across devices of the same model.
constexpr int kRdWaves = 4;
// Register-direct variants whose accumulators and two raw chunk buffers fit
// one wave per SIMD: 4T (CT*OT + 2 (CT + OT)) <= 400 registers.
constexpr bool rd_fits(int T, int CT, int OT) { return 4 * T * (CT * OT + 2 * (CT + OT)) <= 400; }
struct WgradPlan {
  int kind;
  int wgc, ct, otw; // variant: wave grid rows (WGO = 8 / wgc), tiles per wave
  int BC, BO;       // channel tile of one workgroup
  int KR;           // rows per chunk
  int n_ct, n_ot;   // channel tiles
  int S;            // splits
  int64_t rows_per_split;
  int Cin_pad, Cout_pad;
  size_t part_bytes, dbpart_bytes;
  // kind 2 (eql_wgrad_big.h): row-contiguous spectra of x and dy in the
  // workspace, N_pad rows (a multiple of 64) per plane row
  int64_t N_pad;
  size_t xs_bytes, ds_bytes;
};
// dt: element type code.  Plans whose workspace would exceed max_ws fall
// back to the split-row kernels (the allocation-free entry point passes its
// static scratch size).
WgradPlan wgrad_plan(int64_t N, int T, int Cin, int Cout, int dt, size_t max_ws = (size_t)-1);
inline size_t align256z(size_t v) { return (v + 255) / 256 * 256; }
// workspace of a plan: partials, bias partials, then (kind 2) the spectra
inline size_t wgrad_workspace(const WgradPlan& p) {
  return align256z(p.part_bytes) + align256z(p.dbpart_bytes) + align256z(p.xs_bytes) + align256z(p.ds_bytes);
}
// Three-product complex bins in the large-tile kernels (fp32, T = 4;
// 96-channel output tiles).  EQL_GAUSS=0 takes the four-product form
// everywhere, =1 the three-product one everywhere; unset, the forward and
// input gradient take three products and the weight gradient as below.
int gauss_forced();  // -1 unset, 0, 1
inline bool big_gauss(int T, int dt) { return T == 4 && dt == kF32 && gauss_forced() != 0; }

// Large-tile weight gradient (kind 2): T in {2, 4}, and the spectra of x and
// dy addressable with 31-bit offsets.  Taken by default from
// wgrad_big_min_c channels each way, where it measured faster than the
// register-direct kernel (T = 4, 32,768 rows, weight and bias gradient, µs
// large-tile / register-direct: fp16 463 / 864 at c = 768, 261 / 221 at 512;
// fp32 2059 / 3592 at 768, 988 / 888 at 512; bf16 261 / 320 at 512, 109 / 88
// at 256);
// EQL_WGRAD_KIND=2 forces it where it fits.  fp32 at T = 4 takes the
// three-product complex bin with 96-channel o-tiles (big_gauss) where the
// 128-channel tiles alone fill the 256 CUs (c = 2048: 12.04 against 12.71
// ms); with fewer tiles the row splits balance the four-product tiles as
// well and the three products measured 2% slower (c = 1024: 3.48 vs 3.41 ms).
inline int wgrad_big_min_c(int dt) { return dt == kBF16 ? 512 : 768; }
inline int wgrad_big_o_tile(int T, int Cin, int Cout, int dt) {
  if (T != 4 || dt != kF32) return 128;
  const int f = gauss_forced();
  const int64_t tiles128 = (int64_t)((Cin + 127) / 128) * ((Cout + 127) / 128);
  return f == 1 || (f < 0 && tiles128 >= 256) ? 96 : 128;
}
// Rows of the row-contiguous spectra: N in whole 64-row blocks of the
// pre-pass, plus one more block where that count is even, so that the channel
// rows' pitch is an odd multiple of 128 bytes (16-bit) or twice one (fp32)
// and the rows one step reads spread over the L2 sets instead of sharing a
// few (a pitch of 32,768 rows is 64 KB).  The extra rows are zero.
inline int64_t wgrad_big_npad(int64_t N) {
  const int64_t blocks = (N + 63) / 64;
  return (blocks % 2 == 0 ? blocks + 1 : blocks) * 64;
}
inline bool wgrad_big_fits(int64_t N, int T, int Cin, int Cout, int dt) {
  const int64_t eb = dt == kF32 ? 4 : 2;
  const int64_t np = wgrad_big_npad(N);
  const int64_t bo = wgrad_big_o_tile(T, Cin, Cout, dt);
  const int64_t ci = (Cin + 127) / 128 * 128, co = (Cout + bo - 1) / bo * bo;
  const int64_t lim = (int64_t)1 << 31;
  return (dt == kF32 || dt == kF16 || dt == kBF16) && (T == 2 || T == 4) && N > 0 && (int64_t)T * ci * np * eb < lim &&
         (int64_t)T * co * np * eb < lim && (int64_t)64 * (Cin > Cout ? Cin : Cout) * T * eb < lim;
}

// Shape of the partial reduction: NTHR threads per workgroup, runs of IPW
// items (IPW * 16 bytes per split and plane), G = NTHR / (IPW * T) split
// groups (at most 32).  Up to 64 splits: 256 threads and IPW = min(16, 64/T)
// (the headline's 40 splits: 8 items x 4 groups, 10 splits per thread in two
// batches; 10.8 us against 12.1 us with 1024 threads); more splits: 1024
// threads and IPW = 16 where that still gives 128 workgroups, else 8 or 4
// (16-item runs measured as fast as or faster than 4..64).
// EQL_RED_IPW forces IPW (A/B timing).
inline void wgrad_reduce_shape(int T, int S, int64_t items, int& nthr, int& ipw, int& G) {
  int forced = 0;
  if (const char* e = getenv("EQL_RED_IPW")) forced = atoi(e);
  nthr = S <= 64 ? 256 : 1024;
  if ((forced == 4 || forced == 8 || forced == 16 || forced == 32 || forced == 64) && forced * T <= nthr) {
    ipw = forced;
  } else if (nthr == 256) {
    ipw = 64 / T < 1 ? 1 : (64 / T > 16 ? 16 : 64 / T);
  } else {
    for (ipw = 16; ipw > 4; ipw /= 2)
      if ((items + ipw - 1) / ipw >= 128) break;
  }
  G = nthr / (ipw * T);
  if (G > 32) G = 32;
}

// Plan of the single-pass backward (eql_bwd_fused_kernel): the variant (wave
// grid rows, c-tiles, o-tiles per wave of the eql_wgrad_kernel grid) whose
// workgroup tile BC x BO holds every channel pair of the layer, the row
// splits, the input-gradient steps of KR output channels, and the LDS.  ok = 0
// when the layer does not take this path (then eqlinear_backward runs the
// input- and weight-gradient kernels one after the other).  Depends only on
// the problem, not on the device.
struct FusedPlan {
  int ok;
  int wgc, ct, otw, BC, BO;
  int KR, nks, C16;  // rows per chunk (= output channels per step), steps, Cin rounded to 16
  int dbuf, lds;     // two staging buffers; dynamic LDS bytes
  int S;
  int64_t rows_per_split;
  size_t part_bytes, dbpart_bytes;
};
FusedPlan fused_plan(int64_t N, int T, int Cin, int Cout, int dt);  // none for bf16
// Variants of eql_bwd_fused_kernel built for group order T and element
// type (fp16 or fp32): those that fit the 256 registers of a lane at two waves per SIMD
// without spilling (the weight-gradient accumulators, the input-gradient
// tile, two chunks of prefetched raw rows and the transforms; found by
// compiling every variant, and the post-build check refuses a spilling one).
constexpr bool fused_variant_ok(int T, bool f16, int ct, int otw) {
  const int tmax = (ct == 1 && otw == 1) ? (f16 ? 6 : 11)
                   : (ct == 2 && otw == 1) ? (f16 ? 5 : 7)
                   : (ct == 1 && otw == 2) ? (f16 ? 4 : 5)
                   : (ct == 1 && otw == 3) ? (f16 ? 2 : 3)
                                           : 0;
  return T <= tmax;
}
// 4 x 1 waves with one 16-channel block each: fewer registers than 2 x 4
constexpr bool fused_variant_ok(int T, bool f16, int wgc, int ct, int otw) {
  return wgc == 4 && ct == 1 && otw == 1 ? T <= (f16 ? 8 : 11) : fused_variant_ok(T, f16, ct, otw);
}
// LDS bytes of one workgroup of eql_bwd_fused_kernel: one or two staging
// buffers (x planes, dy planes by row, dy planes by output channel), then the
// weight spectrum.  Every staged row is 64 bytes: KR rows (weight-gradient
// staging) or KR output channels (input-gradient staging and weights) of one
// element each.
constexpr int kFusedRowBytes = 64;
inline int fused_lds_bytes(int T, int BC, int BO, int KR, int nks, int C16, bool dbuf) {
  const int stg = T * (BC + BO) * kFusedRowBytes + nks * T * KR * kFusedRowBytes;
  return (dbuf ? 2 : 1) * stg + nks * T * C16 * kFusedRowBytes;
}

struct GemmArgs {
  const void* in;
  const void* wsp;   // plane block of the layout this pass reads
  const void* bias;  // forward only; may be null
  void* out;
  int64_t N;
  int Ci, Co, Ci_pad;
  GemmPlan plan;
  hipStream_t stream;
  GatherGeom geo;    // implicit patch gather only (else zero)
};

struct WgradArgs {
  const void* x;
  const void* dy;
  void* dw;
  void* db;          // may be null
  float* part;
  float* dbpart;
  void* xs;          // kind 2: row-contiguous spectra of x and dy
  void* ds;
  int64_t N;
  int Cin, Cout;
  hipStream_t stream;
};

struct FusedArgs {
  const void* x;
  const void* dy;
  const void* wsp;   // backward-layout plane block of the weight spectrum
  void* dx;
  void* dw;
  void* db;          // may be null
  float* part;
  float* dbpart;
  int64_t N;
  int Cin, Cout, CinB, CoutB;
  hipStream_t stream;
};

// Launches of one group order and element type (eql_inst.hip, one object per
// (T, dtype) so the instantiations build in parallel).
template <int T, int DT>
struct Inst {
  static hipError_t wspec(const void* w, void* wspec, int Cin, int Cout, hipStream_t s);
  static hipError_t gemm(bool bwd, const GemmArgs& a);
  static hipError_t gemm_gather(const GemmArgs& a);
  static hipError_t wgrad(const WgradArgs& a, const WgradPlan& p);
  static hipError_t bwd_fused(const FusedArgs& a, const FusedPlan& p);
};

// Dispatch over T and the element type code dt (eql_dispatch.cpp).
hipError_t launch_wspec(int dt, int T, const void* w, void* wspec, int Cin, int Cout, hipStream_t s);
hipError_t launch_gemm(int dt, int T, bool bwd, const GemmArgs& a);

// Large-tile forward / input gradient (eql_gemm_big.h): T in {2, 4},
// contraction channels a multiple of 32, and every 128-row tile of the input
// and output below 2^31 bytes.  Taken by default for wide layers (both
// channel counts at least kBigMinC), where the spectral products bound the
// pass; EQL_GEMM_BIG=0 never takes it, =1 whenever the shape allows (tests,
// A/B timing).
struct BigArgs {
  const void* in;
  const void* wsp;   // plane block of the layout this pass reads
  const void* bias;  // forward only; may be null
  void* out;
  int64_t N;
  int Ci, Co;        // contraction and output channels of this pass
  int w_rows, w_pitch;  // rows (>= Co) and row pitch (>= Ci) of a spectrum plane
  hipStream_t stream;
};
constexpr int kBigMinC = 256;
int gemm_big_forced();  // -1 unset, 0, 1

inline bool gemm_big_fits(int T, int Ci, int Co, int dt) {
  const int64_t eb = dt == kF32 ? 4 : 2;
  return (dt == kF32 || dt == kF16 || dt == kBF16) && (T == 2 || T == 4) && Ci % 32 == 0 && Co >= 1 &&
         (int64_t)128 * Ci * T * eb < ((int64_t)1 << 31) && (int64_t)128 * Co * T * eb < ((int64_t)1 << 31);
}
inline bool gemm_big_choose(int T, int Ci, int Co, int dt) {
  if (!gemm_big_fits(T, Ci, Co, dt)) return false;
  const int f = gemm_big_forced();
  if (f >= 0) return f == 1;
  return Ci >= kBigMinC && Co >= kBigMinC;
}
hipError_t launch_gemm_big(int dt, int T, bool bwd, const BigArgs& a);
hipError_t launch_gemm_gather(int dt, int T, const GemmArgs& a);
hipError_t launch_wgrad(int dt, int T, const WgradArgs& a, const WgradPlan& p);
// kind 2: the spectrum pre-passes and the product kernel (launch_wgrad then
// runs the reduction)
hipError_t launch_wgrad_big(int dt, int T, const WgradArgs& a, const WgradPlan& p);
hipError_t launch_bwd_fused(int dt, int T, const FusedArgs& a, const FusedPlan& p);

}  // namespace eqk
