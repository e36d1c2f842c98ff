// eql_api.cpp -- the C ABI declared in include/eqlinear.h: argument checks,
// device checks, workspace planning and dispatch to the gfx950 kernels.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "../../include/eqlinear.h"
#include "eql_dihedral.h"
#include "eql_gconv.h"
#include "eql_launch.h"

namespace eqk {

// Split count of one variant: about one workgroup per CU of a 256-CU device,
// fp32 partials (written once, read once) at most half the bytes of x and dy,
// at least two row chunks per split, and each split's rows addressable with
// 31 bits.  Returns the rows per split (0 when N <= 0) and sets S.
static int64_t wgrad_splits(int64_t N, int T, int Cin, int Cout, bool w16, int KR, int64_t tiles,
                            int Cin_pad, int Cout_pad, int& S) {
  if (N <= 0) {
    S = 0;
    return 0;
  }
  int64_t target = 256;
  if (const char* e = getenv("EQL_WGRAD_TARGET")) target = atoi(e) > 0 ? atoi(e) : 256;
  int64_t s = (target + tiles - 1) / tiles;
  const double eb = w16 ? 2.0 : 4.0;
  const double in_bytes = (double)N * (Cin + Cout) * T * eb;
  const double part_per_split = (double)T * Cout_pad * Cin_pad * 4.0;
  const int64_t s_budget = (int64_t)(in_bytes / (2.0 * part_per_split));
  if (s > s_budget) s = s_budget;
  const int64_t max_s = (N + 2 * KR - 1) / (2 * KR);
  if (s > max_s) s = max_s;
  if (s < 1) s = 1;
  // whole groups of 8 splits: the kernel places the tiles of a split on one
  // XCD (split % 8), and a partial group would add idle workgroups and push
  // real ones past the first wave of the grid
  if (s >= 8) s = s / 8 * 8;
  const double row_bytes = (double)(Cin > Cout ? Cin : Cout) * T * eb;
  while ((double)((N + s - 1) / s + KR) * row_bytes >= 2147483648.0) ++s;
  int64_t rows = (N + s - 1) / s;
  rows = (rows + KR - 1) / KR * KR;
  S = (int)((N + rows - 1) / rows);
  return rows;
}

// Plan of the register-direct kernel: the (CT, OT) block tile and split count
// with the smallest estimated time.  One workgroup (kRdWaves waves, one per
// SIMD) per CU, S splits x tiles workgroups; the estimate is the largest of
// the HBM time (x and dy once plus the partials written and read back), the
// L2-to-CU time and the transform (VALU) time of every workgroup loading its
// rows for its channel tile, and the MFMA time, each spread over the CUs the
// grid occupies.
static WgradPlan wgrad_plan_rd(int64_t N, int T, int Cin, int Cout, bool w16) {
  static const int kTiles[][2] = {{1, 1}, {1, 2}, {2, 1}, {2, 2}, {2, 4}, {4, 2}};
  const int cus = 256;
  const int KR = w16 ? 32 : 16;
  const double eb = w16 ? 2.0 : 4.0;
  const int R = 1 + (T % 2 == 0), K = (T - 1) / 2;
  const double n = (double)(N > 0 ? N : 0);
  // VALU cycles per transformed element (packed fp16: two rows per operation)
  const double log2t = T <= 1 ? 1.0 : (T <= 2 ? 1.0 : (T <= 4 ? 2.0 : (T <= 8 ? 3.0 : 4.0)));
  const double cyc = (w16 ? 0.05 : 0.10) * (log2t + 1.0);
  int fc = 0, fo = 0;
  if (const char* e = getenv("EQL_WGRAD_TILE")) {
    if (sscanf(e, "%d,%d", &fc, &fo) != 2) fc = 0;
  }
  WgradPlan p{};
  p.kind = 1;
  double best = -1.0;
  for (const auto& v : kTiles) {
    const int ct = v[0], ot = v[1];
    if (!rd_fits(T, ct, ot)) continue;
    if (fc && (ct != fc || ot != fo)) continue;
    const int BC = 16 * ct, BO = 16 * ot;
    const int nct = (Cin + BC - 1) / BC, not_ = (Cout + BO - 1) / BO;
    const int64_t tiles = (int64_t)nct * not_;
    int64_t S = tiles >= cus ? 1 : cus / tiles;
    const int64_t max_s = (N + (int64_t)kRdWaves * KR - 1) / ((int64_t)kRdWaves * KR);
    if (S > max_s) S = max_s;
    if (S < 1) S = 1;
    const double part = (double)S * T * (nct * BC) * (not_ * BO) * 4.0;
    const double hbm = (n * (Cin + Cout) * T * eb + 2.0 * part) / 5.5e12;
    const double busy = (double)(S * tiles < cus ? S * tiles : cus);
    const double vals = n * T * ((double)nct * BC * not_ + (double)not_ * BO * nct);
    const double l2 = vals * eb / (busy * 154e9);
    const double valu = vals * cyc / (busy * 4.0 * 2.4e9);
    const double mfma = 2.0 * (R + 4 * K) * n * (nct * BC) * (not_ * BO) / ((w16 ? 2.5e15 : 1.573e14) * busy / cus);
    double t = hbm;
    if (l2 > t) t = l2;
    if (valu > t) t = valu;
    if (mfma > t) t = mfma;
    const double cost = t * (1.0 + 1e-9 * tiles);
    if (best < 0 || cost < best) {
      best = cost;
      p.ct = ct; p.otw = ot; p.BC = BC; p.BO = BO; p.n_ct = nct; p.n_ot = not_; p.S = (int)S;
    }
  }
  p.KR = KR;
  p.Cin_pad = p.n_ct * p.BC;
  p.Cout_pad = p.n_ot * p.BO;
  // rows per split: whole chunks, and each split's rows plus the chunks a
  // wave prefetches past its last one addressable with 31-bit offsets
  const double row_bytes = (double)(Cin > Cout ? Cin : Cout) * T * eb;
  int64_t S = p.S;
  while ((double)((N + S - 1) / S + (kRdWaves + 1) * KR) * row_bytes >= 2147483648.0) ++S;
  int64_t rows = N > 0 ? (N + S - 1) / S : 0;
  rows = (rows + KR - 1) / KR * KR;
  p.S = N > 0 ? (int)((N + rows - 1) / rows) : 0;
  p.rows_per_split = rows;
  p.part_bytes = (size_t)p.S * T * p.Cout_pad * p.Cin_pad * sizeof(float);
  p.dbpart_bytes = (size_t)p.S * p.Cout_pad * sizeof(float);
  return p;
}

// Which weight-gradient kernel: EQL_WGRAD_KIND=0/1/2 forces one (tests, A/B timing).
static int wgrad_forced_kind() {
  const char* v = getenv("EQL_WGRAD_KIND");
  return (v != nullptr && v[0] >= '0' && v[0] <= '2' && v[1] == 0) ? v[0] - '0' : -1;
}

// Large-tile plan: 128 x 128 channel tiles, and row splits (whole steps of 32
// rows, at least 8 per split) until about one workgroup per CU.
static WgradPlan wgrad_plan_big(int64_t N, int T, int Cin, int Cout, int dt) {
  WgradPlan p{};
  const size_t eb = dt == kF32 ? 4 : 2;
  p.kind = 2;
  p.BC = 128;
  p.BO = wgrad_big_o_tile(T, Cin, Cout, dt);
  p.KR = dt == kF32 ? 16 : 32;  // rows per step: 64 bytes of each channel row
  p.n_ct = (Cin + 127) / 128;
  p.n_ot = (Cout + p.BO - 1) / p.BO;
  p.Cin_pad = p.n_ct * 128;
  p.Cout_pad = p.n_ot * p.BO;
  p.N_pad = wgrad_big_npad(N);  // whole blocks of the spectrum pre-pass
  const int64_t steps = p.N_pad / 32;
  const int64_t tiles = (int64_t)p.n_ct * p.n_ot;
  // Row splits: each workgroup runs its rows to the end, so the pass lasts
  // about ceil(S * tiles / 256) rounds of workgroups of steps / S steps each.
  // Take the S with the fewest such steps (the smaller S on ties), from 1 to
  // max(8, what first fills the 256 CUs), with at least 8 steps per split.
  const int64_t max_s = steps / 8 > 1 ? steps / 8 : 1;
  int64_t s_hi = (256 + tiles - 1) / tiles;
  if (s_hi < 8) s_hi = 8;
  if (s_hi > max_s) s_hi = max_s;
  int64_t S = 1;
  double best = 0.0;
  for (int64_t s = 1; s <= s_hi; ++s) {
    const double cost = (double)((s * tiles + 255) / 256) / (double)s;
    if (s == 1 || cost < best * 0.999) {
      best = cost;
      S = s;
    }
  }
  const int64_t per = (steps + S - 1) / S;
  p.rows_per_split = per * 32;
  p.S = (int)((steps + per - 1) / per);
  p.part_bytes = (size_t)p.S * T * p.Cout_pad * p.Cin_pad * sizeof(float);
  p.dbpart_bytes = (size_t)p.S * p.Cout_pad * sizeof(float);
  p.xs_bytes = (size_t)T * p.Cin_pad * p.N_pad * eb;
  p.ds_bytes = (size_t)T * p.Cout_pad * p.N_pad * eb;
  return p;
}

static WgradPlan wgrad_plan_staged(int64_t N, int T, int Cin, int Cout, bool w16);

// Kernel choice.  The register-direct kernel writes few partials but reads
// every row once per channel tile and transforms it there; the staged kernel
// transforms each row once per workgroup tile but needs many row splits to
// fill the device, and with channel tiles enough to fill it alone it leaves a
// whole row range to each workgroup.  Measured on MI355X (bench.py): the
// register-direct kernel is faster for layers of at most 48 x 48 channels per
// group element (EQ-ViT-S projection 12.9 vs 22.0 us fp16, 20.3 vs 30.8 us
// fp32; the 16 x 16 layer 7.5 vs 15.0 us) and from 512 x 512 up (T = 4,
// 32768 rows, whole backward: 1.8 vs 2.7 ms at 512 fp32, 28 vs 121 ms at
// 2048 fp32, 7.6 vs 26.8 ms at 2048 fp16), level at 96 x 384 and 256 x 256,
// and slower on Swin stage 1 (24 x 96: 120 vs 79 us) and the 64 x 64 sweep.
// bf16 plans as fp16 (same shapes and tiles).
WgradPlan wgrad_plan(int64_t N, int T, int Cin, int Cout, int dt, size_t max_ws) {
  const bool w16 = dt != kF32;  // 16-bit elements: same shapes for fp16 and bf16
  int forced = wgrad_forced_kind();
  if (wgrad_big_fits(N, T, Cin, Cout, dt) &&
      (forced == 2 || (forced < 0 && Cin >= wgrad_big_min_c(dt) && Cout >= wgrad_big_min_c(dt)))) {
    const WgradPlan p = wgrad_plan_big(N, T, Cin, Cout, dt);
    if (wgrad_workspace(p) <= max_ws) return p;
  }
  if (forced == 2) forced = -1;
  const int lo = Cin < Cout ? Cin : Cout, hi = Cin < Cout ? Cout : Cin;
  if (forced == 1 || (forced < 0 && (hi <= 48 || lo >= 512)))
    return wgrad_plan_rd(N, T, Cin, Cout, w16);
  return wgrad_plan_staged(N, T, Cin, Cout, w16);
}

static WgradPlan wgrad_plan_staged(int64_t N, int T, int Cin, int Cout, bool w16) {
  // Variants (wave grid rows, c-tiles, o-tiles per wave) with at most 96
  // accumulator floats per lane: CT * OTW * T * 4 <= 96.  Pick the one with the
  // smallest estimated time: HBM bytes (x and dy once, the partials written
  // and read back), plus a quarter of the bytes that the channel tiles re-read
  // from L2 (x once per o-tile, dy once per c-tile), or the MFMA time of the
  // padded tiles if larger, divided by the fraction of a 256-CU device the
  // workgroups fill.  Ties go to fewer workgroup tiles.
  static const int kVariants[][3] = {{2, 1, 1}, {2, 2, 1}, {2, 3, 1}, {2, 1, 2},
                                     {2, 1, 3}, {4, 1, 1}, {4, 1, 2}, {4, 1, 3}};
  WgradPlan p{};
  double best = -1.0;
  // EQL_WGRAD_VARIANT=wgc,ct,otw forces one variant where it is valid (A/B timing)
  int fw = 0, fc = 0, fo = 0;
  if (const char* e = getenv("EQL_WGRAD_VARIANT")) {
    if (sscanf(e, "%d,%d,%d", &fw, &fc, &fo) != 3) fw = 0;
  }
  const int KR = w16 ? 32 : 16;
  const double eb = w16 ? 2.0 : 4.0;
  const int R = 1 + (T % 2 == 0), K = (T - 1) / 2;
  const double n = (double)(N > 0 ? N : 0);
  for (const auto& v : kVariants) {
    const int wgc = v[0], ct = v[1], otw = v[2], wgo = 8 / wgc;
    if (fw && (wgc != fw || ct != fc || otw != fo)) continue;
    if (ct * otw * T * 4 > 96) continue;
    const int BC = wgc * 16 * ct, BO = wgo * 16 * otw;
    if ((long)T * (BC + BO) * 64 > 160 * 1024 - 4096) continue;
    const int nct = (Cin + BC - 1) / BC, not_ = (Cout + BO - 1) / BO;
    const int64_t tiles = (int64_t)nct * not_;
    int S = 0;
    wgrad_splits(N, T, Cin, Cout, w16, KR, tiles, nct * BC, not_ * BO, S);
    const double part = (double)S * T * (nct * BC) * (not_ * BO) * 4.0;
    const double hbm = n * (Cin + Cout) * T * eb + 2.0 * part;
    const double l2 = n * T * eb * ((double)Cin * not_ + (double)Cout * nct);
    const double flops = 2.0 * (R + 4 * K) * n * (nct * BC) * (not_ * BO);
    const double mfma_bytes = flops / (w16 ? 2.5e15 : 1.573e14) * 8.0e12;  // as HBM-time bytes
    double mem = hbm + 0.25 * l2;
    if (mfma_bytes > mem) mem = mfma_bytes;
    double fill = (double)S * tiles / 256.0;
    if (fill > 1.0 || fill <= 0.0) fill = 1.0;
    const double cost = mem / fill * (1.0 + 1e-9 * tiles);
    if (best < 0 || cost < best) {
      best = cost;
      p.wgc = wgc; p.ct = ct; p.otw = otw; p.BC = BC; p.BO = BO; p.n_ct = nct; p.n_ot = not_;
    }
  }
  p.KR = KR;
  p.Cin_pad = p.n_ct * p.BC;
  p.Cout_pad = p.n_ot * p.BO;
  p.rows_per_split = wgrad_splits(N, T, Cin, Cout, w16, KR, (int64_t)p.n_ct * p.n_ot, p.Cin_pad,
                                  p.Cout_pad, p.S);
  p.part_bytes = (size_t)p.S * T * p.Cout_pad * p.Cin_pad * sizeof(float);
  p.dbpart_bytes = (size_t)p.S * p.Cout_pad * sizeof(float);
  return p;
}

// Single-pass backward: EQL_BWD_FUSED=0 never takes it, =1 takes it wherever
// a variant fits (tests, A/B timing); unset, the rule of fused_plan decides.
static int bwd_forced_fused() {
  const char* v = getenv("EQL_BWD_FUSED");
  return (v != nullptr && (v[0] == '0' || v[0] == '1') && v[1] == 0) ? v[0] - '0' : -1;
}

// The smallest variant tile that holds every channel pair (a variant built
// for this T, LDS within the CU with one staging buffer; two when they fit),
// about one split per CU of a 256-CU device with at least four chunks each,
// and each split's rows addressable with 31 bits.  Taken for fp16 when at
// least 128 splits result and the fp32 partials, written and read back, move
// no more bytes than the second read of x and dy that the two-kernel path
// makes.  Measured on MI355X (bench.py, whole backward): Swin stage 1
// (401,408 rows, 24 -> 96, T = 4; 17 MB of partials against 385 MB of x and
// dy) 118 against 162 us; the 64 x 64 sweep layers at 32,768 rows, T = 3 and
// 5 (partials as large as x and dy) 36.5 against 42.6 us and 53.9 against
// 64.5 us.  The EQ-ViT-B MLP's 96 x 384 x 8 tile fits no workgroup.  fp32
// stays on the two kernels: its staging does not fit two buffers, and the
// single-buffered pass measured slower (Swin stage 1 shape 494 against
// 383 us, the T = 3 and 5 sweeps 50.0 against 47.4 and 79.3 against 75.3 us).
FusedPlan fused_plan(int64_t N, int T, int Cin, int Cout, int dt) {
  static const int kVariants[][3] = {{2, 1, 1}, {4, 1, 1}, {2, 1, 2}, {2, 2, 1}, {2, 1, 3}};
  FusedPlan p{};
  const int forced = bwd_forced_fused();
  if (forced == 0 || N <= 0 || dt == kBF16) return p;  // fp32 and fp16 only
  const bool f16 = dt == kF16;
  const int KR = f16 ? 32 : 16;
  const int C16 = round_up(Cin, 16);
  const int nks = (Cout + KR - 1) / KR;
  long best = -1;
  for (const auto& v : kVariants) {
    const int wgc = v[0], ct = v[1], otw = v[2];
    const int BC = wgc * 16 * ct, BO = (8 / wgc) * 16 * otw;
    if (!fused_variant_ok(T, f16, wgc, ct, otw) || BC < Cin || BO < Cout || nks * KR > BO) continue;
    if (fused_lds_bytes(T, BC, BO, KR, nks, C16, false) > kLdsBytes) continue;
    const long area = (long)BC * BO;
    if (best < 0 || area < best) {
      best = area;
      p.wgc = wgc; p.ct = ct; p.otw = otw; p.BC = BC; p.BO = BO;
    }
  }
  if (best < 0) return p;
  p.KR = KR;
  p.nks = nks;
  p.C16 = C16;
  p.dbuf = fused_lds_bytes(T, p.BC, p.BO, KR, nks, C16, true) <= kLdsBytes ? 1 : 0;
  p.lds = fused_lds_bytes(T, p.BC, p.BO, KR, nks, C16, p.dbuf != 0);
  int64_t s = 256;
  const int64_t max_s = (N + 4 * KR - 1) / (4 * KR);
  if (s > max_s) s = max_s;
  if (s < 1) s = 1;
  const double eb = f16 ? 2.0 : 4.0;
  const double row_bytes = (double)(Cin > Cout ? Cin : Cout) * T * eb;
  while ((double)((N + s - 1) / s + KR) * row_bytes >= 2147483648.0) ++s;
  int64_t rows = (N + s - 1) / s;
  rows = (rows + KR - 1) / KR * KR;
  p.S = (int)((N + rows - 1) / rows);
  p.rows_per_split = rows;
  p.part_bytes = (size_t)p.S * T * p.BC * p.BO * sizeof(float);
  p.dbpart_bytes = (size_t)p.S * p.BO * sizeof(float);
  if (forced < 0) {
    const double xdy = (double)N * (Cin + Cout) * T * eb;
    if (!f16 || p.S < 128 || 2.0 * (double)p.part_bytes > xdy) return FusedPlan{};
  }
  p.ok = 1;
  return p;
}

}  // namespace eqk

namespace {

constexpr int64_t kMaxN = (int64_t)1 << 36;
constexpr int kMaxC = 65536;

size_t elem_bytes(int dtype) { return dtype == EQL_F32 ? 4 : 2; }
bool valid_dtype(int dtype) { return dtype == EQL_F32 || dtype == EQL_F16 || dtype == EQL_BF16; }

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

struct Range {
  const void* p;
  size_t bytes;
};

bool overlaps(Range a, Range b) {
  if (!a.p || !b.p || a.bytes == 0 || b.bytes == 0) return false;
  const uintptr_t a0 = (uintptr_t)a.p, a1 = a0 + a.bytes;
  const uintptr_t b0 = (uintptr_t)b.p, b1 = b0 + b.bytes;
  return a0 < b1 && b0 < a1;
}

bool any_overlap(const Range* r, int n) {
  for (int i = 0; i < n; ++i)
    for (int j = i + 1; j < n; ++j)
      if (overlaps(r[i], r[j])) return true;
  return false;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

int check_shape(int64_t N, int T, int Cin, int Cout, int dtype) {
  if (!valid_dtype(dtype)) return EQL_ERR_INVALID_ARG;
  if (T < 1 || Cin < 1 || Cout < 1 || N < 0) return EQL_ERR_INVALID_ARG;
  if (T > EQLINEAR_MAX_T || Cin > kMaxC || Cout > kMaxC || N > kMaxN) return EQL_ERR_UNSUPPORTED;
  // the weight spectrum (two padded copies) must stay under 2^31 bytes
  if ((double)T * 2.0 * (Cin + 127) * (Cout + 127) * elem_bytes(dtype) >= 2147483648.0)
    return EQL_ERR_UNSUPPORTED;
  return EQL_OK;
}

// Per-device cache: is this a gfx950 device?  Filled once per device.
constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
int g_arch_ok[kMaxDevices];
int g_cus[kMaxDevices];

int check_device() {
  int count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || count <= 0) {
    (void)hipGetLastError();
    return EQL_ERR_NO_DEVICE;
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return EQL_ERR_NO_DEVICE;
  }
  std::call_once(g_once[dev], [dev] {
    hipDeviceProp_t prop;
    g_arch_ok[dev] = 0;
    g_cus[dev] = 256;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess) {
      g_arch_ok[dev] = strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 0;
      if (prop.multiProcessorCount > 0) g_cus[dev] = prop.multiProcessorCount;
    } else {
      (void)hipGetLastError();
    }
  });
  return g_arch_ok[dev] ? EQL_OK : EQL_ERR_UNSUPPORTED;
}

int launched(hipError_t e) { return e == hipSuccess ? EQL_OK : EQL_ERR_LAUNCH; }

}  // namespace

namespace eqk {
// Read on every plan so that tests can switch it within one process.
int gemm_forced_mode() {
  const char* v = getenv("EQL_GEMM_MODE");
  return (v != nullptr && v[0] >= '0' && v[0] <= '2' && v[1] == 0) ? v[0] - '0' : -1;
}
int gemm_big_forced() {
  const char* v = getenv("EQL_GEMM_BIG");
  return (v != nullptr && (v[0] == '0' || v[0] == '1') && v[1] == 0) ? v[0] - '0' : -1;
}
int gauss_forced() {
  const char* v = getenv("EQL_GAUSS");
  return (v != nullptr && (v[0] == '0' || v[0] == '1') && v[1] == 0) ? v[0] - '0' : -1;
}
// Valid after check_device() succeeded on the current device.
int device_cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices || g_cus[dev] <= 0) {
    (void)hipGetLastError();
    return 256;
  }
  return g_cus[dev];
}
}  // namespace eqk

extern "C" {

int eqlinear_abi_version(void) { return EQLINEAR_ABI_VERSION; }

const char* eqlinear_status_string(int status) {
  switch (status) {
    case EQL_OK: return "ok";
    case EQL_ERR_INVALID_ARG: return "invalid argument (shape, null pointer, dtype or overlapping buffers)";
    case EQL_ERR_UNSUPPORTED: return "unsupported (T > 16, size limit exceeded, or device is not gfx950)";
    case EQL_ERR_ALIGNMENT: return "misaligned pointer (tensors need 16-byte alignment, weights element alignment)";
    case EQL_ERR_WORKSPACE: return "workspace too small or missing";
    case EQL_ERR_NO_DEVICE: return "no HIP device available";
    case EQL_ERR_LAUNCH: return "kernel launch failed";
    case EQL_ERR_SCRATCH: return "problem needs more than the static device scratch of the allocation-free entry point";
    default: return "unknown status";
  }
}

size_t eqlinear_weight_spectrum_bytes(int T, int Cin, int Cout, int dtype) {
  if (check_shape(0, T, Cin, Cout, dtype) != EQL_OK) return 0;
  const eqk::WspecDims d = eqk::wspec_dims(T, Cin, Cout, dtype != EQL_F32);
  const size_t bytes =
      (size_t)T * ((size_t)d.CoF * d.CiF + (size_t)d.CinB * d.CoutB) * elem_bytes(dtype);
  return bytes < ((size_t)1 << 31) ? bytes : 0;  // kernels address the spectrum with 31-bit offsets
}

int eqlinear_weight_spectrum(const void* w, void* wspec, int T, int Cin, int Cout, int dtype,
                             void* stream) {
  int st = check_shape(0, T, Cin, Cout, dtype);
  if (st) return st;
  if (!w || !wspec) return EQL_ERR_INVALID_ARG;
  const size_t e = elem_bytes(dtype);
  if (!aligned(w, e) || !aligned(wspec, 16)) return EQL_ERR_ALIGNMENT;
  const Range r[2] = {{w, (size_t)T * Cin * Cout * e},
                      {wspec, eqlinear_weight_spectrum_bytes(T, Cin, Cout, dtype)}};
  if (any_overlap(r, 2)) return EQL_ERR_INVALID_ARG;
  if ((st = check_device())) return st;
  hipStream_t s = (hipStream_t)stream;
  return launched(eqk::launch_wspec(dtype, T, w, wspec, Cin, Cout, s));
}

static int gemm_common(const void* in, const void* wspec, const void* bias, void* out, int64_t N,
                       int T, int Cin, int Cout, int dtype, void* stream, bool bwd) {
  int st = check_shape(N, T, Cin, Cout, dtype);
  if (st) return st;
  if (!wspec) return EQL_ERR_INVALID_ARG;
  if (N > 0 && (!in || !out)) return EQL_ERR_INVALID_ARG;
  const size_t e = elem_bytes(dtype);
  if (!aligned(wspec, 16) || (in && !aligned(in, 16)) || (out && !aligned(out, 16)) ||
      (bias && !aligned(bias, e)))
    return EQL_ERR_ALIGNMENT;
  const int Ci = bwd ? Cout : Cin;
  const int Co = bwd ? Cin : Cout;
  const Range r[4] = {{in, (size_t)N * Ci * T * e},
                      {out, (size_t)N * Co * T * e},
                      {wspec, eqlinear_weight_spectrum_bytes(T, Cin, Cout, dtype)},
                      {bias, bias ? (size_t)Cout * e : 0}};
  if (any_overlap(r, 4)) return EQL_ERR_INVALID_ARG;
  if ((st = check_device())) return st;
  if (N == 0) return EQL_OK;
  const eqk::WspecDims d = eqk::wspec_dims(T, Cin, Cout, dtype != EQL_F32);
  const size_t fwd_block = (size_t)T * d.CoF * d.CiF * e;  // forward-layout planes
  if (eqk::gemm_big_choose(T, Ci, Co, dtype)) {
    eqk::BigArgs b{};
    b.in = in;
    b.bias = bias;
    b.out = out;
    b.N = N;
    b.Ci = Ci;
    b.Co = Co;
    b.wsp = bwd ? (const void*)((const char*)wspec + fwd_block) : wspec;
    b.w_rows = bwd ? d.CinB : d.CoF;
    b.w_pitch = bwd ? d.CoutB : d.CiF;
    b.stream = (hipStream_t)stream;
    return launched(eqk::launch_gemm_big(dtype, T, bwd, b));
  }
  eqk::GemmArgs a{};
  a.in = in;
  a.bias = bias;
  a.out = out;
  a.N = N;
  a.Ci = Ci;
  a.Co = Co;
  a.stream = (hipStream_t)stream;
  a.plan = eqk::gemm_plan(T, Ci, Co, dtype != EQL_F32);
  eqk::gemm_plan_rows(a.plan, N, T, dtype != EQL_F32, eqk::device_cu_count());
  if (!bwd) {
    a.wsp = wspec;
    a.Ci_pad = d.CiF;
  } else {
    a.wsp = (const char*)wspec + fwd_block;
    a.Ci_pad = d.CoutB;
  }
  return launched(eqk::launch_gemm(dtype, T, bwd, a));
}

int eqlinear_forward(const void* x, const void* wspec, const void* bias, void* y, int64_t N,
                     int T, int Cin, int Cout, int dtype, void* stream) {
  return gemm_common(x, wspec, bias, y, N, T, Cin, Cout, dtype, stream, false);
}

int eqlinear_backward_input(const void* dy, const void* wspec, void* dx, int64_t N, int T,
                            int Cin, int Cout, int dtype, void* stream) {
  return gemm_common(dy, wspec, nullptr, dx, N, T, Cin, Cout, dtype, stream, true);
}

size_t eqlinear_backward_weight_workspace_bytes(int64_t N, int T, int Cin, int Cout, int dtype) {
  if (check_shape(N, T, Cin, Cout, dtype) != EQL_OK || N == 0) return 0;
  return eqk::wgrad_workspace(eqk::wgrad_plan(N, T, Cin, Cout, dtype));
}

static int backward_weight_impl(const void* x, const void* dy, void* dw, void* dbias, void* workspace,
                                size_t workspace_bytes, int64_t N, int T, int Cin, int Cout, int dtype,
                                void* stream, bool static_scratch);

int eqlinear_backward_weight(const void* x, const void* dy, void* dw, void* dbias, void* workspace,
                             size_t workspace_bytes, int64_t N, int T, int Cin, int Cout, int dtype,
                             void* stream) {
  return backward_weight_impl(x, dy, dw, dbias, workspace, workspace_bytes, N, T, Cin, Cout, dtype,
                              stream, false);
}

int eqlinear_backward_weight_noalloc(const void* x, const void* dy, void* dw, void* dbias, int64_t N,
                                     int T, int Cin, int Cout, int dtype, void* stream) {
  return backward_weight_impl(x, dy, dw, dbias, nullptr, 0, N, T, Cin, Cout, dtype, stream, true);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Static scratch of the allocation-free entry point: one array per GPU (the
// loader places a copy in every device's memory).  Host code never uses the
// array's name as an address: the device address is resolved once per device,
// with that device current, and kept.
static __device__ __align__(256) char scratch[EQLINEAR_STATIC_SCRATCH_BYTES];

namespace {
std::once_flag g_scratch_once[kMaxDevices];
void* g_scratch_ptr[kMaxDevices];

// Device address of this device's scratch array, or null if the runtime
// cannot resolve it.  Valid after check_device() succeeded.
void* device_scratch() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return nullptr;
  }
  std::call_once(g_scratch_once[dev], [dev] {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) {
      (void)hipGetLastError();
      ptr = nullptr;
    }
    g_scratch_ptr[dev] = ptr;
  });
  return g_scratch_ptr[dev];
}
}  // namespace

static int backward_weight_impl(const void* x, const void* dy, void* dw, void* dbias, void* workspace,
                                size_t workspace_bytes, int64_t N, int T, int Cin, int Cout, int dtype,
                                void* stream, bool static_scratch) {
  int st = check_shape(N, T, Cin, Cout, dtype);
  if (st) return st;
  if (!dw) return EQL_ERR_INVALID_ARG;
  if (N > 0 && (!x || !dy)) return EQL_ERR_INVALID_ARG;
  const size_t e = elem_bytes(dtype);
  if ((x && !aligned(x, 16)) || (dy && !aligned(dy, 16)) || !aligned(dw, e) ||
      (dbias && !aligned(dbias, e)) || (workspace && !aligned(workspace, 16)))
    return EQL_ERR_ALIGNMENT;
  // the allocation-free entry point plans within its static scratch
  const eqk::WgradPlan p =
      eqk::wgrad_plan(N, T, Cin, Cout, dtype, static_scratch ? EQLINEAR_STATIC_SCRATCH_BYTES : (size_t)-1);
  const size_t need = N > 0 ? eqk::wgrad_workspace(p) : 0;
  if (static_scratch && need > EQLINEAR_STATIC_SCRATCH_BYTES) return EQL_ERR_SCRATCH;
  if (!static_scratch && need > 0 && (!workspace || workspace_bytes < need)) return EQL_ERR_WORKSPACE;
  const Range r[5] = {{x, (size_t)N * Cin * T * e},
                      {dy, (size_t)N * Cout * T * e},
                      {dw, (size_t)T * Cin * Cout * e},
                      {dbias, dbias ? (size_t)Cout * e : 0},
                      {workspace, need}};
  if (any_overlap(r, 5)) return EQL_ERR_INVALID_ARG;
  if ((st = check_device())) return st;
  if (static_scratch && need > 0) {
    workspace = device_scratch();
    if (!workspace) return EQL_ERR_LAUNCH;
  }
  eqk::WgradArgs a{};
  a.x = x;
  a.dy = dy;
  a.dw = dw;
  a.db = dbias;
  a.part = (float*)workspace;
  a.dbpart = workspace ? (float*)((char*)workspace + align256(p.part_bytes)) : nullptr;
  if (p.kind == 2) {
    char* w = (char*)workspace + align256(p.part_bytes) + align256(p.dbpart_bytes);
    a.xs = w;
    a.ds = w + align256(p.xs_bytes);
  }
  a.N = N;
  a.Cin = Cin;
  a.Cout = Cout;
  a.stream = (hipStream_t)stream;
  if (p.kind == 2 && N > 0) {
    st = launched(eqk::launch_wgrad_big(dtype, T, a, p));
    if (st) return st;
  }
  return launched(eqk::launch_wgrad(dtype, T, a, p));
}



// ---------------------------------------------------------------------------
// Whole backward in one call.  With a fused plan, one pass of
// eql_bwd_fused_kernel writes dx and the weight-gradient partials, then the
// partial reduction writes dw and db; otherwise the input-gradient kernel and
// the weight-gradient kernels run one after the other, exactly as the two
// separate entry points do.
extern "C" {

int eqlinear_backward_is_fused(int64_t N, int T, int Cin, int Cout, int dtype) {
  if (check_shape(N, T, Cin, Cout, dtype) != EQL_OK) return 0;
  return eqk::fused_plan(N, T, Cin, Cout, dtype).ok ? 1 : 0;
}

size_t eqlinear_backward_workspace_bytes(int64_t N, int T, int Cin, int Cout, int dtype) {
  if (check_shape(N, T, Cin, Cout, dtype) != EQL_OK || N == 0) return 0;
  const eqk::FusedPlan f = eqk::fused_plan(N, T, Cin, Cout, dtype);
  if (f.ok) return align256(f.part_bytes) + align256(f.dbpart_bytes);
  return eqlinear_backward_weight_workspace_bytes(N, T, Cin, Cout, dtype);
}

int eqlinear_backward(const void* x, const void* dy, const void* wspec, void* dx, void* dw, void* dbias,
                      void* workspace, size_t workspace_bytes, int64_t N, int T, int Cin, int Cout,
                      int dtype, void* stream) {
  int st = check_shape(N, T, Cin, Cout, dtype);
  if (st) return st;
  if (!wspec || !dw) return EQL_ERR_INVALID_ARG;
  if (N > 0 && (!x || !dy || !dx)) return EQL_ERR_INVALID_ARG;
  const size_t e = elem_bytes(dtype);
  if (!aligned(wspec, 16) || (x && !aligned(x, 16)) || (dy && !aligned(dy, 16)) || (dx && !aligned(dx, 16)) ||
      !aligned(dw, e) || (dbias && !aligned(dbias, e)) || (workspace && !aligned(workspace, 16)))
    return EQL_ERR_ALIGNMENT;
  const size_t need = eqlinear_backward_workspace_bytes(N, T, Cin, Cout, dtype);
  if (need > 0 && (!workspace || workspace_bytes < need)) return EQL_ERR_WORKSPACE;
  const Range r[7] = {{x, (size_t)N * Cin * T * e},
                      {dy, (size_t)N * Cout * T * e},
                      {wspec, eqlinear_weight_spectrum_bytes(T, Cin, Cout, dtype)},
                      {dx, (size_t)N * Cin * T * e},
                      {dw, (size_t)T * Cin * Cout * e},
                      {dbias, dbias ? (size_t)Cout * e : 0},
                      {workspace, need}};
  if (any_overlap(r, 7)) return EQL_ERR_INVALID_ARG;
  if ((st = check_device())) return st;
  const eqk::FusedPlan p = eqk::fused_plan(N, T, Cin, Cout, dtype);
  if (!p.ok) {
    st = eqlinear_backward_input(dy, wspec, dx, N, T, Cin, Cout, dtype, stream);
    if (st) return st;
    return eqlinear_backward_weight(x, dy, dw, dbias, workspace, workspace_bytes, N, T, Cin, Cout, dtype,
                                    stream);
  }
  const eqk::WspecDims d = eqk::wspec_dims(T, Cin, Cout, dtype != EQL_F32);
  eqk::FusedArgs a{};
  a.x = x;
  a.dy = dy;
  a.wsp = (const char*)wspec + (size_t)T * d.CoF * d.CiF * e;
  a.dx = dx;
  a.dw = dw;
  a.db = dbias;
  a.part = (float*)workspace;
  a.dbpart = (float*)((char*)workspace + align256(p.part_bytes));
  a.N = N;
  a.Cin = Cin;
  a.Cout = Cout;
  a.CinB = d.CinB;
  a.CoutB = d.CoutB;
  a.stream = (hipStream_t)stream;
  return launched(eqk::launch_bwd_fused(dtype, T, a, p));
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Dihedral group D_T on the C_T kernels (csrc/eql_dihedral.h): the weight
// expansion before the forward pass and the gradient fold after the backward
// pass.  Weight-sized gathers, grid-stride loops of 256-thread workgroups.
namespace {

int dihedral_shape(int T, int Cin, int Cout, int dtype) {
  if (Cin < 1 || Cout < 1) return EQL_ERR_INVALID_ARG;
  if (Cin > kMaxC / 2 || Cout > kMaxC / 2) return EQL_ERR_UNSUPPORTED;
  return check_shape(0, T, 2 * Cin, 2 * Cout, dtype);
}

unsigned gather_grid(int64_t total) {
  const int64_t g = (total + 255) / 256;
  return (unsigned)(g < 1 ? 1 : (g > 4096 ? 4096 : g));
}

template <typename E>
int dihedral_launch(bool expand, const void* in, const void* in_b, void* out, void* out_b, int T,
                    int Cin, int Cout, hipStream_t s) {
  if (expand) {
    const int64_t total = (int64_t)T * 4 * Cin * Cout;
    hipLaunchKernelGGL((eqk::eql_dihedral_expand_kernel<E>), dim3(gather_grid(total)), dim3(256), 0, s,
                       (const E*)in, (const E*)in_b, (E*)out, (E*)out_b, T, Cin, Cout);
  } else {
    const int64_t total = (int64_t)T * 2 * Cin * Cout;
    hipLaunchKernelGGL((eqk::eql_dihedral_fold_kernel<E>), dim3(gather_grid(total)), dim3(256), 0, s,
                       (const E*)in, (const E*)in_b, (E*)out, (E*)out_b, T, Cin, Cout);
  }
  return launched(hipGetLastError());
}

// expand: in = W [2T,Cout,Cin], in_b = b [Cout], out = w2 [T,2Cout,2Cin], out_b = b2 [2Cout]
// fold:   in = dw2 [T,2Cout,2Cin], in_b = db2 [2Cout], out = dW [2T,Cout,Cin], out_b = db [Cout]
int dihedral_common(bool expand, const void* in, const void* in_b, void* out, void* out_b, int T, int Cin,
                    int Cout, int dtype, void* stream) {
  int st = dihedral_shape(T, Cin, Cout, dtype);
  if (st) return st;
  if (!in || !out || (in_b == nullptr) != (out_b == nullptr)) return EQL_ERR_INVALID_ARG;
  const size_t e = elem_bytes(dtype);
  if (!aligned(in, e) || !aligned(out, e) || (in_b && !aligned(in_b, e)) || (out_b && !aligned(out_b, e)))
    return EQL_ERR_ALIGNMENT;
  const size_t in_bytes = expand ? (size_t)2 * T * Cout * Cin * e : (size_t)4 * T * Cout * Cin * e;
  const size_t out_bytes = expand ? (size_t)4 * T * Cout * Cin * e : (size_t)2 * T * Cout * Cin * e;
  const size_t inb_bytes = in_b ? (expand ? (size_t)Cout : (size_t)2 * Cout) * e : 0;
  const size_t outb_bytes = out_b ? (expand ? (size_t)2 * Cout : (size_t)Cout) * e : 0;
  const Range r[4] = {{in, in_bytes}, {in_b, inb_bytes}, {out, out_bytes}, {out_b, outb_bytes}};
  if (any_overlap(r, 4)) return EQL_ERR_INVALID_ARG;
  if ((st = check_device())) return st;
  hipStream_t s = (hipStream_t)stream;
  if (dtype == EQL_F16) return dihedral_launch<_Float16>(expand, in, in_b, out, out_b, T, Cin, Cout, s);
  if (dtype == EQL_BF16) return dihedral_launch<__bf16>(expand, in, in_b, out, out_b, T, Cin, Cout, s);
  return dihedral_launch<float>(expand, in, in_b, out, out_b, T, Cin, Cout, s);
}

}  // namespace

extern "C" {

int eqlinear_dihedral_expand(const void* w, const void* bias, void* w_ct, void* bias_ct, int T, int Cin,
                             int Cout, int dtype, void* stream) {
  return dihedral_common(true, w, bias, w_ct, bias_ct, T, Cin, Cout, dtype, stream);
}

int eqlinear_dihedral_fold(const void* dw_ct, const void* dbias_ct, void* dw, void* dbias, int T, int Cin,
                           int Cout, int dtype, void* stream) {
  return dihedral_common(false, dw_ct, dbias_ct, dw, dbias, T, Cin, Cout, dtype, stream);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Rotation-equivariant group convolution on the C_T kernels
// (csrc/eql_gconv.h): patch gather, its adjoint, weight permutation both ways.
namespace {

int gconv_shape(int T, int Cin, int Cout, int k, int dtype) {
  if (!valid_dtype(dtype)) return EQL_ERR_INVALID_ARG;
  if (Cin < 1 || Cout < 1 || k < 1) return EQL_ERR_INVALID_ARG;
  if (T != 1 && T != 2 && T != 4) return EQL_ERR_UNSUPPORTED;
  if (k % 2 == 0 || k > 7) return EQL_ERR_UNSUPPORTED;
  if (Cin > kMaxC / (k * k) || Cout > kMaxC) return EQL_ERR_UNSUPPORTED;
  return EQL_OK;
}

int gconv_image(int64_t B, int H, int W) {
  if (B < 0 || H < 0 || W < 0) return EQL_ERR_INVALID_ARG;
  if ((double)B * H * W > (double)kMaxN) return EQL_ERR_UNSUPPORTED;
  return EQL_OK;
}

template <typename E, int T, int K>
void gconv_pixels(bool scatter, const void* in, void* out, int64_t n_pix, int H, int W, int Cin, hipStream_t s) {
  // one wave per pixel, kGconvWaves pixels per block; past 2^30 blocks the
  // kernels stride over the pixel groups
  const int64_t groups = (n_pix + eqk::kGconvWaves - 1) / eqk::kGconvWaves;
  const dim3 grid((unsigned)(groups < ((int64_t)1 << 30) ? groups : ((int64_t)1 << 30)));
  if (scatter)
    hipLaunchKernelGGL((eqk::eql_gconv_scatter_kernel<E, T, K>), grid, dim3(256), 0, s, (const E*)in, (E*)out,
                       n_pix, H, W, Cin);
  else if ((uintptr_t)out % (sizeof(E) * T) == 0)
    hipLaunchKernelGGL((eqk::eql_gconv_gather_kernel<E, T, K, true>), grid, dim3(256), 0, s, (const E*)in,
                       (E*)out, n_pix, H, W, Cin);
  else
    hipLaunchKernelGGL((eqk::eql_gconv_gather_kernel<E, T, K, false>), grid, dim3(256), 0, s, (const E*)in,
                       (E*)out, n_pix, H, W, Cin);
}

template <typename E, int T>
int gconv_launch_t(int op, const void* in, void* out, int64_t B, int H, int W, int Cin, int Cout, int k,
                   hipStream_t s) {
  const int64_t n_pix = B * H * W;
  if (op < 2) {
    if (n_pix == 0) return EQL_OK;
    const bool sc = op == 1;
    if (k == 1) gconv_pixels<E, T, 1>(sc, in, out, n_pix, H, W, Cin, s);
    else if (k == 3) gconv_pixels<E, T, 3>(sc, in, out, n_pix, H, W, Cin, s);
    else if (k == 5) gconv_pixels<E, T, 5>(sc, in, out, n_pix, H, W, Cin, s);
    else gconv_pixels<E, T, 7>(sc, in, out, n_pix, H, W, Cin, s);  // gconv_shape admits odd k <= 7
  } else {
    const int64_t total = (int64_t)T * Cout * k * k * Cin;
    if (op == 2)
      hipLaunchKernelGGL((eqk::eql_gconv_pack_kernel<E>), dim3(gather_grid(total)), dim3(256), 0, s,
                         (const E*)in, (E*)out, T, Cin, Cout, k);
    else if (op == 4)
      hipLaunchKernelGGL((eqk::eql_gconv_pack_kernel<E, true>), dim3(gather_grid(total)), dim3(256), 0, s,
                         (const E*)in, (E*)out, T, Cin, Cout, k);
    else
      hipLaunchKernelGGL((eqk::eql_gconv_unpack_kernel<E>), dim3(gather_grid(total)), dim3(256), 0, s,
                         (const E*)in, (E*)out, T, Cin, Cout, k);
  }
  return launched(hipGetLastError());
}

template <typename E>
int gconv_launch(int op, const void* in, void* out, int64_t B, int H, int W, int T, int Cin, int Cout, int k,
                 hipStream_t s) {
  if (T == 4) return gconv_launch_t<E, 4>(op, in, out, B, H, W, Cin, Cout, k, s);
  if (T == 2) return gconv_launch_t<E, 2>(op, in, out, B, H, W, Cin, Cout, k, s);
  return gconv_launch_t<E, 1>(op, in, out, B, H, W, Cin, Cout, k, s);
}

// op 0 gather (in f, out X), 1 scatter (in dX, out df), 2 pack (in psi, out w),
// 3 unpack (in dw, out dpsi), 4 adjoint pack (in psi, out w')
int gconv_common(int op, const void* in, void* out, int64_t B, int H, int W, int T, int Cin, int Cout, int k,
                 int dtype, void* stream) {
  int st = gconv_shape(T, Cin, Cout, k, dtype);
  if (st) return st;
  if (op < 2 && (st = gconv_image(B, H, W))) return st;
  const int64_t n_pix = op < 2 ? B * H * W : 0;
  if ((op >= 2 || n_pix > 0) && (!in || !out)) return EQL_ERR_INVALID_ARG;
  const size_t e = elem_bytes(dtype);
  if ((in && !aligned(in, e)) || (out && !aligned(out, e))) return EQL_ERR_ALIGNMENT;
  const size_t fb = (size_t)n_pix * Cin * T * e, xb = (size_t)n_pix * k * k * Cin * T * e;
  const size_t wb = (size_t)T * Cout * k * k * Cin * e;
  const size_t in_b = op == 0 ? fb : op == 1 ? xb : wb;
  const size_t out_b = op == 0 ? xb : op == 1 ? fb : wb;
  const Range r[2] = {{in, in_b}, {out, out_b}};
  if (any_overlap(r, 2)) return EQL_ERR_INVALID_ARG;
  if ((st = check_device())) return st;
  hipStream_t s = (hipStream_t)stream;
  if (dtype == EQL_F16) return gconv_launch<_Float16>(op, in, out, B, H, W, T, Cin, Cout, k, s);
  if (dtype == EQL_BF16) return gconv_launch<__bf16>(op, in, out, B, H, W, T, Cin, Cout, k, s);
  return gconv_launch<float>(op, in, out, B, H, W, T, Cin, Cout, k, s);
}

}  // namespace

extern "C" {

int eqlinear_gconv_gather(const void* f, void* xcol, int64_t B, int H, int W, int T, int Cin, int k, int dtype,
                          void* stream) {
  return gconv_common(0, f, xcol, B, H, W, T, Cin, 1, k, dtype, stream);
}

int eqlinear_gconv_scatter(const void* dxcol, void* df, int64_t B, int H, int W, int T, int Cin, int k,
                           int dtype, void* stream) {
  return gconv_common(1, dxcol, df, B, H, W, T, Cin, 1, k, dtype, stream);
}

int eqlinear_gconv_forward(const void* f, const void* wspec, const void* bias, void* y, int64_t B, int H, int W,
                           int T, int Cin, int Cout, int k, int dtype, void* stream) {
  int st = gconv_shape(T, Cin, Cout, k, dtype);
  if (st) return st;
  if ((st = gconv_image(B, H, W))) return st;
  if (Cin % 4 != 0) return EQL_ERR_UNSUPPORTED;  // a lane's four gathered channels stay in one block
  const int64_t N = B * H * W;
  const int Ci = k * k * Cin;
  if ((st = check_shape(N, T, Ci, Cout, dtype))) return st;
  if (!wspec || (N > 0 && (!f || !y))) return EQL_ERR_INVALID_ARG;
  const size_t e = elem_bytes(dtype);
  if (!aligned(wspec, 16) || (f && !aligned(f, 16)) || (y && !aligned(y, 16)) || (bias && !aligned(bias, e)))
    return EQL_ERR_ALIGNMENT;
  const size_t fb = (size_t)N * Cin * T * e;
  if (fb >= ((size_t)1 << 31)) return EQL_ERR_UNSUPPORTED;  // one 31-bit buffer range over the features
  const Range r[4] = {{f, fb},
                      {y, (size_t)N * Cout * T * e},
                      {wspec, eqlinear_weight_spectrum_bytes(T, Ci, Cout, dtype)},
                      {bias, bias ? (size_t)Cout * e : 0}};
  if (any_overlap(r, 4)) return EQL_ERR_INVALID_ARG;
  if ((st = check_device())) return st;
  if (N == 0) return EQL_OK;
  const bool w16 = dtype != EQL_F32;
  eqk::GemmArgs a{};
  a.in = f;
  a.wsp = wspec;
  a.bias = bias;
  a.out = y;
  a.N = N;
  a.Ci = Ci;
  a.Co = Cout;
  a.Ci_pad = eqk::wspec_dims(T, Ci, Cout, w16).CiF;
  a.stream = (hipStream_t)stream;
  {
    const unsigned od = T == 4 ? (unsigned)(k / 2 + 1) : (unsigned)k;
    a.geo = eqk::GatherGeom{H, W, Cin, k, eqk::div_magic(W), eqk::div_magic(H), eqk::div_magic(Cin * T),
                            eqk::div_magic(od)};
  }
  a.plan = eqk::gemm_plan(T, Ci, Cout, w16);
  eqk::gemm_plan_rows(a.plan, N, T, w16, eqk::device_cu_count());
  if (a.plan.narrow) return EQL_ERR_UNSUPPORTED;
  if (a.plan.mode == 1) {  // the gathered rows are not kept resident: stream the weights
    a.plan.mode = 0;
    a.plan.lds_bytes = eqk::gemm_lds_c(T, w16, a.plan.OT, eqk::gemm_wblocks(0, a.plan.n_oc, a.plan.n_ks));
  }
  return launched(eqk::launch_gemm_gather(dtype, T, a));
}

int eqlinear_gconv_pack_weight(const void* psi, void* w_ct, int T, int Cin, int Cout, int k, int dtype,
                               void* stream) {
  return gconv_common(2, psi, w_ct, 0, 0, 0, T, Cin, Cout, k, dtype, stream);
}

int eqlinear_gconv_unpack_weight(const void* dw_ct, void* dpsi, int T, int Cin, int Cout, int k, int dtype,
                                 void* stream) {
  return gconv_common(3, dw_ct, dpsi, 0, 0, 0, T, Cin, Cout, k, dtype, stream);
}

int eqlinear_gconv_pack_weight_adjoint(const void* psi, void* w_adj, int T, int Cin, int Cout, int k, int dtype,
                                       void* stream) {
  return gconv_common(4, psi, w_adj, 0, 0, 0, T, Cin, Cout, k, dtype, stream);
}

}  // extern "C"
