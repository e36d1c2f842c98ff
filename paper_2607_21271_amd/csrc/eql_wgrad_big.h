// eql_wgrad_big.h -- weight gradient of wide layers (fp16, bf16, fp32; T in
// {2, 4}): the MFMA-bound regime of Appendix A.2's
//   H_k[c,o] = sum_n conj(Xhat_k[n,c]) dYhat_k[n,o],   db[o] = sum_n dYhat_0[n,o],
// the contraction running over the rows.
//
// The register-direct kernel (eql_wgrad_rd.h) transforms every row once per
// channel tile, and its tiles are small (the T accumulator planes): at 2048
// channels each row is transformed tens of times.  Here the transforms run
// once, in a pre-pass that writes the spectra of x and dy row-contiguous
// (planes [T][C_pad][N_pad], each plane row one channel over all rows, zero
// padded), so that an MFMA operand -- one channel over 8 consecutive rows --
// is 16 contiguous bytes.  The product kernel is then a register-blocked GEMM
// over rows like the large-tile forward (eql_gemm_big.h): a workgroup of four
// waves owns a 128 x 128 (c, o) tile for all T planes, each wave a 64 x 64
// quarter with its T * 64 accumulators in the accumulation registers; per
// step of 64 bytes of each channel row (32 rows of 16-bit spectra, 16 of
// fp32) the x spectrum goes straight into LDS (buffer_load ... lds),
// two steps ahead, and the dy spectrum through registers, one step ahead (the
// pipeline of the large-tile forward).  Row splits fill the device when
// there are fewer tiles than CUs.  Each workgroup writes its fp32 partial in
// the layout of the split-partial reduction (eql_wgrad_reduce_kernel), which
// sums the splits in a fixed order and runs the inverse transform.
//
// GAUSS (fp32, T = 4): the complex bin in three products,
//   A1 += (Xr - Xi) Dr,  A2 += Xr (Di - Dr),  A3 += Xi (Dr + Di),
//   Re H = A1 + A3,  Im H = A1 + A2,
// with 96-channel o-tiles (the third accumulator plane), as in the large-tile
// forward.
#pragma once
#include "eql_gemm_big.h"
#include "eql_wgrad.h"

namespace eqk {

constexpr int kWbBC = 128;  // channel tile (c, and o without GAUSS)
constexpr int kWbKR = 32;   // rows per step (16-bit elements; 16 for fp32)
constexpr int kWbRB = 64;   // bytes of one staged channel per step
constexpr int wgrad_big_bo(bool gauss) { return gauss ? 96 : kWbBC; }

// LDS of the product kernel: three buffers of the T x planes, two of the T dy
// planes (160 KB at T = 4; 136 KB with GAUSS)
constexpr int wgrad_big_lds_bytes(int T, bool gauss = false) {
  return T * (3 * kWbBC + 2 * wgrad_big_bo(gauss)) * kWbRB;
}

// Row-contiguous spectrum: in [N, C, T] -> out[p][c][n] (p < T, c < C_pad,
// n < N_pad), zero for c >= C or n >= N.  A thread transforms one channel of 8
// rows (two rows at a time, as the register-direct kernel does: packed fp16
// for fp16, fp32 then one rounding for bf16; fp32 row by row) and stores 16
// (32 for fp32) bytes per plane.
// Lane l of a wave takes channel l / 8 and rows 8 (l % 8) .. + 7 of the wave's
// 8 channels x 64 rows, so the 8 lanes of a channel store one whole 128-byte
// line per plane; a block (4 waves) covers 32 channels x 64 rows.  1-D grid,
// blocks in (row block, channel block) order.
template <int T, int DT>
__global__ __launch_bounds__(256) void eql_spec_rows_kernel(const void* __restrict__ in, void* __restrict__ out,
                                                            int64_t N, int C, int C_pad, int64_t N_pad,
                                                            int n_cb) {
  constexpr int EB = DT == kF32 ? 4 : 2;
  constexpr int ITB = T * EB;
  constexpr int WPR = (ITB + 3) / 4;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t bid = blockIdx.x;
  const int cb = (int)(bid % n_cb);
  const int64_t rb = bid / n_cb;
  const int c = cb * 32 + wave * 8 + (lane >> 3);
  const int r8 = (lane & 7) * 8;           // first of this thread's 8 rows in the block
  const int64_t n0 = rb * 64 + r8;
  const int64_t rows_here = N - rb * 64 < 64 ? N - rb * 64 : 64;
  // the block's rows as a buffer resource: rows past N read zero
  const __amdgpu_buffer_rsrc_t rs =
      make_rsrc(reinterpret_cast<const char*>(in) + rb * 64 * (int64_t)C * ITB,
                (uint32_t)(rows_here > 0 ? rows_here * C * ITB : 0));
  const bool live = c < C;
  char* const o = reinterpret_cast<char*>(out);
  if constexpr (DT == kF32) {
    float Q[T][8];
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      uint32_t wds[WPR];
      const uint32_t off = (uint32_t)(((r8 + m) * C + (live ? c : C - 1)) * ITB);
      load_row<T, EB>(rs, off, wds);
      float v[T], q[T];
#pragma unroll
      for (int t = 0; t < T; ++t) v[t] = live ? __builtin_bit_cast(float, wds[t]) : 0.0f;
      rdft<T>(v, q);
#pragma unroll
      for (int p = 0; p < T; ++p) Q[p][m] = q[p];
    }
    if (c >= C_pad) return;
#pragma unroll
    for (int p = 0; p < T; ++p) {
      char* dst = o + (((int64_t)p * C_pad + c) * N_pad + n0) * EB;
      *reinterpret_cast<u32x4*>(dst) =
          u32x4{__builtin_bit_cast(uint32_t, Q[p][0]), __builtin_bit_cast(uint32_t, Q[p][1]),
                __builtin_bit_cast(uint32_t, Q[p][2]), __builtin_bit_cast(uint32_t, Q[p][3])};
      *reinterpret_cast<u32x4*>(dst + 16) =
          u32x4{__builtin_bit_cast(uint32_t, Q[p][4]), __builtin_bit_cast(uint32_t, Q[p][5]),
                __builtin_bit_cast(uint32_t, Q[p][6]), __builtin_bit_cast(uint32_t, Q[p][7])};
    }
  } else {
    uint32_t W[T][4];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      uint32_t two[2 * WPR];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        uint32_t wds[WPR];
        // a channel past C reads channel C - 1 and is zeroed below
        const uint32_t off = (uint32_t)(((r8 + 2 * m + h) * C + (live ? c : C - 1)) * ITB);
        load_row<T, EB>(rs, off, wds);
#pragma unroll
        for (int q = 0; q < WPR; ++q) two[h * WPR + q] = live ? wds[q] : 0u;
      }
      if constexpr (DT == kF16) {
        half2v P[T];
        transform_pair<T>(two, P);
#pragma unroll
        for (int p = 0; p < T; ++p) W[p][m] = __builtin_bit_cast(uint32_t, P[p]);
      } else {
        float P0[T], P1[T];
        transform_pair_f32<T>(two, P0, P1);
#pragma unroll
        for (int p = 0; p < T; ++p) W[p][m] = pack2<DT>(P0[p], P1[p]);
      }
    }
    if (c >= C_pad) return;
#pragma unroll
    for (int p = 0; p < T; ++p)
      *reinterpret_cast<u32x4*>(o + (((int64_t)p * C_pad + c) * N_pad + n0) * EB) =
          u32x4{W[p][0], W[p][1], W[p][2], W[p][3]};
  }
}

// Product kernel.  xs, ds: row-contiguous spectra (planes [T][C_pad][N_pad]).
// Block b -> (split, c-tile, o-tile): XCD-contiguous runs, the tiles of one
// split together (they read the same rows), sweeping groups of four c-tiles
// across the o-tiles.  Split s covers rows [s * rows_per_split, ...) in steps
// of 32 (16 for fp32; rows past N are zero in the spectra).  Partial:
// part[s][p][c/4][o][c%4] (Cin_pad / Cout_pad: the padded extents, multiples
// of the c- and o-tiles); bias partial dbpart[s][o] from bin 0 of dy (c-tile 0
// only).
template <int T, int DT, bool GAUSS = false>
__global__ __launch_bounds__(kBigThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void eql_wgrad_big_kernel(const void* __restrict__ xs, const void* __restrict__ ds, float* __restrict__ part,
                          float* __restrict__ dbpart, int64_t N_pad, int Cin_pad, int Cout_pad, int n_ct,
                          int n_ot, int n_splits, int64_t rows_per_split) {
  static_assert(T == 2 || T == 4, "accumulators for T <= 4 planes");
  static_assert(!GAUSS || (T == 4 && DT == kF32), "three-product bins: fp32, T = 4");
  using Bn = Bins<T>;
  using FR = Frag<16>;
  constexpr int EB = DT == kF32 ? 4 : 2;
  constexpr int KR = kWbRB / EB;                // rows per step
  constexpr int KWM = 16 / EB;                  // contraction elements per fragment
  constexpr int NJ = GAUSS ? 3 : 4;             // MFMA o-tiles per wave
  constexpr int BO = 32 * NJ;                   // o-channels of the tile
  constexpr int NA = T + (GAUSS ? 1 : 0);       // accumulator planes
  constexpr int PL = kWbBC * kWbRB;             // bytes of one staged x plane (128 channels)
  constexpr int DPL = BO * kWbRB;               // bytes of one staged dy plane
  constexpr int XB = T * PL;                    // one x buffer (three)
  constexpr int DB = T * DPL;                   // one dy buffer (two)
  constexpr int NWV = kBigThreads / 64;
  constexpr int WDU = XB / 1024 / NWV;          // x wave-loads per wave and step
  constexpr int DU = DB / 16 / kBigThreads;     // dy 16-byte chunks per thread and step
  constexpr int DQ = DU % 4 == 0 ? 4 : 2;       // portions of the dy staging (row tiles that carry one)
  static_assert(3 * XB + 2 * DB == wgrad_big_lds_bytes(T, GAUSS) && XB % (1024 * NWV) == 0 &&
                DB % (16 * kBigThreads) == 0 && DU % DQ == 0, "LDS layout");
  constexpr int DUQ = DU / DQ;                  // dy chunks per portion

  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* const xbase = smem;            // x buffers
  char* const dbase = smem + 3 * XB;   // dy buffers
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave >> 1, wc = wave & 1;
  const int g = lane >> 4, li = lane & 15;

  // block -> (split, ct, ot)
  const int tiles = n_ct * n_ot;
  int split, ct, ot;
  {
    const int G = n_splits * tiles;
    const int bid = blockIdx.x;
    const int q = G / 8, r = G % 8, xcd = bid % 8, idx = bid / 8;
    const int t = xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
    split = t / tiles;
    const int u = t - split * tiles;
    const int gsz = kBigGroup * n_ot;
    const int grp = u / gsz, in = u - grp * gsz;
    const int rows = n_ct - grp * kBigGroup < kBigGroup ? n_ct - grp * kBigGroup : kBigGroup;
    ct = grp * kBigGroup + in % rows;
    ot = in / rows;
  }
  const int c0 = ct * kWbBC, o0 = ot * BO;
  const int64_t n_begin = (int64_t)split * rows_per_split;
  const int64_t n_end = n_begin + rows_per_split < N_pad ? n_begin + rows_per_split : N_pad;
  const int nks = (int)((n_end - n_begin) / KR);

  // The split's rows of the tile's channels as buffer resources, from
  // (plane 0, channel c0 / o0, row n_begin) to the end of each spectrum
  // (loads past it read zero).  Plane p lies Cin_pad (Cout_pad) channel rows
  // further on; the offsets stay below 2^31 bytes (host check).
  const int64_t pitch = N_pad * EB;
  const __amdgpu_buffer_rsrc_t xrs =
      make_rsrc(reinterpret_cast<const char*>(xs) + c0 * pitch + n_begin * EB,
                (uint32_t)(((int64_t)T * Cin_pad - c0) * pitch - n_begin * EB));
  const __amdgpu_buffer_rsrc_t drs =
      make_rsrc(reinterpret_cast<const char*>(ds) + o0 * pitch + n_begin * EB,
                (uint32_t)(((int64_t)T * Cout_pad - o0) * pitch - n_begin * EB));
  // chunk ch of staged channel row r sits at chunk ch ^ ((r >> 1) & 3)
  // x: one LDS slot (16 bytes) per lane and wave-load
  uint32_t xoff[WDU];
#pragma unroll
  for (int v = 0; v < WDU; ++v) {
    const int slot = (v * NWV + wave) * 64 + lane;
    const int p = slot / (kWbBC * 4), rem = slot - p * (kWbBC * 4);
    const int row = rem / 4, cs = rem % 4;
    const int ch = cs ^ ((row >> 1) & 3);
    xoff[v] = (uint32_t)(((int64_t)p * Cin_pad + row) * pitch + ch * 16);
  }
  // dy: chunk u = tid + 256 v of the step's planes, global offset and LDS slot
  uint32_t doff[DU];
  int dlds[DU];
#pragma unroll
  for (int v = 0; v < DU; ++v) {
    const int u = tid + kBigThreads * v;
    const int p = u / (BO * 4), rem = u - p * (BO * 4);
    const int row = rem / 4, ch = rem % 4;
    doff[v] = (uint32_t)(((int64_t)p * Cout_pad + row) * pitch + ch * 16);
    dlds[v] = p * DPL + wl_off<kWbRB>(row, ch * 16);
  }
  u32x4 dr[DU];

  // x rows of step s into x buffer s % 3 (past the split: rows of the next
  // split or past the resource, in a buffer never read again)
  auto load_x = [&](int s) __attribute__((always_inline)) {
#if defined(__HIP_DEVICE_COMPILE__)
    const int so = s * KR * EB;
    char* base = xbase + (s % 3) * XB;
#pragma unroll
    for (int v = 0; v < WDU; ++v)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          xrs, (__attribute__((address_space(3))) void*)(base + (v * NWV + wave) * 1024), 16, xoff[v], so, 0, 0);
#else
    (void)s;
    (void)xrs;
#endif
  };
  // dy chunks [v0, v0 + DUQ) of step s into registers; written to dy buffer b
  auto load_d = [&](int s, int v0) __attribute__((always_inline)) {
    const int so = s * KR * EB;
#pragma unroll
    for (int v = v0; v < v0 + DUQ; ++v)
      dr[v] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(drs, doff[v], so, 0));
  };
  auto store_d = [&](int b, int v0) __attribute__((always_inline)) {
#pragma unroll
    for (int v = v0; v < v0 + DUQ; ++v) *reinterpret_cast<u32x4*>(dbase + b * DB + dlds[v]) = dr[v];
  };
  // Barrier of step s: this wave's LDS writes done and the x rows of s in LDS;
  // the vector-memory instructions issued after those (dy of s and s + 1, x of
  // s + 1) may stay in flight.  No memory fence (a workgroup fence would also
  // wait for the x rows of s + 1); the signal fences keep the compiler from
  // moving memory accesses across.  vmcnt n: bits 3:0 and 15:14; lgkmcnt 11:8.
  constexpr int NV = 2 * DU + WDU;
  static_assert(NV < 64, "vmcnt range");
  constexpr int kWaitBar = (NV & 15) | ((NV >> 4) << 14) | 0x0070;
  auto barrier = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(kWaitBar);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
  };

  floatx4 acc[NA][4][NJ];
#pragma unroll
  for (int p = 0; p < NA; ++p)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) acc[p][i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  // bias gradient: waves of c-quarter 0 in c-tile 0 sum bin 0 of dy
  const bool do_db = dbpart != nullptr && ct == 0 && wr == 0;
  float dbacc[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) dbacc[j] = 0.f;
  // fp32 fragment sums (GAUSS operands)
  auto fsum = [](const FR& a, const FR& b) __attribute__((always_inline)) {
    FR r;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      r.w[q] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(float, a.w[q]) + __builtin_bit_cast(float, b.w[q]));
    return r;
  };
  auto fdiff = [](const FR& a, const FR& b) __attribute__((always_inline)) {
    FR r;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      r.w[q] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(float, a.w[q]) - __builtin_bit_cast(float, b.w[q]));
    return r;
  };

  // Products of one step, as in the large-tile forward: per phase (real bins,
  // then each complex bin) the wave's dy fragments stay in registers and the
  // x fragments are read one 16-channel tile ahead.  Complex bin:
  //   Re H += Xr Dr + Xi Di,   Im H += Xr Di + (-Xi) Dr
  // each accumulator's second product eight MFMAs after its first.
  auto step = [&](int s) __attribute__((always_inline)) {
    const char* xl = xbase + (s % 3) * XB;
    const char* dl = dbase + (s & 1) * DB;
    const int nb = (s + 1) & 1;
    auto colf = [&](int p, FR (&Bp)[NJ]) __attribute__((always_inline)) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) Bp[j] = lds_frag<16, kWbRB>(dl + p * DPL, wc * 16 * NJ + j * 16 + li, g);
    };
    // a portion of the next step's dy chunks, in row tile i (of the first
    // complex bin; of the real bins at T = 2): written to LDS, then reloaded
    // with the step after
    auto stage_d = [&](auto ii) __attribute__((always_inline)) {
      constexpr int i = decltype(ii)::value;
      if constexpr (i % (4 / DQ) == 4 / DQ - 1) {
        store_d(nb, (i / (4 / DQ)) * DUQ);
        load_d(s + 2, (i / (4 / DQ)) * DUQ);
      }
    };
    auto rowf = [&](int p, int i) __attribute__((always_inline)) {
      return lds_frag<16, kWbRB>(xl + p * PL, wr * 64 + i * 16 + li, g);
    };
    {
      constexpr int R = Bn::R;
      FR B[R][NJ];
      FR A[2][R];
#pragma unroll
      for (int p = 0; p < R; ++p) colf(p, B[p]);
#pragma unroll
      for (int p = 0; p < R; ++p) A[0][p] = rowf(p, 0);
      if (do_db) {
        // bin 0 of 8 rows of one output channel per lane and fragment
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const uint32_t wd = B[0][j].w[w];
            if constexpr (DT == kF32) {
              dbacc[j] += __builtin_bit_cast(float, wd);
            } else if constexpr (DT == kF16) {
              dbacc[j] = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2v, wd),
                                                half2v{(_Float16)1.0f, (_Float16)1.0f}, dbacc[j], false);
            } else {
              dbacc[j] += __builtin_bit_cast(float, wd << 16) + __builtin_bit_cast(float, wd & 0xffff0000u);
            }
          }
      }
      static_for<4>([&](auto ii) {
        constexpr int i = decltype(ii)::value;
        if constexpr (i + 1 < 4) {
#pragma unroll
          for (int p = 0; p < R; ++p) A[(i + 1) & 1][p] = rowf(p, i + 1);
        }
#pragma unroll
        for (int p = 0; p < R; ++p)
#pragma unroll
          for (int j = 0; j < NJ; ++j) frag_mma<DT, KWM>(acc[p][i][j], A[i & 1][p], B[p][j]);
        if constexpr (Bn::K == 0) stage_d(ii);
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    if constexpr (GAUSS) {
      static_assert(Bn::K == 1, "one complex bin");
      constexpr int re = Bn::re(1), im = Bn::im(1);
      FR Br[NJ], Bd[NJ], Bu[NJ];
      FR Ar[2], Ai[2];
      colf(re, Br);
      colf(im, Bd);
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        Bu[j] = fsum(Br[j], Bd[j]);   // Dr + Di
        Bd[j] = fdiff(Bd[j], Br[j]);  // Di - Dr
      }
      Ar[0] = rowf(re, 0);
      Ai[0] = rowf(im, 0);
      static_for<4>([&](auto ii) {
        constexpr int i = decltype(ii)::value;
        if constexpr (i + 1 < 4) {
          Ar[(i + 1) & 1] = rowf(re, i + 1);
          Ai[(i + 1) & 1] = rowf(im, i + 1);
        }
        const FR& xre = Ar[i & 1];
        const FR& xim = Ai[i & 1];
        const FR xd = fdiff(xre, xim);
#pragma unroll
        for (int j = 0; j < NJ; ++j) frag_mma<DT, KWM>(acc[re][i][j], xd, Br[j]);
#pragma unroll
        for (int j = 0; j < NJ; ++j) frag_mma<DT, KWM>(acc[im][i][j], xre, Bd[j]);
#pragma unroll
        for (int j = 0; j < NJ; ++j) frag_mma<DT, KWM>(acc[T][i][j], xim, Bu[j]);
        stage_d(ii);
        __builtin_amdgcn_sched_barrier(0);
      });
    } else {
      static_for<Bn::K>([&](auto ki) {
        constexpr int k = decltype(ki)::value + 1;
        constexpr int re = Bn::re(k), im = Bn::im(k);
        FR Br[NJ], Bi[NJ];
        FR Ar[2], Ai[2];
        colf(re, Br);
        colf(im, Bi);
        Ar[0] = rowf(re, 0);
        Ai[0] = rowf(im, 0);
        static_for<4>([&](auto ii) {
          constexpr int i = decltype(ii)::value;
          if constexpr (i + 1 < 4) {
            Ar[(i + 1) & 1] = rowf(re, i + 1);
            Ai[(i + 1) & 1] = rowf(im, i + 1);
          }
          const FR& xre = Ar[i & 1];
          const FR& xim = Ai[i & 1];
          const FR xn = frag_neg<DT, 16>(xim);
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            frag_mma<DT, KWM>(acc[re][i][j], xre, Br[j]);
            frag_mma<DT, KWM>(acc[im][i][j], xre, Bi[j]);
          }
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            frag_mma<DT, KWM>(acc[re][i][j], xim, Bi[j]);
            frag_mma<DT, KWM>(acc[im][i][j], xn, Br[j]);
          }
          if constexpr (k == 1) stage_d(ii);
          __builtin_amdgcn_sched_barrier(0);
        });
      });
    }
  };

  // prologue: dy of step 0 staged, x of steps 0 and 1 and dy of step 1 in
  // flight.  Step s: barrier (buffers of s complete; those read in step s - 1
  // free), x of s + 2 issued, products of s with the dy of s + 1 staged.
  load_x(0);
#pragma unroll
  for (int q = 0; q < DQ; ++q) load_d(0, q * DUQ);
  load_x(1);
#pragma unroll
  for (int q = 0; q < DQ; ++q) store_d(0, q * DUQ);
#pragma unroll
  for (int q = 0; q < DQ; ++q) load_d(1, q * DUQ);
  for (int s = 0; s < nks; ++s) {
    barrier();
    load_x(s + 2);
    step(s);
  }

  // partial: lane (g, li) of tile (i, j) holds c = c0 + wr*64 + 16i + 4g + r
  // (r = 0..3), o = o0 + wc*16*NJ + 16j + li
  const int CQ = Cin_pad / 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int cq = (c0 + wr * 64 + 16 * i) / 4 + g;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int oo = o0 + wc * 16 * NJ + 16 * j + li;
      if constexpr (GAUSS) {
        constexpr int re = Bn::re(1), im = Bn::im(1);
        const floatx4 a1 = acc[re][i][j], a2 = acc[im][i][j], a3 = acc[T][i][j];
        acc[re][i][j] = a1 + a3;
        acc[im][i][j] = a1 + a2;
      }
#pragma unroll
      for (int p = 0; p < T; ++p)
        *reinterpret_cast<floatx4*>(part + ((((int64_t)split * T + p) * CQ + cq) * Cout_pad + oo) * 4) =
            acc[p][i][j];
    }
  }
  if (do_db) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      float v = dbacc[j];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (g == 0) dbpart[(int64_t)split * Cout_pad + o0 + wc * 16 * NJ + 16 * j + li] = v;
    }
  }
}

}  // namespace eqk
