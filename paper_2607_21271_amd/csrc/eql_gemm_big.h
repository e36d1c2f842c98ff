// eql_gemm_big.h -- forward / input-gradient kernel for wide layers: large
// output tiles for the MFMA-bound regime (fp16, bf16 and fp32).
//
// The same computation as eql_gemm_kernel (Alg. 1; Sec. 3.3-3.5: rDFT of the
// activations in registers, per-bin products against the precomputed weight
// spectrum with fp32 accumulation, irDFT and bias in the epilogue), laid out
// for layers whose spectral products dominate the run time.  There the
// operands must be reused from registers: a workgroup computes a 128-row x
// 128-channel output tile for all T planes, each of its four waves a 64 x 64
// quarter (4 x 4 MFMA tiles per plane, T * 64 accumulator registers, which
// live in the accumulation registers at one wave per SIMD).  Per contraction
// step of 32 input channels the workgroup stages the activation spectrum
// (128 rows; two LDS buffers) and the weight spectrum (128 output channels;
// three LDS buffers, loaded two steps ahead straight from global memory);
// each wave reads four row fragments and four channel fragments per plane
// and issues 16 MFMAs per product.  LDS operand traffic per MFMA is a quarter
// of the 16-row tiles of eql_gemm_kernel.  Each step's barrier is an explicit
// wait plus s_barrier with compiler fences only, so loads of later steps stay
// in flight across it.
//
// GAUSS (fp32, T = 4): each complex bin in three products instead of four
// (Eq. 5's product in the three-multiplication form), accumulated apart and
// combined in the epilogue:
//   A1 += (Xr + Xi) Wr,  A2 += Xr (Wi - Wr),  A3 += Xi (Wr + Wi)
//   forward:  Re = A1 - A3,  Im = A1 + A2
//   backward (D = dy spectrum): A2 += Di (Wi - Wr), A3 += Dr (Wr + Wi),
//             Re = A1 + A2,  Im = A1 - A3
// The operand sums are formed in registers from the staged planes.  The third
// accumulator plane takes the channel tile to 96 (4 x 3 MFMA tiles per wave
// and plane, 5 * 48 accumulators per lane).
//
// Workgroups are renumbered so that each XCD (blocks dealt round-robin over
// the 8 of them) takes a contiguous run of tiles, and runs sweep groups of four
// row tiles across all channel tiles, so the workgroups resident on one XCD
// share activation rows and weight rows in its L2.
#pragma once
#include "eql_gemm.h"

namespace eqk {

constexpr int kBigThreads = 256;
constexpr int kBigBM = 128;  // rows per workgroup tile
constexpr int kBigBN = 128;  // output channels per workgroup tile (96 with GAUSS)
constexpr int kBigBK = 32;   // contraction channels per step (16-bit elements; 16 for fp32)
constexpr int kBigRB = 64;   // bytes of one staged row per step (32 16-bit channels)
constexpr int kBigGroup = 4; // row tiles per sweep group

constexpr int big_bn(bool gauss) { return gauss ? 96 : kBigBN; }

// dynamic LDS of one workgroup: two buffers of T activation planes, three of
// T weight planes (160 KB at T = 4; 136 KB with GAUSS)
constexpr int big_lds_bytes(int T, bool gauss = false) { return T * (2 * kBigBM + 3 * big_bn(gauss)) * kBigRB; }

// tile (rt, ct) of block bid out of n_rt * n_ct blocks
__device__ __forceinline__ void big_tile(int bid, int n_rt, int n_ct, int& rt, int& ct) {
  const int G = n_rt * n_ct;
  const int q = G / 8, r = G % 8, xcd = bid % 8, idx = bid / 8;
  const int t = xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
  const int gsz = kBigGroup * n_ct;
  const int grp = t / gsz, in = t - grp * gsz;
  const int rows = n_rt - grp * kBigGroup < kBigGroup ? n_rt - grp * kBigGroup : kBigGroup;
  rt = grp * kBigGroup + in % rows;
  ct = in / rows;
}

// in [N, Ci, T], weight spectrum planes [T][w_rows][w_pitch] (row = output
// channel, w_pitch >= Ci padded with zeros), out [N, Co, T].  Requires
// Ci % 32 == 0 and the per-tile row ranges below 2^31 bytes (host checks).
// A step covers 64 bytes of each staged row: 32 channels of 16-bit elements
// (v_mfma_f32_16x16x32_f16 / bf16), 16 of fp32 (four v_mfma_f32_16x16x4f32
// per fragment pair, a quarter of the contraction each).
// BWD: in = dy, the transposed spectrum, conjugate products, no bias.
template <int T, int DT, bool BWD, bool GAUSS = false>
__global__ __launch_bounds__(kBigThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void eql_gemm_big_kernel(const void* __restrict__ in, const void* __restrict__ wsp,
                         const void* __restrict__ bias, void* __restrict__ out, int64_t N, int Ci, int Co,
                         int w_rows, int w_pitch, int n_rt, int n_ct) {
  static_assert(T == 2 || T == 4, "accumulators for T <= 4 planes");
  static_assert(!GAUSS || (T == 4 && DT == kF32), "three-product bins: fp32, T = 4");
  constexpr int NJ = GAUSS ? 3 : 4;             // MFMA column tiles per wave
  constexpr int BN = 32 * NJ;                   // output channels of the tile
  constexpr int NA = T + (GAUSS ? 1 : 0);       // accumulator planes
  using Bn = Bins<T>;
  using FR = Frag<16>;
  constexpr int EB = DT == kF32 ? 4 : 2;
  constexpr int BK = kBigRB / EB;               // contraction channels per step
  constexpr int KWM = 16 / EB;                  // contraction elements per fragment
  constexpr int HKW = 4;                        // channels of one staging unit
  constexpr int UB = HKW * T * EB;              // raw bytes of a unit: 16, 32 or 64
  constexpr int UPR = BK / HKW;                 // units per row and step
  constexpr int XU = kBigBM * UPR / kBigThreads;  // units per thread
  constexpr int XPL = kBigBM * kBigRB;          // bytes of one activation plane
  constexpr int WPL = BN * kBigRB;              // bytes of one weight plane
  constexpr int XB = T * XPL;                   // one activation buffer
  constexpr int WB = T * WPL;                   // one weight buffer
  constexpr int WCH = T * BN * (kBigRB / 16);   // 16-byte weight chunks per step
  static_assert((kBigBM * UPR) % kBigThreads == 0, "thread split");
  static_assert(2 * XB + 3 * WB == big_lds_bytes(T, GAUSS), "LDS size");

  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* const xbase = smem;           // activation buffers
  char* const wbase = smem + 2 * XB;  // weight buffers
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave >> 1, wc = wave & 1;     // quarter of the tile
  const int g = lane >> 4, li = lane & 15;

  int rt, ct;
  big_tile(blockIdx.x, n_rt, n_ct, rt, ct);
  const int64_t r0 = (int64_t)rt * kBigBM;
  const int len = N - r0 < kBigBM ? (int)(N - r0) : kBigBM;
  const int o0 = ct * BN;
  const int rowb_in = Ci * T * EB;
  const int rowb_out = Co * T * EB;
  // rows of the tile as buffer resources: loads past them read zero, stores
  // past them are dropped
  const __amdgpu_buffer_rsrc_t xrs =
      make_rsrc(reinterpret_cast<const char*>(in) + r0 * rowb_in, (uint32_t)(len * rowb_in));
  const __amdgpu_buffer_rsrc_t wrs = make_rsrc(wsp, (uint32_t)((int64_t)T * w_rows * w_pitch * EB));
  const __amdgpu_buffer_rsrc_t ors =
      make_rsrc(reinterpret_cast<char*>(out) + r0 * rowb_out, (uint32_t)(len * rowb_out));

  // per-thread offsets (step offsets go in the scalar offset)
  uint32_t xoff[XU];
  int xlds[XU];
#pragma unroll
  for (int v = 0; v < XU; ++v) {
    const int u = tid + kBigThreads * v;
    const int row = u / UPR, q = u % UPR;
    xoff[v] = (uint32_t)(row * rowb_in + q * UB);
    xlds[v] = wl_off<kBigRB>(row, q * HKW * EB);
  }
  // weight chunks go from global memory straight into LDS (buffer_load ...
  // lds): a wave-load writes 64 x 16 contiguous bytes (lane l at byte 16 l of
  // the slice), so each lane fetches the chunk the swizzled layout puts at
  // its slot
  constexpr int NWV = kBigThreads / 64;
  constexpr int WDU = WCH / (64 * NWV);  // wave-loads per wave and step
  static_assert(WCH % (64 * NWV) == 0 && (BN * kBigRB) % 1024 == 0, "weight wave-loads");
  uint32_t woff[WDU];
#pragma unroll
  for (int v = 0; v < WDU; ++v) {
    const int slot = (v * NWV + wave) * 64 + lane;  // 16-byte slot of the weight planes
    const int p = slot / (BN * 4), rem = slot - p * (BN * 4);
    const int row = rem / 4, cs = rem % 4;
    const int ch = cs ^ ((row >> 1) & 3);           // source chunk swizzled to slot cs
    woff[v] = (uint32_t)(((int64_t)p * w_rows + o0 + row) * w_pitch * EB + ch * 16);
  }

  // Pipeline, per step s: the weight chunks of s + 2 issued into LDS buffer
  // (s + 2) % 3; the MFMAs of s, real bins then complex bins, and between the
  // row tiles of the first complex bin (of the real bins at T = 2) the four
  // staging units of the activations of s + 1 (loaded during step s - 1),
  // each transformed into LDS buffer (s + 1) & 1 and then reloaded with the
  // raw activations of s + 2.  Weights have two steps to arrive, activations
  // one, and the scheduler spreads the transforms between the MFMAs.
  uint32_t xr[XU][UB / 4];
  // (past the last step the reads land in padding or past the resources, in
  // buffers that are never read again)
  auto load_x = [&](int s, int v) __attribute__((always_inline)) {
    const int xs = s * BK * T * EB;
#pragma unroll
    for (int h = 0; h < UB / 16; ++h) {
      const u32x4 a = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(xrs, xoff[v] + 16 * h, xs, 0));
      xr[v][4 * h] = a[0]; xr[v][4 * h + 1] = a[1]; xr[v][4 * h + 2] = a[2]; xr[v][4 * h + 3] = a[3];
    }
  };
  auto load_w = [&](int s) __attribute__((always_inline)) {
#if defined(__HIP_DEVICE_COMPILE__)
    const int ws = s * BK * EB;
    char* wl = wbase + (s % 3) * WB;
#pragma unroll
    for (int v = 0; v < WDU; ++v)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          wrs, (__attribute__((address_space(3))) void*)(wl + (v * NWV + wave) * 1024), 16, woff[v], ws, 0, 0);
#else
    (void)s;
    (void)wrs;
#endif
  };
  // Barrier of step s: this wave's LDS writes done (lgkmcnt 0) and the weight
  // chunks of s in LDS; the vector-memory instructions issued after those
  // (activations of s and s + 1, weights of s + 1) may stay in flight.  The
  // barrier carries no memory fence (a workgroup fence would also wait for
  // the weight chunks of s + 1, which are still arriving); the signal fences
  // keep the compiler from moving memory accesses across it.  vmcnt n is
  // encoded in bits 3:0 and 15:14, lgkmcnt in 11:8.
  constexpr int NV = 2 * XU * (UB / 16) + WDU;
  static_assert(NV < 64, "vmcnt range");
  constexpr int kWaitBar = (NV & 15) | ((NV >> 4) << 14) | 0x0070;
  auto barrier = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(kWaitBar);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
  };
  // transform the raw activations of unit v into T planes in LDS activation
  // buffer b
  auto publish = [&](int b, int v) __attribute__((always_inline)) {
    char* base = xbase + b * XB;
    if constexpr (DT == kF32) {
      float P[T][HKW];
      raw_to_planes<T, DT, HKW>(xr[v], P);
#pragma unroll
      for (int p = 0; p < T; ++p)
        *reinterpret_cast<u32x4*>(base + p * XPL + xlds[v]) =
            u32x4{__builtin_bit_cast(uint32_t, P[p][0]), __builtin_bit_cast(uint32_t, P[p][1]),
                  __builtin_bit_cast(uint32_t, P[p][2]), __builtin_bit_cast(uint32_t, P[p][3])};
    } else {
      uint32_t W[T][HKW / 2];
      if constexpr (DT == kF16) {
        raw_to_packed_planes<T, HKW>(xr[v], W);
      } else {
        float P[T][HKW];
        raw_to_planes<T, DT, HKW>(xr[v], P);
#pragma unroll
        for (int p = 0; p < T; ++p)
#pragma unroll
          for (int j = 0; j < HKW / 2; ++j) W[p][j] = pack2<DT>(P[p][2 * j], P[p][2 * j + 1]);
      }
#pragma unroll
      for (int p = 0; p < T; ++p) *reinterpret_cast<u32x2*>(base + p * XPL + xlds[v]) = u32x2{W[p][0], W[p][1]};
    }
  };
  // staging units per thread: 4 (16-bit) or 2 (fp32); unit v is staged in
  // row tile UI * v + UI - 1 of the phase that carries them
  static_assert(XU == 4 || XU == 2, "staging units per thread");
  constexpr int UI = 4 / XU;

  floatx4 acc[NA][4][NJ];
#pragma unroll
  for (int p = 0; p < NA; ++p)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) acc[p][i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
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

  // Products of step s from activation buffer s & 1 and weight buffer s % 3,
  // in two phases: the real bins, then each complex bin.  A phase keeps its
  // planes' column fragments in registers and reads row fragments one 16-row
  // tile at a time, the next tile's ahead of the current tile's MFMAs.
  // Complex bins:
  //   forward:  Re += Xr Wr + (-Xi) Wi,  Im += Xr Wi + Xi Wr
  //   backward: Re += Dr Wr + Di Wi,     Im += Di Wr + (-Dr) Wi
  // each accumulator's second product coming eight MFMAs after its first.
  const int nks = Ci / BK;
  auto step = [&](int s) __attribute__((always_inline)) {
    const char* xl = xbase + (s & 1) * XB;
    const char* wl = wbase + (s % 3) * WB;
    auto colf = [&](int p, FR (&Bp)[NJ]) __attribute__((always_inline)) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) Bp[j] = lds_frag<16, kBigRB>(wl + p * WPL, wc * 16 * NJ + j * 16 + li, g);
    };
    auto rowf = [&](int p, int i) __attribute__((always_inline)) {
      return lds_frag<16, kBigRB>(xl + p * XPL, wr * 64 + i * 16 + li, g);
    };
    {
      constexpr int R = Bn::R;
      FR B[R][NJ];
      FR A[2][R];
#pragma unroll
      for (int p = 0; p < R; ++p) colf(p, B[p]);
#pragma unroll
      for (int p = 0; p < R; ++p) A[0][p] = rowf(p, 0);
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
        if constexpr (Bn::K == 0 && i % UI == UI - 1) {
          publish((s + 1) & 1, i / UI);
          load_x(s + 2, i / UI);
        }
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
        Bu[j] = fsum(Br[j], Bd[j]);   // Wr + Wi
        Bd[j] = fdiff(Bd[j], Br[j]);  // Wi - Wr
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
        const FR xs = fsum(xre, xim);
#pragma unroll
        for (int j = 0; j < NJ; ++j) frag_mma<DT, KWM>(acc[re][i][j], xs, Br[j]);
#pragma unroll
        for (int j = 0; j < NJ; ++j) frag_mma<DT, KWM>(acc[im][i][j], BWD ? xim : xre, Bd[j]);
#pragma unroll
        for (int j = 0; j < NJ; ++j) frag_mma<DT, KWM>(acc[T][i][j], BWD ? xre : xim, Bu[j]);
        if constexpr (i % UI == UI - 1) {
          publish((s + 1) & 1, i / UI);
          load_x(s + 2, i / UI);
        }
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
          const FR xn = frag_neg<DT, 16>(BWD ? xre : xim);
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            frag_mma<DT, KWM>(acc[re][i][j], xre, Br[j]);
            if constexpr (!BWD) frag_mma<DT, KWM>(acc[im][i][j], xre, Bi[j]);
            else frag_mma<DT, KWM>(acc[im][i][j], xim, Br[j]);
          }
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            if constexpr (!BWD) {
              frag_mma<DT, KWM>(acc[re][i][j], xn, Bi[j]);
              frag_mma<DT, KWM>(acc[im][i][j], xim, Br[j]);
            } else {
              frag_mma<DT, KWM>(acc[re][i][j], xim, Bi[j]);
              frag_mma<DT, KWM>(acc[im][i][j], xn, Bi[j]);
            }
          }
          // one staging unit of the next step per row tile (first complex
          // bin), interleaved with these MFMAs by the scheduler
          if constexpr (k == 1 && i % UI == UI - 1) {
            publish((s + 1) & 1, i / UI);
            load_x(s + 2, i / UI);
          }
          __builtin_amdgcn_sched_barrier(0);
        });
      });
    }
  };

  // prologue: activations of step 0 staged, weights of steps 0 and 1 and raw
  // activations of step 1 in flight.  The barrier of step s makes buffers
  // s & 1 / s % 3 complete and frees those read in step s - 1.
  load_w(0);
#pragma unroll
  for (int v = 0; v < XU; ++v) load_x(0, v);
  load_w(1);
#pragma unroll
  for (int v = 0; v < XU; ++v) publish(0, v);
#pragma unroll
  for (int v = 0; v < XU; ++v) load_x(1, v);
  for (int s = 0; s < nks; ++s) {
    barrier();
    load_w(s + 2);
    step(s);
  }

  // D = X W^T: lane (g, li) of tile (i, j) holds channel o0 + wc*16*NJ + j*16 + li
  // of rows wr*64 + i*16 + 4g .. +3; the 16 lanes of a lane group store 16
  // consecutive channels of one row (16*T contiguous elements)
  using E = typename Elem<DT>::T;
  const E* __restrict__ bp = reinterpret_cast<const E*>(bias);
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int o = o0 + wc * 16 * NJ + j * 16 + li;
    float bv = 0.0f;
    if constexpr (!BWD) {
      if (bp != nullptr) bv = (float)bp[o < Co ? o : Co - 1];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = wr * 64 + i * 16 + 4 * g + r;
        float Pl[T], ul[T];
#pragma unroll
        for (int p = 0; p < T; ++p) Pl[p] = acc[p][i][j][r];
        if constexpr (GAUSS) {
          constexpr int re = Bn::re(1), im = Bn::im(1);
          const float a1 = acc[re][i][j][r], a2 = acc[im][i][j][r], a3 = acc[T][i][j][r];
          Pl[re] = BWD ? a1 + a2 : a1 - a3;
          Pl[im] = BWD ? a1 - a3 : a1 + a2;
        }
        // a constant added to every group position is T times it added to bin 0
        Pl[0] = __builtin_fmaf((float)T, bv, Pl[0]);
        irdft<T>(Pl, ul);
        const uint32_t off = (row < len && o < Co) ? (uint32_t)((row * Co + o) * T * EB) : kDropOffset;
        store_run_rsrc<DT, T>(ors, off, ul);
      }
  }
}

}  // namespace eqk
