// eql_bwd_fused.h -- single-pass backward of the C_T equivariant linear layer
// for gfx950: input, weight and bias gradients from one read of x and dy.
//
// The paper runs every stage of the layer as one GEMM-like dataflow so that
// no intermediate makes a round trip through global memory (Sec. 3.5), and
// computes the gradients in the Fourier basis of the forward pass (Appendix
// A.2, "Forward and backward passes").  Here one workgroup of 8 waves holds the whole
// weight-gradient tile of the layer (BC >= Cin input x BO >= Cout output
// channels, every plane) for one split of the rows, so each row of x and dy
// is loaded and transformed once and feeds all three gradients.  Per chunk of
// KR rows:
//
//   staging  the raw x and dy of the chunk are transformed (packed fp16 pairs
//            of rows, or fp32) and their planes written to LDS: x planes
//            [p][c][row] and dy planes [p][o][row] with the row index
//            contiguous (the weight gradient contracts over rows), and a
//            second copy of the dy planes [step][p][row][o] with the output
//            channel contiguous (the input gradient contracts over output
//            channels, KR of them per step);
//   dW       H_k[c,o] += sum_n conj(Xhat_k[n,c]) dYhat_k[n,o], as in
//            eql_wgrad_kernel: wave (wc, wo) of a WGC x WGO grid owns CT x OTW
//            blocks of 16 x 16 channels;
//   dX       dXhat_k[n,c] = sum_o dYhat_k[n,o] conj(What_k[o,c]) on tiles of
//            16 rows x 16 input channels, dealt round-robin to the waves, with
//            the weight spectrum (backward layout) resident in LDS for the
//            whole kernel; the inverse transform runs in registers and dx is
//            written once;
//   db       bin 0 of dy, summed per output channel.
//
// The fp32 weight-gradient partial of the split goes to
// part[split][p][c/4][o][c%4] and the bias partial to dbpart[split][o], the
// layout that eql_wgrad_reduce_kernel sums in a fixed order.
//
// The whole tile in one workgroup is what bounds this kernel's reach: the
// accumulators (BC * BO * T fp32 over 512 lanes) must fit the registers, and
// each split writes one BC x BO x T partial, so the pass pays off where the
// rows per split dwarf the tile (the host decides).
#pragma once
#include "eql_launch.h"
#include "eql_wgrad.h"

namespace eqk {

template <int T, int DT, int WGC, int CT, int OTW>
__global__ __launch_bounds__(512) void eql_bwd_fused_kernel(
    const void* __restrict__ x, const void* __restrict__ dy, const void* __restrict__ wsp,
    void* __restrict__ dx, float* __restrict__ part, float* __restrict__ dbpart, int64_t N, int Cin,
    int Cout, int64_t rows_per_split, int n_splits, int CinB, int CoutB, int nks, int dbuf) {
  // fp32 and fp16 (bf16 layers take the two-pass backward)
  static_assert(DT != kBF16, "single-pass backward: fp32 or fp16");
  constexpr bool F16 = DT == kF16;
  using Bn = Bins<T>;
  constexpr int WGO = 8 / WGC;
  constexpr int EB = F16 ? 2 : 4;
  constexpr int KW = F16 ? 8 : 4;            // contraction values per lane and fragment
  constexpr int KR = 4 * KW;                 // rows per chunk = output channels per dX step
  constexpr int FB = KW * EB;                // 16 bytes
  constexpr int RB = KR * EB;                // 64 bytes
  static_assert(RB == kFusedRowBytes, "staging row");
  using FR = Frag<FB>;
  constexpr int BC = WGC * 16 * CT;
  constexpr int BO = WGO * 16 * OTW;
  static_assert((KR / 2) % 8 == 0 && BC % 8 == 0 && BO % 8 == 0, "wgrad_item tiling");
  constexpr int NIX = BC * KR / 2;           // (channel, row pair) items of x per chunk
  constexpr int NID = BO * KR / 2;
  constexpr int UX = (NIX + 511) / 512;
  constexpr int UD = (NID + 511) / 512;
  constexpr int WPR = (T * EB + 3) / 4;      // words of one (row, channel)
  constexpr int RAW = 2 * WPR;               // words of one item (two rows)
  constexpr int XSB = T * BC * RB, DSB = T * BO * RB;
  constexpr int RT = KR / 16;                // 16-row tiles per chunk

  // dynamic LDS: one or two staging buffers [xs | ds | dr], then the weights
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int C16 = (Cin + 15) & ~15;
  const int DRB = nks * T * KR * RB;
  const int STG = XSB + DSB + DRB;
  char* const wl = smem + (dbuf ? 2 : 1) * STG;
  float* const dred = reinterpret_cast<float*>(smem);

  const int split = blockIdx.x;
  if (split >= n_splits) return;
  const int64_t n_begin = (int64_t)split * rows_per_split;
  const int64_t n_end = (n_begin + rows_per_split < N) ? n_begin + rows_per_split : N;
  const int64_t len = n_end - n_begin;
  const int nchunks = (int)((len + KR - 1) / KR);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4;
  const int li = lane & 15;
  const int wc = wave / WGO;
  const int wo = wave - wc * WGO;

  // rows of this split as buffer ranges: bytes past the split read as zero,
  // stores past it are dropped
  const int rowx = Cin * T * EB, rowd = Cout * T * EB;
  const __amdgpu_buffer_rsrc_t xrs =
      make_rsrc(reinterpret_cast<const char*>(x) + n_begin * rowx, (uint32_t)(len * rowx));
  const __amdgpu_buffer_rsrc_t drs =
      make_rsrc(reinterpret_cast<const char*>(dy) + n_begin * rowd, (uint32_t)(len * rowd));
  const __amdgpu_buffer_rsrc_t dxrs =
      make_rsrc(reinterpret_cast<char*>(dx) + n_begin * rowx, (uint32_t)(len * rowx));
  constexpr int ITB = T * EB;  // bytes of one (row, channel)

  // ---- weight spectrum, backward layout B[p][c][o] ([T][CinB][CoutB]), into
  // LDS once: block (step s, plane p) holds rows c < C16 of the KR output
  // channels of step s, wl[(s*T + p)][c][KR], rows swizzled as the staging.
  {
    const char* wb = reinterpret_cast<const char*>(wsp);
    constexpr int UPR = RB / 16;  // 16-byte units per row
    const int units = nks * T * C16 * UPR;
    for (int u0 = tid; u0 < units; u0 += 4 * 512) {
      u32x4 v[4];
      int lo[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int u = u0 + 512 * j;
        lo[j] = -1;
        if (u < units) {
          const int chk = u % UPR;
          const int rest = u / UPR;
          const int c = rest % C16;
          const int sp = rest / C16;  // s * T + p
          const int p = sp % T, s = sp / T;
          v[j] = *reinterpret_cast<const u32x4*>(wb + ((int64_t)(p * CinB + c) * CoutB + s * KR) * EB + chk * 16);
          lo[j] = sp * C16 * RB + wl_off<RB>(c, chk * 16);
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (lo[j] >= 0) *reinterpret_cast<u32x4*>(wl + lo[j]) = v[j];
    }
  }

  // Raw rows of one chunk.  Every thread issues the same loads on every call
  // (items past the tile or the layer's channels, and rows past the split,
  // read from offsets beyond the buffer range and come back zero), so the
  // compiler's memory-counter waits stay exact across the loop.
  // NSET register sets: chunk c is loaded into set c % NSET, NSET chunks
  // ahead of its transform, so NSET chunks of loads are in flight per thread.
  constexpr int NSET = 2;
  uint32_t rx[NSET][UX][RAW], rd[NSET][UD][RAW];
  auto issue = [&](auto set, int chunk) __attribute__((always_inline)) {
    constexpr int R = decltype(set)::value;
    const int n0 = chunk * KR;  // row offset within the split
#pragma unroll
    for (int u = 0; u < UX; ++u) {
      const int item = tid + 512 * u;
      int c, rp;
      wgrad_item<BC>(item, c, rp);
      const bool ok = (NIX % 512 == 0 || item < NIX) && c < Cin;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        uint32_t w[WPR];
        const uint32_t off = ok ? (uint32_t)(((int64_t)(n0 + 2 * rp + h) * Cin + c) * ITB) : kDropOffset;
        load_row<T, EB>(xrs, off, w);
#pragma unroll
        for (int q = 0; q < WPR; ++q) rx[R][u][h * WPR + q] = w[q];
      }
    }
#pragma unroll
    for (int u = 0; u < UD; ++u) {
      const int item = tid + 512 * u;
      int o, rp;
      wgrad_item<BO>(item, o, rp);
      const bool ok = (NID % 512 == 0 || item < NID) && o < Cout;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        uint32_t w[WPR];
        const uint32_t off = ok ? (uint32_t)(((int64_t)(n0 + 2 * rp + h) * Cout + o) * ITB) : kDropOffset;
        load_row<T, EB>(drs, off, w);
#pragma unroll
        for (int q = 0; q < WPR; ++q) rd[R][u][h * WPR + q] = w[q];
      }
    }
  };

  float dbacc[UD];
#pragma unroll
  for (int u = 0; u < UD; ++u) dbacc[u] = 0.0f;

  const int n_dr = nks * KR;  // output channels of the input-gradient staging
  auto publish = [&](auto set, int buf) __attribute__((always_inline)) {
    constexpr int R = decltype(set)::value;
    char* const xs = smem + buf * STG;
    char* const ds = xs + XSB;
    char* const dr = ds + DSB;
#pragma unroll
    for (int u = 0; u < UX; ++u) {
      const int item = tid + 512 * u;
      if (NIX % 512 != 0 && item >= NIX) continue;
      int c, rp;
      wgrad_item<BC>(item, c, rp);
      if constexpr (F16) {
        half2v P[T];
        transform_pair<T>(rx[R][u], P);
#pragma unroll
        for (int p = 0; p < T; ++p)
          *reinterpret_cast<uint32_t*>(&xs[p * BC * RB + wl_off<RB>(c, rp * 2 * EB)]) = __builtin_bit_cast(uint32_t, P[p]);
      } else {
        float P0[T], P1[T];
        transform_rows<T>(rx[R][u], P0, P1);
#pragma unroll
        for (int p = 0; p < T; ++p)
          *reinterpret_cast<u32x2*>(&xs[p * BC * RB + wl_off<RB>(c, rp * 2 * EB)]) =
              u32x2{__builtin_bit_cast(uint32_t, P0[p]), __builtin_bit_cast(uint32_t, P1[p])};
      }
    }
#pragma unroll
    for (int u = 0; u < UD; ++u) {
      const int item = tid + 512 * u;
      if (NID % 512 != 0 && item >= NID) continue;
      int o, rp;
      wgrad_item<BO>(item, o, rp);
      const bool to_dr = o < n_dr;
      const int s = o / KR;
      const int ob = (o - s * KR) * EB;  // byte of o within its step's row
      char* const drs_base = dr + s * T * KR * RB;
      if constexpr (F16) {
        half2v P[T];
        transform_pair<T>(rd[R][u], P);
        dbacc[u] = __builtin_amdgcn_fdot2(P[0], half2v{(_Float16)1.0f, (_Float16)1.0f}, dbacc[u], false);
#pragma unroll
        for (int p = 0; p < T; ++p) {
          const uint32_t wv = __builtin_bit_cast(uint32_t, P[p]);
          *reinterpret_cast<uint32_t*>(&ds[p * BO * RB + wl_off<RB>(o, rp * 2 * EB)]) = wv;
          if (to_dr) {
            char* const blk = drs_base + p * KR * RB;
            *reinterpret_cast<uint16_t*>(&blk[wl_off<RB>(2 * rp, ob)]) = (uint16_t)(wv & 0xffffu);
            *reinterpret_cast<uint16_t*>(&blk[wl_off<RB>(2 * rp + 1, ob)]) = (uint16_t)(wv >> 16);
          }
        }
      } else {
        float P0[T], P1[T];
        transform_rows<T>(rd[R][u], P0, P1);
        dbacc[u] += P0[0] + P1[0];
#pragma unroll
        for (int p = 0; p < T; ++p) {
          const uint32_t w0 = __builtin_bit_cast(uint32_t, P0[p]);
          const uint32_t w1 = __builtin_bit_cast(uint32_t, P1[p]);
          *reinterpret_cast<u32x2*>(&ds[p * BO * RB + wl_off<RB>(o, rp * 2 * EB)]) = u32x2{w0, w1};
          if (to_dr) {
            char* const blk = drs_base + p * KR * RB;
            *reinterpret_cast<uint32_t*>(&blk[wl_off<RB>(2 * rp, ob)]) = w0;
            *reinterpret_cast<uint32_t*>(&blk[wl_off<RB>(2 * rp + 1, ob)]) = w1;
          }
        }
      }
    }
  };

  floatx4 acc[T][CT][OTW];
#pragma unroll
  for (int p = 0; p < T; ++p)
#pragma unroll
    for (int a = 0; a < CT; ++a)
#pragma unroll
      for (int b = 0; b < OTW; ++b) acc[p][a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  // weight gradient of one staged chunk: D[c][o] = sum_n A[c][n] B[n][o]
  auto mma_chunk = [&](int buf) __attribute__((always_inline)) {
    const char* const xs = smem + buf * STG;
    const char* const ds = xs + XSB;
#pragma unroll
    for (int b = 0; b < OTW; ++b) {
      const int ol = (wo * OTW + b) * 16 + li;
      FR Bf[T];
#pragma unroll
      for (int p = 0; p < T; ++p) Bf[p] = lds_frag<FB, RB>(&ds[p * BO * RB], ol, g);
#pragma unroll
      for (int a = 0; a < CT; ++a) {
        const int cl = (wc * CT + a) * 16 + li;
        FR A[T];
#pragma unroll
        for (int p = 0; p < T; ++p) A[p] = lds_frag<FB, RB>(&xs[p * BC * RB], cl, g);
        frag_mma<DT, KW>(acc[0][a][b], A[0], Bf[0]);
        if constexpr (Bn::kEven) frag_mma<DT, KW>(acc[1][a][b], A[1], Bf[1]);
        static_for<Bn::K>([&](auto ki) {
          constexpr int k = decltype(ki)::value + 1;
          constexpr int r = Bn::re(k);
          constexpr int i = Bn::im(k);
          frag_mma<DT, KW>(acc[r][a][b], A[r], Bf[r]);
          frag_mma<DT, KW>(acc[i][a][b], A[r], Bf[i]);
          frag_mma<DT, KW>(acc[r][a][b], A[i], Bf[i]);
          frag_mma<DT, KW>(acc[i][a][b], frag_neg<DT, FB>(A[i]), Bf[r]);
        });
      }
    }
  };

  // input gradient of one staged chunk: D[n][c] = sum_o dYhat[n][o] conj(What[o][c])
  //   Re += Dr Wr + Di Wi,   Im += Di Wr + (-Dr) Wi
  // on tiles of 16 rows x 16 input channels, one per wave (RT * C16 / 16 <= 8
  // tiles per chunk).  Lane (g, i) of a tile ends with input channel i of rows
  // 4g .. 4g+3 in every plane; the inverse transforms go to registers
  // (dxv, dxoff) and dx_store writes them later, the 16 lanes of a lane group
  // storing 16 consecutive channels of one row (16*T contiguous elements).
  // Every wave issues the same stores on every chunk (a wave without a tile,
  // rows past the split and channels past Cin store to an offset beyond the
  // buffer range, which writes nothing), so the stores never make the
  // counter waits of the next chunk's loads inexact.
  static_assert(RT * BC / 16 <= 8, "one input-gradient tile per wave");
  const int n_tiles = RT * (C16 / 16);
  float dxv[4][T];
  uint32_t dxoff[4];
  auto dx_compute = [&](int buf, int chunk) __attribute__((always_inline)) {
    const char* const dr = smem + buf * STG + XSB + DSB;
    const bool has_tile = wave < n_tiles;  // uniform across the wave
    const int rt = wave % RT;
    const int cti = wave / RT;
    const int c = cti * 16 + li;
    if (has_tile) {
      floatx4 ax[T];
#pragma unroll
      for (int p = 0; p < T; ++p) ax[p] = floatx4{0.f, 0.f, 0.f, 0.f};
      for (int s = 0; s < nks; ++s) {
        // operands one bin at a time (at most four fragments live)
        const char* const ab = dr + s * T * KR * RB;
        const char* const wb = wl + s * T * C16 * RB;
        auto A = [&](int p) __attribute__((always_inline)) { return lds_frag<FB, RB>(ab + p * KR * RB, rt * 16 + li, g); };
        auto W = [&](int p) __attribute__((always_inline)) { return lds_frag<FB, RB>(wb + p * C16 * RB, cti * 16 + li, g); };
        frag_mma<DT, KW>(ax[0], A(0), W(0));
        if constexpr (Bn::kEven) frag_mma<DT, KW>(ax[1], A(1), W(1));
        static_for<Bn::K>([&](auto ki) {
          constexpr int k = decltype(ki)::value + 1;
          constexpr int r = Bn::re(k);
          constexpr int i = Bn::im(k);
          const FR ar = A(r), ai = A(i), wr = W(r), wi = W(i);
          frag_mma<DT, KW>(ax[r], ar, wr);
          frag_mma<DT, KW>(ax[i], ai, wr);
          frag_mma<DT, KW>(ax[r], ai, wi);
          frag_mma<DT, KW>(ax[i], frag_neg<DT, FB>(ar), wi);
        });
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float Pl[T];
#pragma unroll
        for (int p = 0; p < T; ++p) Pl[p] = ax[p][q];
        irdft<T>(Pl, dxv[q]);
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t n = (int64_t)chunk * KR + rt * 16 + 4 * g + q;  // row within the split
      dxoff[q] = (has_tile && n < len && c < Cin) ? (uint32_t)((n * Cin + c) * ITB) : kDropOffset;
    }
  };
  auto dx_store = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < 4; ++q) store_run_rsrc<DT, T>(dxrs, dxoff[q], dxv[q]);
  };
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    dxoff[q] = kDropOffset;
#pragma unroll
    for (int t = 0; t < T; ++t) dxv[q][t] = 0.0f;
  }

  // Chunk loop, unrolled by NSET so that each chunk's register set is a
  // compile-time index.  The loads of chunk ch+NSET are issued while chunk ch
  // is computed; each wave's waits for a chunk's loads come before its dx
  // stores of the current chunk are issued.
  if (dbuf) {
    // chunk ch staged in buffer ch & 1; one barrier per chunk:
    //   barrier; MFMAs of ch (both gradients); transform chunk ch+1 into the
    //   other buffer; dx stores of ch; loads of chunk ch+1+NSET.  (Splitting
    //   the waves of a SIMD into transform-first and multiply-first, as the
    //   weight-gradient kernel does, measured slower here: 138 against 121 us
    //   on Swin stage 1.)
    auto step = [&](auto set, int ch) __attribute__((always_inline)) {
      using Q = std::integral_constant<int, (decltype(set)::value + 1) % NSET>;  // set of chunk ch+1
      const int b = ch & 1;
      __syncthreads();  // chunk ch staged (and the weights at ch = 0); chunk ch-1 finished
      mma_chunk(b);
      dx_compute(b, ch);
      publish(Q{}, b ^ 1);  // chunk ch+1 (zeros past the end)
      dx_store();
      issue(Q{}, ch + 1 + NSET);
    };
    static_for<NSET>([&](auto si) { issue(si, decltype(si)::value); });
    publish(std::integral_constant<int, 0>{}, 0);
    issue(std::integral_constant<int, 0>{}, NSET);
    for (int ch = 0; ch < nchunks; ch += NSET) {
      bool done = false;
      static_for<NSET>([&](auto si) {
        if (!done) {
          if (ch + decltype(si)::value >= nchunks) done = true;
          else step(si, ch + decltype(si)::value);
        }
      });
      if (done) break;
    }
  } else {
    //   transform chunk ch; barrier; dx stores of ch-1; loads of chunk
    //   ch+NSET; MFMAs of ch; barrier
    auto step = [&](auto set, int ch) __attribute__((always_inline)) {
      publish(set, 0);
      __syncthreads();   // spectra of chunk ch (and the weights) visible
      dx_store();        // chunk ch-1 (nothing at ch = 0)
      issue(set, ch + NSET);
      mma_chunk(0);
      dx_compute(0, ch);
      __syncthreads();   // staging free for the next chunk
    };
    static_for<NSET>([&](auto si) { issue(si, decltype(si)::value); });
    for (int ch = 0; ch < nchunks; ch += NSET) {
      bool done = false;
      static_for<NSET>([&](auto si) {
        if (!done) {
          if (ch + decltype(si)::value >= nchunks) done = true;
          else step(si, ch + decltype(si)::value);
        }
      });
      if (done) break;
    }
    dx_store();
  }

  // ---- weight-gradient partial: part[split][p][c/4][o][c%4] (padded extents BC, BO)
  constexpr int CQ = BC / 4;
#pragma unroll
  for (int a = 0; a < CT; ++a) {
    const int cq = ((wc * CT + a) * 16) / 4 + g;
#pragma unroll
    for (int b = 0; b < OTW; ++b) {
      const int oo = (wo * OTW + b) * 16 + li;
#pragma unroll
      for (int p = 0; p < T; ++p) {
        float* dst = part + ((((int64_t)split * T + p) * CQ + cq) * BO + oo) * 4;
        *reinterpret_cast<floatx4*>(dst) = acc[p][a][b];
      }
    }
  }
  if (dbpart != nullptr) {
    // thread q's dbacc[u] belongs to output channel o of item q + 512u
    // (wgrad_item); thread t < BO sums, in a fixed order, the entries of o = t
    float dsum = 0.0f;
#pragma unroll
    for (int u = 0; u < UD; ++u) {
      __syncthreads();
      dred[tid] = dbacc[u];
      __syncthreads();
      if (tid < BO) {
        for (int w = 0; w < 8; ++w) {
          if ((w + 8 * u) % (BO / 8) != (tid >> 3)) continue;
          for (int rl = 0; rl < 8; ++rl) {
            const int q = w * 64 + rl * 8 + (tid & 7);
            if (NID % 512 == 0 || q + 512 * u < NID) dsum += dred[q];
          }
        }
      }
    }
    if (tid < BO) dbpart[(int64_t)split * BO + tid] = dsum;
  }
}

}  // namespace eqk
