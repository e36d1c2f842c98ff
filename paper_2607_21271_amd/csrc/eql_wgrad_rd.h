// eql_wgrad_rd.h -- weight- and bias-gradient kernel with register-direct
// operands, for gfx950.
//
//   H_k[c,o]  = sum_n conj(Xhat_k[n,c]) dYhat_k[n,o]          (one split of rows)
//   db[o]     = sum_n dYhat_0[n,o]
// (Appendix A.2 "Forward and backward passes"; the inverse transform to dw and
// the sum over splits run in eql_wgrad_reduce_kernel.)
//
// The MFMA contracts over rows: D[c][o] = sum_n A[c][n] B[n][o], and the
// operand a lane holds is one channel over KR/4 consecutive rows (fp16:
// v_mfma_f32_16x16x32_f16, lane (i, g) holds rows 8g..8g+7 of channel i; fp32:
// four v_mfma_f32_16x16x4f32 per 16 rows, lane (i, g) holds rows 4g..4g+3).
// In the [N, C, T] layout the T group elements of one (row, channel) are
// contiguous, so a lane loads exactly the elements of its operand (one run of
// T elements per row), transforms each row along the group axis in registers
// and has the T operand planes without any exchange through LDS:
//   fp16: rows (2m, 2m+1) are transformed together in packed fp16 arithmetic
//         (transform_pair), so plane p of the pair is already the packed
//         operand word (row 2m low, row 2m+1 high);
//   fp32: one transform per row, plane p of row 4g+s feeding MFMA s.
//
// Work split.  A workgroup of NW waves owns one tile of CT x OT blocks of
// 16 x 16 channels for one split of rows; its waves take the split's chunks
// of KR rows in turn (wave w: chunks w, w + NW, ...), each accumulating the
// whole tile, and add their tiles through LDS in a fixed order at the end.
// So the transforms are not repeated inside a workgroup, no barrier runs in
// the main loop, and the number of splits -- the fp32 partial spectra written
// and read back once -- stays small: the host sizes the grid to one
// workgroup per CU.  The raw rows of a wave's next chunk are loaded while the
// current chunk is transformed and multiplied.
//
// Complex bin (r, i):  Re H += Xr Dr + Xi Di,   Im H += Xr Di + (-Xi) Dr.
#pragma once
#include "eql_common.h"
#include "eql_gemm.h"
#include "eql_wgrad.h"

namespace eqk {

template <int T, int DT, int CT, int OT>
struct RdShape {
  static constexpr bool W16 = DT != kF32;
  static constexpr int EB = W16 ? 2 : 4;
  static constexpr int KR = W16 ? 32 : 16;        // rows per chunk
  static constexpr int RPL = KR / 4;              // rows per lane
  static constexpr int WPR = (T * EB + 3) / 4;    // raw words of one (row, channel)
  static constexpr int RAW = RPL * WPR;           // raw words of one block per lane
  static constexpr int OPW = 4;                   // operand words per plane per lane
  static constexpr int BLK = CT + OT;             // blocks loaded per chunk
  static constexpr int BC = 16 * CT, BO = 16 * OT;
};

// Accumulator bytes a wave hands to LDS at the end: one floatx4 per lane for
// every (plane, c-block, o-block).
template <int T, int CT, int OT>
constexpr int rd_wave_acc_bytes() { return T * CT * OT * 64 * 16; }

template <int T, int DT, int CT, int OT, int NW>
__global__ __launch_bounds__(64 * NW) void eql_wgrad_rd_kernel(
    const void* __restrict__ x, const void* __restrict__ dy, float* __restrict__ part,
    float* __restrict__ dbpart, int64_t N, int Cin, int Cout, int64_t rows_per_split, int n_ct,
    int n_ot, int n_splits, int Cin_pad, int Cout_pad) {
  constexpr bool F16 = DT == kF16;
  constexpr bool W16 = DT != kF32;
  using S = RdShape<T, DT, CT, OT>;
  using Bn = Bins<T>;
  constexpr int EB = S::EB, KR = S::KR, RPL = S::RPL, WPR = S::WPR, RAW = S::RAW;
  constexpr int ITB = T * EB;  // bytes of one (row, channel)

  // Workgroup w of the ones in use; the hardware deals consecutive workgroup
  // ids to the 8 XCDs in turn, so w = (id % 8) * Q + id / 8 gives each XCD a
  // contiguous range of w: the tiles of one split (which read the same rows)
  // mostly share an L2.
  const int tiles = n_ct * n_ot;
  const int G = n_splits * tiles;
  const int Q = (G + 7) / 8;
  const int w = (int)(blockIdx.x & 7) * Q + (int)(blockIdx.x >> 3);
  if (w >= G) return;
  const int split = w / tiles;
  const int tile = w - split * tiles;
  const int ct = tile / n_ot;
  const int ot = tile - ct * n_ot;
  const int64_t n_begin = (int64_t)split * rows_per_split;
  const int64_t n_end = (n_begin + rows_per_split < N) ? n_begin + rows_per_split : N;
  const int nchunks = (int)((n_end - n_begin + KR - 1) / KR);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4;
  const int li = lane & 15;

  const int rowx = Cin * ITB, rowd = Cout * ITB;
  const __amdgpu_buffer_rsrc_t xrs =
      make_rsrc(reinterpret_cast<const char*>(x) + n_begin * rowx, (uint32_t)((n_end - n_begin) * rowx));
  const __amdgpu_buffer_rsrc_t drs =
      make_rsrc(reinterpret_cast<const char*>(dy) + n_begin * rowd, (uint32_t)((n_end - n_begin) * rowd));

  // Per-lane byte offsets of row 0 of the lane's rows in chunk 0, one per
  // block.  A channel past the tensor (tile padding) reads the last channel
  // instead: its sums land only in padded rows or columns of the partial,
  // which the reduction never reads.
  uint32_t boff[S::BLK];
#pragma unroll
  for (int a = 0; a < CT; ++a) {
    const int c = min(ct * S::BC + 16 * a + li, Cin - 1);
    boff[a] = (uint32_t)(((int64_t)RPL * g * Cin + c) * ITB);
  }
#pragma unroll
  for (int b = 0; b < OT; ++b) {
    const int o = min(ot * S::BO + 16 * b + li, Cout - 1);
    boff[CT + b] = (uint32_t)(((int64_t)RPL * g * Cout + o) * ITB);
  }

  // raw words of one chunk: [block][row][word].  A block's loads go out as
  // soon as its previous contents are transformed, so they are in flight
  // during the rest of the chunk; loads of chunks past the split (the wave's
  // last prefetch) read zero, and no branch skips a load, so the compiler's
  // memory-counter waits stay exact.
  uint32_t raw[S::BLK][RAW];
  auto issue_block = [&](int bl, int chunk) __attribute__((always_inline)) {
    const bool isx = bl < CT;
    const __amdgpu_buffer_rsrc_t rs = isx ? xrs : drs;
    const uint32_t rstride = (uint32_t)(isx ? rowx : rowd);
    // rows past the split (the resource's end) read as zero; the host keeps
    // every offset below 2^31
    const uint32_t base = boff[bl] + (uint32_t)(chunk * KR) * rstride;
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
      uint32_t wds[WPR];
      load_row<T, EB>(rs, base + (uint32_t)i * rstride, wds);
#pragma unroll
      for (int q = 0; q < WPR; ++q) raw[bl][i * WPR + q] = wds[q];
    }
  };

  // operand planes: fp16 [block][plane] 4 packed words (8 rows); fp32
  // [block][plane] 4 floats (rows 4g..4g+3, one per MFMA)
  floatx4 acc[T][CT][OT];
#pragma unroll
  for (int p = 0; p < T; ++p)
#pragma unroll
    for (int a = 0; a < CT; ++a)
#pragma unroll
      for (int b = 0; b < OT; ++b) acc[p][a][b] = floatx4{0.f, 0.f, 0.f, 0.f};
  float dbacc[OT];
#pragma unroll
  for (int b = 0; b < OT; ++b) dbacc[b] = 0.0f;

  // Transform one block of the chunk into its T operand planes.  bf16: fp32
  // transforms, each plane value rounded once; the block's fp32 bin 0 is
  // added to dbs (output-gradient blocks pass their bias sum, others a dummy).
  auto transform = [&](int bl, u32x4 (&op)[T], float& dbs) __attribute__((always_inline)) {
    if constexpr (DT == kBF16) {
#pragma unroll
      for (int m = 0; m < RPL / 2; ++m) {
        uint32_t two[2 * WPR];
#pragma unroll
        for (int q = 0; q < 2 * WPR; ++q) two[q] = raw[bl][2 * m * WPR + q];
        float P0[T], P1[T];
        transform_pair_f32<T>(two, P0, P1);
        dbs += P0[0] + P1[0];
#pragma unroll
        for (int p = 0; p < T; ++p) op[p][m] = pack2<DT>(P0[p], P1[p]);
      }
    } else if constexpr (F16) {
#pragma unroll
      for (int m = 0; m < RPL / 2; ++m) {
        uint32_t two[2 * WPR];
#pragma unroll
        for (int q = 0; q < 2 * WPR; ++q) two[q] = raw[bl][2 * m * WPR + q];
        half2v P[T];
        transform_pair<T>(two, P);
#pragma unroll
        for (int p = 0; p < T; ++p) op[p][m] = __builtin_bit_cast(uint32_t, P[p]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < RPL; ++i) {
        float v[T], P[T];
#pragma unroll
        for (int t = 0; t < T; ++t) v[t] = __builtin_bit_cast(float, raw[bl][i * WPR + t]);
        rdft<T>(v, P);
#pragma unroll
        for (int p = 0; p < T; ++p) op[p][i] = __builtin_bit_cast(uint32_t, P[p]);
      }
    }
  };
  auto mma = [&](floatx4& d, const u32x4& A, const u32x4& B) __attribute__((always_inline)) {
    if constexpr (F16) {
      d = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8, A),
                                                 __builtin_bit_cast(half8, B), d, 0, 0, 0);
    } else if constexpr (DT == kBF16) {
      typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
      d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, A),
                                                  __builtin_bit_cast(bf16x8, B), d, 0, 0, 0);
    } else {
      // (elements copied to scalars first: __builtin_bit_cast of a vector
      // element expression read element 0 whatever the index)
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const uint32_t as = A[s], bs = B[s];
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(__builtin_bit_cast(float, as),
                                                 __builtin_bit_cast(float, bs), d, 0, 0, 0);
      }
    }
  };

  // One chunk: the output-gradient blocks are transformed first and stay live;
  // then each activation block is transformed and multiplied with all of them.
  // Each block's loads for the wave's next chunk go out right after its
  // transform, so they are in flight during the rest of this chunk.
  auto compute = [&](int next_chunk) __attribute__((always_inline)) {
    u32x4 opd[OT][T];
#pragma unroll
    for (int b = 0; b < OT; ++b) {
      transform(CT + b, opd[b], dbacc[b]);
      issue_block(CT + b, next_chunk);
      // keep the loads here: sunk below the MFMAs they would leave only the
      // MFMA time to cover their latency
      __builtin_amdgcn_sched_barrier(0);
      // bias gradient: bin 0 of the output-gradient rows (bf16: summed in the
      // transform, from fp32)
      // (vector elements are copied to scalars before a bit cast, see mma)
      if constexpr (DT != kBF16) {
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const uint32_t w0 = opd[b][0][m];
          if constexpr (F16)
            dbacc[b] = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2v, w0),
                                              half2v{(_Float16)1.0f, (_Float16)1.0f}, dbacc[b], false);
          else
            dbacc[b] += __builtin_bit_cast(float, w0);
        }
      }
    }
    constexpr uint32_t kSign = W16 ? 0x80008000u : 0x80000000u;
#pragma unroll
    for (int a = 0; a < CT; ++a) {
      u32x4 X[T];
      float unused = 0.0f;  // activation blocks add nothing to the bias
      transform(a, X, unused);
      issue_block(a, next_chunk);
      __builtin_amdgcn_sched_barrier(0);
      // -Xi of every complex bin (sign bits)
      u32x4 xneg[Bn::K > 0 ? Bn::K : 1];
      static_for<Bn::K>([&](auto ki) {
        constexpr int k = decltype(ki)::value + 1;
        xneg[k - 1] = X[Bn::im(k)] ^ u32x4{kSign, kSign, kSign, kSign};
      });
#pragma unroll
      for (int b = 0; b < OT; ++b) {
        const u32x4* D = opd[b];
        mma(acc[0][a][b], X[0], D[0]);
        if constexpr (Bn::kEven) mma(acc[1][a][b], X[1], D[1]);
        static_for<Bn::K>([&](auto ki) {
          constexpr int k = decltype(ki)::value + 1;
          constexpr int re = Bn::re(k), im = Bn::im(k);
          mma(acc[re][a][b], X[re], D[re]);
          mma(acc[im][a][b], X[re], D[im]);
          mma(acc[re][a][b], X[im], D[im]);
          mma(acc[im][a][b], xneg[k - 1], D[re]);
        });
      }
    }
  };

  if (wave < nchunks) {
#pragma unroll
    for (int bl = 0; bl < S::BLK; ++bl) issue_block(bl, wave);
    for (int q = wave; q < nchunks; q += NW) compute(q + NW);
  }

  // ---- the waves' tiles added in wave order through LDS, then one partial
  // per workgroup: part[split][p][c/4][o][c%4]
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr int WAB = rd_wave_acc_bytes<T, CT, OT>();
  floatx4* const red = reinterpret_cast<floatx4*>(smem);
  if (wave > 0) {
#pragma unroll
    for (int p = 0; p < T; ++p)
#pragma unroll
      for (int a = 0; a < CT; ++a)
#pragma unroll
        for (int b = 0; b < OT; ++b)
          red[(wave - 1) * (WAB / 16) + ((p * CT + a) * OT + b) * 64 + lane] = acc[p][a][b];
  }
  // bias partial: the four lane groups of a wave, then the waves, in order
  float* const dred = reinterpret_cast<float*>(smem + (NW - 1) * WAB);
#pragma unroll
  for (int b = 0; b < OT; ++b) {
    float v = dbacc[b];
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    if (g == 0) dred[(wave * OT + b) * 16 + li] = v;
  }
  __syncthreads();
  if (wave != 0) return;
  for (int wv = 1; wv < NW; ++wv) {
#pragma unroll
    for (int p = 0; p < T; ++p)
#pragma unroll
      for (int a = 0; a < CT; ++a)
#pragma unroll
        for (int b = 0; b < OT; ++b) acc[p][a][b] += red[(wv - 1) * (WAB / 16) + ((p * CT + a) * OT + b) * 64 + lane];
  }
  const int CQ = Cin_pad / 4;
#pragma unroll
  for (int a = 0; a < CT; ++a) {
    const int cq = (ct * S::BC + 16 * a) / 4 + g;
#pragma unroll
    for (int b = 0; b < OT; ++b) {
      const int oo = ot * S::BO + 16 * b + li;
#pragma unroll
      for (int p = 0; p < T; ++p)
        *reinterpret_cast<floatx4*>(part + ((((int64_t)split * T + p) * CQ + cq) * Cout_pad + oo) * 4) =
            acc[p][a][b];
    }
  }
  if (ct == 0 && dbpart != nullptr && g == 0) {
#pragma unroll
    for (int b = 0; b < OT; ++b) {
      float s = 0.0f;
      for (int wv = 0; wv < NW; ++wv) s += dred[(wv * OT + b) * 16 + li];
      dbpart[(int64_t)split * Cout_pad + ot * S::BO + 16 * b + li] = s;
    }
  }
}

}  // namespace eqk
