// eql_wgrad.h -- weight- and bias-gradient kernels of the C_T equivariant
// linear layer for gfx950.
//
//   H_k[c,o]  = sum_n conj(Xhat_k[n,c]) dYhat_k[n,o]          (one split of rows)
//   dw[j,o,c] = (1/T) sum_{k=0}^{T-1} H_k[c,o] e^{+2 pi i k j/T}
//   db[o]     = sum_n dYhat_0[n,o] = sum_n sum_t dy[n,o,t]
// (the gradients with respect to the original parameters, Appendix A.2
// "Forward and backward passes").  Complex bin (r, i):
//   Re H += Xr Dr + Xi Di,   Im H += Xr Di + (-Xi) Dr.
//
// eql_wgrad_kernel: one workgroup of 8 waves (WGC x WGO grid) owns BC input x
// BO output channels, all T planes, for one split of rows.  Per chunk of KR
// rows the raw x and dy of the next chunk are loaded into registers while the
// MFMAs of the current chunk run; every (row, channel) is transformed once
// per workgroup and its planes staged in LDS with the row index contiguous
// (the MFMA contraction index), so D[c][o] = sum_n A[c][n] B[n][o].  The fp32
// partial goes to part[split][p][c/4][o][c%4] (each lane's four consecutive
// c form one 16-byte run, and the 16 lanes of a quarter write 256 contiguous
// bytes); tiles with ct == 0 also write the split's bias partial.
//
// eql_wgrad_reduce_kernel: fixed-order sum over splits, inverse transform over
// the planes, dw (and db) in the output dtype.
#pragma once
#include "eql_common.h"
#include "eql_gemm.h"

namespace eqk {

// The T elements of one (row, channel), EB bytes each, packed into words
// (element e in half e%2 of word e/2 for 16-bit data).  Every (row, channel)
// starts at a multiple of T*EB bytes, so the widest load width dividing T*EB
// is always aligned; it is fixed at compile time (one load shape per kernel).
template <int T, int EB>
__device__ __forceinline__ void load_row(__amdgpu_buffer_rsrc_t rs, uint32_t off,
                                         uint32_t (&w)[(T * EB + 3) / 4]) {
  constexpr int NB = T * EB;
  if constexpr (NB % 4 == 0) {
    constexpr int W = NB % 16 == 0 ? 16 : NB % 8 == 0 ? 8 : 4;
    load_raw<NB, W>(rs, off, 0, w);
  } else {
#pragma unroll
    for (int q = 0; q < (NB + 3) / 4; ++q) {
      const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(rs, off + 4 * q, 0, 0);
      const uint32_t hi = (4 * q + 2 < NB) ? __builtin_amdgcn_raw_buffer_load_b16(rs, off + 4 * q + 2, 0, 0) : 0u;
      w[q] = (lo & 0xffffu) | (hi << 16);
    }
  }
}

// Spectra of the two rows of one item.  fp16: element t of both rows in one
// packed register (row 0 low), transformed together in fp16 arithmetic, so
// plane p comes out as the staged word (row 0, row 1).  fp32: one transform
// per row.  Each row's element t sits in raw word t / 2 (fp16, half t % 2) or
// t (fp32) of its WPR words.
template <int T>
__device__ __forceinline__ void transform_pair(const uint32_t (&r)[2 * ((2 * T + 3) / 4)], half2v (&P)[T]) {
  constexpr int WPR = (2 * T + 3) / 4;
  half2v v[T];
  static_for<T>([&](auto ti) {
    constexpr int t = decltype(ti)::value;
    v[t] = pair_halves<t % 2, t % 2>(r[t / 2], r[WPR + t / 2]);
  });
  rdft<T, H2Ops>(v, P);
}
// bf16: both rows widened to fp32 (exact) and transformed in fp32; the
// caller rounds plane p of the two rows into one staged word.
template <int T>
__device__ __forceinline__ void transform_pair_f32(const uint32_t (&r)[2 * ((2 * T + 3) / 4)], float (&P0)[T],
                                                   float (&P1)[T]) {
  constexpr int WPR = (2 * T + 3) / 4;
  float v0[T], v1[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int sh = (t % 2) ? 0 : 16;  // half t % 2 of word t / 2 into the top 16 bits
    v0[t] = __builtin_bit_cast(float, (r[t / 2] << sh) & 0xffff0000u);
    v1[t] = __builtin_bit_cast(float, (r[WPR + t / 2] << sh) & 0xffff0000u);
  }
  rdft<T>(v0, P0);
  rdft<T>(v1, P1);
}
template <int T>
__device__ __forceinline__ void transform_rows(const uint32_t (&r)[2 * T], float (&P0)[T], float (&P1)[T]) {
  float v0[T], v1[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    v0[t] = __builtin_bit_cast(float, r[t]);
    v1[t] = __builtin_bit_cast(float, r[T + t]);
  }
  rdft<T>(v0, P0);
  rdft<T>(v1, P1);
}

// Item order of the staging threads: a wave takes 8 channels x 8 row pairs, so
// each of its loads covers 8 rows x 8 channels (whole 128-byte lines for
// 16-byte items) and its 64 LDS stores, with the chunk swizzle of wl_off, fall
// on 64 distinct banks.  B (channels in the tile) is a multiple of 8.
template <int B>
__device__ __forceinline__ void wgrad_item(int item, int& ch, int& rp) {
  const int lo = item & 63, hi = item >> 6;
  ch = (hi % (B / 8)) * 8 + (lo & 7);
  rp = (hi / (B / 8)) * 8 + (lo >> 3);
}

template <int T, int DT, int WGC, int WGO, int CT, int OTW>
__global__ __launch_bounds__(512) void eql_wgrad_kernel(const void* __restrict__ x,
                                                        const void* __restrict__ dy,
                                                        float* __restrict__ part,
                                                        float* __restrict__ dbpart, int64_t N,
                                                        int Cin, int Cout, int64_t rows_per_split,
                                                        int n_ct, int n_ot, int n_splits, int Cin_pad,
                                                        int Cout_pad) {
  using Bn = Bins<T>;
  constexpr bool W16 = DT != kF32;           // 16-bit elements (fp16 or bf16)
  constexpr int EB = W16 ? 2 : 4;
  constexpr int KW = W16 ? 8 : 4;            // rows per lane group per fragment
  constexpr int KR = 4 * KW;                 // rows per chunk (one MFMA contraction step)
  constexpr int FB = KW * EB;                // 16 bytes
  constexpr int RB = KR * EB;                // 64 bytes: one channel's chunk of rows
  using FR = Frag<FB>;
  static_assert(WGC * WGO == 8, "8 waves");
  constexpr int BC = WGC * 16 * CT;
  constexpr int BO = WGO * 16 * OTW;
  static_assert((KR / 2) % 8 == 0 && BC % 8 == 0 && BO % 8 == 0, "wgrad_item tiling");
  constexpr int NIX = BC * KR / 2;           // (channel, row pair) items of x per chunk
  constexpr int NID = BO * KR / 2;
  constexpr int UX = (NIX + 511) / 512;
  constexpr int UD = (NID + 511) / 512;
  constexpr int WPR = (T * EB + 3) / 4;      // words of one (row, channel)
  constexpr int RAW = 2 * WPR;               // words of one item (two rows)

  // Staging: spectra of one chunk, x planes [p][c][row] then dy planes
  // [p][o][row].  Double buffered when two copies fit in LDS (DB): then the
  // transform of chunk ch+1 and the MFMAs of chunk ch run between the same two
  // barriers, the two waves that share a SIMD in opposite order, so one's VALU
  // work overlaps the other's MFMAs.  The bias sums reuse the area afterwards.
  constexpr int XSB = T * BC * RB, DSB = T * BO * RB;
  constexpr bool DB = 2 * (XSB + DSB) <= 160 * 1024;
  constexpr int SMEM = (DB ? 2 : 1) * (XSB + DSB);
  static_assert(SMEM >= 512 * 4, "bias scratch");
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  float* const dred = reinterpret_cast<float*>(smem);

  // XCD-aware tile order: workgroup b runs on XCD b % 8, so the tiles of one
  // split (which all read the split's rows of x and dy) are given the same
  // b % 8 and consecutive b / 8; they then share one L2 and the rows are read
  // from HBM once.  The grid holds whole groups of 8 splits; workgroups past
  // the last split exit before any barrier.
  const int per_split = n_ct * n_ot;
  const int xcd = blockIdx.x & 7;
  const int j = blockIdx.x >> 3;
  const int split = (j / per_split) * 8 + xcd;
  if (split >= n_splits) return;
  const int rem = j - (j / per_split) * per_split;
  const int ct = rem / n_ot;
  const int ot = rem - ct * n_ot;
  const int64_t n_begin = (int64_t)split * rows_per_split;
  const int64_t n_end = (n_begin + rows_per_split < N) ? n_begin + rows_per_split : N;
  const int nchunks = (int)((n_end - n_begin + KR - 1) / KR);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int g = lane >> 4;
  const int li = lane & 15;
  const int wc = wave / WGO;
  const int wo = wave - wc * WGO;

  // rows of this split as buffer ranges: bytes past the split read as zero
  const int rowx = Cin * T * EB, rowd = Cout * T * EB;
  const __amdgpu_buffer_rsrc_t xrs =
      make_rsrc(reinterpret_cast<const char*>(x) + n_begin * rowx, (uint32_t)((n_end - n_begin) * rowx));
  const __amdgpu_buffer_rsrc_t drs =
      make_rsrc(reinterpret_cast<const char*>(dy) + n_begin * rowd, (uint32_t)((n_end - n_begin) * rowd));
  constexpr int ITB = T * EB;  // bytes of one (row, channel)

  uint32_t rx[UX][RAW], rd[UD][RAW];
  // item u of this thread: (channel, row pair) = wgrad_item(tid + 512 u)
  auto issue = [&](int chunk) __attribute__((always_inline)) {
    const int n0 = chunk * KR;  // row offset within the split
#pragma unroll
    for (int u = 0; u < UX; ++u) {
      const int item = tid + 512 * u;
      int c, rp;
      wgrad_item<BC>(item, c, rp);
      const int cg = ct * BC + c;
      if ((NIX % 512 == 0 || item < NIX) && cg < Cin) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          uint32_t w[WPR];
          load_row<T, EB>(xrs, (uint32_t)(((int64_t)(n0 + 2 * rp + h) * Cin + cg) * ITB), w);
#pragma unroll
          for (int q = 0; q < WPR; ++q) rx[u][h * WPR + q] = w[q];
        }
      } else {
#pragma unroll
        for (int q = 0; q < RAW; ++q) rx[u][q] = 0u;
      }
    }
#pragma unroll
    for (int u = 0; u < UD; ++u) {
      const int item = tid + 512 * u;
      int o, rp;
      wgrad_item<BO>(item, o, rp);
      const int og = ot * BO + o;
      if ((NID % 512 == 0 || item < NID) && og < Cout) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          uint32_t w[WPR];
          load_row<T, EB>(drs, (uint32_t)(((int64_t)(n0 + 2 * rp + h) * Cout + og) * ITB), w);
#pragma unroll
          for (int q = 0; q < WPR; ++q) rd[u][h * WPR + q] = w[q];
        }
      } else {
#pragma unroll
        for (int q = 0; q < RAW; ++q) rd[u][q] = 0u;
      }
    }
  };

  float dbacc[UD];
#pragma unroll
  for (int u = 0; u < UD; ++u) dbacc[u] = 0.0f;

  // transform the prefetched items and stage their planes (two rows each)
  auto publish = [&](int buf) __attribute__((always_inline)) {
    char* const xs = smem + buf * (XSB + DSB);
    char* const ds = xs + XSB;
#pragma unroll
    for (int u = 0; u < UX; ++u) {
      const int item = tid + 512 * u;
      if (NIX % 512 != 0 && item >= NIX) continue;
      int c, rp;
      wgrad_item<BC>(item, c, rp);
      if constexpr (DT == kF16) {
        half2v P[T];
        transform_pair<T>(rx[u], P);
#pragma unroll
        for (int p = 0; p < T; ++p)
          *reinterpret_cast<uint32_t*>(&xs[p * BC * RB + wl_off<RB>(c, rp * 2 * EB)]) = __builtin_bit_cast(uint32_t, P[p]);
      } else if constexpr (DT == kBF16) {
        float P0[T], P1[T];
        transform_pair_f32<T>(rx[u], P0, P1);
#pragma unroll
        for (int p = 0; p < T; ++p)
          *reinterpret_cast<uint32_t*>(&xs[p * BC * RB + wl_off<RB>(c, rp * 2 * EB)]) = pack2<DT>(P0[p], P1[p]);
      } else {
        float P0[T], P1[T];
        transform_rows<T>(rx[u], P0, P1);
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
      if constexpr (DT == kF16) {
        half2v P[T];
        transform_pair<T>(rd[u], P);
        // bin 0 of both rows, summed in fp32
        dbacc[u] = __builtin_amdgcn_fdot2(P[0], half2v{(_Float16)1.0f, (_Float16)1.0f}, dbacc[u], false);
#pragma unroll
        for (int p = 0; p < T; ++p)
          *reinterpret_cast<uint32_t*>(&ds[p * BO * RB + wl_off<RB>(o, rp * 2 * EB)]) = __builtin_bit_cast(uint32_t, P[p]);
      } else if constexpr (DT == kBF16) {
        float P0[T], P1[T];
        transform_pair_f32<T>(rd[u], P0, P1);
        dbacc[u] += P0[0] + P1[0];
#pragma unroll
        for (int p = 0; p < T; ++p)
          *reinterpret_cast<uint32_t*>(&ds[p * BO * RB + wl_off<RB>(o, rp * 2 * EB)]) = pack2<DT>(P0[p], P1[p]);
      } else {
        float P0[T], P1[T];
        transform_rows<T>(rd[u], P0, P1);
        dbacc[u] += P0[0] + P1[0];
#pragma unroll
        for (int p = 0; p < T; ++p)
          *reinterpret_cast<u32x2*>(&ds[p * BO * RB + wl_off<RB>(o, rp * 2 * EB)]) =
              u32x2{__builtin_bit_cast(uint32_t, P0[p]), __builtin_bit_cast(uint32_t, P1[p])};
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

  auto mma_chunk = [&](int buf) __attribute__((always_inline)) {
    const char* const xs = smem + buf * (XSB + DSB);
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

  if constexpr (DB) {
    // chunk ch staged in buffer ch & 1; raw loads run two chunks ahead of the MFMAs
    if (nchunks > 0) {
      issue(0);
      publish(0);
    }
    if (nchunks > 1) issue(1);
    const bool transform_first = wave < 4;
    for (int ch = 0; ch < nchunks; ++ch) {
      __syncthreads();  // chunk ch staged; every wave done with chunk ch-1's buffer
      const bool more = ch + 1 < nchunks;
      if (transform_first) {
        if (more) {
          publish((ch + 1) & 1);
          if (ch + 2 < nchunks) issue(ch + 2);
        }
        mma_chunk(ch & 1);
      } else {
        mma_chunk(ch & 1);
        if (more) {
          publish((ch + 1) & 1);
          if (ch + 2 < nchunks) issue(ch + 2);
        }
      }
    }
  } else {
    if (nchunks > 0) issue(0);
    for (int ch = 0; ch < nchunks; ++ch) {
      publish(0);
      __syncthreads();                       // spectra of chunk ch visible
      if (ch + 1 < nchunks) issue(ch + 1);   // in flight during the MFMAs
      mma_chunk(0);
      __syncthreads();                       // staging free for the next chunk
    }
  }

  // ---- partials: part[split][p][c/4][o][c%4]
  const int CQ = Cin_pad / 4;
#pragma unroll
  for (int a = 0; a < CT; ++a) {
    const int cq = (ct * BC + (wc * CT + a) * 16) / 4 + g;
#pragma unroll
    for (int b = 0; b < OTW; ++b) {
      const int oo = ot * BO + (wo * OTW + b) * 16 + li;
#pragma unroll
      for (int p = 0; p < T; ++p) {
        float* dst = part + ((((int64_t)split * T + p) * CQ + cq) * Cout_pad + oo) * 4;
        *reinterpret_cast<floatx4*>(dst) = acc[p][a][b];
      }
    }
  }
  if (ct == 0 && dbpart != nullptr) {
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
    if (tid < BO) dbpart[(int64_t)split * Cout_pad + ot * BO + tid] = dsum;
  }
}

// Fixed-order sum of the S split partials, then the inverse transform over
// the planes (the same inverse as the forward epilogue).  An item is one
// 16-byte run of the partial layout: four consecutive input channels c of one
// padded output channel o, flat index cq * Cout_pad + o, so consecutive items
// are contiguous within a plane.  A workgroup of NTHR threads (256 or 1024)
// takes IPW consecutive items with all T planes (IPW * T slots) and splits the
// splits G ways (IPW * T * G <= NTHR): thread (q, e) reads slot e = p * IPW + i (plane p
// of item i, so a plane's IPW items are one contiguous run of IPW * 16 bytes)
// of splits q, q+G, q+2G, ...  Its loads are issued in batches of 8 before any
// of them is added, so each thread keeps up to 8 loads in flight.  The G group
// sums are added in a fixed order through LDS, and one thread per (item,
// channel) transforms the planes and writes dw.  Workgroups past the items sum
// the bias-gradient partials, NTHR / G output channels each, the same way.
// Every summation order depends only on (S, G), so results are bitwise
// reproducible.
constexpr int kRedBatch = 8;
template <int NB>
__device__ __forceinline__ floatx4 sum_splits(const float* src, int64_t stride, int first, int step, int S) {
  floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int sp = first; sp < S; sp += NB * step) {
    floatx4 v[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int s2 = sp + b * step;
      v[b] = s2 < S ? *reinterpret_cast<const floatx4*>(src + s2 * stride) : floatx4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) acc += v[b];
  }
  return acc;
}

template <int T, int DT, int NTHR>
__global__ __launch_bounds__(NTHR) void eql_wgrad_reduce_kernel(const float* __restrict__ part,
                                                                       const float* __restrict__ dbpart,
                                                                       void* __restrict__ dw,
                                                                       void* __restrict__ db, int S,
                                                                       int Cin, int Cout, int Cin_pad,
                                                                       int Cout_pad, int IPW, int G) {
  using E = typename Elem<DT>::T;
  __shared__ floatx4 red[NTHR];
  const int NS = NTHR / G;         // slot lanes (>= IPW * T)
  const int CQ = Cin_pad / 4;
  const int64_t items = (int64_t)CQ * Cout_pad;
  const int64_t nblk = (items + IPW - 1) / IPW;
  const int tid = threadIdx.x;
  const int q = tid / NS;          // split group
  const int e = tid - q * NS;      // slot lane
  if ((int64_t)blockIdx.x >= nblk) {  // bias gradient: NS output channels per workgroup
    if (db == nullptr) return;
    const int o = (int)((int64_t)blockIdx.x - nblk) * NS + e;
    float s = 0.0f;
    if (q < G && o < Cout) {
      for (int sp = q; sp < S; sp += kRedBatch * G) {
        float v[kRedBatch];
#pragma unroll
        for (int b = 0; b < kRedBatch; ++b) {
          const int s2 = sp + b * G;
          v[b] = s2 < S ? dbpart[(int64_t)s2 * Cout_pad + o] : 0.0f;
        }
#pragma unroll
        for (int b = 0; b < kRedBatch; ++b) s += v[b];
      }
    }
    float* const rs = reinterpret_cast<float*>(red);
    rs[tid] = s;
    __syncthreads();
    if (q == 0 && o < Cout) {
      float t = rs[e];
      for (int g = 1; g < G; ++g) t += rs[g * NS + e];
      reinterpret_cast<E*>(db)[o] = (E)t;
    }
    return;
  }
  const int64_t plane_stride = items * 4;
  const int64_t split_stride = (int64_t)T * plane_stride;
  const int64_t it0 = (int64_t)blockIdx.x * IPW;
  floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
  if (q < G && e < IPW * T) {
    const int p = e / IPW;
    const int i = e - p * IPW;
    const int64_t it = it0 + i;
    if (it < items) acc = sum_splits<kRedBatch>(part + p * plane_stride + it * 4, split_stride, q, G, S);
  }
  red[tid] = acc;
  __syncthreads();
  if (tid < IPW * 4) {
    const int il = tid >> 2, ce = tid & 3;
    const int64_t it = it0 + il;
    if (it < items) {
      const int cq = (int)(it / Cout_pad);
      const int o = (int)(it - (int64_t)cq * Cout_pad);
      const int c = cq * 4 + ce;
      if (o < Cout && c < Cin) {
        float Pl[T], u[T];
#pragma unroll
        for (int p = 0; p < T; ++p) {
          const int sl = p * IPW + il;
          float v = red[sl][ce];
          for (int g = 1; g < G; ++g) v += red[g * NS + sl][ce];
          Pl[p] = v;
        }
        irdft<T>(Pl, u);
        E* d = reinterpret_cast<E*>(dw);
#pragma unroll
        for (int j = 0; j < T; ++j) d[((int64_t)j * Cout + o) * Cin + c] = (E)u[j];
      }
    }
  }
}

}  // namespace eqk
