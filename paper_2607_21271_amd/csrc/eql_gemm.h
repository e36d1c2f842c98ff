// eql_gemm.h -- forward and input-gradient kernel of the C_T equivariant linear
// layer for gfx950: rDFT prologue -> per-bin MFMA products -> irDFT (+bias)
// epilogue, fused in one pass over the rows (Alg. 1 steps 1-4; Sec. 3.5).
//
// Work split.  The grid is persistent: workgroup w owns rows
// [w*N/G, (w+1)*N/G), so every CU streams the same number of rows.  A
// workgroup is 8 waves in 4 pairs; its rows are dealt out in rounds of 64, row
// q of a round going to pair q % 4, tile row q / 4.  The two waves of a pair
// share those 16 rows and split every o-chunk between them.
//
// Activations.  Per contraction step each lane loads, for one row, HKW
// channels with all T group positions (HKW*T contiguous elements), transforms
// them in registers and writes their T planes to the pair's spectrum buffer in
// LDS (double buffered); both waves then read complete MFMA operands from it.
// With RES the spectrum of all contraction steps stays in registers across
// o-chunks, so each activation is loaded and transformed once.
//
// Weights.  Per step a block of T planes x OC output channels x KSTEP
// contraction channels is prefetched into registers, written to the idle half
// of a double buffer in LDS and read as MFMA operands by all eight waves.  One
// barrier per step orders both exchanges.
//
// MFMA computes D[n][o] = sum_c X[n][c] W[o][c] (activation spectrum as the
// row operand); each lane ends with one output channel of 4 rows for every
// plane, so the inverse transform and bias run in registers, and the 16 lanes
// of a lane group store 16 consecutive channels (16*T contiguous elements) of
// one row.
#pragma once
#include "eql_common.h"
#include "eql_config.h"

namespace eqk {

template <int T, int DT>
struct GemmShape {
  static constexpr bool W16 = DT != kF32;  // 16-bit elements (fp16 or bf16)
  static constexpr int EB = W16 ? 2 : 4;
  static constexpr int kw_fit = 128 / (T * EB);  // channels whose T values fill <= 128 bytes
  static constexpr int KW = W16 ? (kw_fit >= 8 ? 8 : 4)
                                : (kw_fit >= 8 ? 8 : kw_fit >= 4 ? 4 : kw_fit >= 2 ? 2 : 1);
  static constexpr int KSTEP = 4 * KW;  // contraction channels per step (4 lane groups)
  static constexpr int FB = KW * EB;    // operand fragment bytes per lane
  static constexpr int RB = 4 * FB;     // bytes of one weight row per step
  static constexpr int NBH = KW / 2 * T * EB;  // raw activation bytes per lane per step
  // widest load (<= 16 bytes) dividing a lane's run; valid when the row stride
  // Ci*T*EB is a multiple of it, else the narrow kernel loads single elements
  static constexpr int WV = NBH % 16 == 0 ? 16 : NBH % 8 == 0 ? 8 : 4;
};

template <int FB>
struct Frag {
  uint32_t w[FB / 4];
};

template <int DT, int KW>
__device__ __forceinline__ void frag_mma(floatx4& acc, const Frag<KW*(DT != kF32 ? 2 : 4)>& a,
                                         const Frag<KW*(DT != kF32 ? 2 : 4)>& b) {
  if constexpr (DT == kF16 && KW == 8) {
    const u32x4 av = {a.w[0], a.w[1], a.w[2], a.w[3]};
    const u32x4 bv = {b.w[0], b.w[1], b.w[2], b.w[3]};
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8, av),
                                                 __builtin_bit_cast(half8, bv), acc, 0, 0, 0);
  } else if constexpr (DT == kF16 && KW == 4) {
    typedef _Float16 half4 __attribute__((ext_vector_type(4)));
    const u32x2 av = {a.w[0], a.w[1]};
    const u32x2 bv = {b.w[0], b.w[1]};
    acc = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(half4, av),
                                                __builtin_bit_cast(half4, bv), acc, 0, 0, 0);
  } else if constexpr (DT == kBF16 && KW == 8) {
    typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
    const u32x4 av = {a.w[0], a.w[1], a.w[2], a.w[3]};
    const u32x4 bv = {b.w[0], b.w[1], b.w[2], b.w[3]};
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av),
                                                  __builtin_bit_cast(bf16x8, bv), acc, 0, 0, 0);
  } else if constexpr (DT == kBF16 && KW == 4) {
    typedef short short4v __attribute__((ext_vector_type(4)));
    const u32x2 av = {a.w[0], a.w[1]};
    const u32x2 bv = {b.w[0], b.w[1]};
    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(short4v, av),
                                                    __builtin_bit_cast(short4v, bv), acc, 0, 0, 0);
  } else {
#pragma unroll
    for (int s = 0; s < KW; ++s)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__builtin_bit_cast(float, a.w[s]),
                                                 __builtin_bit_cast(float, b.w[s]), acc, 0, 0, 0);
  }
}

// sign flip of every element (the sign is the top bit of fp16, bf16 and fp32)
template <int DT, int FB>
__device__ __forceinline__ Frag<FB> frag_neg(const Frag<FB>& a) {
  Frag<FB> r;
#pragma unroll
  for (int j = 0; j < FB / 4; ++j) r.w[j] = a.w[j] ^ (DT != kF32 ? 0x80008000u : 0x80000000u);
  return r;
}

// Swizzled LDS rows of RB bytes: 16-byte chunk c of row r lives at chunk
// c ^ ((r >> 1) & (RB/16 - 1)).
template <int RB>
__device__ __forceinline__ int wl_off(int row, int byte) {
  constexpr int NCH = RB / 16;
  const int ch = byte >> 4;
  return row * RB + ((ch ^ ((row >> 1) & (NCH - 1))) << 4) + (byte & 15);
}

template <int FB, int RB>
__device__ __forceinline__ Frag<FB> lds_frag(const char* base, int row, int g) {
  Frag<FB> f;
  if constexpr (FB == 32) {
    const u32x4 a = *reinterpret_cast<const u32x4*>(base + wl_off<RB>(row, g * 32));
    const u32x4 b = *reinterpret_cast<const u32x4*>(base + wl_off<RB>(row, g * 32 + 16));
    f.w[0] = a[0]; f.w[1] = a[1]; f.w[2] = a[2]; f.w[3] = a[3];
    f.w[4] = b[0]; f.w[5] = b[1]; f.w[6] = b[2]; f.w[7] = b[3];
  } else if constexpr (FB == 16) {
    const u32x4 a = *reinterpret_cast<const u32x4*>(base + wl_off<RB>(row, g * 16));
    f.w[0] = a[0]; f.w[1] = a[1]; f.w[2] = a[2]; f.w[3] = a[3];
  } else {
    static_assert(FB == 8, "fragment size");
    const u32x2 a = *reinterpret_cast<const u32x2*>(base + wl_off<RB>(row, g * 8));
    f.w[0] = a[0]; f.w[1] = a[1];
  }
  return f;
}

// Buffer resource over [base, base + bytes): loads past the end return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// One lane's L contiguous output elements through a buffer resource, at byte
// offset off; a lane passes kDropOffset (past any resource) to store nothing.
// No branch skips a store, so every path through a loop issues the same
// memory operations and the compiler's memory-counter waits stay exact.
constexpr uint32_t kDropOffset = 0x80000000u;
template <int DT, int L>
__device__ __forceinline__ void store_run_rsrc(__amdgpu_buffer_rsrc_t rs, uint32_t off, const float (&v)[L]) {
  using E = typename Elem<DT>::T;
  constexpr int EBY = Elem<DT>::bytes;
  constexpr int NB = L * EBY;
  constexpr int VEC = (NB % 16 == 0) ? 16 : (NB % 8 == 0) ? 8 : (NB % 4 == 0) ? 4 : 2;
  constexpr int PER = VEC / EBY;
#pragma unroll
  for (int s = 0; s < L / PER; ++s) {
    E tmp[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) tmp[q] = (E)v[s * PER + q];
    const uint32_t o = off + s * VEC;
    if constexpr (VEC == 16) {
      u32x4 w;
      __builtin_memcpy(&w, tmp, 16);
      __builtin_amdgcn_raw_buffer_store_b128(w, rs, o, 0, 0);
    } else if constexpr (VEC == 8) {
      u32x2 w;
      __builtin_memcpy(&w, tmp, 8);
      __builtin_amdgcn_raw_buffer_store_b64(w, rs, o, 0, 0);
    } else if constexpr (VEC == 4) {
      uint32_t w;
      __builtin_memcpy(&w, tmp, 4);
      __builtin_amdgcn_raw_buffer_store_b32(w, rs, o, 0, 0);
    } else {
      uint16_t w;
      __builtin_memcpy(&w, tmp, 2);
      __builtin_amdgcn_raw_buffer_store_b16(w, rs, o, 0, 0);
    }
  }
}

// Raw bytes of one lane for one step: NB bytes at byte offset off (+ soff) of
// the resource, with loads of W bytes (W = 2: 16-bit loads paired into words).
// The width is a compile-time constant so that every kernel has a single load
// shape: with the width chosen at run time among several load shapes feeding
// the same registers, the register allocator in this toolchain produced code
// that overwrote live raw words in some kernels.  Bytes past the resource
// read as zero.
template <int NB, int W>
__device__ __forceinline__ void load_raw(__amdgpu_buffer_rsrc_t rs, uint32_t off, int soff,
                                         uint32_t (&r)[NB / 4]) {
  static_assert(NB % W == 0 && NB % 4 == 0, "load width");
  if constexpr (W == 16) {
#pragma unroll
    for (int v = 0; v < NB / 16; ++v) {
      const u32x4 x = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16 * v, soff, 0));
      r[4 * v] = x[0]; r[4 * v + 1] = x[1]; r[4 * v + 2] = x[2]; r[4 * v + 3] = x[3];
    }
  } else if constexpr (W == 8) {
#pragma unroll
    for (int v = 0; v < NB / 8; ++v) {
      const u32x2 x = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rs, off + 8 * v, soff, 0));
      r[2 * v] = x[0]; r[2 * v + 1] = x[1];
    }
  } else if constexpr (W == 4) {
#pragma unroll
    for (int v = 0; v < NB / 4; ++v) r[v] = __builtin_amdgcn_raw_buffer_load_b32(rs, off + 4 * v, soff, 0);
  } else {
#pragma unroll
    for (int v = 0; v < NB / 4; ++v) {
      const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(rs, off + 4 * v, soff, 0);
      const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(rs, off + 4 * v + 2, soff, 0);
      r[v] = (lo & 0xffffu) | (hi << 16);
    }
  }
}

// Zero the elements past nvalid (a ragged last channel group).
template <int NB, int EB>
__device__ __forceinline__ void mask_raw(int nvalid_elems, uint32_t (&r)[NB / 4]) {
  if (nvalid_elems >= NB / EB) return;
#pragma unroll
  for (int v = 0; v < NB / 4; ++v) {
    if constexpr (EB == 2) {
      if (2 * v + 1 >= nvalid_elems) r[v] = (2 * v < nvalid_elems) ? (r[v] & 0xffffu) : 0u;
    } else {
      if (v >= nvalid_elems) r[v] = 0u;
    }
  }
}

// Implicit patch gather (group convolution): a lane's raw words hold T
// vectors, vector j being the HKW elements vec_j[cc*T + s] = f[pixel + R^j d0,
// c + cc, s] of one window orbit (M = HKW / T input channels c + cc, every
// group position s).  The gathered channel (cc, u) at group position j is
// vec_j[cc*T + (u + j) mod T] (the shear u = s - j); this rewrites the words
// into the plain order, element (cc*T + u)*T + j.  The centre of the window is
// already in plain order (keep).
template <int T, int HKW, int EB>
__device__ __forceinline__ void gather_shear(uint32_t (&r)[HKW * T * EB / 4], bool keep) {
  constexpr int NW = HKW * T * EB / 4;
  // source element of plain element i = (cc*T + u)*T + j
  constexpr auto src = [](int i) {
    const int j = i % T, u = (i / T) % T, cc = i / (T * T);
    return j * HKW + cc * T + (u + j) % T;
  };
  // every index below is a compile-time constant: the sheared words are
  // built into their own array and the lane's choice applied per word (a
  // per-element choice of source index became a runtime-indexed array)
  uint32_t o[NW];
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    if constexpr (EB == 4) {
      o[w] = r[src(w)];
    } else {
      const int s0 = src(2 * w), s1 = src(2 * w + 1);
      const uint32_t lo = (r[s0 / 2] >> (16 * (s0 % 2))) & 0xffffu;
      const uint32_t hi = (r[s1 / 2] >> (16 * (s1 % 2))) & 0xffffu;
      o[w] = lo | (hi << 16);
    }
  }
  const uint32_t km = keep ? 0xffffffffu : 0u;
#pragma unroll
  for (int w = 0; w < NW; ++w) r[w] = (r[w] & km) | (o[w] & ~km);
}

// n / d and n mod d for n < 2^31 and a launch-constant divisor d with its
// multiplier m = floor(2^32 / d) (2^32 - 1 for d = 1): the product estimate
// is exact or one low
__device__ __forceinline__ uint32_t gather_div(uint32_t n, uint32_t d, uint32_t m, uint32_t& r) {
  uint32_t q = __umulhi(n, m);
  r = n - q * d;
  if (r >= d) {
    ++q;
    r -= d;
  }
  return q;
}

// Transform the HKW channels held raw by one lane; P[p][j] is plane p of channel j.
template <int T, int DT, int HKW>
__device__ __forceinline__ void raw_to_planes(const uint32_t (&r)[HKW * T * (DT != kF32 ? 2 : 4) / 4],
                                              float (&P)[T][HKW]) {
  constexpr int NW = HKW * T * (DT != kF32 ? 2 : 4) / 4;
  float f[DT != kF32 ? 2 * NW : NW];
  raw_to_floats<DT, NW>(r, f);
#pragma unroll
  for (int j = 0; j < HKW; ++j) {
    float v[T], q[T];
#pragma unroll
    for (int t = 0; t < T; ++t) v[t] = f[j * T + t];
    rdft<T>(v, q);
#pragma unroll
    for (int p = 0; p < T; ++p) P[p][j] = q[p];
  }
}

// fp16: the HKW channels of one lane taken in pairs (2j, 2j+1), element t of
// both in one packed register, and transformed together in fp16 arithmetic;
// W[p][j] is then plane p of the pair, the word that is staged.  Element t of
// channel c is half (c*T + t) % 2 of raw word (c*T + t) / 2.
template <int T, int HKW>
__device__ __forceinline__ void raw_to_packed_planes(const uint32_t (&r)[HKW * T / 2],
                                                     uint32_t (&W)[T][HKW / 2]) {
  static_for<HKW / 2>([&](auto ji) {
    constexpr int j = decltype(ji)::value;
    half2v v[T], P[T];
    static_for<T>([&](auto ti) {
      constexpr int t = decltype(ti)::value;
      constexpr int ia = (2 * j) * T + t, ib = (2 * j + 1) * T + t;
      v[t] = pair_halves<ia % 2, ib % 2>(r[ia / 2], r[ib / 2]);
    });
    rdft<T, H2Ops>(v, P);
#pragma unroll
    for (int p = 0; p < T; ++p) W[p][j] = __builtin_bit_cast(uint32_t, P[p]);
  });
}

// How the weight blocks reach LDS (MODE):
//   kStream  two block buffers; the block of the next step is prefetched into
//            registers while the current one feeds the MFMAs
//   kRes     as kStream, and each wave's operand spectrum of all NKR
//            contraction steps stays in registers across o-chunks
//            (requires ceil(Ci / KSTEP) == NKR)
//   kStat    every block of the layer is loaded into LDS once per workgroup;
//            inside the row loop only activations move
enum GemmMode { kStream = 0, kRes = 1, kStat = 2 };

// LDS arena of one workgroup: two spectrum buffers, then the weight blocks.
template <int T, int DT, int OT>
struct GemmLds {
  static constexpr int RB = GemmShape<T, DT>::RB;
  static constexpr int XBLK = kGemmPairs * T * 16 * RB;  // pairs x T planes x 16 rows
  static constexpr int WBLK = T * 32 * OT * RB; // T planes x OC channels
  static constexpr int bytes(int n_wblocks) { return 2 * XBLK + n_wblocks * WBLK; }
};

// Kernel parameters: the workgroup is 8 waves, wave w = 2*rg + oh.  Waves rg
// own rows; the pair (rg, 0), (rg, 1) shares 16 rows and splits each o-chunk:
// wave oh computes OT output tiles of 16, so an o-chunk holds OC = 32*OT
// channels.
//
// Per contraction step a lane of wave oh transforms HKW = KW/2 channels of its
// row and writes their planes to the pair's spectrum buffer in LDS; after a
// barrier both waves read complete MFMA operands from it.  Weight blocks are
// double buffered in LDS: the next block is loaded into registers while the
// current one feeds the MFMAs, then written to the idle buffer.
//
// GATHER (forward of the group convolution, T in {1, 2, 4}): `in` is the feature map
// f [N pixels, geo.Cin, T] and row n of the layer's input is the gathered
// patch row of pixel n (k*k*Cin channels: window orbits, then the centre),
// read straight from f instead of a materialised patch buffer.
template <int T, int DT, bool BWD, int OT, int MODE, int NKR, bool NARROW, bool GATHER>
__global__ __launch_bounds__(kGemmThreads) void eql_gemm_kernel(const void* __restrict__ in,
                                                       const void* __restrict__ wsp,
                                                       const void* __restrict__ bias,
                                                       void* __restrict__ out, int64_t N, int Ci,
                                                       int Co, int Ci_pad, int Co_pad, int n_oc,
                                                       int n_ks, GatherGeom geo) {
  using S = GemmShape<T, DT>;
  using Bn = Bins<T>;
  using FR = Frag<S::FB>;
  using E = typename Elem<DT>::T;
  constexpr int EB = S::EB;
  constexpr int KW = S::KW;
  constexpr int HKW = KW / 2;
  constexpr int KSTEP = S::KSTEP;
  constexpr int FB = S::FB;
  constexpr int RB = S::RB;             // bytes of one row (weights or spectrum) per step
  constexpr int NBH = S::NBH;           // raw activation bytes per lane per step
  constexpr int OC = 32 * OT;
  constexpr bool RES = MODE == kRes;
  constexpr int WBLK = GemmLds<T, DT, OT>::WBLK;  // bytes of one weight block
  constexpr int NU = WBLK / 16;         // 16-byte units per block
  constexpr int NTH = kGemmThreads;
  constexpr int UPT = (NU + NTH - 1) / NTH; // weight units per thread
  constexpr int XBLK = GemmLds<T, DT, OT>::XBLK;  // bytes of one spectrum buffer
  static_assert(KW >= 2, "contraction split");
  static_assert(!GATHER || (!BWD && !NARROW && (T == 1 || T == 2 || T == 4) && HKW % T == 0),
                "implicit gather: forward, T in {1, 2, 4}");

  // dynamic LDS: xl[2][XBLK], then the weight blocks (2 streamed, 2 * NKR with a
  // resident spectrum, n_oc * n_ks resident)
  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* const xlb = smem;
  char* const wlb = smem + 2 * XBLK;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: branches on it stay scalar
  const int rg = wave >> 1;
  const int oh = wave & 1;
  const int g = lane >> 4;
  const int li = lane & 15;
  const int64_t r0 = (int64_t)blockIdx.x * N / gridDim.x;
  const int64_t r1 = ((int64_t)blockIdx.x + 1) * N / gridDim.x;
  const int64_t len = r1 - r0;
  const int rounds = (int)((len + kGemmRoundRows - 1) / kGemmRoundRows);
  const int nks = RES ? NKR : n_ks;
  const int64_t wplane = (int64_t)Co_pad * Ci_pad * EB;
  const char* wbase = reinterpret_cast<const char*>(wsp);
  const char* xin = reinterpret_cast<const char*>(in);
  const int rowb = Ci * T * EB;
  constexpr int LW = NARROW ? EB : S::WV;  // load width; the host checks rowb % LW == 0
  // rows of this workgroup (GATHER: the whole feature map, below 2^31 bytes)
  const __amdgpu_buffer_rsrc_t xrs =
      GATHER ? make_rsrc(xin, (uint32_t)(N * geo.Cin * T * EB)) : make_rsrc(xin + r0 * rowb, (uint32_t)(len * rowb));
  if (rounds == 0) return;

  // ---- weight block (oc, kc): global -> registers -> LDS buffer.  Per-thread
  // unit offsets are fixed; a step only moves a uniform base.
  // register sets of prefetched weight blocks: 2 when streamed (a block is
  // issued two steps before it is stored to LDS), NKR with a resident
  // spectrum (block (oc, kc) always uses set kc)
  // Streamed weights whose blocks split into whole wave-loads of 64 x 16
  // bytes go from global memory straight into LDS (buffer_load ... lds): no
  // staging registers, no LDS store instructions.  Lane l of a wave-load
  // writes LDS bytes [16 l, 16 l + 16) of the wave's 1 KB slice, so each lane
  // loads the 16-byte chunk that the swizzled layout puts there.
  constexpr int NWV = NTH / 64;
  // (not at T = 4 and 8, where the EQ-ViT and EQ-Swin layers measured level
  // per pass and 1-2% slower per training step with it)
  constexpr bool DMA = MODE == kStream && NU % (64 * NWV) == 0 && T != 4 && T != 8;
  // Operand reads of the next o-tile ahead of the current tile's MFMAs, where
  // that measured faster (16-bit types at T = 3 and 16: 6-10% on the input
  // gradient, and at T = 16 on the forward; at T = 5, 8 and 12 level or
  // slower per pass, at T = 4 6% faster per forward pass but 2% slower per
  // training step; with a resident spectrum the registers are not there).
  constexpr bool PIPE = !RES && DT != kF32 && (T == 3 || T == 16);
  constexpr int UPD = DMA ? NU / (64 * NWV) : 1;  // wave-loads per wave and block
  int gdma[UPD];
  if constexpr (DMA) {
#pragma unroll
    for (int u = 0; u < UPD; ++u) {
      const int unit = (u * NWV + wave) * 64 + lane;  // LDS slot of the block
      const int p = unit / (OC * RB / 16);
      const int rem = unit - p * (OC * RB / 16);
      const int row = rem / (RB / 16);
      const int cs = rem - row * (RB / 16);
      const int ch = cs ^ ((row >> 1) & (RB / 16 - 1));  // source chunk swizzled to slot cs
      gdma[u] = (int)(p * wplane + (int64_t)row * Ci_pad * EB + ch * 16);
    }
  }
  constexpr int NWS = DMA ? 1 : RES ? (NKR > 1 ? NKR : 1) : 2;
  constexpr int UPTR = DMA ? 1 : UPT;  // staging registers per set
  u32x4 wr[NWS][UPTR];
  int goff[UPTR];
  int loff[UPTR];
#pragma unroll
  for (int u = 0; u < UPTR; ++u) {
    const int unit = tid + NTH * u;
    const int p = unit / (OC * RB / 16);
    const int rem = unit - p * (OC * RB / 16);
    const int row = rem / (RB / 16);
    const int ch = rem - row * (RB / 16);
    goff[u] = (unit < NU) ? (int)(p * wplane + (int64_t)row * Ci_pad * EB + ch * 16) : 0;
    loff[u] = (unit < NU) ? p * OC * RB + wl_off<RB>(row, ch * 16) : 0;
  }
  // Buffer loads: per-thread offsets stay in fixed VGPRs and the block offset
  // goes in the scalar offset, so issuing a load writes no VGPR before it (an
  // address computed into the destination registers made the compiler wait
  // for every load in flight first).  The spectrum is below 2^31 bytes.
  const __amdgpu_buffer_rsrc_t wrs = make_rsrc(wbase, (uint32_t)((int64_t)T * wplane));
  auto issue_w = [&](auto set, int oc, int kc) __attribute__((always_inline)) {
    constexpr int S = decltype(set)::value;
    const int boff = (oc * OC * Ci_pad + kc * KSTEP) * EB;
#pragma unroll
    for (int u = 0; u < UPTR; ++u)
      if (NU % NTH == 0 || tid + NTH * u < NU)
        wr[S][u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(wrs, goff[u], boff, 0));
  };
  auto store_w = [&](auto set, int blk) __attribute__((always_inline)) {
    constexpr int S = decltype(set)::value;
#pragma unroll
    for (int u = 0; u < UPTR; ++u)
      if (NU % NTH == 0 || tid + NTH * u < NU) *reinterpret_cast<u32x4*>(wlb + blk * WBLK + loff[u]) = wr[S][u];
  };
  // weight block (oc, kc) straight into LDS block blk (each wave its slices).
  // The builtin exists for the device pass only (the host pass, which never
  // runs kernel code, emits unusable IR for it when intermediate files are
  // kept, as this build does for the post-build check).
  auto dma_w = [&](int blk, int oc, int kc) __attribute__((always_inline)) {
#if defined(__HIP_DEVICE_COMPILE__)
    const int boff = (oc * OC * Ci_pad + kc * KSTEP) * EB;
#pragma unroll
    for (int u = 0; u < UPD; ++u)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          wrs, (__attribute__((address_space(3))) void*)(wlb + blk * WBLK + (u * NWV + wave) * 1024), 16,
          gdma[u], boff, 0, 0);
#else
    (void)blk; (void)oc; (void)kc;
#endif
  };

  // ---- raw activations of (round m, step kc): HKW channels of this lane's row.
  // Issued unconditionally, also for the round after the last one (those rows
  // lie past the buffer resource and read as zero); offsets stay below 2^31
  // because the grid keeps one round of slack.
  // raw activation sets (compile-time index): one per contraction step with
  // a resident spectrum (a round's loads are issued together), else one
  constexpr int NXS = RES ? NKR : 1;
  uint32_t xr[NXS][NBH / 4];
  int xr_valid[NXS];  // valid elements per set (the rest belong to the next row)
  bool xr_plain[NXS];  // GATHER: the words are already in plain order (window centre)
  auto issue_x = [&](auto set, int m, int kc) __attribute__((always_inline)) {
    constexpr int X = decltype(set)::value;
    const int q = m * kGemmRoundRows + kGemmPairs * li + rg;
    const int c0 = oh * (KSTEP / 2) + g * HKW;  // channel within the step
    const int cabs = kc * KSTEP + c0;
    if constexpr (GATHER) {
      // T loads of HKW elements each: the lane's gathered channels are M =
      // HKW / T input channels c.. of one window orbit O (all T sheared
      // positions), or HKW channels of the centre.  The host keeps Cin a
      // multiple of HKW, so a lane never straddles two blocks.  Pixels outside
      // the image, rows past the workgroup's and channels past k*k*Cin read
      // zero (dropped offsets).  Divisions by launch constants are multiplies
      // (GatherGeom), offsets 32-bit (the feature map is below 2^31 bytes).
      constexpr int VB = HKW * EB;  // bytes per vector
      const uint32_t CT = (uint32_t)geo.Cin * T;
      const uint32_t p = (uint32_t)(r0 + q);
      const bool row_ok = q < len && cabs < Ci;
      uint32_t x, y, rem;
      const uint32_t py = gather_div(p, (uint32_t)geo.W, geo.mW, x);
      gather_div(py, (uint32_t)geo.H, geo.mH, y);
      uint32_t cr;
      const uint32_t O = gather_div((uint32_t)cabs, CT, geo.mCT, cr);
      const int h = geo.k >> 1;
      const bool centre = (int)O >= (geo.k * geo.k - 1) / T;  // past the last orbit block
      // orbit base point (a0, b0)
      int a0, b0;
      if constexpr (T == 4) {
        const uint32_t qa = gather_div(O, (uint32_t)(h + 1), geo.mO, rem);
        a0 = 1 + (int)qa;
        b0 = (int)rem;
      } else if constexpr (T == 2) {
        const uint32_t qa = gather_div(O, (uint32_t)geo.k, geo.mO, rem);
        const bool upper = (int)qa < h;
        a0 = upper ? 1 + (int)qa : 0;
        b0 = upper ? (int)rem - h : 1 + (int)rem;
      } else {
        const uint32_t idx = O + (O >= (uint32_t)((geo.k * geo.k - 1) / 2) ? 1u : 0u);
        const uint32_t qa = gather_div(idx, (uint32_t)geo.k, geo.mO, rem);
        a0 = (int)qa - h;
        b0 = (int)rem - h;
      }
      if (centre) { a0 = 0; b0 = 0; }
      // byte offset of the lane's first channel in a pixel row: orbit lanes
      // read channel c = cr / T of T pixels, centre lanes T consecutive
      // vectors of their own pixel
      const uint32_t coff = centre ? ((uint32_t)cabs - O * CT) * T * EB : (cr / T) * T * EB;
      const uint32_t rowf = CT * EB;
      xr_valid[X] = HKW * T;
      xr_plain[X] = centre;
      static_for<T>([&](auto ji) {
        constexpr int j = decltype(ji)::value;
        // R^j (a0, b0): R(a, b) = (-b, a) at T = 4, (-a, -b) at T = 2
        int a = a0, b = b0;
        if constexpr (T == 4) {
          if constexpr (j == 1) { a = -b0; b = a0; }
          if constexpr (j == 2) { a = -a0; b = -b0; }
          if constexpr (j == 3) { a = b0; b = -a0; }
        } else if constexpr (T == 2) {
          if constexpr (j == 1) { a = -a0; b = -b0; }
        }
        const bool in_img = (uint32_t)((int)y + a) < (uint32_t)geo.H && (uint32_t)((int)x + b) < (uint32_t)geo.W;
        const uint32_t pix = p + (uint32_t)(a * geo.W + b);
        const uint32_t off = (row_ok && in_img) ? pix * rowf + coff + (centre ? (uint32_t)(j * VB) : 0u)
                                                : kDropOffset;
        if constexpr (VB == 16) {
          const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(xrs, off, 0, 0));
          xr[X][4 * j] = v[0]; xr[X][4 * j + 1] = v[1]; xr[X][4 * j + 2] = v[2]; xr[X][4 * j + 3] = v[3];
        } else {
          static_assert(VB == 8, "gather vector");
          const u32x2 v = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(xrs, off, 0, 0));
          xr[X][2 * j] = v[0]; xr[X][2 * j + 1] = v[1];
        }
      });
    } else {
      const uint32_t voff = (uint32_t)(((int64_t)q * Ci + c0) * T * EB);
      xr_valid[X] = (Ci - cabs >= HKW) ? HKW * T : (Ci - cabs > 0 ? (Ci - cabs) * T : 0);
      load_raw<NBH, LW>(xrs, voff, kc * KSTEP * T * EB, xr[X]);
    }
  };
  // transform and publish this lane's part of the step's operand spectrum
  auto publish_x = [&](auto set, int xb) __attribute__((always_inline)) {
    constexpr int X = decltype(set)::value;
    if constexpr (GATHER) gather_shear<T, HKW, EB>(xr[X], xr_plain[X]);
    mask_raw<NBH, EB>(xr_valid[X], xr[X]);
    const int byte = (oh * (KSTEP / 2) + g * HKW) * EB;
    if constexpr (DT != kF32) {
      uint32_t W[T][HKW / 2];
      if constexpr (DT == kF16) {
        raw_to_packed_planes<T, HKW>(xr[X], W);
      } else {
        float P[T][HKW];
        raw_to_planes<T, DT, HKW>(xr[X], P);
#pragma unroll
        for (int p = 0; p < T; ++p)
#pragma unroll
          for (int j = 0; j < HKW / 2; ++j) W[p][j] = pack2<DT>(P[p][2 * j], P[p][2 * j + 1]);
      }
#pragma unroll
      for (int p = 0; p < T; ++p) {
        char* dst = xlb + xb * XBLK + (rg * T + p) * 16 * RB + wl_off<RB>(li, byte);
        if constexpr (HKW == 4) *reinterpret_cast<u32x2*>(dst) = u32x2{W[p][0], W[p][1]};
        else *reinterpret_cast<uint32_t*>(dst) = W[p][0];
      }
      return;
    }
    float P[T][HKW];
    raw_to_planes<T, DT, HKW>(xr[X], P);
#pragma unroll
    for (int p = 0; p < T; ++p) {
      {
        char* dst = xlb + xb * XBLK + (rg * T + p) * 16 * RB + wl_off<RB>(li, byte);
        if constexpr (HKW == 4) {
          *reinterpret_cast<u32x4*>(dst) = u32x4{__builtin_bit_cast(uint32_t, P[p][0]), __builtin_bit_cast(uint32_t, P[p][1]),
                                                 __builtin_bit_cast(uint32_t, P[p][2]), __builtin_bit_cast(uint32_t, P[p][3])};
        } else if constexpr (HKW == 2) {
          *reinterpret_cast<u32x2*>(dst) = u32x2{__builtin_bit_cast(uint32_t, P[p][0]), __builtin_bit_cast(uint32_t, P[p][1])};
        } else {
          *reinterpret_cast<uint32_t*>(dst) = __builtin_bit_cast(uint32_t, P[p][0]);
        }
      }
    }
  };
  auto read_x = [&](int xb, FR (&B)[T]) {
#pragma unroll
    for (int p = 0; p < T; ++p) B[p] = lds_frag<FB, RB>(xlb + xb * XBLK + (rg * T + p) * 16 * RB, li, g);
  };

  floatx4 acc[T][OT];
  // With a resident spectrum the subtracted product of each complex bin has
  // its own accumulator (difference taken in the epilogue) instead of a
  // negated operand, which would stay live across o-chunks.
  constexpr int NXA = RES && Bn::K > 0 ? Bn::K : 1;
  floatx4 accx[NXA][OT];
  FR xres[RES ? NKR : 1][T];
  FR bcur[T];
  const E* __restrict__ bp = reinterpret_cast<const E*>(bias);
  // output rows of this workgroup as a buffer resource, below 2^31 bytes (the
  // launcher sizes the grid so)
  const __amdgpu_buffer_rsrc_t ors =
      make_rsrc(reinterpret_cast<char*>(out) + r0 * Co * T * EB, (uint32_t)(len * Co * T * EB));

  // One step: weights of (oc, kc) in LDS block blk, X the activation spectrum.
  // The sign of each complex product sits on a negated copy of one X plane
  // (Im for the forward, Re for the input gradient), made once per step:
  //   forward:  Re += Wr Xr + Wi (-Xi),   Im += Wi Xr + Wr Xi
  //   backward: Re += Wr Dr + Wi Di,      Im += Wr Di + Wi (-Dr)
  auto mma_step = [&](int oc, int blk, FR (&X)[T]) {
    FR Xneg[Bn::K > 0 && !RES ? Bn::K : 1];
    if constexpr (!RES) {
      static_for<Bn::K>([&](auto ki) {
        constexpr int k = decltype(ki)::value + 1;
        Xneg[k - 1] = frag_neg<DT, FB>(X[BWD ? Bn::re(k) : Bn::im(k)]);
      });
    }
    // With PIPE the operand reads of tile a + 1 are issued before the MFMAs of
    // tile a; otherwise each tile reads its operands just before its MFMAs.
    // Tiles past Co skip their MFMAs.
    auto tile_mma = [&](int a, const FR (&W)[T]) __attribute__((always_inline)) {
      frag_mma<DT, KW>(acc[0][a], X[0], W[0]);
      if constexpr (Bn::kEven) frag_mma<DT, KW>(acc[1][a], X[1], W[1]);
      static_for<Bn::K>([&](auto ki) {
        constexpr int k = decltype(ki)::value + 1;
        constexpr int r = Bn::re(k);
        constexpr int i = Bn::im(k);
        if constexpr (RES && !BWD) {
          frag_mma<DT, KW>(acc[r][a], X[r], W[r]);
          frag_mma<DT, KW>(acc[i][a], X[r], W[i]);
          frag_mma<DT, KW>(accx[k - 1][a], X[i], W[i]);   // subtracted from Re
          frag_mma<DT, KW>(acc[i][a], X[i], W[r]);
        } else if constexpr (RES) {
          frag_mma<DT, KW>(acc[r][a], X[r], W[r]);
          frag_mma<DT, KW>(acc[i][a], X[i], W[r]);
          frag_mma<DT, KW>(acc[r][a], X[i], W[i]);
          frag_mma<DT, KW>(accx[k - 1][a], X[r], W[i]);   // subtracted from Im
        } else if constexpr (!BWD) {
          frag_mma<DT, KW>(acc[r][a], X[r], W[r]);
          frag_mma<DT, KW>(acc[i][a], X[r], W[i]);
          frag_mma<DT, KW>(acc[r][a], Xneg[k - 1], W[i]);
          frag_mma<DT, KW>(acc[i][a], X[i], W[r]);
        } else {
          frag_mma<DT, KW>(acc[r][a], X[r], W[r]);
          frag_mma<DT, KW>(acc[i][a], X[i], W[r]);
          frag_mma<DT, KW>(acc[r][a], X[i], W[i]);
          frag_mma<DT, KW>(acc[i][a], Xneg[k - 1], W[i]);
        }
      });
    };
    if constexpr (PIPE) {
      FR Wb[2][T];
      auto load_w = [&](int a, FR (&W)[T]) __attribute__((always_inline)) {
        const int ot = oh * OT + a;
#pragma unroll
        for (int p = 0; p < T; ++p) W[p] = lds_frag<FB, RB>(wlb + blk * WBLK + p * OC * RB, ot * 16 + li, g);
      };
      load_w(0, Wb[0]);
#pragma unroll
      for (int a = 0; a < OT; ++a) {
        if (a + 1 < OT) load_w(a + 1, Wb[(a + 1) & 1]);
        if (oc * OC + (oh * OT + a) * 16 >= Co) continue;  // uniform across the wave
        tile_mma(a, Wb[a & 1]);
      }
    } else {
#pragma unroll
      for (int a = 0; a < OT; ++a) {
        const int ot = oh * OT + a;                 // o-tile within the chunk
        if (oc * OC + ot * 16 >= Co) continue;      // uniform across the wave
        FR W[T];
#pragma unroll
        for (int p = 0; p < T; ++p) W[p] = lds_frag<FB, RB>(wlb + blk * WBLK + p * OC * RB, ot * 16 + li, g);
        tile_mma(a, W);
      }
    }
  };

  // D = X W^T: lane (g, i) holds output channel ot*16 + i of the pair's rows
  // 4g .. 4g+3.  The 16 lanes of a lane group write 16 consecutive channels of
  // one row, a contiguous span of 16*T elements (whole cache lines).
  // Tiles past Co (zero accumulators) run too, with every store dropped.
  // With active false the inverse transforms are skipped and the same
  // stores are issued, all dropped (one wave group of the resident-spectrum
  // loop runs its epilogue at another point of the iteration than the other;
  // identical memory operations on both keep the waits exact).
  auto epilogue_if = [&](int m, int oc, bool active) __attribute__((always_inline)) {
#pragma unroll
    for (int a = 0; a < OT; ++a) {
      const int ot = oh * OT + a;
      const int o = oc * OC + ot * 16 + li;
      float bv = 0.0f;
      if constexpr (!BWD) {
        // (a uniform branch; waiting for this load also waits for every
        // memory operation issued before it)
        if (bp != nullptr) bv = (float)bp[o < Co ? o : Co - 1];
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int q = m * kGemmRoundRows + kGemmPairs * (4 * g + r) + rg;
        float ul[T];
#pragma unroll
        for (int t = 0; t < T; ++t) ul[t] = 0.0f;
        if (active) {  // uniform across the wave
          float Pl[T];
#pragma unroll
          for (int p = 0; p < T; ++p) Pl[p] = acc[p][a][r];
          if constexpr (RES) {
            static_for<Bn::K>([&](auto ki) {
              constexpr int k = decltype(ki)::value + 1;
              constexpr int pl = BWD ? Bn::im(k) : Bn::re(k);
              Pl[pl] -= accx[k - 1][a][r];
            });
          }
          // a constant added to every group position is T times it added to bin 0
          Pl[0] = __builtin_fmaf((float)T, bv, Pl[0]);
          irdft<T>(Pl, ul);
        }
        const uint32_t off = (active && q < len && o < Co) ? (uint32_t)((q * Co + o) * T * EB) : kDropOffset;
        store_run_rsrc<DT, T>(ors, off, ul);
      }
    }
  };
  auto epilogue = [&](int m, int oc) __attribute__((always_inline)) { epilogue_if(m, oc, true); };

  auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int p = 0; p < T; ++p)
#pragma unroll
      for (int a = 0; a < OT; ++a) acc[p][a] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < NXA; ++k)
#pragma unroll
      for (int a = 0; a < OT; ++a) accx[k][a] = floatx4{0.f, 0.f, 0.f, 0.f};
  };

  // Pipelining.  Every global load is issued right after a barrier and
  // consumed in the same loop iteration, after that step's MFMAs: the
  // compiler's memory-counter waits are exact only for loads whose issue and
  // use lie on one straight path (across a loop back edge or around a branch
  // that issues other memory operations it falls back to waiting for nearly
  // everything in flight).  Epilogue stores come last in an iteration, so no
  // wait of that iteration covers them.
  int buf = 0;
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  if constexpr (MODE == kStat) {
    // All weight blocks into LDS once; then a step only exchanges activations:
    //   barrier; issue activations of s+1; read operands, MFMA(s);
    //   publish X(s+1) to xl[(s+1) & 1]; epilogue if s ends an o-chunk.
    issue_x(I0{}, 0, 0);
    {
      // block b = oc * nks + kc holds planes x OC rows x KSTEP channels; unit
      // u of the arena is 16 bytes of it.  Four loads in flight per thread.
      const int n_units = n_oc * nks * NU;
      for (int u0 = tid; u0 < n_units; u0 += 4 * NTH) {
        u32x4 v[4];
        int lo[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int u = u0 + NTH * j;
          lo[j] = -1;
          if (u < n_units) {
            const int blk = u / NU;
            const int in_blk = u - blk * NU;
            const int boc = blk / nks;
            const int bkc = blk - boc * nks;
            const int p = in_blk / (OC * RB / 16);
            const int rem = in_blk - p * (OC * RB / 16);
            const int row = rem / (RB / 16);
            const int ch = rem - row * (RB / 16);
            const char* src = wbase + p * wplane + ((int64_t)(boc * OC + row) * Ci_pad + bkc * KSTEP) * EB + ch * 16;
            v[j] = *reinterpret_cast<const u32x4*>(src);
            lo[j] = blk * WBLK + p * OC * RB + wl_off<RB>(row, ch * 16);
          }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (lo[j] >= 0) *reinterpret_cast<u32x4*>(wlb + lo[j]) = v[j];
      }
    }
    publish_x(I0{}, 0);
    for (int m = 0; m < rounds; ++m) {
      for (int oc = 0; oc < n_oc; ++oc) {
        zero_acc();
        for (int kc = 0; kc < nks; ++kc) {
          int nkc = kc + 1, nm = m;
          if (nkc == nks) { nkc = 0; if (oc + 1 == n_oc) ++nm; }
          __syncthreads();
          issue_x(I0{}, nm, nkc);  // past the last round: rows beyond the resource read as zero
          read_x(buf, bcur);
          mma_step(oc, oc * nks + kc, bcur);
          publish_x(I0{}, buf ^ 1);
          buf ^= 1;
        }
        epilogue(m, oc);
      }
    }
    return;
  }

  if constexpr (RES) {
    // Resident spectrum: the NKR weight blocks of an o-chunk sit together in
    // one of two LDS regions (block kc of region r at LDS block r * NKR + kc).
    // Iteration (m, oc):
    //   oc == 0: the round's raw activations are issued together (for the
    //     first round in the prologue), then published and read into xres one
    //     step per barrier; else one barrier
    //   issue the next o-chunk's blocks (register set kc for block kc); the
    //   NKR steps run from the current region; the next blocks go to the
    //   other region.
    static_for<NKR>([&](auto ki) { issue_w(ki, 0, decltype(ki)::value); });
    static_for<NKR>([&](auto ki) { issue_x(ki, 0, decltype(ki)::value); });
    static_for<NKR>([&](auto ki) { store_w(ki, decltype(ki)::value); });
    int reg = 0;
    for (int m = 0; m < rounds; ++m) {
      for (int oc = 0; oc < n_oc; ++oc) {
        if (oc == 0) {
          if (m > 0) static_for<NKR>([&](auto ki) { issue_x(ki, m, decltype(ki)::value); });
          static_for<NKR>([&](auto kci) {
            constexpr int kc = decltype(kci)::value;
            publish_x(kci, buf);
            __syncthreads();
            read_x(buf, xres[kc]);
            buf ^= 1;
          });
        } else {
          __syncthreads();
        }
        const int noc = oc + 1 < n_oc ? oc + 1 : 0;
        static_for<NKR>([&](auto ki) { issue_w(ki, noc, decltype(ki)::value); });
        zero_acc();
        static_for<NKR>([&](auto kci) {
          constexpr int kc = decltype(kci)::value;
          mma_step(oc, reg * NKR + kc, xres[kc]);
          // keep each step's operand reads with its MFMAs (hoisting all of
          // them ahead would need more registers than two waves per SIMD have)
          __builtin_amdgcn_sched_barrier(0);
        });
        static_for<NKR>([&](auto ki) { store_w(ki, (reg ^ 1) * NKR + decltype(ki)::value); });
        epilogue(m, oc);
        reg ^= 1;
      }
    }
  } else {
    // Streamed weights, step s with coordinates (m, oc, kc); weight block of
    // step s in register set s & 1 and LDS buffer s & 1, spectrum in xl[s & 1]:
    //   publish X(s); barrier: X(s), W(s) visible, step s-1 finished everywhere
    //   issue W(s+2) into set s & 1 (stored to LDS at step s-1), activations
    //     of s+1; MFMA(s); store W(s+1) (issued at step s-1) to LDS (s+1) & 1
    // so each weight load has two steps to arrive.
    const int total = rounds * n_oc * nks;
    int s = 0, m = 0, oc = 0, kc = 0;
    if constexpr (DMA) {
      dma_w(0, 0, 0);
      issue_x(I0{}, 0, 0);
    } else {
      issue_w(I0{}, 0, 0);
      issue_x(I0{}, 0, 0);
      if (total > 1) issue_w(I1{}, nks > 1 ? 0 : (n_oc > 1 ? 1 : 0), nks > 1 ? 1 : 0);
      store_w(I0{}, 0);
    }
    auto step = [&](auto par) __attribute__((always_inline)) {
      constexpr int P = decltype(par)::value;
      if (kc == 0) zero_acc();
      int m1 = m, oc1 = oc, kc1 = kc + 1;  // step s+1
      if (kc1 == nks) { kc1 = 0; if (++oc1 == n_oc) { oc1 = 0; ++m1; } }
      int oc2 = oc1, kc2 = kc1 + 1;        // weight block of step s+2
      if (kc2 == nks) { kc2 = 0; if (++oc2 == n_oc) oc2 = 0; }
      publish_x(I0{}, P);
      if constexpr (DMA) {
        // W(s), loaded into LDS block P during step s-1, complete for this
        // wave (vmcnt 0; the compiler does not track LDS-direct loads), then
        // visible to all after the barrier, which also frees block 1 - P
        // (read in step s-1) for W(s+1)
        __builtin_amdgcn_s_waitcnt(0x0F70);
        __syncthreads();
        dma_w(1 - P, oc1, kc1);  // past the last step: a valid block, never read
      } else {
        __syncthreads();
        if (s + 2 < total) issue_w(par, oc2, kc2);
      }
      issue_x(I0{}, m1, kc1);
      read_x(P, bcur);
      mma_step(oc, P, bcur);
      if constexpr (!DMA) {
        if (s + 1 < total) store_w(std::integral_constant<int, 1 - P>{}, 1 - P);
      }
      if (kc == nks - 1) epilogue(m, oc);
      m = m1; oc = oc1; kc = kc1; ++s;
    };
    while (true) {
      step(I0{});
      if (s >= total) break;
      step(I1{});
      if (s >= total) break;
    }
  }
}

}  // namespace eqk
