// eql_kernels.h -- gfx950 kernel templates of the C_T equivariant linear layer.
//
//   eql_wspec_kernel        weight spectrum (Alg. 1 step 1 applied to the shared
//                           parameters, Sec. 3.2.1 Eq. 4), stored as T real planes
//   (eql_gemm_kernel, the forward and input-gradient kernel, is in eql_gemm.h)
//   eql_wgrad_kernel        weight gradient, split over rows: spectra of x and dy,
//                           per-bin conj(X)^T dY on MFMA, fp32 partials per split
//   eql_wgrad_reduce_kernel fixed-order sum of the split partials, irDFT, db
//
// Layout conventions (row-major): x[N,Cin,T], y[N,Cout,T], w[T,Cout,Cin].
#pragma once
#include "eql_common.h"

namespace eqk {

// ---------------------------------------------------------------------------
// Weight spectrum.  For every (o, c): the T lags w[0..T-1, o, c] are transformed
// by the same real DFT as the activations, giving What_k[o, c] in plane form.
// Two zero-padded copies are written:
//   forward  layout  F[p][o][c], dims [T][CoF][CiF]     (A operand of the forward)
//   backward layout  B[p][c][o], dims [T][CinB][CoutB]  (A operand of the input gradient)
// Threads [0, CoF*CiF) fill F with c fastest; the next CinB*CoutB threads fill
// B with o fastest, so both sets of stores are coalesced.
template <int T, bool F16>
__global__ __launch_bounds__(256) void eql_wspec_kernel(const void* __restrict__ w,
                                                        void* __restrict__ wspec, int Cin, int Cout,
                                                        int CoF, int CiF, int CinB, int CoutB) {
  using E = typename Elem<F16>::T;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t nF = (int64_t)CoF * CiF;
  const int64_t nB = (int64_t)CinB * CoutB;
  int o, c;
  bool toF;
  if (idx < nF) {
    o = (int)(idx / CiF);
    c = (int)(idx - (int64_t)o * CiF);
    toF = true;
  } else if (idx < nF + nB) {
    const int64_t j = idx - nF;
    c = (int)(j / CoutB);
    o = (int)(j - (int64_t)c * CoutB);
    toF = false;
  } else {
    return;
  }
  float v[T];
  const E* wp = reinterpret_cast<const E*>(w);
  const bool ok = o < Cout && c < Cin;
#pragma unroll
  for (int j = 0; j < T; ++j) v[j] = ok ? (float)wp[((int64_t)j * Cout + o) * Cin + c] : 0.0f;
  float P[T];
  rdft<T>(v, P);
  E* F = reinterpret_cast<E*>(wspec);
  if (toF) {
#pragma unroll
    for (int p = 0; p < T; ++p) F[((int64_t)p * CoF + o) * CiF + c] = (E)P[p];
  } else {
    E* Bl = F + (int64_t)T * CoF * CiF;
#pragma unroll
    for (int p = 0; p < T; ++p) Bl[((int64_t)p * CinB + c) * CoutB + o] = (E)P[p];
  }
}

// ---------------------------------------------------------------------------
// Weight gradient, one split of rows.
//   H_k[c,o] = sum_n conj(Xhat_k[n,c]) dYhat_k[n,o]
// complex bin (r, i):  Re H += Xr Dr + Xi Di,  Im H += Xr Di - Xi Dr.
// One workgroup of 4 waves (2 x 2) owns BC input x BO output channels, all T
// planes, over rows [split*rows_per_split, ...).  Per chunk of KR rows the
// prologue transforms x and dy rows and stages both spectra in LDS with the
// row index contiguous (the MFMA contraction index); MFMA computes
// D[c][o] = sum_n A[c][n] B[n][o].  The fp32 partial goes to
// part[split][p][o][c] (dims [S][T][Cout_pad][Cin_pad]); tiles with ct == 0
// also write the split's bias-gradient partial sum_n dYhat_0[n,o] (kept in
// fp32 before any rounding) to dbpart[split][o].
template <int T, bool F16, int BC, int BO>
__global__ __launch_bounds__(256) void eql_wgrad_kernel(const void* __restrict__ x,
                                                        const void* __restrict__ dy,
                                                        float* __restrict__ part,
                                                        float* __restrict__ dbpart, int64_t N,
                                                        int Cin, int Cout, int64_t rows_per_split,
                                                        int n_ct, int n_ot, int n_tiles, int Cin_pad,
                                                        int Cout_pad) {
  using MM = Mma<F16>;
  using Bn = Bins<T>;
  constexpr int EB = Elem<F16>::bytes;
  constexpr int KR = 64 / EB;  // rows per chunk (32 f16, 16 f32)
  constexpr int RGX = KR * BC / 256;
  constexpr int RGD = KR * BO / 256;
  constexpr int WC = BC / 2;
  constexpr int WD = BO / 2;
  constexpr int CT = WC / 16;
  constexpr int OT = WD / 16;
  static_assert(RGX >= 1 && RGD >= 1 && CT >= 1 && OT >= 1, "tile shape");

  __shared__ __attribute__((aligned(16))) char xs[T * BC * 64];
  __shared__ __attribute__((aligned(16))) char ds[T * BO * 64];

  const int tile = xcd_tile(blockIdx.x, gridDim.x, n_tiles);
  if (tile < 0) return;
  const int per_split = n_ct * n_ot;
  const int split = tile / per_split;
  const int rem = tile - split * per_split;
  const int ct = rem / n_ot;
  const int ot = rem - ct * n_ot;
  const int64_t n_begin = (int64_t)split * rows_per_split;
  const int64_t n_end = (n_begin + rows_per_split < N) ? n_begin + rows_per_split : N;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int g = lane >> 4;
  const int li = lane & 15;
  const int wc = wave >> 1;
  const int wo = wave & 1;

  floatx4 acc[T][CT][OT];
#pragma unroll
  for (int p = 0; p < T; ++p)
#pragma unroll
    for (int a = 0; a < CT; ++a)
#pragma unroll
      for (int b = 0; b < OT; ++b) acc[p][a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int pc = tid % BC;
  const int prg = tid / BC;
  const int po = tid % BO;
  const int prgd = tid / BO;
  const int c = ct * BC + pc;
  const int o = ot * BO + po;
  const bool x_vec = ((int64_t)Cin * T * EB) % run_vec_bytes<F16, T>() == 0;
  const bool d_vec = ((int64_t)Cout * T * EB) % run_vec_bytes<F16, T>() == 0;
  float dbacc = 0.0f;

  for (int64_t n0 = n_begin; n0 < n_end; n0 += KR) {
    float Px[T][RGX];
    float Pd[T][RGD];
#pragma unroll
    for (int r = 0; r < RGX; ++r) {
      const int64_t n = n0 + prg * RGX + r;
      float v[T], s[T];
      if (n < n_end && c < Cin) {
        load_run<F16, T>(x, (n * Cin + c) * T, x_vec, v);
      } else {
#pragma unroll
        for (int t = 0; t < T; ++t) v[t] = 0.0f;
      }
      rdft<T>(v, s);
#pragma unroll
      for (int p = 0; p < T; ++p) Px[p][r] = s[p];
    }
#pragma unroll
    for (int r = 0; r < RGD; ++r) {
      const int64_t n = n0 + prgd * RGD + r;
      float v[T], s[T];
      if (n < n_end && o < Cout) {
        load_run<F16, T>(dy, (n * Cout + o) * T, d_vec, v);
      } else {
#pragma unroll
        for (int t = 0; t < T; ++t) v[t] = 0.0f;
      }
      rdft<T>(v, s);
      dbacc += s[0];
#pragma unroll
      for (int p = 0; p < T; ++p) Pd[p][r] = s[p];
    }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < T; ++p) {
      pack_store_lds<F16, RGX>(xs, p * BC * 64 + lds_off(pc, prg * RGX * EB), Px[p]);
      pack_store_lds<F16, RGD>(ds, p * BO * 64 + lds_off(po, prgd * RGD * EB), Pd[p]);
    }
    __syncthreads();

#pragma unroll
    for (int a = 0; a < CT; ++a) {
      const int cl = wc * WC + a * 16 + li;
      u32x4 A[T];
#pragma unroll
      for (int p = 0; p < T; ++p)
        A[p] = *reinterpret_cast<const u32x4*>(xs + p * BC * 64 + lds_off(cl, g * 16));
#pragma unroll
      for (int b = 0; b < OT; ++b) {
        const int ol = wo * WD + b * 16 + li;
        u32x4 Bf[T];
#pragma unroll
        for (int p = 0; p < T; ++p)
          Bf[p] = *reinterpret_cast<const u32x4*>(ds + p * BO * 64 + lds_off(ol, g * 16));
        MM::run(acc[0][a][b], A[0], Bf[0]);
        if constexpr (Bn::kEven) MM::run(acc[1][a][b], A[1], Bf[1]);
        static_for<Bn::K>([&](auto ki) {
          constexpr int k = decltype(ki)::value + 1;
          constexpr int r = Bn::re(k);
          constexpr int i = Bn::im(k);
          MM::run(acc[r][a][b], A[r], Bf[r]);
          MM::run(acc[r][a][b], A[i], Bf[i]);
          MM::run(acc[i][a][b], A[r], Bf[i]);
          MM::run(acc[i][a][b], MM::neg(A[i]), Bf[r]);
        });
      }
    }
  }

  // ---- partials: lane holds D[c = 4g + r][o = li] of each 16 x 16 sub-tile
#pragma unroll
  for (int a = 0; a < CT; ++a) {
    const int cc = ct * BC + wc * WC + a * 16 + 4 * g;
#pragma unroll
    for (int b = 0; b < OT; ++b) {
      const int oo = ot * BO + wo * WD + b * 16 + li;
#pragma unroll
      for (int p = 0; p < T; ++p) {
        float* dst = part + (((int64_t)split * T + p) * Cout_pad + oo) * Cin_pad + cc;
        *reinterpret_cast<floatx4*>(dst) = acc[p][a][b];
      }
    }
  }
  if (ct == 0 && dbpart != nullptr) {
    __syncthreads();
    float* red = reinterpret_cast<float*>(xs);
    red[tid] = dbacc;
    __syncthreads();
    if (tid < BO) {
      float s = 0.0f;
#pragma unroll
      for (int q = 0; q < 256 / BO; ++q) s += red[q * BO + tid];
      dbpart[(int64_t)split * Cout_pad + ot * BO + tid] = s;
    }
  }
}

// Fixed-order sum of the S split partials, then the inverse transform over
// the planes: dw[j,o,c] = (1/T) sum_k H_k[c,o] e^{+2 pi i k j/T}, conjugate bins
// folded into weight 2 (the same inverse as the forward epilogue).  A
// workgroup takes 256 consecutive (o, c) pairs: thread t sums plane p of pair
// t for every p (coalesced over c), then transforms its pair.  The last
// workgroup (when db is requested) sums the bias-gradient partials.
template <int T, bool F16>
__global__ __launch_bounds__(256) void eql_wgrad_reduce_kernel(const float* __restrict__ part,
                                                               const float* __restrict__ dbpart,
                                                               void* __restrict__ dw,
                                                               void* __restrict__ db, int S,
                                                               int Cin, int Cout, int Cin_pad,
                                                               int Cout_pad) {
  using E = typename Elem<F16>::T;
  const int64_t pairs = (int64_t)Cout * Cin;
  const int64_t nblk = (pairs + 255) / 256;
  const int tid = threadIdx.x;
  if ((int64_t)blockIdx.x == nblk) {  // bias gradient
    if (db == nullptr) return;
    for (int o = tid; o < Cout; o += 256) {
      float s = 0.0f;
      for (int sp = 0; sp < S; ++sp) s += dbpart[(int64_t)sp * Cout_pad + o];
      reinterpret_cast<E*>(db)[o] = (E)s;
    }
    return;
  }
  const int64_t idx = (int64_t)blockIdx.x * 256 + tid;
  if (idx >= pairs) return;
  const int o = (int)(idx / Cin);
  const int c = (int)(idx - (int64_t)o * Cin);
  const int64_t split_stride = (int64_t)T * Cout_pad * Cin_pad;
  const float* src = part + (int64_t)o * Cin_pad + c;
  float P[T];
#pragma unroll
  for (int p = 0; p < T; ++p) P[p] = 0.0f;
  int sp = 0;
  for (; sp + 4 <= S; sp += 4) {
#pragma unroll
    for (int p = 0; p < T; ++p) {
      const float* q = src + (int64_t)p * Cout_pad * Cin_pad + sp * split_stride;
      const float a0 = q[0], a1 = q[split_stride], a2 = q[2 * split_stride], a3 = q[3 * split_stride];
      P[p] = (((P[p] + a0) + a1) + a2) + a3;
    }
  }
  for (; sp < S; ++sp) {
#pragma unroll
    for (int p = 0; p < T; ++p) P[p] += src[(int64_t)p * Cout_pad * Cin_pad + sp * split_stride];
  }
  float u[T];
  irdft<T>(P, u);
  E* d = reinterpret_cast<E*>(dw);
#pragma unroll
  for (int j = 0; j < T; ++j) d[((int64_t)j * Cout + o) * Cin + c] = (E)u[j];
}

}  // namespace eqk
