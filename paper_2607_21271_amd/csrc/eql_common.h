// eql_common.h -- device building blocks shared by the gfx950 kernels of the
// C_T equivariant linear layer (Flash EQ-Linear, arXiv 2607.21271).
//
//  * compile-time twiddles cos/sin(2*pi*m/T), evaluated in double and rounded
//    once to float, so no device sin/cos is ever called;
//  * the real DFT along the group axis, keeping the non-redundant bins
//    k = 0..floor(T/2) (Alg. 1 step 1, Sec. 3.2.1 Eq. 4), and its inverse with
//    conjugate pairs folded into weights 2 (Alg. 1 steps 3-4, Eq. 6-7 and the
//    conjugate-pair form of Appendix A.1);
//  * MFMA fragment helpers for v_mfma_f32_16x16x32_f16 and
//    v_mfma_f32_16x16x4_f32.
//
// Spectral planes.  A length-T real signal is held as exactly T reals:
//   plane 0            Re X_0                       (bin 0 is real)
//   plane 1            X_{T/2}        (even T only; the Nyquist bin is real)
//   plane R+2(k-1)     Re X_k,  k = 1..K
//   plane R+2(k-1)+1   Im X_k
// with R = 1 + [T even] real bins and K = floor((T-1)/2) complex bins, so that
// R + 2K = T.  The forward transform is unnormalised, X_k = sum_t x_t e^{-2 pi i k t/T};
// the inverse carries the 1/T.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "eql_config.h"

namespace eqk {

// ---------------------------------------------------------------------------
// Compile-time twiddles.
constexpr double kPi = 3.14159265358979323846264338327950288;

constexpr double cos_series(double x) {  // |x| <= pi; Taylor series, 40 terms
  double term = 1.0, sum = 1.0;
  const double x2 = x * x;
  for (int i = 1; i < 40; ++i) {
    term *= -x2 / ((2.0 * i - 1.0) * (2.0 * i));
    sum += term;
  }
  return sum;
}

// cos(2*pi*m/T) with exact values at the quarter points.
constexpr double cos2pi(long m, long T) {
  m %= T;
  if (m < 0) m += T;
  if (m == 0) return 1.0;
  if (2 * m == T) return -1.0;
  if (4 * m == T || 4 * m == 3 * T) return 0.0;
  double x = 2.0 * kPi * (double)m / (double)T;
  if (x > kPi) x -= 2.0 * kPi;
  return cos_series(x);
}

// sin(2*pi*m/T) = cos(2*pi*(4m - T)/(4T)).
constexpr double sin2pi(long m, long T) { return cos2pi(4 * m - T, 4 * T); }

template <int T>
struct Bins {
  static constexpr int R = 1 + (T % 2 == 0 ? 1 : 0);  // real bins
  static constexpr int K = (T - 1) / 2;               // complex bins
  static constexpr int S = (T - 1) / 2;               // symmetric pairs (s, T-s)
  static constexpr bool kEven = (T % 2 == 0);
  static constexpr int re(int k) { return R + 2 * (k - 1); }
  static constexpr int im(int k) { return R + 2 * (k - 1) + 1; }
};

template <typename F, int... I>
__host__ __device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
// f(integral_constant<int, i>) for i = 0..N-1, fully unrolled at compile time.
template <int N, typename F>
__host__ __device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Arithmetic of the transforms, as a policy: F32Ops holds one value per
// element in fp32 (H2Ops, with the element types below, holds two independent
// signals in the halves of a packed fp16 register).
struct F32Ops {
  using V = float;
  static __device__ __forceinline__ V zero() { return 0.0f; }
  static __device__ __forceinline__ V fma(float c, V x, V y) { return __builtin_fmaf(c, x, y); }
  static __device__ __forceinline__ V mul(float c, V x) { return c * x; }
};

// acc += C * v for a compile-time constant C; terms with C = 0 vanish and
// C = +-1 become an add or a subtract.
template <float C, typename A = F32Ops>
__device__ __forceinline__ void axpy_c(typename A::V& acc, typename A::V v) {
  if constexpr (C == 1.0f) {
    acc += v;
  } else if constexpr (C == -1.0f) {
    acc -= v;
  } else if constexpr (C != 0.0f) {
    acc = A::fma(C, v, acc);
  }
}

// ---------------------------------------------------------------------------
// Real DFT of v[0..T-1] into T spectral planes (layout above).  Input pairs
// (s, T-s) are folded into e_s = v_s + v_{T-s} and d_s = v_s - v_{T-s} so
// that each bin takes about T/2 multiply-adds:
//   Re X_k = v_0 + (-1)^k v_{T/2} + sum_s e_s cos(2 pi k s/T)
//   Im X_k = -sum_s d_s sin(2 pi k s/T)
template <int T, typename A = F32Ops>
__device__ __forceinline__ void rdft_direct(const typename A::V (&v)[T], typename A::V (&P)[T]) {
  using V = typename A::V;
  using B = Bins<T>;
  constexpr int S = B::S;
  V e[S + 1], d[S + 1];
  static_for<S>([&](auto si) {
    constexpr int s = decltype(si)::value + 1;
    e[s] = v[s] + v[T - s];
    d[s] = v[s] - v[T - s];
  });
  V a = v[0];
  static_for<S>([&](auto si) { a += e[decltype(si)::value + 1]; });
  if constexpr (B::kEven) a += v[T / 2];
  P[0] = a;
  if constexpr (B::kEven) {
    V b = v[0];
    static_for<S>([&](auto si) {
      constexpr int s = decltype(si)::value + 1;
      if constexpr (s & 1) b -= e[s]; else b += e[s];
    });
    if constexpr ((T / 2) & 1) b -= v[T / 2]; else b += v[T / 2];
    P[1] = b;
  }
  static_for<B::K>([&](auto ki) {
    constexpr int k = decltype(ki)::value + 1;
    V re = v[0];
    V im = A::zero();
    static_for<S>([&](auto si) {
      constexpr int s = decltype(si)::value + 1;
      axpy_c<(float)cos2pi((long)k * s, T), A>(re, e[s]);
      axpy_c<(float)-sin2pi((long)k * s, T), A>(im, d[s]);
    });
    if constexpr (B::kEven) {
      if constexpr (k & 1) re -= v[T / 2]; else re += v[T / 2];
    }
    P[B::re(k)] = re;
    P[B::im(k)] = im;
  });
}

// Inverse real DFT of T spectral planes, u_t = (1/T) sum_{k=0}^{T-1} X_k e^{2 pi i k t/T},
// with the conjugate bins folded in:
//   u_t = (X_0 + (-1)^t X_{T/2})/T + (2/T) sum_{k=1}^{K} (Re X_k cos(2 pi k t/T) - Im X_k sin(2 pi k t/T)).
// Output pairs (t, T-t) share the even part E_t and differ in the sign of the odd part O_t.
template <int T>
__device__ __forceinline__ void irdft_direct(const float (&P)[T], float (&u)[T]) {
  using B = Bins<T>;
  constexpr int S = B::S;
  constexpr float inv = (float)(1.0 / T);
  float A = P[0] * inv;
  float Bn = 0.0f;
  if constexpr (B::kEven) Bn = P[1] * inv;
  const float base_e = A + Bn;  // (-1)^t = +1
  const float base_o = A - Bn;  // (-1)^t = -1
  static_for<S>([&](auto ti) {
    constexpr int t = decltype(ti)::value + 1;
    float E = 0.0f, O = 0.0f;
    static_for<B::K>([&](auto ki) {
      constexpr int k = decltype(ki)::value + 1;
      axpy_c<(float)(2.0 * cos2pi((long)k * t, T) / T)>(E, P[B::re(k)]);
      axpy_c<(float)(2.0 * sin2pi((long)k * t, T) / T)>(O, P[B::im(k)]);
    });
    const float base = (t & 1) ? base_o : base_e;
    u[t] = base + (E - O);
    u[T - t] = base + (E + O);
  });
  float u0 = base_e;
  static_for<B::K>([&](auto ki) {
    constexpr int k = decltype(ki)::value + 1;
    axpy_c<(float)(2.0 / T)>(u0, P[B::re(k)]);
  });
  u[0] = u0;
  if constexpr (B::kEven) {
    float uh = ((T / 2) & 1) ? base_o : base_e;
    static_for<B::K>([&](auto ki) {
      constexpr int k = decltype(ki)::value + 1;
      axpy_c<(float)((k & 1 ? -2.0 : 2.0) / T)>(uh, P[B::re(k)]);
    });
    u[T / 2] = uh;
  }
}

// ---------------------------------------------------------------------------
// FFT forms for T = 4, 8, 16 (same planes, same results up to rounding order).
//
// T = 4: two length-2 butterflies.  Planes: 0 X0, 1 X2, 2 Re X1, 3 Im X1.
template <typename A = F32Ops>
__device__ __forceinline__ void rdft4(const typename A::V (&v)[4], typename A::V (&P)[4]) {
  const typename A::V a0 = v[0] + v[2], a1 = v[1] + v[3];
  P[0] = a0 + a1;
  P[1] = a0 - a1;
  P[2] = v[0] - v[2];
  P[3] = v[3] - v[1];
}
__device__ __forceinline__ void irdft4(const float (&P)[4], float (&u)[4]) {
  const float e = (P[0] + P[1]) * 0.25f, o = (P[0] - P[1]) * 0.25f;
  u[0] = __builtin_fmaf(0.5f, P[2], e);
  u[2] = __builtin_fmaf(-0.5f, P[2], e);
  u[1] = __builtin_fmaf(-0.5f, P[3], o);
  u[3] = __builtin_fmaf(0.5f, P[3], o);
}

// T = 8: radix-2 split on (s, s+4), a DFT4 of the sums for the even bins and a
// twiddled DFT4 of the differences for the odd bins.
// Planes: 0 X0, 1 X4, 2/3 Re/Im X1, 4/5 Re/Im X2, 6/7 Re/Im X3.
constexpr float kR2 = 0.70710678118654752440f;  // 1/sqrt(2)
template <typename A = F32Ops>
__device__ __forceinline__ void rdft8(const typename A::V (&v)[8], typename A::V (&P)[8]) {
  using V = typename A::V;
  const V a0 = v[0] + v[4], a1 = v[1] + v[5], a2 = v[2] + v[6], a3 = v[3] + v[7];
  const V b0 = v[0] - v[4], b1 = v[1] - v[5], b2 = v[2] - v[6], b3 = v[3] - v[7];
  const V s02 = a0 + a2, s13 = a1 + a3;
  P[0] = s02 + s13;
  P[1] = s02 - s13;
  P[4] = a0 - a2;
  P[5] = a3 - a1;
  const V p = b1 - b3, q = b1 + b3;
  P[2] = A::fma(kR2, p, b0);
  P[6] = A::fma(-kR2, p, b0);
  P[3] = A::fma(-kR2, q, -b2);
  P[7] = A::fma(-kR2, q, b2);
}
// Inverse: even outputs from X0+X4, Re X2 and the sums/differences of bins 1
// and 3; odd outputs from X0-X4, Im X2 and bins 1, 3 rotated by e^{i pi/4}.
__device__ __forceinline__ void irdft8(const float (&P)[8], float (&u)[8]) {
  constexpr float h = 0.125f, q = 0.25f, qr = 0.25f * kR2;
  const float A = (P[0] + P[1]) * h, Bo = (P[0] - P[1]) * h;
  const float S = P[2] + P[6], D = P[7] - P[3];
  const float e1 = __builtin_fmaf(q, P[4], A), e2 = __builtin_fmaf(-q, P[4], A);
  u[0] = __builtin_fmaf(q, S, e1);
  u[4] = __builtin_fmaf(-q, S, e1);
  u[2] = __builtin_fmaf(q, D, e2);
  u[6] = __builtin_fmaf(-q, D, e2);
  const float t1 = P[2] - P[3], t2 = P[6] + P[7], t3 = P[6] - P[7], t4 = P[2] + P[3];
  const float sd = t1 - t2, dd = t3 - t4;
  const float o1 = __builtin_fmaf(-q, P[5], Bo), o2 = __builtin_fmaf(q, P[5], Bo);
  u[1] = __builtin_fmaf(qr, sd, o1);
  u[5] = __builtin_fmaf(-qr, sd, o1);
  u[3] = __builtin_fmaf(qr, dd, o2);
  u[7] = __builtin_fmaf(-qr, dd, o2);
}

// T = 16: two DFT8 of the even and odd samples, combined with the twiddles
// w^k = e^{-i pi k/8}: X_k = E_k + w^k O_k and X_{8-k} = conj(E_k - w^k O_k).
// Planes: 0 X0, 1 X8, 2k/2k+1 Re/Im X_k for k = 1..7.
template <typename A = F32Ops>
__device__ __forceinline__ void rdft16(const typename A::V (&v)[16], typename A::V (&P)[16]) {
  using V = typename A::V;
  V ve[8], vo[8], E[8], O[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) { ve[i] = v[2 * i]; vo[i] = v[2 * i + 1]; }
  rdft8<A>(ve, E);
  rdft8<A>(vo, O);
  // E, O planes: 0 X0, 1 X4, 2/3 X1, 4/5 X2, 6/7 X3 (length-8 spectra)
  P[0] = E[0] + O[0];
  P[1] = E[0] - O[0];
  // k = 4: w^4 = -i and E_4, O_4 are the (real) Nyquist bins of E and O
  P[8] = E[1];
  P[9] = -O[1];
  constexpr float c1 = 0.92387953251128675613f, s1 = 0.38268343236508977173f;  // cos, sin(pi/8)
  // k = 1: Z = w O1 = (c - i s)(Or + i Oi)
  {
    const V zr = A::fma(c1, O[2], A::mul(s1, O[3]));
    const V zi = A::fma(c1, O[3], A::mul(-s1, O[2]));
    P[2] = E[2] + zr; P[3] = E[3] + zi;      // X1
    P[14] = E[2] - zr; P[15] = zi - E[3];    // X7 = conj(E1 - Z)
  }
  // k = 2: w^2 = (1 - i)/sqrt2, uses E2/O2 planes 4/5
  {
    const V zr = A::mul(kR2, O[4] + O[5]);
    const V zi = A::mul(kR2, O[5] - O[4]);
    P[4] = E[4] + zr; P[5] = E[5] + zi;      // X2
    P[12] = E[4] - zr; P[13] = zi - E[5];    // X6
  }
  // k = 3: w^3 = (s - i c), uses E3/O3 planes 6/7
  {
    const V zr = A::fma(s1, O[6], A::mul(c1, O[7]));
    const V zi = A::fma(s1, O[7], A::mul(-c1, O[6]));
    P[6] = E[6] + zr; P[7] = E[7] + zi;      // X3
    P[10] = E[6] - zr; P[11] = zi - E[7];    // X5
  }
}
// Inverse: even outputs are irdft8 of A_k = X_k + X_{k+8}, odd outputs irdft8
// of B_k = (X_k - X_{k+8}) e^{i pi k/8}, each times 1/2.
__device__ __forceinline__ void irdft16(const float (&P)[16], float (&u)[16]) {
  // X_k (k = 1..7): Re P[2k], Im P[2k+1]; X_0 = P[0], X_8 = P[1].
  // X_{k+8} = conj(X_{8-k}) for k = 1..4.
  float A[8], Bq[8];
  A[0] = 0.5f * (P[0] + P[1]);
  Bq[0] = 0.5f * (P[0] - P[1]);
  A[1] = 0.5f * (2.0f * P[8]);   // A_4 = 2 Re X4, length-8 Nyquist plane
  Bq[1] = 0.5f * (-2.0f * P[9]); // B_4 = -2 Im X4
  constexpr float c1 = 0.92387953251128675613f, s1 = 0.38268343236508977173f;
  // k = 1: A1 = X1 + conj(X7); B1 = (X1 - conj(X7)) e^{i pi/8}
  {
    const float ar = P[2] + P[14], ai = P[3] - P[15];
    const float dr = P[2] - P[14], di = P[3] + P[15];
    A[2] = 0.5f * ar; A[3] = 0.5f * ai;
    Bq[2] = 0.5f * __builtin_fmaf(c1, dr, -s1 * di);
    Bq[3] = 0.5f * __builtin_fmaf(c1, di, s1 * dr);
  }
  // k = 2: with X6; rotation e^{i pi/4}
  {
    const float ar = P[4] + P[12], ai = P[5] - P[13];
    const float dr = P[4] - P[12], di = P[5] + P[13];
    A[4] = 0.5f * ar; A[5] = 0.5f * ai;
    Bq[4] = (0.5f * kR2) * (dr - di);
    Bq[5] = (0.5f * kR2) * (di + dr);
  }
  // k = 3: with X5; rotation e^{i 3pi/8} = (s1 + i c1)
  {
    const float ar = P[6] + P[10], ai = P[7] - P[11];
    const float dr = P[6] - P[10], di = P[7] + P[11];
    A[6] = 0.5f * ar; A[7] = 0.5f * ai;
    Bq[6] = 0.5f * __builtin_fmaf(s1, dr, -c1 * di);
    Bq[7] = 0.5f * __builtin_fmaf(s1, di, c1 * dr);
  }
  float ue[8], uo[8];
  irdft8(A, ue);
  irdft8(Bq, uo);
#pragma unroll
  for (int m = 0; m < 8; ++m) { u[2 * m] = ue[m]; u[2 * m + 1] = uo[m]; }
}

// Dispatch: FFT forms where written, the symmetric direct form otherwise.
template <int T, typename A = F32Ops>
__device__ __forceinline__ void rdft(const typename A::V (&v)[T], typename A::V (&P)[T]) {
  if constexpr (T == 4) rdft4<A>(v, P);
  else if constexpr (T == 8) rdft8<A>(v, P);
  else if constexpr (T == 16) rdft16<A>(v, P);
  else rdft_direct<T, A>(v, P);
}
template <int T>
__device__ __forceinline__ void irdft(const float (&P)[T], float (&u)[T]) {
  if constexpr (T == 4) irdft4(P, u);
  else if constexpr (T == 8) irdft8(P, u);
  else if constexpr (T == 16) irdft16(P, u);
  else irdft_direct<T>(P, u);
}

// ---------------------------------------------------------------------------
// Element types, by their codes (eql_config.h).  Products accumulate in
// fp32; the inverse transforms and the weight spectrum are computed in fp32.
// Forward transforms of fp16 data run in packed fp16 arithmetic (H2Ops);
// those of bf16 data (8 significand bits, too few for transform arithmetic)
// in fp32, each result rounded once to bf16 as an MFMA operand.
template <int DT>
struct Elem;
template <>
struct Elem<kF16> {
  using T = _Float16;
  static constexpr int bytes = 2;
};
template <>
struct Elem<kBF16> {
  using T = __bf16;
  static constexpr int bytes = 2;
};
template <>
struct Elem<kF32> {
  using T = float;
  static constexpr int bytes = 4;
};

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));

// Transform arithmetic on two independent signals held in the two halves of
// packed fp16 registers (v_pk_add/v_pk_fma_f16), twiddles rounded to fp16.
struct H2Ops {
  using V = half2v;
  static __device__ __forceinline__ V zero() { return V{(_Float16)0.0f, (_Float16)0.0f}; }
  static __device__ __forceinline__ V fma(float c, V x, V y) {
    const _Float16 h = (_Float16)c;
    return __builtin_elementwise_fma(V{h, h}, x, y);
  }
  static __device__ __forceinline__ V mul(float c, V x) {
    const _Float16 h = (_Float16)c;
    return V{h, h} * x;
  }
};

// One packed register from two fp16 words: half ha of word a in the low half,
// half hb of word b in the high half.
template <int ha, int hb>
__device__ __forceinline__ half2v pair_halves(uint32_t a, uint32_t b) {
  constexpr uint32_t sel = (ha ? 0x0302u : 0x0100u) | ((hb ? 0x0706u : 0x0504u) << 16);
  return __builtin_bit_cast(half2v, __builtin_amdgcn_perm(b, a, sel));
}
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Raw words -> floats (fp16: two elements per word, low half first; fp32:
// one).  Each fp16 word is read exactly once, by one asm statement that
// converts both halves.  (With the halves read by separate instructions the
// compiler, in some kernels, reused a word's register after its first read
// and the second read then saw the converted value.)
__device__ __forceinline__ void f16x2_to_f32(uint32_t w, float& lo, float& hi) {
  asm("v_cvt_f32_f16_e32 %0, %2\n\t"
      "v_cvt_f32_f16_sdwa %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_1"
      : "=&v"(lo), "=v"(hi)
      : "v"(w));
}
// bf16 word -> the floats of its two halves (low half first); exact
__device__ __forceinline__ void bf16x2_to_f32(uint32_t w, float& lo, float& hi) {
  lo = __builtin_bit_cast(float, w << 16);
  hi = __builtin_bit_cast(float, w & 0xffff0000u);
}
template <int DT, int NW>
__device__ __forceinline__ void raw_to_floats(const uint32_t* r, float (&f)[DT != kF32 ? 2 * NW : NW]) {
#pragma unroll
  for (int v = 0; v < NW; ++v) {
    if constexpr (DT == kF16) f16x2_to_f32(r[v], f[2 * v], f[2 * v + 1]);
    else if constexpr (DT == kBF16) bf16x2_to_f32(r[v], f[2 * v], f[2 * v + 1]);
    else f[v] = __builtin_bit_cast(float, r[v]);
  }
}

// Two floats rounded to the 16-bit type (round to nearest even) and packed,
// a in the low half; fp32: a alone.
template <int DT>
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  if constexpr (DT != kF32) {
    using E = typename Elem<DT>::T;
    const uint16_t lo = __builtin_bit_cast(uint16_t, (E)a);
    const uint16_t hi = __builtin_bit_cast(uint16_t, (E)b);
    return (uint32_t)lo | ((uint32_t)hi << 16);
  } else {
    return __builtin_bit_cast(uint32_t, a);
  }
}

// ---------------------------------------------------------------------------
// Contiguous store of L elements at an element offset, converting from float.
// VEC is the widest power-of-two byte width (<= 16) that divides L * elem
// bytes; the caller states whether the start is VEC-aligned.
template <int DT, int L>
__device__ __forceinline__ void store_run(void* base, int64_t elem_off, bool vec_ok, int n_valid,
                                          const float (&v)[L]) {
  using E = typename Elem<DT>::T;
  constexpr int NB = L * Elem<DT>::bytes;
  constexpr int VEC = (NB % 16 == 0) ? 16 : (NB % 8 == 0) ? 8 : (NB % 4 == 0) ? 4 : 2;
  E* p = reinterpret_cast<E*>(base) + elem_off;
  if (vec_ok && n_valid >= L && VEC >= 4) {
    constexpr int PER = VEC / Elem<DT>::bytes;
#pragma unroll
    for (int s = 0; s < L / PER; ++s) {
      E tmp[PER];
#pragma unroll
      for (int q = 0; q < PER; ++q) tmp[q] = (E)v[s * PER + q];
      if constexpr (VEC == 16) {
        u32x4 w;
        __builtin_memcpy(&w, tmp, 16);
        *reinterpret_cast<u32x4*>(p + s * PER) = w;
      } else if constexpr (VEC == 8) {
        u32x2 w;
        __builtin_memcpy(&w, tmp, 8);
        *reinterpret_cast<u32x2*>(p + s * PER) = w;
      } else {
        uint32_t w;
        __builtin_memcpy(&w, tmp, 4);
        *reinterpret_cast<uint32_t*>(p + s * PER) = w;
      }
    }
  } else {
#pragma unroll
    for (int q = 0; q < L; ++q)
      if (q < n_valid) p[q] = (E)v[q];
  }
}

}  // namespace eqk
