"""The group-axis transforms of the HIP kernels, compiled for the host, against numpy's FFT.

The real DFT / inverse real DFT device functions in
paper_2607_21271_amd/csrc/eql_common.h are plain float arithmetic; this test
extracts them, builds them with g++ and checks every T in 1..16 (direct and
FFT forms) against numpy.fft on random data, plus inverse(forward(v)) == v.
CPU only.  This checks the GPU path's building blocks, not the oracle.
"""
import ctypes
import os
import subprocess
import tempfile

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR = os.path.join(ROOT, "paper_2607_21271_amd", "csrc", "eql_common.h")

DRIVER = r'''
#include "tx.h"
extern "C" void run(int T, int fwd, const float* in, float* out, int n) {
#define CASE(t) case t: for (int r = 0; r < n; ++r) { float a[t], b[t]; \
    for (int i = 0; i < t; ++i) a[i] = in[r * t + i]; \
    if (fwd) eqk::rdft<t>(a, b); else eqk::irdft<t>(a, b); \
    for (int i = 0; i < t; ++i) out[r * t + i] = b[i]; } break;
  switch (T) { CASE(1) CASE(2) CASE(3) CASE(4) CASE(5) CASE(6) CASE(7) CASE(8)
               CASE(9) CASE(10) CASE(11) CASE(12) CASE(13) CASE(14) CASE(15) CASE(16) }
}
'''


@pytest.fixture(scope="module")
def txlib():
    src = open(HDR).read()
    a = src.index("namespace eqk {")
    b = src.index("// ---------------------------------------------------------------------------\n// Element types")
    body = (src[a:b].replace("__host__ __device__ __forceinline__", "inline")
            .replace("__device__ __forceinline__", "inline") + "}\n")
    d = tempfile.mkdtemp()
    with open(os.path.join(d, "tx.h"), "w") as f:
        f.write("#include <cmath>\n#include <cstdint>\n#include <type_traits>\n#include <utility>\n"
                "#define __builtin_fmaf fmaf\n" + body)
    with open(os.path.join(d, "tx.cpp"), "w") as f:
        f.write(DRIVER)
    so = os.path.join(d, "libtx.so")
    subprocess.run(["g++", "-O2", "-std=c++20", "-shared", "-fPIC", os.path.join(d, "tx.cpp"),
                    "-o", so], check=True)
    return ctypes.CDLL(so)


def planes(X, T):
    """numpy complex spectrum -> the kernels' T real planes (bin 0, Nyquist, Re/Im pairs)."""
    R, K = 1 + (T % 2 == 0), (T - 1) // 2
    out = np.zeros(X.shape[:-1] + (T,))
    out[..., 0] = X[..., 0].real
    if T % 2 == 0:
        out[..., 1] = X[..., T // 2].real
    for k in range(1, K + 1):
        out[..., R + 2 * (k - 1)] = X[..., k].real
        out[..., R + 2 * (k - 1) + 1] = X[..., k].imag
    return out


@pytest.mark.parametrize("T", range(1, 17))
def test_transform_matches_numpy(txlib, T):
    P = ctypes.POINTER(ctypes.c_float)
    rs = np.random.RandomState(100 + T)
    v = rs.standard_normal((400, T)).astype(np.float32)
    fwd = np.empty_like(v)
    txlib.run(T, 1, v.ctypes.data_as(P), fwd.ctypes.data_as(P), v.shape[0])
    ref = planes(np.fft.fft(v.astype(np.float64), axis=1), T)
    assert np.max(np.abs(fwd - ref)) <= 1e-6 * np.max(np.abs(ref))
    back = np.empty_like(v)
    txlib.run(T, 0, fwd.ctypes.data_as(P), back.ctypes.data_as(P), v.shape[0])
    assert np.max(np.abs(back - v)) <= 1e-6 * np.max(np.abs(v))
    # the inverse alone, on a spectrum of an independent real signal
    w = rs.standard_normal((400, T))
    inv = np.empty((400, T), np.float32)
    spec = planes(np.fft.fft(w, axis=1), T).astype(np.float32)
    txlib.run(T, 0, spec.ctypes.data_as(P), inv.ctypes.data_as(P), 400)
    assert np.max(np.abs(inv - w)) <= 1e-6 * np.max(np.abs(w))


# ---------------------------------------------------------------------------
# fp16 activations: the kernels transform x and dy in packed fp16 arithmetic
# (H2Ops in eql_common.h: two independent signals in the halves of a register,
# v_pk_add / v_pk_fma / v_pk_mul with twiddles rounded to fp16).  The same
# transform templates are built here with a host stand-in for H2Ops whose
# every add, multiply and fused multiply-add rounds its exact result to the
# nearest fp16 (ties to even), as the packed fp16 instructions do.

H2_DRIVER = r'''
#include <cmath>
#include "tx.h"
static double r16(double v) {           // round to binary16, nearest-even, with overflow to inf
  if (v == 0.0 || std::isnan(v) || std::isinf(v)) return v;
  int ex; std::frexp(std::fabs(v), &ex);  // |v| = m 2^ex, m in [0.5, 1)
  int e = ex - 1; if (e < -14) e = -14;  // subnormal spacing 2^-24
  const double step = std::ldexp(1.0, e - 10);
  const double r = std::nearbyint(std::fabs(v) / step) * step;
  return std::copysign(r > 65504.0 ? INFINITY : r, v);
}
struct H2 {
  double lo = 0.0, hi = 0.0;
  H2() = default;
  H2(double a, double b) : lo(r16(a)), hi(r16(b)) {}
  H2 operator+(H2 o) const { return H2(lo + o.lo, hi + o.hi); }
  H2 operator-(H2 o) const { return H2(lo - o.lo, hi - o.hi); }
  H2 operator-() const { H2 r; r.lo = -lo; r.hi = -hi; return r; }
  H2& operator+=(H2 o) { return *this = *this + o; }
  H2& operator-=(H2 o) { return *this = *this - o; }
};
struct HostH2Ops {
  using V = H2;
  static V zero() { return H2(0.0, 0.0); }
  static double h(float c) { return r16((double)c); }  // twiddle rounded to fp16
  static V fma(float c, V x, V y) { return H2(std::fma(h(c), x.lo, y.lo), std::fma(h(c), x.hi, y.hi)); }
  static V mul(float c, V x) { return H2(h(c) * x.lo, h(c) * x.hi); }
};
// in: n rows of two signals (lo, hi), each already fp16; out: the planes of both
extern "C" void run_h2(int T, const double* lo, const double* hi, double* plo, double* phi, int n) {
#define CASE(t) case t: for (int r = 0; r < n; ++r) { H2 a[t], b[t]; \
    for (int i = 0; i < t; ++i) a[i] = H2(lo[r * t + i], hi[r * t + i]); \
    eqk::rdft<t, HostH2Ops>(a, b); \
    for (int i = 0; i < t; ++i) { plo[r * t + i] = b[i].lo; phi[r * t + i] = b[i].hi; } } break;
  switch (T) { CASE(1) CASE(2) CASE(3) CASE(4) CASE(5) CASE(6) CASE(7) CASE(8)
               CASE(9) CASE(10) CASE(11) CASE(12) CASE(13) CASE(14) CASE(15) CASE(16) }
}
'''


@pytest.fixture(scope="module")
def h2lib():
    src = open(HDR).read()
    a = src.index("namespace eqk {")
    b = src.index("// ---------------------------------------------------------------------------\n// Element types")
    body = (src[a:b].replace("__host__ __device__ __forceinline__", "inline")
            .replace("__device__ __forceinline__", "inline") + "}\n")
    d = tempfile.mkdtemp()
    with open(os.path.join(d, "tx.h"), "w") as f:
        f.write("#include <cmath>\n#include <cstdint>\n#include <type_traits>\n#include <utility>\n"
                "#define __builtin_fmaf fmaf\n" + body)
    with open(os.path.join(d, "h2.cpp"), "w") as f:
        f.write(H2_DRIVER)
    so = os.path.join(d, "libh2.so")
    subprocess.run(["g++", "-O2", "-std=c++20", "-ffp-contract=off", "-shared", "-fPIC",
                    os.path.join(d, "h2.cpp"), "-o", so], check=True)
    return ctypes.CDLL(so)


def _run_h2(lib, T, lo, hi):
    P = ctypes.POINTER(ctypes.c_double)
    lo = np.ascontiguousarray(lo, np.float64)
    hi = np.ascontiguousarray(hi, np.float64)
    plo, phi = np.empty_like(lo), np.empty_like(hi)
    lib.run_h2(T, lo.ctypes.data_as(P), hi.ctypes.data_as(P), plo.ctypes.data_as(P),
               phi.ctypes.data_as(P), lo.shape[0])
    return plo, phi


U16 = 2.0 ** -11   # unit roundoff of binary16


@pytest.mark.parametrize("T", range(1, 17))
def test_packed_fp16_transform_accuracy(h2lib, T):
    """Each plane is within (number of rounded operations on its longest path) x
    u16 x sum|v| of the exact spectrum of the fp16 inputs, and the two halves
    of a register carry independent signals."""
    rs = np.random.RandomState(300 + T)
    lo = rs.standard_normal((500, T)).astype(np.float16).astype(np.float64)
    hi = (3.0 * rs.standard_normal((500, T))).astype(np.float16).astype(np.float64)
    plo, phi = _run_h2(h2lib, T, lo, hi)
    # longest chain of roundings: log2(T) + 2 butterfly/twiddle stages for the
    # FFT forms (T = 4, 8, 16), T/2 + 2 accumulations for the direct form
    depth = {4: 3, 8: 5, 16: 7}.get(T, T // 2 + 3)
    for sig, got in ((lo, plo), (hi, phi)):
        ref = planes(np.fft.fft(sig, axis=1), T)
        bound = depth * U16 * np.abs(sig).sum(axis=1, keepdims=True)
        assert np.all(np.abs(got - ref) <= bound), (T, float(np.max(np.abs(got - ref) / bound)))
    # swapping the halves swaps the results: no cross-talk between the signals
    plo2, phi2 = _run_h2(h2lib, T, hi, lo)
    assert np.array_equal(plo2, phi) and np.array_equal(phi2, plo)


@pytest.mark.parametrize("T", [4, 8, 16, 5])
def test_packed_fp16_transform_overflow_threshold(h2lib, T):
    """A partial sum above 65504 overflows to inf: with every element at
    65504 / T the bins stay finite, at twice that bin 0 overflows."""
    v = np.full((1, T), np.float16(60000.0 / T), np.float64)
    p, _ = _run_h2(h2lib, T, v, v)
    assert np.all(np.isfinite(p))
    p, _ = _run_h2(h2lib, T, 2 * v, 2 * v)
    assert np.isinf(p[0, 0])
