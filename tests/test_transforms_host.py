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
    b = src.index("// ---------------------------------------------------------------------------\n// Element types.")
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
