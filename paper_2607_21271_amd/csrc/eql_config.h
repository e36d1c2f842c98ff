// eql_config.h -- compile-time configuration shared by host and device code.
#pragma once

namespace eqk {

// Wave pairs per workgroup of the forward / input-gradient kernel: a workgroup
// is 128 * kGemmPairs threads and takes rounds of 16 * kGemmPairs rows.
#ifndef EQL_GEMM_PAIRS
#define EQL_GEMM_PAIRS 4
#endif
constexpr int kGemmPairs = EQL_GEMM_PAIRS;
constexpr int kGemmThreads = 128 * kGemmPairs;
constexpr int kGemmRoundRows = 16 * kGemmPairs;

// Element type codes, equal to the C ABI's dtype values: IEEE binary32,
// IEEE binary16, bfloat16.
constexpr int kF32 = 0, kF16 = 1, kBF16 = 2;

// Geometry of the implicit patch gather of the forward kernel (the group
// convolution read straight from its features): images of H x W pixels,
// Cin input channels per group element, k x k window.  Unused (zero) by the
// plain layer.
struct GatherGeom {
  int H, W, Cin, k;
  // division by a launch constant d as a multiply: m = floor(2^32 / d)
  // (2^32 - 1 for d = 1) gives floor(n * m / 2^32) in {n / d - 1, n / d}
  // for n < 2^31, and one correction step makes it exact (div_magic below).
  // For W, H, Cin * T (channels of a gathered orbit block) and the orbit
  // divisor (k / 2 + 1 for T = 4, k for T = 2 and 1).
  unsigned mW, mH, mCT, mO;
};

// the multiplier of GatherGeom for divisor d >= 1
inline unsigned div_magic(unsigned d) { return d == 1 ? 0xffffffffu : (unsigned)((1ull << 32) / d); }

}  // namespace eqk
