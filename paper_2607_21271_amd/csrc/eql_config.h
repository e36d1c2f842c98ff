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

}  // namespace eqk
