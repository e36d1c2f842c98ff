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

}  // namespace eqk
