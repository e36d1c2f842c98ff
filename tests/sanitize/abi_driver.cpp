// Exercises the host side of libeqlinear (argument checks, size queries, the
// weight-gradient and single-pass planning, the dihedral entry points) for the
// address and undefined-behaviour sanitizers, without a GPU: every call below
// returns before any kernel
// launch, either with an argument error or, for valid arguments on a machine
// without a HIP device, EQL_ERR_NO_DEVICE.  The device pointers are fake and
// never dereferenced.
#include <stdint.h>
#include <stdio.h>

#include "eqlinear.h"

static int bad = 0;
#define EXPECT(cond)                                         \
  do {                                                       \
    if (!(cond)) {                                           \
      printf("failed: %s (line %d)\n", #cond, __LINE__);     \
      bad = 1;                                               \
    }                                                        \
  } while (0)

int main(int argc, char** argv) {
  const bool no_device = argc > 1;  // the caller checked that no GPU is visible
  char* A = (char*)0x10000000;
  const size_t MB = 1 << 20;
  for (int s = -1; s < 10; ++s) EXPECT(eqlinear_status_string(s) != nullptr);
  EXPECT(eqlinear_abi_version() == EQLINEAR_ABI_VERSION);
  // size queries and the weight-gradient plans over a range of shapes
  const int Cs[] = {1, 7, 16, 24, 33, 48, 64, 96, 130, 384, 512, 2048};
  const int64_t Ns[] = {0, 1, 31, 257, 12608, 401408, (int64_t)1 << 24};
  size_t total = 0;
  for (int T = 1; T <= 16; ++T)
    for (int ci : Cs)
      for (int co : Cs)
        for (int dt = 0; dt < 2; ++dt) {
          total += eqlinear_weight_spectrum_bytes(T, ci, co, dt);
          for (int64_t n : Ns) {
            total += eqlinear_backward_weight_workspace_bytes(n, T, ci, co, dt);
            // the single-pass plan and the whole-backward workspace
            total += eqlinear_backward_workspace_bytes(n, T, ci, co, dt);
            total += (size_t)eqlinear_backward_is_fused(n, T, ci, co, dt);
          }
        }
  EXPECT(total > 0);
  EXPECT(eqlinear_weight_spectrum_bytes(17, 4, 4, 0) == 0);
  EXPECT(eqlinear_backward_weight_workspace_bytes(-1, 4, 4, 4, 0) == 0);
  EXPECT(eqlinear_backward_weight_workspace_bytes(100, 4, 4, 4, 9) == 0);
  // argument errors
  EXPECT(eqlinear_forward(A, A + 8 * MB, nullptr, A + 16 * MB, 10, 0, 4, 4, 0, nullptr) == EQL_ERR_INVALID_ARG);
  EXPECT(eqlinear_forward(A + 4, A + 8 * MB, nullptr, A + 16 * MB, 10, 4, 4, 4, 0, nullptr) == EQL_ERR_ALIGNMENT);
  EXPECT(eqlinear_forward(A, A + 8 * MB, nullptr, A + 16, 10, 4, 4, 4, 0, nullptr) == EQL_ERR_INVALID_ARG);
  EXPECT(eqlinear_forward(A, A + 8 * MB, nullptr, A + 16 * MB, 10, 17, 4, 4, 0, nullptr) == EQL_ERR_UNSUPPORTED);
  EXPECT(eqlinear_backward_input(A, nullptr, A + 16 * MB, 10, 4, 4, 4, 0, nullptr) == EQL_ERR_INVALID_ARG);
  const size_t need = eqlinear_backward_weight_workspace_bytes(1000, 8, 16, 16, EQL_F32);
  EXPECT(eqlinear_backward_weight(A, A + 8 * MB, A + 16 * MB, A + 17 * MB, A + 24 * MB, need - 1, 1000,
                                  8, 16, 16, EQL_F32, nullptr) == EQL_ERR_WORKSPACE);
  EXPECT(eqlinear_backward_weight_noalloc(A, A + (1 << 30), A + 2 * ((size_t)1 << 30), nullptr, 1000,
                                          16, 2048, 2048, EQL_F32, nullptr) == EQL_ERR_SCRATCH);
  EXPECT(eqlinear_weight_spectrum(A + 2, A + MB, 4, 4, 4, 0, nullptr) == EQL_ERR_ALIGNMENT);
  // whole backward and the dihedral entry points: argument errors
  const size_t needb = eqlinear_backward_workspace_bytes(1000, 4, 24, 96, EQL_F16);
  EXPECT(eqlinear_backward(A, A + 8 * MB, A + 16 * MB, A + 24 * MB, A + 32 * MB, nullptr, A + 40 * MB,
                           needb - 1, 1000, 4, 24, 96, EQL_F16, nullptr) == EQL_ERR_WORKSPACE);
  EXPECT(eqlinear_backward(A, A + 8 * MB, A + 16 * MB, A + 16, A + 32 * MB, nullptr, A + 40 * MB, needb,
                           1000, 4, 24, 96, EQL_F16, nullptr) == EQL_ERR_INVALID_ARG);
  EXPECT(eqlinear_backward(A, A + 8 * MB, nullptr, A + 24 * MB, A + 32 * MB, nullptr, A + 40 * MB, needb,
                           1000, 4, 24, 96, EQL_F16, nullptr) == EQL_ERR_INVALID_ARG);
  EXPECT(eqlinear_dihedral_expand(A, nullptr, A + 8 * MB, nullptr, 4, 1 << 30, 8, 0, nullptr) ==
         EQL_ERR_UNSUPPORTED);
  EXPECT(eqlinear_dihedral_expand(A, A + MB, A + 8 * MB, nullptr, 4, 8, 8, 0, nullptr) == EQL_ERR_INVALID_ARG);
  EXPECT(eqlinear_dihedral_fold(A, nullptr, A + 4, nullptr, 4, 8, 8, 0, nullptr) == EQL_ERR_INVALID_ARG);
  EXPECT(eqlinear_dihedral_fold(A + 2, nullptr, A + 8 * MB, nullptr, 4, 8, 8, 0, nullptr) == EQL_ERR_ALIGNMENT);
  if (no_device) {
    EXPECT(eqlinear_backward(A, A + 8 * MB, A + 16 * MB, A + 24 * MB, A + 32 * MB, nullptr, A + 40 * MB,
                             needb, 1000, 4, 24, 96, EQL_F16, nullptr) == EQL_ERR_NO_DEVICE);
    EXPECT(eqlinear_dihedral_expand(A, A + MB, A + 8 * MB, A + 9 * MB, 4, 8, 8, 1, nullptr) ==
           EQL_ERR_NO_DEVICE);
    EXPECT(eqlinear_forward(A, A + 8 * MB, nullptr, A + 16 * MB, 100, 4, 8, 8, 0, nullptr) == EQL_ERR_NO_DEVICE);
    EXPECT(eqlinear_weight_spectrum(A, A + MB, 4, 8, 8, 1, nullptr) == EQL_ERR_NO_DEVICE);
    EXPECT(eqlinear_backward_weight(A, A + 8 * MB, A + 16 * MB, A + 17 * MB, A + 24 * MB, need, 1000, 8,
                                    16, 16, EQL_F32, nullptr) == EQL_ERR_NO_DEVICE);
    EXPECT(eqlinear_backward_weight_noalloc(A, A + 8 * MB, A + 16 * MB, A + 17 * MB, 1000, 8, 16, 16,
                                            EQL_F32, nullptr) == EQL_ERR_NO_DEVICE);
  }
  printf(bad ? "abi driver: FAILED\n" : "abi driver: ok\n");
  return bad;
}
