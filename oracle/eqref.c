/*
 * eqref.c -- fp64 CPU oracle for the equivariant linear layer over the cyclic
 * group C_T (Flash EQ-Linear, arXiv 2607.21271).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the correctness reference that the
 * GPU library is checked against.  Only the tests, the smoke check and the
 * CPU-baseline leg of the benchmark may load it.  It shares no code, header,
 * table or helper with the HIP library, and the HIP library never calls it.
 *
 * What it computes.  The paper writes the layer as a block-circulant matrix
 * acting on the group axis (Sec. 3.1, Eq. 1) and equivalently as a circular
 * convolution along the group axis composed with a channel contraction
 * (Sec. 3.1, Eq. 2).  The method is exact (Sec. 3.4), so the oracle evaluates
 * that defining sum directly -- no DFT, no twiddles, no reordering:
 *
 *   y [n,o,t] = ( sum_j sum_c w[j,o,c] * x[n,c,(t-j) mod T] ) + b[o]
 *
 * with the lag direction (t-j) of a circular convolution.  Eq. 2 as printed
 * indexes the shared block by (s-t), a correlation, while the convolution
 * theorem the paper applies (Sec. 3.1, Eq. 3; Alg. 1; the p4 kernel products
 * of Appendix A.2) multiplies forward DFTs of both operands, which is a
 * convolution; the oracle follows the convolution reading.  Weights are laid
 * out w[T,Cout,Cin] with j the lag.
 *
 * Gradients of L = <dy, y> (the training-step tensors of Sec. 4.3, Table 4):
 *
 *   dx[n,c,s] = sum_j sum_o w[j,o,c] * dy[n,o,(s+j) mod T]
 *   dw[j,o,c] = sum_n sum_t dy[n,o,t] * x[n,c,(t-j) mod T]
 *   db[o]     = sum_n sum_t dy[n,o,t]
 *
 * Summation order is fixed as written (lag outer, channel inner, bias last;
 * rows outer, group index inner), so a roll of x along the group axis rolls y
 * bit-exactly.  Build with strict IEEE semantics: -O2 -fno-fast-math
 * -ffp-contract=off (no fused multiply-add contraction).
 *
 * All tensors are row-major, contiguous, float64.
 */
#include <stdint.h>
#include <stdlib.h>

#define IDX3(a, b, c, B, C) (((int64_t)(a) * (B) + (b)) * (C) + (c))

static int wrap(int i, int T) {
  int r = i % T;
  return r < 0 ? r + T : r;
}

int eqref_version(void) { return 1; }

/* Forward pass: the circular-convolution sum of Sec. 3.1, Eq. 2 (convolution
 * lag direction), plus the group-shared bias broadcast over rows and group
 * positions (Sec. 3.1, Eq. 1).  b may be NULL (no bias). */
void eqref_forward(const double* x, const double* w, const double* b, double* y,
                   int64_t N, int T, int Cin, int Cout) {
#pragma omp parallel for schedule(static)
  for (int64_t n = 0; n < N; ++n) {
    for (int o = 0; o < Cout; ++o) {
      for (int t = 0; t < T; ++t) {
        double acc = 0.0;
        for (int j = 0; j < T; ++j) {
          const int s = wrap(t - j, T);
          for (int c = 0; c < Cin; ++c)
            acc += w[IDX3(j, o, c, Cout, Cin)] * x[IDX3(n, c, s, Cin, T)];
        }
        if (b) acc += b[o];
        y[IDX3(n, o, t, Cout, T)] = acc;
      }
    }
  }
}

/* Input gradient: the adjoint of the forward map with respect to x.  Output
 * group position t = s + j receives x[.,.,s] through lag j, so the gradient
 * gathers dy at (s+j) mod T. */
void eqref_backward_input(const double* dy, const double* w, double* dx,
                          int64_t N, int T, int Cin, int Cout) {
#pragma omp parallel for schedule(static)
  for (int64_t n = 0; n < N; ++n) {
    for (int c = 0; c < Cin; ++c) {
      for (int s = 0; s < T; ++s) {
        double acc = 0.0;
        for (int j = 0; j < T; ++j) {
          const int t = wrap(s + j, T);
          for (int o = 0; o < Cout; ++o)
            acc += w[IDX3(j, o, c, Cout, Cin)] * dy[IDX3(n, o, t, Cout, T)];
        }
        dx[IDX3(n, c, s, Cin, T)] = acc;
      }
    }
  }
}

/* Weight and bias gradients: the adjoint with respect to the shared
 * parameters w[j,o,c] and b[o] (gradients are taken with respect to the
 * original parameters, Appendix A.2 "Forward and backward passes").  db may
 * be NULL.  Rows are summed in increasing order. */
void eqref_backward_weight(const double* x, const double* dy, double* dw, double* db,
                           int64_t N, int T, int Cin, int Cout) {
#pragma omp parallel for schedule(static)
  for (int64_t jo = 0; jo < (int64_t)T * Cout; ++jo) {
    const int j = (int)(jo / Cout);
    const int o = (int)(jo % Cout);
    double* acc = (double*)calloc((size_t)(Cin > 0 ? Cin : 1), sizeof(double));
    for (int64_t n = 0; n < N; ++n) {
      for (int t = 0; t < T; ++t) {
        const double g = dy[IDX3(n, o, t, Cout, T)];
        const int s = wrap(t - j, T);
        for (int c = 0; c < Cin; ++c) acc[c] += g * x[IDX3(n, c, s, Cin, T)];
      }
    }
    for (int c = 0; c < Cin; ++c) dw[IDX3(j, o, c, Cout, Cin)] = acc[c];
    free(acc);
  }
  if (db) {
#pragma omp parallel for schedule(static)
    for (int o = 0; o < Cout; ++o) {
      double acc = 0.0;
      for (int64_t n = 0; n < N; ++n)
        for (int t = 0; t < T; ++t) acc += dy[IDX3(n, o, t, Cout, T)];
      db[o] = acc;
    }
  }
}

/* Selected entries of dw, each by the same sum as eqref_backward_weight
 * (rows outer, group index inner): out[e] = dw[j[e], o[e], c[e]].  Lets a
 * test check a full-size weight gradient at sampled entries without paying
 * for the whole tensor. */
void eqref_backward_weight_entries(const double* x, const double* dy,
                                   const int32_t* j, const int32_t* o, const int32_t* c,
                                   int64_t n_entries, double* out,
                                   int64_t N, int T, int Cin, int Cout) {
#pragma omp parallel for schedule(static)
  for (int64_t e = 0; e < n_entries; ++e) {
    double acc = 0.0;
    for (int64_t n = 0; n < N; ++n)
      for (int t = 0; t < T; ++t) {
        const int s = wrap(t - j[e], T);
        acc += dy[IDX3(n, o[e], t, Cout, T)] * x[IDX3(n, c[e], s, Cin, T)];
      }
    out[e] = acc;
  }
}
