/* Runs every entry point of oracle/eqref.c on exactly-sized heap buffers, for
 * the address and undefined-behaviour sanitizers: group orders 1..16, ragged
 * channel counts, zero rows, with and without a bias.  Also checks one
 * identity per call so the calls are not dead: dw summed over lags and
 * channels equals sum_n sum_t dy * sum_c x (lag-summed weights see the
 * channel sums of x), db = sum dy, and an entry of dw equals the full dw. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void eqref_forward(const double*, const double*, const double*, double*, int64_t, int, int, int);
void eqref_backward_input(const double*, const double*, double*, int64_t, int, int, int);
void eqref_backward_weight(const double*, const double*, double*, double*, int64_t, int, int, int);
void eqref_backward_weight_entries(const double*, const double*, const int32_t*, const int32_t*,
                                   const int32_t*, int64_t, double*, int64_t, int, int, int);

static double* fill(size_t n, unsigned* seed) {
  double* p = (double*)malloc((n ? n : 1) * sizeof(double));
  for (size_t i = 0; i < n; ++i) p[i] = (double)(rand_r(seed) % 2001 - 1000) / 1000.0;
  return p;
}

int main(void) {
  unsigned seed = 7;
  int bad = 0;
  const int shapes[][4] = {{1, 3, 2, 5}, {2, 1, 1, 0}, {3, 5, 7, 9}, {4, 16, 16, 33}, {5, 2, 9, 4},
                           {8, 7, 3, 11}, {12, 4, 5, 6}, {16, 3, 2, 7}, {7, 1, 13, 1}};
  for (size_t k = 0; k < sizeof(shapes) / sizeof(shapes[0]); ++k) {
    const int T = shapes[k][0], Cin = shapes[k][1], Cout = shapes[k][2];
    const int64_t N = shapes[k][3];
    double* x = fill((size_t)N * Cin * T, &seed);
    double* w = fill((size_t)T * Cout * Cin, &seed);
    double* b = fill((size_t)Cout, &seed);
    double* dy = fill((size_t)N * Cout * T, &seed);
    double* y = fill((size_t)N * Cout * T, &seed);
    double* dx = fill((size_t)N * Cin * T, &seed);
    double* dw = fill((size_t)T * Cout * Cin, &seed);
    double* db = fill((size_t)Cout, &seed);
    eqref_forward(x, w, b, y, N, T, Cin, Cout);
    eqref_forward(x, w, NULL, y, N, T, Cin, Cout);
    eqref_backward_input(dy, w, dx, N, T, Cin, Cout);
    eqref_backward_weight(x, dy, dw, db, N, T, Cin, Cout);
    eqref_backward_weight(x, dy, dw, NULL, N, T, Cin, Cout);
    double lhs = 0.0, rhs = 0.0, sdy = 0.0, sdb = 0.0;
    for (int64_t i = 0; i < (int64_t)T * Cout * Cin; ++i) lhs += dw[i];
    for (int64_t n = 0; n < N; ++n) {
      double sx = 0.0;
      for (int c = 0; c < Cin; ++c)
        for (int t = 0; t < T; ++t) sx += x[(n * Cin + c) * T + t];
      double sd = 0.0;
      for (int o = 0; o < Cout; ++o)
        for (int t = 0; t < T; ++t) sd += dy[(n * Cout + o) * T + t];
      rhs += sd * sx;
      sdy += sd;
    }
    for (int o = 0; o < Cout; ++o) sdb += db[o];
    if (fabs(lhs - rhs) > 1e-9 * (1.0 + fabs(rhs))) { printf("dw sum T=%d\n", T); bad = 1; }
    if (fabs(sdb - sdy) > 1e-9 * (1.0 + fabs(sdy))) { printf("db sum T=%d\n", T); bad = 1; }
    int32_t je[3] = {0, T - 1, T / 2}, oe[3] = {0, Cout - 1, Cout / 2}, ce[3] = {Cin - 1, 0, Cin / 2};
    double out[3];
    eqref_backward_weight_entries(x, dy, je, oe, ce, 3, out, N, T, Cin, Cout);
    for (int e = 0; e < 3; ++e) {
      const double ref = dw[((int64_t)je[e] * Cout + oe[e]) * Cin + ce[e]];
      if (fabs(out[e] - ref) > 1e-12 * (1.0 + fabs(ref))) { printf("entry T=%d\n", T); bad = 1; }
    }
    free(x); free(w); free(b); free(dy); free(y); free(dx); free(dw); free(db);
  }
  printf(bad ? "oracle driver: FAILED\n" : "oracle driver: ok\n");
  return bad;
}
