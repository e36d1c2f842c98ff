/*
 * eqref_dihedral.c -- fp64 CPU oracle for the equivariant linear layer over
 * the dihedral group D_T (the T rotations and T reflections of a regular
 * T-gon).
 *
 * TEST INFRASTRUCTURE ONLY.  The correctness reference that the GPU path of
 * the dihedral layer is checked against; only the tests may load it.  It
 * shares no code, header, table or helper with the HIP library (nor with the
 * C_T oracle in eqref.c).
 *
 * What it computes.  The paper's layer over the rotation group C_T shares one
 * Cout x Cin weight block per group element and mixes the group axis by the
 * group's own law: output position t takes block w[(t - s) mod T] against
 * input position s (Sec. 3.1, Eq. 1-2, with the convolution lag direction).
 * Sec. 5 names reflection groups as the next groups to cover.  The same
 * weight-sharing rule over D_T, written with the group law itself:
 *
 *   y[n,o,g] = ( sum_{h in D_T} sum_c W[h^-1 g][o][c] * x[n,c,h] ) + b[o]
 *
 * so that y of a translated input (x'(h) = x(u^-1 h)) is the translated
 * output (y'(g) = y(u^-1 g)) for every u in D_T.  Over C_T (m = 0 only) this
 * is exactly the C_T layer: h^-1 g = t - s.
 *
 * Elements.  g = (t, m) stands for r^t s^m: t in Z_T the rotation, m in {0,1}
 * the reflection.  Since s r s = r^-1:
 *   (t1, m1)(t2, m2) = (t1 + (-1)^m1 t2 mod T, m1 xor m2)
 *   (t, m)^-1        = (-(-1)^m t mod T, m)
 * Storage index of g: m*T + t.  Layouts (row-major, float64):
 *   x, dx [N, Cin, 2T]   y, dy [N, Cout, 2T]   W, dW [2T, Cout, Cin]   b, db [Cout]
 *
 * Gradients of L = <dy, y>:
 *   dx[n,c,h] = sum_g sum_o W[h^-1 g][o][c] * dy[n,o,g]
 *   dW[u][o][c] = sum_n sum_h dy[n,o,h u] * x[n,c,h]
 *   db[o]     = sum_n sum_g dy[n,o,g]
 *
 * Summation orders are fixed as written.  Build with -O2 -fno-fast-math
 * -ffp-contract=off.
 */
#include <stdint.h>
#include <stdlib.h>

/* storage index of the product of the elements with storage indices a, b */
static int d_mul(int a, int b, int T) {
  const int ta = a % T, ma = a / T, tb = b % T, mb = b / T;
  int t = ma ? ta - tb : ta + tb;
  t %= T;
  if (t < 0) t += T;
  return (ma ^ mb) * T + t;
}

/* storage index of the inverse of the element with storage index a */
static int d_inv(int a, int T) {
  const int ta = a % T, ma = a / T;
  int t = ma ? ta : (T - ta) % T;
  return ma * T + t;
}

int eqref_dihedral_version(void) { return 1; }

void eqref_dihedral_forward(const double* x, const double* W, const double* b, double* y,
                            int64_t N, int T, int Cin, int Cout) {
  const int G = 2 * T;
#pragma omp parallel for schedule(static)
  for (int64_t n = 0; n < N; ++n) {
    for (int o = 0; o < Cout; ++o) {
      for (int g = 0; g < G; ++g) {
        double acc = 0.0;
        for (int h = 0; h < G; ++h) {
          const int u = d_mul(d_inv(h, T), g, T);
          for (int c = 0; c < Cin; ++c)
            acc += W[((int64_t)u * Cout + o) * Cin + c] * x[(n * Cin + c) * G + h];
        }
        if (b) acc += b[o];
        y[(n * Cout + o) * G + g] = acc;
      }
    }
  }
}

void eqref_dihedral_backward_input(const double* dy, const double* W, double* dx, int64_t N, int T,
                                   int Cin, int Cout) {
  const int G = 2 * T;
#pragma omp parallel for schedule(static)
  for (int64_t n = 0; n < N; ++n) {
    for (int c = 0; c < Cin; ++c) {
      for (int h = 0; h < G; ++h) {
        const int hi = d_inv(h, T);
        double acc = 0.0;
        for (int g = 0; g < G; ++g) {
          const int u = d_mul(hi, g, T);
          for (int o = 0; o < Cout; ++o)
            acc += W[((int64_t)u * Cout + o) * Cin + c] * dy[(n * Cout + o) * G + g];
        }
        dx[(n * Cin + c) * G + h] = acc;
      }
    }
  }
}

void eqref_dihedral_backward_weight(const double* x, const double* dy, double* dW, double* db,
                                    int64_t N, int T, int Cin, int Cout) {
  const int G = 2 * T;
#pragma omp parallel for collapse(2) schedule(static)
  for (int u = 0; u < G; ++u) {
    for (int o = 0; o < Cout; ++o) {
      for (int c = 0; c < Cin; ++c) {
        double acc = 0.0;
        for (int64_t n = 0; n < N; ++n)
          for (int h = 0; h < G; ++h)
            acc += dy[(n * Cout + o) * G + d_mul(h, u, T)] * x[(n * Cin + c) * G + h];
        dW[((int64_t)u * Cout + o) * Cin + c] = acc;
      }
    }
  }
  if (db) {
    for (int o = 0; o < Cout; ++o) {
      double acc = 0.0;
      for (int64_t n = 0; n < N; ++n)
        for (int g = 0; g < G; ++g) acc += dy[(n * Cout + o) * G + g];
      db[o] = acc;
    }
  }
}

/* The group law itself, for the tests: products and inverses of storage
 * indices. */
int eqref_dihedral_mul(int a, int b, int T) { return d_mul(a, b, T); }
int eqref_dihedral_inv(int a, int T) { return d_inv(a, T); }
