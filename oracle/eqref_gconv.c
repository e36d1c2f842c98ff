/*
 * eqref_gconv.c -- fp64 CPU oracle for the rotation-equivariant group
 * convolution on a square grid (the group C_T of rotations by 360/T degrees,
 * T in {1, 2, 4}, acting on the image plane and on the group axis of the
 * features).
 *
 * TEST INFRASTRUCTURE ONLY.  The correctness reference for the GPU path of
 * the group convolution; only the tests may load it.  It shares no code,
 * header, table or helper with the HIP library or the other oracles.
 *
 * What it computes.  Sec. 5 names equivariant convolutions as the next
 * operators to carry the method to.  Features are f[b, y, x, c, s] (pixel
 * (y, x), channel c, group element s); the layer shares one weight block per
 * (spatial offset, group lag) and rotates the offset with the output's group
 * element, which is the group convolution over the plane and C_T:
 *
 *   out[b,y,x,o,r] = sum_{(dy,dx) in window} sum_s sum_c
 *                      psi[R^-r (dy,dx)][(s - r) mod T][o][c] * f[b, y+dy, x+dx, c, s]
 *                    + bias[o]
 *
 * with f zero outside the image ("same" padding), the window the k x k
 * offsets (dy, dx) in [-k/2, k/2]^2 (k odd), and R the rotation of offsets by
 * 360/T degrees: R(a, b) = (-b, a) for T = 4, (-a, -b) for T = 2, the identity
 * for T = 1.  Rotating the image about its centre by R (a square image) and
 * shifting the group axis by one maps the output the same way.
 *
 * Layouts (row-major, float64): f, df [B, H, W, Cin, T]; out, dout
 * [B, H, W, Cout, T]; psi, dpsi [k, k, T, Cout, Cin] indexed by
 * (dy + k/2, dx + k/2, lag); bias, dbias [Cout].
 *
 * Gradients of L = <dout, out>:
 *   df[b,y',x',c,s]    = sum_{(y,x)} sum_r sum_o psi[R^-r (y'-y, x'-x)][(s - r) mod T][o][c] * dout[b,y,x,o,r]
 *   dpsi[d][l][o][c]   = sum_{b,y,x} sum_r f[b, (y,x) + R^r d, c, (l + r) mod T] * dout[b,y,x,o,r]
 *   dbias[o]           = sum dout[b,y,x,o,r]
 *
 * Summation orders are fixed as written.  Build with -O2 -fno-fast-math
 * -ffp-contract=off.
 */
#include <stdint.h>
#include <stdlib.h>

/* offset (a, b) rotated by R^n, n >= 0 */
static void rot(int n, int T, int a, int b, int* ra, int* rb) {
  const int q = T == 4 ? 1 : (T == 2 ? 2 : 0); /* quarter turns per step of R */
  int turns = ((n % T + T) % T) * q;
  int x = a, y = b;
  for (int i = 0; i < turns; ++i) {
    const int nx = -y, ny = x; /* one quarter turn: (a, b) -> (-b, a) */
    x = nx;
    y = ny;
  }
  *ra = x;
  *rb = y;
}

#define PSI(dy, dx, l, o, c) \
  psi[((((int64_t)((dy) + h) * k + ((dx) + h)) * T + (l)) * Cout + (o)) * Cin + (c)]

int eqref_gconv_version(void) { return 1; }

void eqref_gconv_forward(const double* f, const double* psi, const double* bias, double* out, int B,
                         int H, int W, int T, int Cin, int Cout, int k) {
  const int h = k / 2;
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b)
    for (int y = 0; y < H; ++y)
      for (int x = 0; x < W; ++x)
        for (int o = 0; o < Cout; ++o)
          for (int r = 0; r < T; ++r) {
            double acc = 0.0;
            for (int dy = -h; dy <= h; ++dy)
              for (int dx = -h; dx <= h; ++dx) {
                const int yy = y + dy, xx = x + dx;
                if (yy < 0 || yy >= H || xx < 0 || xx >= W) continue;
                int ry, rx;
                rot(-r, T, dy, dx, &ry, &rx);
                for (int s = 0; s < T; ++s) {
                  const int l = ((s - r) % T + T) % T;
                  for (int c = 0; c < Cin; ++c)
                    acc += PSI(ry, rx, l, o, c) *
                           f[((((int64_t)b * H + yy) * W + xx) * Cin + c) * T + s];
                }
              }
            if (bias) acc += bias[o];
            out[((((int64_t)b * H + y) * W + x) * Cout + o) * T + r] = acc;
          }
}

void eqref_gconv_backward_input(const double* dout, const double* psi, double* df, int B, int H, int W,
                                int T, int Cin, int Cout, int k) {
  const int h = k / 2;
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b)
    for (int yp = 0; yp < H; ++yp)
      for (int xp = 0; xp < W; ++xp)
        for (int c = 0; c < Cin; ++c)
          for (int s = 0; s < T; ++s) {
            double acc = 0.0;
            /* outputs (y, x) whose window holds (yp, xp): offset (yp - y, xp - x) */
            for (int dy = -h; dy <= h; ++dy)
              for (int dx = -h; dx <= h; ++dx) {
                const int y = yp - dy, x = xp - dx;
                if (y < 0 || y >= H || x < 0 || x >= W) continue;
                for (int r = 0; r < T; ++r) {
                  int ry, rx;
                  rot(-r, T, dy, dx, &ry, &rx);
                  const int l = ((s - r) % T + T) % T;
                  for (int o = 0; o < Cout; ++o)
                    acc += PSI(ry, rx, l, o, c) *
                           dout[((((int64_t)b * H + y) * W + x) * Cout + o) * T + r];
                }
              }
            df[((((int64_t)b * H + yp) * W + xp) * Cin + c) * T + s] = acc;
          }
}

void eqref_gconv_backward_weight(const double* f, const double* dout, double* dpsi, double* dbias, int B,
                                 int H, int W, int T, int Cin, int Cout, int k) {
  const int h = k / 2;
#pragma omp parallel for collapse(2) schedule(static)
  for (int dy = -h; dy <= h; ++dy)
    for (int dx = -h; dx <= h; ++dx)
      for (int l = 0; l < T; ++l)
        for (int o = 0; o < Cout; ++o)
          for (int c = 0; c < Cin; ++c) {
            double acc = 0.0;
            for (int b = 0; b < B; ++b)
              for (int y = 0; y < H; ++y)
                for (int x = 0; x < W; ++x)
                  for (int r = 0; r < T; ++r) {
                    int ry, rx;
                    rot(r, T, dy, dx, &ry, &rx);
                    const int yy = y + ry, xx = x + rx;
                    if (yy < 0 || yy >= H || xx < 0 || xx >= W) continue;
                    const int s = (l + r) % T;
                    acc += f[((((int64_t)b * H + yy) * W + xx) * Cin + c) * T + s] *
                           dout[((((int64_t)b * H + y) * W + x) * Cout + o) * T + r];
                  }
            const int64_t idx = ((((int64_t)(dy + h) * k + (dx + h)) * T + l) * Cout + o) * Cin + c;
            dpsi[idx] = acc;
          }
  if (dbias) {
    for (int o = 0; o < Cout; ++o) {
      double acc = 0.0;
      for (int64_t n = 0; n < (int64_t)B * H * W; ++n)
        for (int r = 0; r < T; ++r) acc += dout[(n * Cout + o) * T + r];
      dbias[o] = acc;
    }
  }
}
