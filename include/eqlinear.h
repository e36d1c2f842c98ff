/*
 * eqlinear.h -- C ABI of the MI355X (gfx950) library for the equivariant linear
 * layer over the cyclic group C_T, computed the Flash EQ-Linear way
 * (arXiv 2607.21271): real DFT along the group axis, one GEMM per non-redundant
 * frequency bin, inverse real DFT.
 *
 * The operation (Sec. 3.1, Eq. 1-2, read with the convolution lag direction
 * that the convolution theorem of Eq. 3 and Alg. 1 imply):
 *
 *     y[n,o,t] = sum_{j=0}^{T-1} sum_{c=0}^{Cin-1} w[j,o,c] * x[n,c,(t-j) mod T] + b[o]
 *
 * Layouts (row-major, contiguous, group axis innermost as in Appendix A.2
 * "Memory layout and vectorization"):
 *     x, dx   [N, Cin, T]        y, dy   [N, Cout, T]
 *     w, dw   [T, Cout, Cin]     (j = lag)
 *     b, db   [Cout]
 * A caller whose weights follow Eq. 2's printed index (s - t) reverses the lag
 * axis: w[j] = W_paper[(T - j) mod T].
 *
 * Common rules for every entry point:
 *   - dtype is EQL_F32, EQL_F16 or EQL_BF16 and applies to every tensor of
 *     the call.
 *     EQL_F32: every transform, product and accumulation is fp32.
 *     EQL_F16 (IEEE binary16): the forward real DFTs of the activations x and
 *     of the output gradients dy run in packed fp16 arithmetic (two signals per
 *     register, twiddles rounded to fp16), since their results are fp16 MFMA
 *     operands; the weight spectrum, every product's accumulation, the inverse
 *     transforms and the bias are fp32.  db sums each pair of rows' fp16 bin 0
 *     into fp32.  A transform partial sum above 65504 in magnitude overflows
 *     to +-inf, so |x| and |dy| must stay below about 65504 / T.
 *     EQL_BF16 (bfloat16: fp32's exponent range, 8 significand bits): the
 *     forward real DFTs run in fp32 on the exactly widened inputs and each
 *     spectrum value is rounded once to bf16 as an MFMA operand; the weight
 *     spectrum, accumulation, inverse transforms and bias (db from the fp32
 *     bin 0) are fp32.  eqlinear_backward always takes the two passes for
 *     bf16.
 *     Each output is rounded once (round-to-nearest-even).
 *   - All pointers are device pointers owned by the caller.  The library never
 *     allocates, frees or synchronises; work is enqueued on `stream` (a
 *     hipStream_t passed as void*, NULL = the null stream) and the call returns
 *     as soon as it is enqueued.
 *   - Arguments are checked before any HIP call.  On any error nothing is
 *     enqueued and no output is touched.  Checks: 1 <= T <= 16 (T > 16 is
 *     EQL_ERR_UNSUPPORTED), 1 <= Cin, Cout <= 65536, 0 <= N <= 2^36, non-null
 *     pointers (bias and dbias may be NULL; with N = 0 the row tensors may be
 *     NULL), 16-byte aligned x, y, dy, dx, wspec and workspace and
 *     element-aligned w, dw, bias, dbias (EQL_ERR_ALIGNMENT), no byte overlap
 *     between any two tensors of a call (EQL_ERR_INVALID_ARG), and a large
 *     enough workspace (EQL_ERR_WORKSPACE).  Then: no visible HIP device is
 *     EQL_ERR_NO_DEVICE, a device other than gfx950 is EQL_ERR_UNSUPPORTED, and
 *     a failed launch is EQL_ERR_LAUNCH.
 *   - Outputs are overwritten, never accumulated into.
 *   - Results are bitwise reproducible for the same inputs, shape, dtype and
 *     device model: no atomics, fixed summation orders.
 *   - Calls are thread-safe: the library's only shared state is a per-device
 *     property cache filled once and a kernel-occupancy cache guarded by a
 *     mutex.  Concurrent calls that share no output buffer may run on
 *     different streams.
 */
#ifndef EQLINEAR_H
#define EQLINEAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EQLINEAR_ABI_VERSION 8
#define EQLINEAR_MAX_T 16

typedef enum { EQL_F32 = 0, EQL_F16 = 1, EQL_BF16 = 2 } eql_dtype_t;

typedef enum {
  EQL_OK = 0,
  EQL_ERR_INVALID_ARG = 1,
  EQL_ERR_UNSUPPORTED = 2,
  EQL_ERR_ALIGNMENT = 3,
  EQL_ERR_WORKSPACE = 4,
  EQL_ERR_NO_DEVICE = 5,
  EQL_ERR_LAUNCH = 6,
  EQL_ERR_SCRATCH = 7
} eql_status_t;

/* Bytes of the static device scratch array that
 * eqlinear_backward_weight_noalloc uses in place of a workspace (per GPU,
 * held until the process ends). */
#define EQLINEAR_STATIC_SCRATCH_BYTES ((size_t)64 << 20)

/* EQLINEAR_ABI_VERSION of the built library. */
int eqlinear_abi_version(void);

/* Static, NUL-terminated description of a status code ("unknown status" for
 * values outside eql_status_t).  Never NULL. */
const char* eqlinear_status_string(int status);

/* Bytes of the opaque weight-spectrum buffer for (T, Cin, Cout, dtype); 0 if
 * the arguments are invalid. */
size_t eqlinear_weight_spectrum_bytes(int T, int Cin, int Cout, int dtype);

/* Weight spectrum (Alg. 1 step 1 for the shared parameters; Sec. 3.2.1 Eq. 4):
 *     What_k[o,c] = sum_j w[j,o,c] e^{-2 pi i j k / T},   k = 0..floor(T/2),
 * kept as T real planes (the imaginary parts of bin 0 and, for even T, of bin
 * T/2 are zero and not stored), in the frequency-domain plane form that the
 * paper's kernels keep their weights in (Sec. 3.5).  w is [T,Cout,Cin] in
 * `dtype`; wspec is an opaque device buffer of
 * eqlinear_weight_spectrum_bytes() bytes, fully overwritten (padding
 * included).  For EQL_F16 and EQL_BF16 the spectrum is computed in fp32 and
 * rounded once to the 16-bit type.  It stays valid until w changes and serves eqlinear_forward and
 * eqlinear_backward_input of the same (T, Cin, Cout, dtype). */
int eqlinear_weight_spectrum(const void* w, void* wspec, int T, int Cin, int Cout, int dtype,
                             void* stream);

/* Forward pass (Alg. 1; Sec. 3.2.1 Eq. 4-7): rDFT of x along the group axis,
 * one product Yhat_k = What_k Xhat_k per bin k = 0..floor(T/2) (complex bins
 * as real block products, conjugate bins never formed), inverse rDFT, plus
 * bias.  x [N,Cin,T] in, y [N,Cout,T] out, bias [Cout] or NULL.  N = 0 is a
 * no-op.  x and y must not overlap (y is written directly in its final
 * layout, never staged through x). */
int eqlinear_forward(const void* x, const void* wspec, const void* bias, void* y, int64_t N,
                     int T, int Cin, int Cout, int dtype, void* stream);

/* Input gradient (the backward pass computed in the Fourier basis of the
 * forward, Appendix A.2 "Forward and backward passes"): dYhat = rDFT(dy),
 *     dXhat_k[n,c] = sum_o dYhat_k[n,o] conj(What_k[o,c]),
 * dx = irDFT(dXhat), i.e. dx[n,c,s] = sum_j sum_o w[j,o,c] dy[n,o,(s+j) mod T].
 * dy [N,Cout,T] in, dx [N,Cin,T] out; wspec as produced by
 * eqlinear_weight_spectrum.  N = 0 is a no-op. */
int eqlinear_backward_input(const void* dy, const void* wspec, void* dx, int64_t N, int T,
                            int Cin, int Cout, int dtype, void* stream);

/* Bytes of device workspace that eqlinear_backward_weight needs for this
 * problem (fp32 partial sums of the row splits; for wide layers with T = 2 or
 * 4 also the transformed x and dy, stored with the rows contiguous, about
 * (Cin + Cout) T N times the element size in bytes); 0 if the arguments are
 * invalid or N = 0. */
size_t eqlinear_backward_weight_workspace_bytes(int64_t N, int T, int Cin, int Cout, int dtype);

/* Weight and bias gradients with respect to the original parameters (Appendix
 * A.2 "Forward and backward passes"; the dW and db of Sec. 4.3 Table 4):
 *     H_k[c,o]  = sum_n conj(Xhat_k[n,c]) dYhat_k[n,o]          (fp32, split over rows)
 *     dw[j,o,c] = (1/T) sum_{k=0}^{T-1} H_k[c,o] e^{+2 pi i j k / T}
 *               = sum_n sum_t dy[n,o,t] x[n,c,(t-j) mod T]
 *     db[o]     = sum_n sum_t dy[n,o,t]
 * The row splits are summed in a fixed order by a second kernel (no atomics).
 * x [N,Cin,T] and dy [N,Cout,T] in; dw [T,Cout,Cin] and dbias [Cout] (or NULL
 * to skip it) out.  workspace is caller-owned device memory of at least
 * eqlinear_backward_weight_workspace_bytes() bytes (may be NULL when that is
 * 0); its contents on entry do not matter.  N = 0 writes zeros to dw and
 * dbias. */
int eqlinear_backward_weight(const void* x, const void* dy, void* dw, void* dbias, void* workspace,
                             size_t workspace_bytes, int64_t N, int T, int Cin, int Cout, int dtype,
                             void* stream);

/* Bytes of device workspace that eqlinear_backward needs for this problem
 * (fp32 partial sums of the weight gradient's row splits, for whichever path
 * eqlinear_backward_is_fused reports); 0 if the arguments are invalid or
 * N = 0. */
size_t eqlinear_backward_workspace_bytes(int64_t N, int T, int Cin, int Cout, int dtype);

/* 1 if eqlinear_backward runs this problem as one fused pass, 0 if it runs
 * the input- and weight-gradient kernels one after the other (or the
 * arguments are invalid).  Depends only on the arguments (and on the
 * EQL_BWD_FUSED environment variable: 0 never fuses, 1 fuses whenever the
 * layer fits). */
int eqlinear_backward_is_fused(int64_t N, int T, int Cin, int Cout, int dtype);

/* The whole backward pass of the layer in one call: dx as
 * eqlinear_backward_input computes it, dw and dbias as
 * eqlinear_backward_weight computes them (same operations, same layouts,
 * same precision rules).  Where every (input, output) channel pair of the
 * layer fits one workgroup's accumulators and the rows are many against them
 * (eqlinear_backward_is_fused), this runs as one pass that reads each row of
 * x and dy once and feeds all three gradients from the same spectra, the
 * single fused dataflow of Sec. 3.5 applied to the backward pass of Appendix
 * A.2 ("Forward and backward passes"); then a fixed-order reduction of the
 * weight gradient's row splits.  Otherwise the two gradient passes run one
 * after the other on `stream`.  x [N,Cin,T], dy [N,Cout,T] and wspec (of w,
 * from eqlinear_weight_spectrum) in; dx [N,Cin,T], dw [T,Cout,Cin] and dbias
 * [Cout] (or NULL to skip it) out.  workspace is caller-owned device memory of
 * at least eqlinear_backward_workspace_bytes() bytes (may be NULL when that
 * is 0).  The fused and two-pass paths sum in different orders, so their
 * results agree to rounding, not bitwise; each is bitwise reproducible.
 * N = 0 writes zeros to dw and dbias and leaves dx (empty) alone. */
int eqlinear_backward(const void* x, const void* dy, const void* wspec, void* dx, void* dw, void* dbias,
                      void* workspace, size_t workspace_bytes, int64_t N, int T, int Cin, int Cout,
                      int dtype, void* stream);

/* The equivariant linear layer over the dihedral group D_T (the T rotations
 * and T reflections of a regular T-gon), the reflection-group generalisation
 * that Sec. 5 names, run on the C_T entry points.  Group elements (t, m) =
 * r^t s^m are stored at m*T + t, so x [N,Cin,2T], y [N,Cout,2T], the weight
 * W [2T,Cout,Cin] (one Cout x Cin block per element) and b [Cout]; the layer
 * shares weights by the group law as the C_T layer does (Sec. 3.1, Eq. 1-2):
 *     y[n,o,g] = sum_h sum_c W[h^-1 g][o][c] x[n,c,h] + b[o].
 * Read as [N,2Cin,T] and [N,2Cout,T] (channel 2c+m), x and y are the input and
 * output of the C_T layer with 2Cin -> 2Cout channels and the weight
 *     w_ct[j][2o+mg][2c+mh] = W[(mg xor mh) T + ((-1)^mh j mod T)][o][c],
 * bias_ct[2o+mg] = b[o], so eqlinear_weight_spectrum, eqlinear_forward and
 * eqlinear_backward with (T, 2Cin, 2Cout) compute it, at the C_T layer's
 * T/2 saving over the dense sum.
 *
 * eqlinear_dihedral_expand writes w_ct [T,2Cout,2Cin] from W, and bias_ct
 * [2Cout] from bias (both NULL, or both non-NULL).
 * eqlinear_dihedral_fold writes the gradients with respect to W and b from
 * those of the C_T layer: dw [2T,Cout,Cin] from dw_ct [T,2Cout,2Cin] (each W
 * entry sums its two places in w_ct, in fp32, rounded once) and dbias [Cout]
 * from dbias_ct [2Cout] (both NULL, or both non-NULL).
 * Checks as for the other entry points (Cin, Cout <= 32768, element-aligned
 * pointers, no overlap); asynchronous on `stream`. */
int eqlinear_dihedral_expand(const void* w, const void* bias, void* w_ct, void* bias_ct, int T, int Cin,
                             int Cout, int dtype, void* stream);
int eqlinear_dihedral_fold(const void* dw_ct, const void* dbias_ct, void* dw, void* dbias, int T, int Cin,
                           int Cout, int dtype, void* stream);

/* The rotation-equivariant group convolution on a square grid, the
 * equivariant-convolution generalisation that Sec. 5 names, run on the C_T
 * entry points.  T in {1, 2, 4}: rotations by 360/T degrees act on the image
 * plane and on the group axis.  Features f [B,H,W,Cin,T], output
 * [B,H,W,Cout,T], weight psi [k,k,T,Cout,Cin] (k odd, at most 7; one
 * Cout x Cin block per window offset (a, b) and group lag, stored at
 * (a + k/2, b + k/2, lag)), bias [Cout]:
 *     out[n,o,r] = sum_{(a,b)} sum_s sum_c psi[R^-r (a,b)][(s - r) mod T][o][c]
 *                  * f[n + (a,b), c, s] + bias[o]
 * with f zero outside the image and R(a, b) = (-b, a) (T = 4), (-a, -b)
 * (T = 2).  Splitting the window into rotation orbits turns it into ONE C_T
 * layer with k*k*Cin input channels: eqlinear_gconv_gather writes its input
 * xcol [B*H*W, k*k*Cin, T] from f, eqlinear_gconv_pack_weight its weight
 * w_ct [T, Cout, k*k*Cin] from psi; eqlinear_weight_spectrum /
 * eqlinear_forward / eqlinear_backward with (T, k*k*Cin, Cout) then give the
 * output and the C_T gradients, eqlinear_gconv_scatter folds the gradient of
 * xcol back to df [B,H,W,Cin,T] (the adjoint of the gather, an fp32 sum of
 * each pixel's k*k entries) and eqlinear_gconv_unpack_weight the gradient of
 * w_ct back to dpsi [k,k,T,Cout,Cin] (a permutation).  The orbit order and
 * channel layout of xcol are documented in csrc/eql_gconv.h.  Checks as for
 * the other entry points (T not in {1, 2, 4} or k even or above 7 is
 * EQL_ERR_UNSUPPORTED); B, H or W = 0 is a no-op for the gather and scatter. */
int eqlinear_gconv_gather(const void* f, void* xcol, int64_t B, int H, int W, int T, int Cin, int k, int dtype,
                          void* stream);
int eqlinear_gconv_scatter(const void* dxcol, void* df, int64_t B, int H, int W, int T, int Cin, int k,
                           int dtype, void* stream);
int eqlinear_gconv_pack_weight(const void* psi, void* w_ct, int T, int Cin, int Cout, int k, int dtype,
                               void* stream);
int eqlinear_gconv_unpack_weight(const void* dw_ct, void* dpsi, int T, int Cin, int Cout, int k, int dtype,
                                 void* stream);

/* The weight of the adjoint convolution: the input gradient of the group
 * convolution is itself a group convolution of the output gradient,
 *     df[n, c, s] = sum_(a,b) sum_l sum_o psi'[R^-s (a,b)][l][c][o] dy[n + (a,b), o, (s + l) mod T]
 *     psi'[(a,b)][l][c][o] = psi[-R^-l (a,b)][-l mod T][o][c]
 * (the adjoint of the forward map above, Sec. 5), so it runs as the forward
 * of a layer with Cout inputs and Cin outputs and no bias.  Writes that
 * layer's C_T weight w_adj [T, Cin, k*k*Cout] from psi [k,k,T,Cout,Cin] (a
 * permutation); its spectrum (eqlinear_weight_spectrum with T, k*k*Cout,
 * Cin) feeds eqlinear_gconv_forward(dy, ..., Cin = Cout, Cout = Cin) or the
 * gather + eqlinear_forward pair, with no patch buffer of dy's gradient and
 * no scatter.  Checks as for eqlinear_gconv_pack_weight. */
int eqlinear_gconv_pack_weight_adjoint(const void* psi, void* w_adj, int T, int Cin, int Cout, int k, int dtype,
                                       void* stream);

/* The group convolution's forward pass without the patch buffer: y
 * [B,H,W,Cout,T] = eqlinear_forward of the gathered patches (T, k*k*Cin ->
 * Cout) with wspec the spectrum of eqlinear_gconv_pack_weight's w_ct and the
 * optional bias [Cout], the forward kernel reading each patch straight from f
 * [B,H,W,Cin,T] (Sec. 5's equivariant convolution on the method's kernels).
 * Same arithmetic, bit for bit, as eqlinear_gconv_gather followed by
 * eqlinear_forward.  Requires Cin a multiple of 4 and f below 2^31 bytes
 * (else EQL_ERR_UNSUPPORTED); f, y and wspec 16-byte aligned; other checks as
 * for eqlinear_forward and the gather.  B, H or W = 0 is a no-op. */
int eqlinear_gconv_forward(const void* f, const void* wspec, const void* bias, void* y, int64_t B, int H, int W,
                           int T, int Cin, int Cout, int k, int dtype, void* stream);

/* eqlinear_backward_weight without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid allocation).  Same operation and arguments (minus
 * the workspace) as eqlinear_backward_weight; the workspace contents live in
 * a file-scope static device array of EQLINEAR_STATIC_SCRATCH_BYTES per GPU
 * instead, and the call performs no allocation of any kind.  Wherever
 * eqlinear_backward_weight_workspace_bytes() <= EQLINEAR_STATIC_SCRATCH_BYTES
 * it runs the same kernels and gives the same bits; for wide layers whose
 * plan needs more (the transformed x and dy above) it plans the split-row
 * kernels instead, whose partials are smaller (same result up to rounding).
 * A problem whose partials still need more than the array returns
 * EQL_ERR_SCRATCH before any HIP call.
 * Every call on one GPU uses that GPU's one array, and every partial a call
 * reads it first writes in the same call, so nothing carries over between
 * calls; but two calls whose executions overlap on one GPU (different
 * streams, or host threads without ordering) race on the array and give
 * wrong results.  The first call on a device resolves the array's address
 * on that device once (EQL_ERR_LAUNCH if the runtime cannot). */
int eqlinear_backward_weight_noalloc(const void* x, const void* dy, void* dw, void* dbias, int64_t N,
                                     int T, int Cin, int Cout, int dtype, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* EQLINEAR_H */
