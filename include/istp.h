/*
 * istp.h: C ABI of the multiple-input, multiple-output irrep-signal tensor
 * products (arXiv 2602.21466, Section 4.3 and Appendix D) on MI355X (gfx950).
 *
 * Three products of two feature rows x1, x2, each the (s, s, s) case of the
 * irrep-signal tensor product with every input irrep lifted into one signal
 * and every output irrep read back from the one pointwise product:
 *
 *   ISTP_GAUNT  (s = 0, the Gaunt tensor product, Section 3.3).  A row holds
 *               one copy of each degree l = 0..L at index l^2 + l + m
 *               ((L+1)^2 values).  The output row holds degrees 0..2L at
 *               l^2 + l + m ((2L+1)^2 values): the integral over the sphere
 *               of f1 f2 conj(Y_l^m) with f_i = sum_lm x_i[l^2+l+m] Y_l^m.
 *
 *   ISTP_VECTOR (s = 1, the vector signal tensor product, Section 5).  A row
 *               holds the coefficients of the tensor harmonics Y^{l,1}_{j,m}
 *               of Definition 4.1 for the labels (j, l), l = 0..L,
 *               j = l-1, l, l+1 (j >= 0; for l = 0 only j = 1), ordered by l,
 *               then j, then m = -j..j: label (j, l) starts at
 *               istp_label_offset(1, j, l) = 3 l^2 + {0, 2l-1, 4l}[j-l+1]
 *               (3 (L+1)^2 values).  The output row holds the coefficients, in
 *               the same basis and order up to l = 2L (3 (2L+1)^2 values), of
 *               the 1 (x) 1 -> 1 coupled pointwise product
 *               g_q = sum C^{1 q}_{1 q1 1 q2} f1_q1 f2_q2 of the two vector
 *               signals f_i = sum x_i^{(j,l)}_m Y^{l,1}_{j,m}.
 *
 *   ISTP_TENSOR (s = 2, the general irrep-signal product of Section 4.3 with
 *               rank-2 tensor harmonics Y^{l,2}_{j,m}, Definition 4.1).  Labels
 *               (j, l), l = 0..L, j = |l-2|..l+2, ordered by l, then j, then
 *               m: label (j, l) starts at istp_label_offset(2, j, l) =
 *               5 l^2 + j^2 - (l-2)^2 (5 (L+1)^2 values).  The output holds the
 *               2 (x) 2 -> 2 coupled pointwise product
 *               g_q = sum C^{2 q}_{2 q1 2 q2} f1_q1 f2_q2 in the same basis up
 *               to l = 2L (5 (2L+1)^2 values).  The coupling is symmetric;
 *               gradients (istp_backward) exist up to L = 11 (fp32) and
 *               L = 9 (fp64).
 *
 * Basis: complex spherical harmonics with the Condon-Shortley phase; inputs
 * and outputs are real.  By Theorem 4.2 each output label (j3, l3) of the
 * vector product is a sum over input label pairs of K times the CGTP path
 * (x1^{(j1,l1)} (x) x2^{(j2,l2)})^{(j3)}.
 *
 * The result is computed the paper's way on an exact grid: lift (Legendre
 * synthesis on MFMA, then longitude FFTs), pointwise product, longitude FFTs,
 * Legendre projection on MFMA, recombination.  Grid: n_theta = 2L + 2
 * Gauss-Legendre rings, n_phi = smallest 2^a 3^b >= 4L + 1 longitudes, exact
 * for every output.
 *
 * Status codes are those of cgtp.h (CGTP_OK, CGTP_EINVAL, ...), and
 * cgtp_strerror / cgtp_last_hip_error apply.
 */
#ifndef ISTP_H
#define ISTP_H

#include <stdint.h>

#include "cgtp.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct istp_plan_s *istp_plan_t;

enum { ISTP_GAUNT = 0, ISTP_VECTOR = 1, ISTP_TENSOR = 2 };

/* Largest L: the projection accumulators must fit the register file. */
#define ISTP_MAX_L_FP32 33
#define ISTP_MAX_L_FP64 12
/* spin 2 (ISTP_TENSOR) bounds: staging its rows and rank-2 couplings */
#define ISTP_TENSOR_MAX_L_FP32 20
#define ISTP_TENSOR_MAX_L_FP64 12

/*
 * Builds the grid, the MFMA weight tables and the recombination table on the
 * current HIP device and uploads them (device memory owned by the plan).
 *   L     >= 0 (CGTP_EINVAL below; CGTP_EUNSUP above the limits above)
 *   spin  ISTP_GAUNT, ISTP_VECTOR or ISTP_TENSOR (else CGTP_EINVAL)
 *   dtype CGTP_FP32 or CGTP_FP64 (else CGTP_EDTYPE)
 * Returns CGTP_ENOMEM / CGTP_EHIP on allocation or copy failure; *plan_out is
 * written only on success.
 */
int istp_plan(int32_t L, int32_t spin, int32_t dtype, istp_plan_t *plan_out);

/*
 * out[n, :] = product of x1[n, :] and x2[n, :] for n < N.
 *   x1, x2: device arrays [N, istp_num_inputs(L, spin)], row-major, of the
 *           plan's dtype; out: device array [N, istp_num_outputs(L, spin)].
 *   All three 16-byte aligned; out must not overlap x1 or x2 (x1 == x2 is
 *   allowed); the current device must be the plan's.  Else CGTP_EINVAL.
 *   N == 0 returns CGTP_OK without a launch; N < 0 is CGTP_EINVAL.
 * Runs asynchronously on hip_stream (NULL: the default stream) and allocates
 * nothing; execution errors surface at the caller's next synchronisation.
 */
int istp_forward(istp_plan_t plan, const void *x1, const void *x2, void *out, int64_t N,
                 void *hip_stream);

/* Frees the plan's device tables.  NULL is a no-op. */
int istp_destroy(istp_plan_t plan);

/*
 * Multiplicity channels and label weights (the layer around the product).
 * A layer holds C channels of the input feature; equivariant linear maps
 * before and after the product can only scale each irrep label (Schur's
 * lemma; the degrees-of-freedom count of Appendix E), so each channel's
 * product is
 *   out[n, c] = wo[c] . P(w1[c] . x1[n, c], w2[c] . x2[n, c] or x2[n])
 * with "w . x" scaling every column of label k by w[k].
 *   channels:         C >= 1.
 *   x2_shared:        0: x2 is [N, C, n_in]; 1: x2 is [N, n_in], row n met by
 *                     every channel of pair n.
 *   weights_per_pair: 0: weight rows per channel, w1 / w2 [C, istp_num_labels(L)],
 *                     wo [C, istp_num_labels(2L)]; 1: per (pair, channel),
 *                     [N, C, ...].
 *   reserved:         must be 0.
 */
typedef struct {
    int32_t channels;
    int32_t x2_shared;
    int32_t weights_per_pair;
    int32_t reserved;
} istp_channels;

/*
 * Channel-wise forward product with label weights, asynchronously on
 * hip_stream.  x1: [N, C, istp_num_inputs(L, spin)]; out: [N, C,
 * istp_num_outputs(L, spin)]; x2 and the weights as described at
 * istp_channels; device arrays of the plan's dtype, row-major, contiguous;
 * x1, x2 and out 16-byte aligned, weights element-aligned.  Any of w1, w2,
 * wo may be NULL (all ones); ch == NULL means one channel, x2 not shared.
 * Label k of a weight row is the one istp_label_index returns.  CGTP_EINVAL
 * for a bad channel description, out overlapping any input, or byte counts
 * that overflow; otherwise as istp_forward.
 */
int istp_forward_weighted(istp_plan_t plan, const void *x1, const void *x2, const void *w1, const void *w2,
                          const void *wo, void *out, int64_t N, const istp_channels *ch, void *hip_stream);

/*
 * The signal products in the real spherical-harmonic basis.  Spin 0: real
 * harmonics with the Condon-Shortley phase carried over,
 *   Y^R_{l,m} = sqrt(2) (-1)^m Re Y_l^m (m > 0), Y_l^0 (m = 0),
 *               sqrt(2) (-1)^m Im Y_l^{|m|} (m < 0),
 * index l^2 + l + m.  x1, x2: [N, (L+1)^2] real-basis rows; out: [N, (2L+1)^2]
 * the real-basis coefficients of the integral of f1 f2 Y^R_{l3 m3}.  Spin 1
 * and 2 (rows in istp_forward's label layout): a real field's coefficients of
 * label (j, l) satisfy c_{-m} = sigma (-1)^m conj(c_m), sigma = (-1)^(l+s-j)
 * (the tensor harmonics' conjugation rule, Definition 4.1); each label with
 * sigma = +1 takes the scalar real basis above, each with sigma = -1 the
 * scalar real basis of i c.  The output is the real field of the coupled
 * pointwise product (Section 4.3); for spin 1, whose coupling is i / sqrt 2
 * times the cross product, the real basis of i times the product, so that two
 * constant fields give their cross product over sqrt 2 (label (1, 0) holds a
 * constant field's Cartesian (y, z, x) components times Y_0^0).
 * Spin 0 and 1: one launch of a kernel for real-basis rows (the real field's
 * symmetry makes each ring's scalar signal real and the spin-1 components
 * f_-1 = -conj f_+1, so the lift, products and projection take real and
 * imaginary parts where the complex product takes +m and -m); no workspace
 * (istp_real_workspace_bytes returns 0; workspace may be NULL,
 * workspace_bytes must be >= 0).  Spin 2: the inputs are
 * converted to the real and imaginary parts of their complex coefficients,
 * three products of those parts run on the plan's kernel (Karatsuba's form:
 * P(a1, a2), P(b1, b2), P(a1 + b1, a2 + b2)), and the result is read back in
 * the real basis; workspace: caller-owned device memory of
 * istp_real_workspace_bytes(plan, N) bytes or more, 256-byte aligned, not
 * overlapping the other buffers (its contents are scratch).  Otherwise as
 * istp_forward.
 */
int istp_forward_real(istp_plan_t plan, const void *x1, const void *x2, void *out, int64_t N, void *workspace,
                      int64_t workspace_bytes, void *hip_stream);

/* Workspace bytes istp_forward_real needs for N pairs (0 for spin 0 and 1); -1 for N < 0 or overflow. */
int64_t istp_real_workspace_bytes(istp_plan_t plan, int64_t N);

/*
 * istp_forward_real for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same kernels, with the workspace of spin 2 taken from a
 * static device array of ISTP_STATIC_SCRATCH_BYTES (64 MiB) that the library
 * holds on each GPU it runs on until the process ends (spins 0 and 1 need
 * none).  Same arguments and rules as istp_forward_real without the
 * workspace; the plan's device must be current.  CGTP_ESCRATCH when
 * istp_real_workspace_bytes(plan, N) exceeds the array (fp32 spin 2: above
 * 2479 pairs at L = 8, 670 at L = 16).  The
 * entry point calls no allocating routine; every call on a GPU shares that
 * GPU's array, so calls that overlap in time on one GPU (concurrent streams)
 * race and must be ordered by the caller.  Nothing in the array needs to
 * start at zero.
 */
#define ISTP_STATIC_SCRATCH_BYTES (64LL << 20)
int istp_forward_real_static(istp_plan_t plan, const void *x1, const void *x2, void *out, int64_t N,
                             void *hip_stream);

/*
 * Gradients of sum(grad_out * out) for istp_forward_real, in the real basis.
 * The integrals of three real harmonics are fully symmetric, so
 *   grad_x1 = Q(grad_out, x2),  grad_x2 = Q(grad_out, x1),
 * with Q the real-basis product of a degree-2L and a degree-L row projected on
 * degrees <= L (on the plan's gradient grid; no time reversal): one launch of
 * the real-basis kernel per gradient where the plan holds its real-basis
 * gradient product (no workspace), else three products between conversions.
 * Layouts and rules as istp_backward; workspace: caller-owned, 256-byte
 * aligned, istp_real_backward_workspace_bytes(plan, N) bytes or more (0: may
 * be NULL), reused by the two gradients.  CGTP_EUNSUP for spin 1 or 2 plans
 * and where the plan has no gradient product.
 */
int istp_backward_real(istp_plan_t plan, const void *x1, const void *x2, const void *grad_out, void *grad_x1,
                       void *grad_x2, int64_t N, void *workspace, int64_t workspace_bytes, void *hip_stream);

/* Workspace bytes istp_backward_real needs for N pairs; -1 where it does not apply. */
int64_t istp_real_backward_workspace_bytes(istp_plan_t plan, int64_t N);

/*
 * Gradients of sum(grad_out * out) for istp_forward_weighted with x2 per
 * channel (x2_shared must be 0: its gradient would sum over the channels,
 * CGTP_EUNSUP).  By the chain rule through the label weights,
 *   grad_x1 = w1 . P'(wo . grad_out, w2 . x2~),  grad_x2 = +-w2 . P'(wo . grad_out, w1 . x1~),
 * with P' and x~ as for istp_backward; the channel kernel runs them on the
 * gradient grid.  Layouts as istp_forward_weighted (grad_x1, grad_x2 like x1);
 * rules as istp_backward.  CGTP_EUNSUP where the plan's gradient product needs
 * lifts beyond 36 degrees (L > 17) or does not exist.  Gradients with respect
 * to the weights are not computed.
 */
int istp_backward_weighted(istp_plan_t plan, const void *x1, const void *x2, const void *w1, const void *w2,
                           const void *wo, const void *grad_out, void *grad_x1, void *grad_x2, int64_t N,
                           const istp_channels *ch, void *hip_stream);

/* Irrep labels in a row of degree bound L: L + 1 (spin 0), 3 L + 1 (spin 1); -1 if invalid. */
int64_t istp_num_labels(int32_t L, int32_t spin);

/* Position of label (j, l) in a weight row: l (spin 0, j == l); 2 l - 1 + j (spin 1,
   the row order of the labels); -1 if it is not a label. */
int64_t istp_label_index(int32_t spin, int32_t j, int32_t l);

/* Values per input row: (L+1)^2 (spin 0), 3 (L+1)^2 (spin 1); -1 if invalid. */
int64_t istp_num_inputs(int32_t L, int32_t spin);

/* Values per output row: (2L+1)^2 (spin 0), 3 (2L+1)^2 (spin 1); -1 if invalid. */
int64_t istp_num_outputs(int32_t L, int32_t spin);

/*
 * First value of irrep label (j, l) in a row: spin 0 needs j == l and gives
 * l^2; spin 1 gives 3 l^2 + {0, 2l-1, 4l}[j-l+1].  -1 if not a label.
 */
int64_t istp_label_offset(int32_t spin, int32_t j, int32_t l);

/*
 * Plan facts: grid sizes, pairs per work-group, and the model counts per
 * pair.  flops_per_pair counts the method's arithmetic on the exact grid (one
 * complex FFT = 5 n log2 n): Legendre synthesis 2 per (l, m) per input
 * component per ring pair; 2 C complex FFTs per ring pair (north and south in
 * one transform); the products on the half circle (6 per complex multiply,
 * 2 per complex add); C complex FFTs per ring pair back; Legendre projection
 * 2 per (l3, m) per component per ring pair; recombination 2 per term.
 * bytes_per_pair = (2 inputs + 1 output) values in HBM.  Any pointer may be
 * NULL.
 */
int istp_plan_query(istp_plan_t plan, int32_t *n_theta, int32_t *n_phi, int32_t *pairs_per_group,
                    double *flops_per_pair, double *bytes_per_pair);

/*
 * Gradients (vector-Jacobian product) of istp_forward: with g = dLoss/dout
 * ([N, istp_num_outputs], real),
 *   grad_x1[n, :] = dLoss/dx1[n, :],  grad_x2[n, :] = dLoss/dx2[n, :].
 * The product is bilinear, so each is again a signal product, the adjoint of
 * the forward pipeline: by the symmetry of the integral of three harmonics,
 *   grad_x1 = P(g, x2~),  grad_x2 = +-P(g, x1~)  (- for the vector product,
 *   which is antisymmetric),
 * where P is the same kind of product of a degree-2L and a degree-L signal
 * projected on degrees <= L (the same exact grid), and x~ is the input
 * time-reversed: x~[(j,l), m] = (-1)^(m + j - l + s) x[(j,l), -m].
 *   x1, x2, grad_x1, grad_x2: [N, istp_num_inputs]; grad_out: [N,
 *   istp_num_outputs]; all 16-byte aligned device arrays of the plan's dtype.
 *   Either gradient pointer may be NULL (not computed), not both.  A gradient
 *   may not overlap any input or the other gradient (CGTP_EINVAL).
 * CGTP_EUNSUP when the plan's gradient product is outside the kernel's limits
 * (the degree-2L lift's LDS and register budget; istp_backward_query says).
 * Asynchronous on hip_stream; allocates nothing.
 */
int istp_backward(istp_plan_t plan, const void *x1, const void *x2, const void *grad_out, void *grad_x1,
                  void *grad_x2, int64_t N, void *hip_stream);

/*
 * The gradient product's facts: pairs per work-group, and the model counts
 * per pair of both gradients (two launches; the counting rules of
 * istp_plan_query).  CGTP_EUNSUP when the plan has no gradient product.
 */
int istp_backward_query(istp_plan_t plan, int32_t *pairs_per_group, double *flops_per_pair,
                        double *bytes_per_pair);

/*
 * Host-only: the geometry a plan for (L, spin, dtype) would use, without a
 * device.  Writes 48 int32 values to desc_out: the forward product's
 * descriptor, then the gradient product's (all zero when outside the
 * kernel's limits).  Each descriptor: first and second input degree bounds,
 * output degree bound, spin, components, north rings R, ring pairs per group
 * G, n_phi, its factors A and B, pairs per work-group, values per first
 * input, second input and output row, lift and projection MFMA tiles, lift
 * operand elements, end-phase elements per pair, lift and projection
 * weight-table elements, projection row length, LDS bytes per work-group,
 * lift operand columns, flags.  Status codes as istp_plan.
 */
int istp_plan_describe(int32_t L, int32_t spin, int32_t dtype, int32_t *desc_out);

#ifdef __cplusplus
}
#endif

#endif /* ISTP_H */
