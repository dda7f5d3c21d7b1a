/*
 * cgtp.h - C ABI of the MI355X (gfx950) full Clebsch-Gordan tensor product.
 *
 * The library computes, for N pairs of real irrep features x1, x2 holding one
 * copy of every degree 0..L (the (0 + 1 + ... + L) representation of
 * Appendix B), every Clebsch-Gordan path
 *
 *   z^(l1,l2,l3)_m3 = sum_{m1,m2} C^{l3 m3}_{l1 m1 l2 m2} x1^(l1)_m1 x2^(l2)_m2
 *
 * (the CGTP of Section 1 and Appendix F.1), the paper's way: each (l1, l2)
 * block is one irrep-signal tensor product (Section 4.3).  Both inputs are
 * lifted to scalar and toroidal vector signals on a sphere grid (tensor
 * spherical harmonics, Definition 4.1), multiplied pointwise (scalar-scalar
 * product and cross product, Section 5.1, or scalar-vector and dot product
 * for the alternate cover), transformed back, and each path is divided by the
 * factor the generalized Gaunt formula (Theorem 4.2) fixes.  Corollary 5.3 is
 * what makes one such product per block enough.
 *
 * Conventions: complex spherical basis with Condon-Shortley phase
 * (quantum-mechanics conventions, footnote of Section 3.3); coefficients are
 * real numbers in that basis.  Index of (l, m) in a feature row: l^2 + l + m.
 *
 * Errors: every entry point returns a cgtp_status code; nothing is printed,
 * no exception crosses the ABI, and a call that fails validation launches no
 * GPU work.
 */
#ifndef CGTP_H
#define CGTP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
enum cgtp_status {
    CGTP_OK = 0,
    CGTP_EINVAL = -1, /* bad argument: NULL pointer, negative size, misaligned or overlapping buffers */
    CGTP_EGRID = -2,  /* grid too small to integrate the products exactly (it would alias) */
    CGTP_EDTYPE = -3, /* unknown dtype */
    CGTP_ENOMEM = -4, /* host or device allocation failed */
    CGTP_EHIP = -5,   /* a HIP runtime call failed; cgtp_last_hip_error() has the HIP code */
    CGTP_EUNSUP = -6, /* valid request this build does not support (L above CGTP_MAX_L, FFT size) */
    CGTP_ESCRATCH = -7 /* request larger than a no-allocation entry point's static scratch */
};

enum cgtp_dtype { CGTP_FP32 = 0, CGTP_FP64 = 1 };

/* Which products recover the paths (Corollary 5.3 leaves the choice open). */
enum cgtp_cover {
    /* even l1+l2+l3: scalar-scalar product (the Gaunt product, Section 3.3);
       odd: cross product of the two toroidal vector lifts (l = j, s = 1),
       projected on the l3 - 1 vector harmonics (Section 5.1). */
    CGTP_COVER_DEFAULT = 0,
    /* even: dot product of the toroidal lifts; odd: scalar x1 times toroidal
       x2.  Blocks (l1, l2) with a degree-0 input use the scalar-scalar
       product.  A block in which the dot-product factor of some even path
       vanishes by accident (l1(l1+1) + l2(l2+1) = l3(l3+1), e.g. (3, 5, 6))
       uses the scalar-scalar product for all its even paths; likewise the
       cross product for its odd paths if a scalar-vector factor vanishes.
       Same result as the default cover up to rounding. */
    CGTP_COVER_ALTERNATE = 1
};

#define CGTP_MAX_L 32

/*
 * Grid choice.  A zero field takes the default.
 *   n_theta: 0 -> per-block minimal exact Gauss-Legendre grid (2*floor((l1+l2)/2)+2
 *            nodes); else one grid for all blocks with this many nodes, which
 *            must be even and >= 2L+2 (else CGTP_EGRID for < 2L+1, CGTP_EUNSUP
 *            for odd values).
 *   n_phi:   0 -> per-block smallest 2^a 3^b >= 2(l1+l2)+1 longitudes; else one
 *            size for all blocks, which must be >= 4L+1 (else CGTP_EGRID), at
 *            most 144 and of the form 2^a 3^b (else CGTP_EUNSUP).
 *   dtype:   CGTP_FP32 or CGTP_FP64; inputs and output share it.
 *   cover:   enum cgtp_cover.
 */
typedef struct {
    int32_t n_theta;
    int32_t n_phi;
    int32_t dtype;
    int32_t cover;
} cgtp_grid;

typedef struct cgtp_plan_s *cgtp_plan_t;

/*
 * Builds a plan for degree L on the current HIP device: quadrature nodes,
 * normalised associated Legendre tables, Clebsch-Gordan tables for the lifts
 * and the recombination, and 1/K for every path (Theorem 4.2), uploaded to
 * device memory the plan owns.  grid == NULL takes every default.
 * Returns CGTP_EINVAL (L < 0, plan_out NULL), CGTP_EUNSUP (L > CGTP_MAX_L,
 * or a block whose projection accumulators do not fit one work-group: fp64
 * plans support L <= 19), CGTP_EDTYPE, CGTP_EGRID, CGTP_ENOMEM or CGTP_EHIP;
 * *plan_out is set only on success.  Not timed work: call once per (L, grid).
 */
int cgtp_plan(int32_t L, const cgtp_grid *grid, cgtp_plan_t *plan_out);

/*
 * Full CGTP of N pairs, asynchronously on hip_stream (NULL: the default
 * stream).  x1, x2: device arrays [N, (L+1)^2]; out: device array
 * [N, (L+1)^4]; all row-major, contiguous, of the plan's dtype, 16-byte
 * aligned.  Path (l1, l2, l3) of pair n occupies out[n, cgtp_path_offset(L,
 * l1, l2, l3) + l3 + m3], m3 = -l3..l3.  The caller owns all three buffers;
 * this call allocates nothing.  x1 == x2 is allowed; out overlapping an input
 * is CGTP_EINVAL.  N == 0 returns CGTP_OK with no launch.  Launch failures
 * return CGTP_EHIP; faults during execution surface when the caller
 * synchronises.  A plan may be used from several streams at once.  The
 * current device must be the one the plan was built on (else CGTP_EINVAL).
 */
int cgtp_forward(cgtp_plan_t plan, const void *x1, const void *x2, void *out, int64_t N,
                 void *hip_stream);

/*
 * Multiplicity channels and path weights.  A network layer carries C copies
 * (channels) of every irrep; the method is applied to each channel, and the
 * output of every path is scaled by a weight, the per-irrep linear maps
 * around the tensor product that the expressivity count of Appendix E
 * allows (Schur's lemma leaves one scalar per path).
 *   channels:          C >= 1.
 *   x2_shared:         0: x2 is [N, C, (L+1)^2], channel c of pair n meets
 *                      channel c of x1; 1: x2 is [N, (L+1)^2], row n meets
 *                      every channel of pair n (e.g. spherical harmonics of
 *                      an edge direction).
 *   weights_per_pair:  0: weights [C, P], shared by all pairs (a layer's
 *                      parameters); 1: weights [N, C, P] (per-pair weights,
 *                      e.g. from a radial network).  P = cgtp_num_paths(L).
 *   reserved:          must be 0.
 */
typedef struct {
    int32_t channels;
    int32_t x2_shared;
    int32_t weights_per_pair;
    int32_t reserved;
} cgtp_channels;

/*
 * Channel-wise CGTP with path weights, asynchronously on hip_stream.
 *   out[n, c, cgtp_path_offset(L, l1, l2, l3) + l3 + m3]
 *     = w[(n,) c, cgtp_path_index(L, l1, l2, l3)] * z^(l1,l2,l3)_m3(x1[n, c], x2[n, c] or x2[n])
 * x1: [N, C, (L+1)^2]; out: [N, C, (L+1)^4]; x2 and weights as described at
 * cgtp_channels; all device arrays of the plan's dtype, row-major and
 * contiguous; x1, x2 and out 16-byte aligned, weights element-aligned.
 * weights == NULL means every weight is 1; ch == NULL means one channel,
 * x2 not shared.  CGTP_EINVAL for a bad channel description, out overlapping
 * any input, or sizes whose byte count overflows.  Otherwise as cgtp_forward
 * (which equals this call with C = 1 and no weights).
 */
int cgtp_forward_weighted(cgtp_plan_t plan, const void *x1, const void *x2, const void *weights, void *out,
                          int64_t N, const cgtp_channels *ch, void *hip_stream);

/*
 * Gradients of sum(grad_out * out) for cgtp_forward:
 *   grad_x1[n, (l1, m1)] = sum over paths and m2, m3 of C^{l3 m3}_{l1 m1 l2 m2} x2[n, (l2, m2)] grad_out[n, (l1, l2, l3), m3]
 *   grad_x2[n, (l2, m2)] = sum over paths and m1, m3 of C^{l3 m3}_{l1 m1 l2 m2} x1[n, (l1, m1)] grad_out[n, (l1, l2, l3), m3]
 * (the CGTP is bilinear: each gradient is the transpose of a linear map).
 * Computed by the method of the forward call run backwards, block by block
 * (Section 4.3): the adjoint of every stage (recombination and 1/K, Legendre
 * projection, longitude analysis, pointwise products, longitude synthesis,
 * lift), on the same grids and with the same tables, so the result equals the
 * double sum above up to rounding.
 *   x1, x2, grad_x1, grad_x2: device arrays [N, (L+1)^2]; grad_out: [N,
 *   (L+1)^4] in cgtp_forward's output layout; all of the plan's dtype,
 *   row-major, contiguous, 16-byte aligned.  Either gradient pointer may be
 *   NULL (not written), not both.
 *   workspace: caller-owned device memory, 256-byte aligned, at least
 *   cgtp_backward_workspace_bytes(plan, N) bytes (each block's contribution
 *   to both gradients of every pair, summed afterwards in a fixed order, so
 *   results do not depend on scheduling).  Contents on entry are ignored.
 * CGTP_EINVAL for NULL inputs, misalignment, a short workspace, or a
 * gradient or the workspace overlapping any other buffer; CGTP_EUNSUP when a
 * block of the plan does not fit the gradient kernel or N (L+1)^2 exceeds
 * 2^31 - 1.  Asynchronous on hip_stream; allocates nothing; N == 0 returns
 * CGTP_OK with no launch.  The plan's device must be current.
 */
int cgtp_backward(cgtp_plan_t plan, const void *x1, const void *x2, const void *grad_out, void *grad_x1,
                  void *grad_x2, int64_t N, void *workspace, int64_t workspace_bytes, void *hip_stream);

/* Workspace bytes cgtp_backward needs for N pairs: 2 (L+1)^3 N elements; -1 for a NULL plan, N < 0 or overflow. */
int64_t cgtp_backward_workspace_bytes(cgtp_plan_t plan, int64_t N);

/*
 * Model counts per pair of cgtp_backward (both gradients): the forward's
 * algorithmic flops (cgtp_plan_query) plus the adjoint's extra work, i.e. the
 * products' adjoint forms both factors' gradients (the products term twice)
 * and the transposed synthesis costs what the lift does; compulsory bytes:
 * x1, x2, grad_x1, grad_x2 and grad_out, each once.  Either pointer may be
 * NULL.  CGTP_EINVAL for a NULL plan, CGTP_EUNSUP where cgtp_backward is.
 */
int cgtp_backward_query(cgtp_plan_t plan, double *flops_per_pair, double *bytes_per_pair);

/*
 * The full CGTP in the real spherical-harmonic basis (the paper works with real
 * signals on the sphere, Section 3.3).  Real harmonics, Condon-Shortley phase
 * kept, index l^2 + l + m:
 *   Y^R_{l,m} = sqrt(2) (-1)^m Re Y_l^m (m > 0),  Y_l^0 (m = 0),  sqrt(2) (-1)^m Im Y_l^|m| (m < 0).
 * x1, x2 hold real-basis coefficients [N, (L+1)^2]; out [N, (L+1)^4] in
 * cgtp_forward's layout holds every path in the real basis: the complex-basis
 * CGTP of the inputs' (Hermitian) complex coefficients, path by path read back
 * in the real basis, odd l1 + l2 + l3 paths (anti-Hermitian) after a factor i.
 * So the even paths are the real Gaunt integrals over K (Theorem 4.2 read in the
 * real basis) and path (1, 1, 1) is the cross product over sqrt(2) in the real
 * basis' (y, z, x) order.  One launch of the block kernel's real-basis
 * variant: the inputs' Hermitian coefficients make every lifted signal real
 * (or i times real, or a conjugate pair), so a cross block still needs two
 * transforms per input; the end phase forms the real-basis outputs.
 *   workspace, workspace_bytes: unused (kept for callers of an earlier version
 *   that needed one); workspace may be NULL, workspace_bytes must be >= 0.
 * Rules otherwise as cgtp_forward.  Allocates nothing; asynchronous on
 * hip_stream.
 */
int cgtp_forward_real(cgtp_plan_t plan, const void *x1, const void *x2, void *out, int64_t N, void *workspace,
                      int64_t workspace_bytes, void *hip_stream);

/* Workspace bytes cgtp_forward_real needs for N pairs: 0; -1 for a NULL plan or N < 0. */
int64_t cgtp_real_workspace_bytes(cgtp_plan_t plan, int64_t N);

/* Number of paths of degree L: sum over l1, l2 <= L of 2 min(l1, l2) + 1; -1 for L < 0. */
int64_t cgtp_num_paths(int32_t L);

/* Index of path (l1, l2, l3) in the (l1, l2, l3) order of all paths of degree L
   (the layout of a weight row); -1 if it is not a path. */
int64_t cgtp_path_index(int32_t L, int32_t l1, int32_t l2, int32_t l3);

/* Frees the plan's device tables.  NULL is a no-op. */
int cgtp_destroy(cgtp_plan_t plan);

/* (L+1)^4, the output count per pair; -1 for L < 0. */
int64_t cgtp_num_outputs(int32_t L);

/* Offset of path (l1, l2, l3) within one pair's output: l1^2 (L+1)^2 +
   (2 l1 + 1) l2^2 + l3^2 - (l1 - l2)^2; -1 if (l1, l2, l3) is not a path of
   degree L. */
int64_t cgtp_path_offset(int32_t L, int32_t l1, int32_t l2, int32_t l3);

/*
 * Plan facts: the largest grid used (n_theta, n_phi), the smallest |K| over
 * the recovered paths, the algorithmic flops per pair of the method (every
 * block on its minimal exact grid: lifts, longitude transforms at
 * 2.5 n log2 n flops per Hermitian transform of n points, pointwise products,
 * Legendre projection, recombination; the default cover's products whatever
 * the plan's cover), and the compulsory HBM bytes per pair
 * (inputs read once, output written once).  Any pointer may be NULL.
 */
int cgtp_plan_query(cgtp_plan_t plan, int32_t *n_theta, int32_t *n_phi, double *min_abs_K,
                    double *flops_per_pair, double *bytes_per_pair);

/* Static text for a status code. */
const char *cgtp_strerror(int code);

/* HIP error code of the last CGTP_EHIP on this thread (0 if none). */
int cgtp_last_hip_error(void);

/* ---- host-side math the plan is built from (no GPU needed) ---- */

/*
 * Per-path normalisation K of Theorem 4.2 for the product the given cover uses
 * on path (j1, j2, j3): raw projection = K * z.  *kind receives 0 for the
 * scalar-scalar product, 1 for the cross product, 2 for scalar-vector, 3 for
 * the dot product (the alternate cover's fall-backs are per block, as
 * described at CGTP_COVER_ALTERNATE).  Returns CGTP_EINVAL if (j1, j2, j3) violates the triangle
 * rule or any degree is negative.
 */
int cgtp_path_norm(int32_t j1, int32_t j2, int32_t j3, int32_t cover, double *K, int32_t *kind);

/* Wigner 9j symbol {a b c; d e f; g h i} (sum over products of three 6j
   symbols; the recoupling coefficient defined in Appendix F.1), for testing the closed forms. */
double cgtp_wigner_9j(int32_t a, int32_t b, int32_t c, int32_t d, int32_t e, int32_t f, int32_t g,
                      int32_t h, int32_t i);

/* Clebsch-Gordan coefficient C^{j m}_{j1 m1 1 q} for coupling with a vector
   (closed forms of the j2 = 1 table); 0 outside the selection rules. */
double cgtp_cg_vector(int32_t j1, int32_t m1, int32_t q, int32_t j, int32_t m);

/* C^{l3 0}_{l1 0 l2 0} from the closed form of the 3j symbol with zero
   projections; 0 when l1 + l2 + l3 is odd or the triangle rule fails. */
double cgtp_cg_zero(int32_t l1, int32_t l2, int32_t l3);

/* n Gauss-Legendre nodes (descending, x[0] closest to +1) and weights. */
int cgtp_gauss_legendre(int32_t n, double *x, double *w);

/* Normalised associated Legendre values P^m_l(x) with Condon-Shortley phase,
   Y_l^m = P^m_l(cos theta) e^{i m phi}, for 0 <= m <= l <= lmax, written at
   out[l (l + 1) / 2 + m]. */
int cgtp_legendre(int32_t lmax, double x, double *out);

/* Grid a block (l1, l2) uses under the given grid request: number of
   Gauss-Legendre nodes (even; the kernel visits n_theta / 2 northern rings)
   and longitudes. */
int cgtp_block_grid(int32_t L, const cgtp_grid *grid, int32_t l1, int32_t l2, int32_t *n_theta,
                    int32_t *n_phi);

#ifdef __cplusplus
}
#endif

#endif /* CGTP_H */
