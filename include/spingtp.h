/*
 * spingtp.h -- C ABI of the spin-weighted Gaunt tensor product (SpinGTP) on
 * AMD MI355X (gfx950).
 *
 * The operation (paper Sec. 3.2 eq. generalized_gaunt, Sec. 3.3 eq. real_swsh,
 * App. B proof of the runtime proposition, App. C):
 *
 *   For every unit (edge n, channel c) independently, with real-basis spin-weighted
 *   spherical-harmonic (SWSH) coefficients x1 (degree <= L1) and x2 (degree <= L2),
 *   both carrying the spins listed in `spins`:
 *     a_i   = Q x_i                                (real -> complex, App. C)
 *     f_i,s = sum_{l,m} a_i[s,l,m] sY_lm           (spin-weighted fields on S^2)
 *     h_s3  = sum_{s1+s2=s3} f_1,s1 * f_2,s2       (pointwise product, s3 in spins)
 *     c[s3,l3,m3] = int h_s3 conj(s3Y_l3m3) dOmega (l3 <= Lout)
 *     out   = Re(Q^dagger c)                       (complex -> real, App. C)
 *   i.e. out[k3] = sum G x1 x2 with G the spin-weighted Gaunt coefficients.
 *   Spin pairs with the same s3 are summed with no normalisation; products with
 *   s3 outside `spins` (e.g. s3 = +-2 for spins {-1,0,+1}) are dropped.  This is the
 *   elementwise channel mode ("uuu", App. E.1) with unit path weights.
 *
 * Layout of x1, x2, out (all dense, row-major, same dtype):
 *   x1  [N][C][n_spins][(L1+1)^2],  x2 [N][C][n_spins][(L2+1)^2],
 *   out [N][C][n_spins][(Lout+1)^2].
 *   The spin axis holds the real-basis sector spins[i] (spins strictly ascending,
 *   the -|s| sector first as in App. C).  Inside a spin block the flat index is
 *   l^2 + l + k with k = -l..l ascending.  Slots with l < |s| are ignored on input
 *   and written as 0 on output.
 *
 * Real basis at m = 0 for |s| > 0 (the paper's eq. real_swsh sets sR_l0 = sY_l0):
 *   SPINGTP_BASIS_REAL_PAPER      that definition literally (default);
 *   SPINGTP_BASIS_REAL_M0_PAIRED  the m = 0 pair (s,0),(-s,0) mixed as
 *                                 (1/sqrt2)(1, (-1)^s) and (i/sqrt2)(1, -(-1)^s),
 *                                 which makes the real basis closed under rotation;
 *   SPINGTP_BASIS_PARITY          the parity-labelled basis of Sec. 3.4 eq.
 *                                 parity_basis, built on the paper basis:
 *                                 R_p = (R_{-s} + p (-1)^l R_s)/sqrt2, p = +-1, for
 *                                 |s| > 0; the coefficient of p = +1 is stored in
 *                                 the -|s| block and that of p = -1 in the +|s|
 *                                 block (s = 0 unchanged).
 *
 * Threading and ownership: a plan is immutable after creation; concurrent
 * spingtp_forward calls with one plan on different streams or threads are safe.
 * The caller owns x1, x2 and out.  No call keeps global error state.
 */
#ifndef SPINGTP_H
#define SPINGTP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct spingtp_plan_s* spingtp_plan; /* opaque */

typedef enum {
    SPINGTP_OK = 0,
    SPINGTP_ERR_INVALID_ARG = 1,   /* bad degree, spin list, pointer, alignment or size */
    SPINGTP_ERR_UNSUPPORTED = 2,   /* valid by the paper but not built in this library */
    SPINGTP_ERR_OUT_OF_MEMORY = 3, /* device allocation failed */
    SPINGTP_ERR_HIP = 4,           /* a HIP runtime call or kernel launch failed */
    SPINGTP_ERR_INTERNAL = 5,      /* plan self-check failed (a library bug) */
    SPINGTP_ERR_TOO_LARGE = 6      /* the request needs more than the library's fixed device scratch */
} spingtp_status;

typedef enum { SPINGTP_FP32 = 0, SPINGTP_BF16 = 1 } spingtp_dtype;

#define SPINGTP_BASIS_REAL_PAPER 0u
#define SPINGTP_BASIS_REAL_M0_PAIRED 1u
#define SPINGTP_BASIS_PARITY 2u

/* Kernel choice, OR-ed into the flags of spingtp_plan_create: use the fp32
 * vector-ALU kernels even where a matrix-core kernel is built (family 4 below).
 * The other entry points accept and ignore it. */
#define SPINGTP_KERNEL_VALU 0x100u

/* Route of spingtp_forward_v1, OR-ed into the flags of spingtp_plan_create
 * (at most one of the two): SPINGTP_V1_FOURIER takes the Fourier-route kernels
 * (the ones spingtp_forward uses, reading x2 per edge) even where the
 * precontracted kernel (family 5 below) is the default; SPINGTP_V1_PRECONTRACT
 * takes the precontracted kernel wherever it is built (SPINGTP_ERR_UNSUPPORTED
 * where it is not).  Without either, the precontracted kernel is used for row
 * lengths n_spins (L+1)^2 <= 75 in L1 and Lout (degree <= 4 with spins
 * {-1, 0, +1}, where it is the faster route) and for shapes with no
 * Fourier-route kernel. */
#define SPINGTP_V1_FOURIER 0x200u
#define SPINGTP_V1_PRECONTRACT 0x400u

/* Also build the tables of spingtp_forward_v1_weighted (per-channel path weights),
 * OR-ed into the flags of spingtp_plan_create. */
#define SPINGTP_CHANNEL_WEIGHTS 0x1000u
/* plan also holds the entry tables of spingtp_forward_fully_connected and
 * spingtp_backward_fully_connected (mode uvw).  With this flag spingtp_pre_table_host
 * returns the forward's entry table, and with SPINGTP_TABLES_BACKWARD as well the tables
 * of the gradients w.r.t. x1 and then x2, one after the other (the tensor read as
 * T[k2, k3 -> k1] and T[k1, k3 -> k2]); each starts with the 8-word header described
 * with the plan's tables in the source (n_paths, n_blocks, the row widths of its two
 * inputs and its output, max block width, first word of the path records, first word
 * of the entries; a path record is 6 words, an entry 2). */
#define SPINGTP_FULLY_CONNECTED 0x2000u

/* For spingtp_plan_tables_host only: return the tables spingtp_backward uses
 * (input 2's m = 0 mixing with the conjugation folded in). */
#define SPINGTP_TABLES_BACKWARD 0x800u

/*
 * Create a plan for degrees (L1, L2, Lout) and a spin set.
 *   0 <= L1, L2 <= 16, 0 <= Lout <= L1 + L2 (the product of degrees l1, l2 has
 *   degree <= l1 + l2, App. B proof); otherwise SPINGTP_ERR_INVALID_ARG.
 *   spins/n_spins: host array, strictly ascending and symmetric; {0},
 *   {-1, 0, +1} and {-2, -1, 0, +1, +2} (s_max = 2) are supported, other valid
 *   sets give SPINGTP_ERR_UNSUPPORTED.  Spins {-2..2} run on the direct kernel
 *   (family 6) and, for spingtp_forward_v1, on the precontracted kernel.
 *   dtype: element type of x1, x2 and out.  Arithmetic: the vector-ALU kernels
 *   compute in fp32.  The matrix-core kernel (L1 = L2 = Lout = 4..8, spins
 *   {-1, 0, +1}) runs the two phi transforms as fp16 matrix products with fp32
 *   accumulation: for fp32 plans every operand is split into fp16 high and low
 *   parts (three products per term, relative error near 2^-21 per term, like
 *   fp32), for bf16 plans only the high parts are used (near 2^-11).  Every
 *   other step is fp32.  bf16 output is rounded to nearest even.
 *   flags: one SPINGTP_BASIS_* value, optionally OR SPINGTP_KERNEL_VALU and one of
 *   SPINGTP_V1_FOURIER, SPINGTP_V1_PRECONTRACT.
 * A shape with no Fourier kernel (families 1-4) runs spingtp_forward on the
 * direct kernel (family 6) where its LDS tile fits (64 n_spins ((L1+1)^2 +
 * (L2+1)^2 + (Lout+1)^2) floats plus padding within 160 KB, rows of at most 254
 * slots); beyond that, with spins {0} or {-1, 0, +1}, on the large-degree kernel
 * (family 3) of L = max(L1, L2, Lout): x1 and x2 are padded with zeros to degree
 * L as the kernel stages them and the degree-L product is stored up to Lout,
 * which is exact since that kernel's grid integrates degree 3 L >= L1 + L2 + Lout
 * (forward, spingtp_forward_v1 and the gradients of spingtp_backward and
 * spingtp_backward_v1, the degree-L ones of the padded functions, truncated).
 * A shape that only the precontracted kernel of
 * spingtp_forward_v1 covers gives a plan for that entry point, and
 * spingtp_forward and spingtp_plan_kernel_info then return
 * SPINGTP_ERR_UNSUPPORTED.
 * The plan tables (Gauss-Legendre weights and SWSH values on the quadrature
 * nodes, trigonometric tables, real-basis mixing constants) are computed in
 * float64 on the host, rounded to fp32 and copied synchronously to the current
 * HIP device, which the plan is bound to.  *out_plan receives the handle; on any
 * error it is set to NULL and nothing is leaked.
 */
spingtp_status spingtp_plan_create(int L1, int L2, int Lout, const int* spins, int n_spins,
                                   spingtp_dtype dtype, unsigned flags, spingtp_plan* out_plan);

/*
 * Paths of the instruction-weighted product (Sec. 3.4 eq. spin_gtp): the block
 * triples (rho1, rho2 -> rho3) on which the tensor T of spingtp_dense_tensor_host
 * has a nonzero entry.  A block is the set of slots of one spin index i and degree
 * l, labelled i (L+1) + l with the L of its input or output (in the parity basis
 * these blocks are the irreps (l, |s|, p) of the paper).  Host only, no GPU; same
 * argument rules as spingtp_plan_create.  Writes min(capacity, total) triples
 * (b1, b2, b3), 3 ints each, to `triples` (may be NULL when capacity is 0) in
 * ascending lexicographic order and the total to *count.
 */
spingtp_status spingtp_paths_host(int L1, int L2, int Lout, const int* spins, int n_spins, unsigned flags,
                                  int* triples, size_t capacity, size_t* count);

/*
 * A plan for the path-weighted product y[k3] = sum W[path(k1,k2,k3)] T[k1][k2][k3]
 * x1[k1] x2[k2]: one weight per path of spingtp_paths_host, in its order, shared
 * by every channel (the per-instruction weights of Sec. 3.4 eq. spin_gtp in the
 * elementwise channel mode; channel mixing is not part of this call).  weights:
 * host float64 array of n_weights finite values; n_weights must equal the path
 * count, else SPINGTP_ERR_INVALID_ARG.  The weights are folded into the plan's
 * tensor tables, so a plan holds one weight set.  Routes: spingtp_forward and both
 * gradients on the direct kernel (family 6), spingtp_forward_v1 on the
 * precontracted kernel where built (else the direct kernel); the Fourier kernels
 * compute the unweighted sum over all paths and are not used
 * (SPINGTP_V1_FOURIER gives SPINGTP_ERR_UNSUPPORTED).  Shapes the direct kernel
 * does not fit give a plan for spingtp_forward_v1 only, or
 * SPINGTP_ERR_UNSUPPORTED.  Otherwise as spingtp_plan_create.
 */
spingtp_status spingtp_plan_create_weighted(int L1, int L2, int Lout, const int* spins, int n_spins,
                                            spingtp_dtype dtype, unsigned flags, const double* weights,
                                            size_t n_weights, spingtp_plan* out_plan);

/*
 * out = SpinGTP(x1, x2) for N*C units, asynchronously on `stream` (a hipStream_t;
 * NULL = the null stream of the plan's device).
 *   x1, x2, out: device pointers of the plan's dtype in the layout above, each
 *   16-byte aligned; out must not overlap x1 or x2 (undefined otherwise).
 *   N, C >= 0; N*C == 0 is a no-op that returns SPINGTP_OK without touching
 *   memory.  Null pointers (when N*C > 0), misalignment or negative sizes give
 *   SPINGTP_ERR_INVALID_ARG before anything is launched.
 * out is overwritten (not accumulated).  No allocation and no host
 * synchronisation.  A launch failure gives SPINGTP_ERR_HIP; a plan whose shape
 * only spingtp_forward_v1 supports gives SPINGTP_ERR_UNSUPPORTED.
 */
spingtp_status spingtp_forward(spingtp_plan plan, const void* x1, const void* x2, void* out,
                               int64_t N, int64_t C, void* stream);

/*
 * out = SpinGTP(x1, x2) when the second input is an edge feature shared by the C
 * channels of its edge (edge multiplicity V = 1; paper Sec. 3.4, the
 * precontraction equations, and App. E, depthwise mode with unit weights):
 *   out[n][c] = SpinGTP(x1[n][c], x2[n]),
 *   x1 [N][C][n_spins][(L1+1)^2],  x2 [N][n_spins][(L2+1)^2],
 *   out [N][C][n_spins][(Lout+1)^2];  same dtype, same slot conventions.
 * Route: the precontracted kernel (family 5: per edge
 * K[k1][k3] = sum_k2 T[k1][k2][k3] x2[n][k2], then out[n][c] = x1[n][c] K, fp32
 * arithmetic; built for degrees <= 6 with spins {-1, 0, +1}, <= 7 with spin {0})
 * or the kernel of spingtp_forward reading x2 once per edge, as chosen at plan
 * creation (SPINGTP_V1_FOURIER / SPINGTP_V1_PRECONTRACT above).  Arguments, alignment, asynchrony and
 * errors as for spingtp_forward; no allocation.
 */
spingtp_status spingtp_forward_v1(spingtp_plan plan, const void* x1, const void* x2, void* out,
                                  int64_t N, int64_t C, void* stream);

/*
 * The depthwise product with per-channel path weights and the edge input shared
 * by the channels (Sec. 3.4, the precontraction equations; App. E.1, mode uvu with
 * V = 1):
 *   out[n][c][k3] = sum over paths p of weights[c][p] sum_{k1,k2 on p}
 *                   T[k1][k2][k3] x1[n][c][k1] x2[n][k2],
 * paths p in the order of spingtp_paths_host (block triples rho1, rho2 -> rho3).
 *   weights: device fp32 [C][n_paths], 4-byte aligned, read only.
 *   x1, x2, out, N, C, stream: as spingtp_forward_v1.
 * Needs a plan created with SPINGTP_CHANNEL_WEIGHTS (else SPINGTP_ERR_UNSUPPORTED).
 * Route: the entry-list kernel of spingtp_forward_weighted with the x2 row shared
 * by the tile's channels (four waves per 64-channel tile walk the tensor's nonzeros
 * by output slot; measured faster on the depthwise runtime table's shapes), where
 * the plan's lists hold the shape and the plan was not created with
 * SPINGTP_V1_PRECONTRACT; otherwise the precontracted kernel over path slots
 * q = (p, k1): per edge the kernel
 * K[q][k3] = sum_{k2 on p} T x2 is built once, and each channel's operand is
 * weights[c][p] x1[c][k1]; the contraction then runs over all path slots (at L = 2
 * with spins {-1, 0, +1}: 263 in the parity basis, 471 in the paper basis, whose
 * +-1 blocks split paths; 27 without weights).  Built for shapes whose
 * path slots fit 480 and output rows 48 (the depthwise runtime table's shapes,
 * degree <= 2 with spins {-1, 0, +1}, (1, 3, 3), degree <= 4 with spin {0}).
 * Plan creation with SPINGTP_CHANNEL_WEIGHTS fails with SPINGTP_ERR_UNSUPPORTED
 * when neither route nor the gradients' lists hold the shape.
 * Gradients: spingtp_backward_v1_weighted.  Asynchronous, no allocation.
 */
spingtp_status spingtp_forward_v1_weighted(spingtp_plan plan, const void* x1, const void* x2,
                                           const float* weights, void* out, int64_t N, int64_t C, void* stream);

/*
 * Gradients of spingtp_forward_v1_weighted for dL/dout = grad_out.  The product is
 * linear in each of x1, x2 and the weights, so
 *   grad_x1[n][c][k1]  = sum_p weights[c][p] sum_{k2,k3 on p} T x2[n][k2] grad_out[n][c][k3],
 *   grad_x2[n][k2]     = sum_c sum_p weights[c][p] sum_{k1,k3 on p} T x1[n][c][k1] grad_out[n][c][k3],
 *   grad_weights[c][p] = sum_n sum_{k1,k2,k3 on p} T x1[n][c][k1] x2[n][k2] grad_out[n][c][k3].
 *   x1, grad_out, grad_x1: device [N][C][n_spins][(L+1)^2] of the plan's dtype (L1,
 *     Lout, L1), 16-byte aligned; x2, grad_x2: [N][n_spins][(L2+1)^2];
 *   weights: device fp32 [C][n_paths] (as the forward), grad_weights: device fp32
 *     [C][n_paths] (written, not accumulated; zero when N = 0); 4-byte aligned;
 *   workspace: device memory of spingtp_backward_v1_weighted_workspace_size bytes
 *     or more, 4-byte aligned, overwritten (partial sums over channel tiles and
 *     edge ranges, added in a fixed order, so results do not depend on scheduling).
 * All three outputs are required and must not overlap the inputs.  Kernel: one
 * wave per 64-channel tile and range of edges walks the tensor's nonzeros in three
 * orders (by k1, by k2, by path) with the tile's weights in LDS; built where the
 * slot counts and the path count are <= 1022 and the LDS tile fits 160 KB (the
 * depthwise runtime table's shapes), otherwise SPINGTP_ERR_UNSUPPORTED, as for
 * plans created without SPINGTP_CHANNEL_WEIGHTS.  Asynchronous on `stream`, no
 * allocation.
 */
spingtp_status spingtp_backward_v1_weighted(spingtp_plan plan, const void* x1, const void* x2,
                                            const float* weights, const void* grad_out, void* grad_x1,
                                            void* grad_x2, float* grad_weights, void* workspace,
                                            size_t workspace_bytes, int64_t N, int64_t C, void* stream);

/* Bytes of workspace spingtp_backward_v1_weighted needs for N edges x C channels
 * (fp32 partial sums; 0 when N or C is 0).  SPINGTP_ERR_UNSUPPORTED as for it. */
spingtp_status spingtp_backward_v1_weighted_workspace_size(spingtp_plan plan, int64_t N, int64_t C, size_t* bytes);

/*
 * Elementwise product with one weight per (channel, path) and a per-unit second
 * input (Sec. 3.4 eq. spin_gtp with per-channel path weights; App. E.1 mode uuu):
 *   out[n][c][k3] = sum over paths p of weights[c][p] sum_{k1,k2 on p}
 *                   T[k1][k2][k3] x1[n][c][k1] x2[n][c][k2],
 * paths in the order of spingtp_paths_host.
 *   x1, x2, out: as spingtp_forward (x2 [N][C][n_spins][(L2+1)^2], per unit);
 *   weights: device fp32 [C][n_paths], 4-byte aligned, read only.
 * Needs a plan created with SPINGTP_CHANNEL_WEIGHTS whose entry lists hold the
 * shape (as spingtp_backward_v1_weighted; the tile here is the weight, x1, x2 and
 * output rows of 64 channels, 64 (P + NC1 + NC2 + NCO + 4) floats <= 160 KB), else
 * SPINGTP_ERR_UNSUPPORTED.  Kernel: four waves per 64-channel tile and range of
 * edges walk the tensor's nonzeros ordered by output slot.  Asynchronous, no
 * allocation.
 */
spingtp_status spingtp_forward_weighted(spingtp_plan plan, const void* x1, const void* x2, const float* weights,
                                        void* out, int64_t N, int64_t C, void* stream);

/*
 * Gradients of spingtp_forward_weighted for dL/dout = grad_out:
 *   grad_x1[n][c][k1]  = sum_p weights[c][p] sum_{k2,k3 on p} T x2[n][c][k2] grad_out[n][c][k3],
 *   grad_x2[n][c][k2]  = sum_p weights[c][p] sum_{k1,k3 on p} T x1[n][c][k1] grad_out[n][c][k3],
 *   grad_weights[c][p] = sum_n sum_{k1,k2,k3 on p} T x1[n][c][k1] x2[n][c][k2] grad_out[n][c][k3].
 * Arguments and rules as spingtp_backward_v1_weighted, with x2 and grad_x2
 * [N][C][n_spins][(L2+1)^2] per unit and the workspace of
 * spingtp_backward_weighted_workspace_size (grad_weights partial sums per edge
 * range, added in a fixed order).  SPINGTP_ERR_UNSUPPORTED where the plan's lists
 * do not hold the shape or the tile (64 (2 P + NC1 + NCO + 2 NC2 + 6) floats)
 * exceeds 160 KB.  Asynchronous, no allocation.
 */
spingtp_status spingtp_backward_weighted(spingtp_plan plan, const void* x1, const void* x2, const float* weights,
                                         const void* grad_out, void* grad_x1, void* grad_x2, float* grad_weights,
                                         void* workspace, size_t workspace_bytes, int64_t N, int64_t C, void* stream);

/* Bytes of workspace spingtp_backward_weighted needs for N edges x C channels.
 * SPINGTP_ERR_UNSUPPORTED as for it. */
spingtp_status spingtp_backward_weighted_workspace_size(spingtp_plan plan, int64_t N, int64_t C, size_t* bytes);

/*
 * The depthwise product with V second-input channels per edge (App. E.1, mode uvu,
 * one weight per path and channel pair):
 *   out[n][u][k3] = sum_{v < V} sum over paths p of weights[v][u][p] sum_{k1,k2 on p}
 *                   T[k1][k2][k3] x1[n][u][k1] x2[n][v][k2].
 *   x1, out: [N][C][...] as spingtp_forward_v1 (u < C); x2: device [N][V][n_spins]
 *   [(L2+1)^2] of the plan's dtype, 16-byte aligned; weights: device fp32 [V][C][n_paths]
 *   (the slice of channel v is the weight layout of spingtp_forward_v1_weighted);
 *   V >= 1.
 * Runs the entry-list kernel of spingtp_forward_v1_weighted on groups of up to four
 * channels v per launch (each tensor entry takes x1[k1] sum_v W_v[p] x2_v[k2]; as many
 * channels as its LDS holds while two workgroups still fit a compute unit), reading
 * the x2 rows of an edge V n_spins (L2+1)^2 elements apart and adding into out after
 * the first launch (bf16 outputs round at every add).  V = 1 gives the results of
 * spingtp_forward_v1_weighted bit for bit.  Needs a plan created with
 * SPINGTP_CHANNEL_WEIGHTS whose entry lists hold the shape, else
 * SPINGTP_ERR_UNSUPPORTED.  Asynchronous on `stream`, no allocation.
 */
spingtp_status spingtp_forward_depthwise(spingtp_plan plan, const void* x1, const void* x2, const float* weights,
                                         void* out, int64_t N, int64_t C, int64_t V, void* stream);

/*
 * Gradients of spingtp_forward_depthwise: grad_x1 [N][C][...] (the sum over v),
 * grad_x2 [N][V][...] and grad_weights [V][C][n_paths] (fp32), each channel v's part
 * computed as by spingtp_backward_v1_weighted (deterministic).  The workspace
 * (spingtp_backward_depthwise_workspace_size, that of spingtp_backward_v1_weighted
 * for N, C) is reused by every v, so calls on one stream are ordered.  Rules as
 * spingtp_backward_v1_weighted.
 */
spingtp_status spingtp_backward_depthwise(spingtp_plan plan, const void* x1, const void* x2, const float* weights,
                                          const void* grad_out, void* grad_x1, void* grad_x2, float* grad_weights,
                                          void* workspace, size_t workspace_bytes, int64_t N, int64_t C, int64_t V,
                                          void* stream);

/* Bytes of workspace spingtp_backward_depthwise needs (independent of V >= 1). */
spingtp_status spingtp_backward_depthwise_workspace_size(spingtp_plan plan, int64_t N, int64_t C, int64_t V,
                                                         size_t* bytes);

/*
 * Gradients of a scalar loss through out = SpinGTP(x1, x2) of spingtp_forward:
 * given grad_out = dLoss/dout, writes
 *   grad_x1[n][c][k1] = sum_{k2,k3} T[k1][k2][k3] x2[n][c][k2] grad_out[n][c][k3],
 *   grad_x2[n][c][k2] = sum_{k1,k3} T[k1][k2][k3] x1[n][c][k1] grad_out[n][c][k3]
 * (the chain rule on the real bilinear map T of spingtp_dense_tensor_host).
 * Route: let J be the real matrix of complex conjugation on real-basis
 * coefficients (App. A.1: conj(sY_lm) = (-1)^(s+m) (-s)Y_l(-m); a signed
 * permutation, see spingtp_conj_map_host).  Conjugating the Gaunt integral of
 * Sec. 3.2 eq. generalized_gaunt gives T[k1][k2][k3] = sum_j T'[k3][j][k1] J[j][k2]
 * with T' the tensor of degrees (Lout, L2, L1), so grad_x1 = SpinGTP'(grad_out,
 * J x2) and grad_x2 = SpinGTP''(grad_out, J x1): one launch of the plan's forward
 * kernel each, on backward tables where J is folded into the input-2 mixing of
 * the m = 0 slots of the |s| = 1 sectors (the only slots J moves: with
 * SPINGTP_BASIS_REAL_PAPER they swap between s = +1 and -1 with a sign change; J is
 * the identity for SPINGTP_BASIS_REAL_M0_PAIRED and spins {0}; with
 * SPINGTP_BASIS_PARITY the kernel mixes its tiles into the paper basis first, where
 * that J applies, since P^T J P x = P^T J (P x)).  That route serves plans with
 * L1 = L2 = Lout and a Fourier spingtp_forward kernel.  Other plans whose tile
 * fits the direct kernel (family 6: spins {-2..2}, shapes without a Fourier
 * kernel, mixed degrees) run the two gradients on it, from tables listing the
 * nonzeros of T by k1 and by k2 (spingtp_direct_table_host roles 1 and 2; no J).
 * Otherwise SPINGTP_ERR_UNSUPPORTED.
 *   x1, x2, grad_out: as x1, x2, out of spingtp_forward; grad_x1, grad_x2: same
 *   shapes as x1, x2 (either may be NULL: not computed), overwritten; slots with
 *   l < |s| are written 0.  Same dtype, 16-byte alignment and error rules as
 *   spingtp_forward; outputs must not overlap inputs.
 * Asynchronous on `stream`, ordered on it; no allocation; same arithmetic as the
 * forward kernel of the plan.
 */
spingtp_status spingtp_backward(spingtp_plan plan, const void* x1, const void* x2, const void* grad_out,
                                void* grad_x1, void* grad_x2, int64_t N, int64_t C, void* stream);

/*
 * Gradients through spingtp_forward_v1 (x2 shared by the C channels of an edge):
 *   grad_x1[n][c][k1] = sum_{k2,k3} T[k1][k2][k3] x2[n][k2] grad_out[n][c][k3],
 *   grad_x2[n][k2]    = sum_c sum_{k1,k3} T[k1][k2][k3] x1[n][c][k1] grad_out[n][c][k3].
 * Route (same identity as spingtp_backward): grad_x1 = SpinGTP_v1(grad_out, J x2) on
 * the plan's spingtp_forward_v1 kernel (the precontracted kernel reads a second
 * tensor table with J folded into its x2 indices and signs; the Fourier kernel
 * reads the backward tables); grad_x2: the per-unit products
 * SpinGTP(grad_out[n][c], J x1[n][c]) of the plan's spingtp_forward kernel go to
 * `workspace` ([N][C][n_spins (L2+1)^2], the plan's dtype), then a second kernel
 * sums them over c in order (fp32 sums; bf16 output rounded to nearest even).
 * On plans whose gradients run on the direct kernel (see spingtp_backward), both
 * steps use its role tables instead (grad_x1 with x2 read once per edge), except
 * that grad_x1 stays on the precontracted kernel where the plan has its
 * conjugated table.  Plans with neither: SPINGTP_ERR_UNSUPPORTED.
 *   x1 [N][C][...], x2 [N][...], grad_out [N][C][...]; grad_x1 [N][C][...] and
 *   grad_x2 [N][n_spins (L2+1)^2] (either may be NULL: not computed), overwritten;
 *   slots with l < |s| are written 0.  C = 0 writes grad_x2 = 0.
 *   workspace: device memory of spingtp_backward_v1_workspace_size bytes or more,
 *   16-byte aligned, overlapping no other argument (needed only for grad_x2; may
 *   be NULL otherwise).  Too small or missing: SPINGTP_ERR_INVALID_ARG.
 * Same dtype, alignment and error rules as spingtp_forward; asynchronous on
 * `stream`, ordered on it; no allocation.
 */
spingtp_status spingtp_backward_v1(spingtp_plan plan, const void* x1, const void* x2, const void* grad_out,
                                   void* grad_x1, void* grad_x2, void* workspace, size_t workspace_bytes,
                                   int64_t N, int64_t C, void* stream);

/*
 * spingtp_backward_v1 for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same gradients, computed by the same kernels in the same order (bit-identical
 * results), with the per-unit products of grad_x2 staged in a fixed device array
 * of SPINGTP_NOALLOC_SCRATCH_BYTES (64 MiB) that the library holds on each GPU
 * it runs on until the process ends, instead of a caller workspace.
 *   Arguments as for spingtp_backward_v1 without workspace/workspace_bytes.
 *   grad_x2 != NULL with spingtp_backward_v1_workspace_size(plan, N, C) above
 *   SPINGTP_NOALLOC_SCRATCH_BYTES: SPINGTP_ERR_TOO_LARGE, nothing launched
 *   (grad_x1 alone has no limit).  The first call on a device looks up the
 *   array's device address (hipGetSymbolAddress, the plan's device current);
 *   failure: SPINGTP_ERR_HIP.  No hipMalloc or hipFree, no allocation.
 *   Every call on one GPU shares that GPU's array (each call overwrites the rows
 *   it reads, so nothing carries over): calls that overlap in time on one GPU,
 *   on different streams or threads, race and give undefined gradients.
 */
#define SPINGTP_NOALLOC_SCRATCH_BYTES (64u << 20)
spingtp_status spingtp_backward_v1_noalloc(spingtp_plan plan, const void* x1, const void* x2, const void* grad_out,
                                           void* grad_x1, void* grad_x2, int64_t N, int64_t C, void* stream);

/*
 * Host-only self-test of plan creation's device upload, for tests of its failure
 * handling (no GPU needed).  Builds the host tables exactly as spingtp_plan_create
 * (same arguments and rules), then runs the same upload routine with host memory
 * standing in for device memory, failing allocation number fail_at (0-based; -1:
 * none fails).  *n_allocs = allocations attempted, *n_live = allocations still held
 * when the upload returned (0 after a failure: everything allocated so far was
 * released; those of a successful upload are released afterwards by this call).
 * Returns the upload's status: SPINGTP_ERR_OUT_OF_MEMORY for the injected failure.
 */
spingtp_status spingtp_plan_upload_selftest_host(int L1, int L2, int Lout, const int* spins, int n_spins,
                                                 spingtp_dtype dtype, unsigned flags, int fail_at, int* n_allocs,
                                                 int* n_live);

/*
 * Fully connected product (mode uvw of App. E.1; Sec. 3.5 eq. spin_gtp), U channels of
 * x1, V of x2, W of the output, one weight per (path, u, v, w):
 *   R_p[n][u][v][m3] = sum over the nonzeros (k1, k2, m3) of path p of T x1[n][u][k1] x2[n][v][k2],
 *   out[n][w][k3]    = sum_p sum_{u,v} weights[p][u][v][w] R_p[n][u][v][k3]  (k3 in p's output block),
 * paths (block triples) numbered as by spingtp_paths_host.
 *   x1 [N][U][n_spins][(L1+1)^2], x2 [N][V][n_spins][(L2+1)^2], fp32, 16-byte aligned;
 *   weights [n_paths][U][V][W] fp32, 4-byte aligned; out [N][W][n_spins][(Lout+1)^2],
 *   16-byte aligned, overwritten (0 in blocks no path reaches and in slots l < |s|).
 *   N, U, V, W >= 0, U, V, W <= 65536, U V <= 2^24; N W = 0 is a no-op, U V = 0 writes 0.
 * Needs an fp32 plan created with SPINGTP_FULLY_CONNECTED (else SPINGTP_ERR_UNSUPPORTED).
 * Products and sums in fp32: the per-path products R on the vector ALU, the channel
 * mixing on the matrix cores.  Asynchronous on `stream`, no allocation; deterministic.
 */
spingtp_status spingtp_forward_fully_connected(spingtp_plan plan, const void* x1, const void* x2,
                                               const float* weights, void* out, int64_t N, int64_t U, int64_t V,
                                               int64_t W, void* stream);

/*
 * Gradients of spingtp_forward_fully_connected (reverse mode; App. E.1 mode uvw, Sec. 3.5
 * eq. spin_gtp, chain rule through R_p and the channel mixing) for g = grad_out = dL/dout:
 *   grad_x1[n][u][k1]       = sum_p sum_{v,w} weights[p][u][v][w] sum_{(k1,k2,k3) in p} T x2[n][v][k2] g[n][w][k3],
 *   grad_x2[n][v][k2]       = sum_p sum_{u,w} weights[p][u][v][w] sum_{(k1,k2,k3) in p} T x1[n][u][k1] g[n][w][k3],
 *   grad_weights[p][u][v][w] = sum_n sum_{k3 in p's output block} R_p[n][u][v][k3] g[n][w][k3].
 *   x1, x2, weights: as for the forward; grad_out [N][W][n_spins][(Lout+1)^2] fp32,
 *   16-byte aligned; grad_x1, grad_x2 shaped like x1 and x2 (16-byte aligned) and
 *   grad_weights like weights (4-byte aligned), each overwritten, or nullptr to skip
 *   that gradient.  Slots with l < |s| and blocks no path reaches get 0; with N = 0,
 *   grad_weights is 0.  U, V, W <= 65536 and U V, V W, U W <= 2^24.
 * Needs an fp32 plan created with SPINGTP_FULLY_CONNECTED (else SPINGTP_ERR_UNSUPPORTED).
 * fp32 products and sums (grad_x1 and grad_x2 on the forward's kernel with the tensor's
 * axes exchanged, grad_weights on the matrix cores with the edges as the reduction);
 * asynchronous on `stream`, no allocation; deterministic (every element has one owner
 * that sums in a fixed order).
 */
spingtp_status spingtp_backward_fully_connected(spingtp_plan plan, const void* x1, const void* x2,
                                                const float* weights, const void* grad_out, void* grad_x1,
                                                void* grad_x2, float* grad_weights, int64_t N, int64_t U, int64_t V,
                                                int64_t W, void* stream);

/* Bytes of workspace spingtp_backward_v1 needs for grad_x2 with N x C units:
 * N C n_spins (L2+1)^2 elements of the plan's dtype.  SPINGTP_ERR_UNSUPPORTED as
 * for spingtp_backward_v1. */
spingtp_status spingtp_backward_v1_workspace_size(spingtp_plan plan, int64_t N, int64_t C, size_t* bytes);

/*
 * Host-only: the conjugation map J of degree L (one word per destination slot j
 * of a [n_spins][(L+1)^2] vector: (J x)[j] = x[w & 0xffff], negated if bit 16 of
 * w is set, 0 if bit 17 is set (slots with l < |s|)), derived from the real basis
 * columns of App. C and the conjugation relation of App. A.1.  Same argument
 * rules as spingtp_plan_create with L1 = L2 = Lout = L.  Writes min(capacity,
 * total) words to `words` (may be NULL when capacity is 0) and the total to *count.
 */
spingtp_status spingtp_conj_map_host(int L, const int* spins, int n_spins, unsigned flags, uint32_t* words,
                                     size_t capacity, size_t* count);

/* Free the plan's device tables.  The caller must ensure that no forward using
 * the plan is still running.  NULL is accepted (no-op). */
spingtp_status spingtp_plan_destroy(spingtp_plan plan);

/* Static English description of a status code. */
const char* spingtp_status_string(spingtp_status s);

/*
 * Host-only inspection of the plan tables in float64, before rounding.  Needs no
 * GPU.  Same argument rules as spingtp_plan_create.  Writes at most `capacity`
 * doubles to `tables` (may be NULL when capacity is 0) and the full count to
 * *n_tables; `dims` (may be NULL) receives 8 ints:
 *   {n_theta, n_phi, L1, L2, Lout, n_spins, per_theta_block, global_block}.
 * The table layout is the one documented in csrc/layout.h of the library source.
 * With SPINGTP_TABLES_BACKWARD in `flags`: the tables of spingtp_backward
 * (SPINGTP_ERR_UNSUPPORTED if the conjugation map cannot be folded into them).
 */
spingtp_status spingtp_plan_tables_host(int L1, int L2, int Lout, const int* spins, int n_spins,
                                        unsigned flags, double* tables, size_t capacity,
                                        size_t* n_tables, int* dims);

/*
 * The explicit real bilinear tensor of the operation, dense, in float64, on the host
 * (no GPU needed): out[k3] = sum_{k1,k2} T[k1][k2][k3] x1[k1] x2[k2] with
 * k1 < NC1 = n_spins (L1+1)^2, k2 < NC2, k3 < NCO in the layout above.  T is built
 * from the spin-weighted Gaunt coefficients G (Sec. 3.2 eq. generalized_gaunt, by
 * exact Gauss-Legendre quadrature of triple SWSH products) mapped through the real
 * basis (App. C): T = Re(conj(Q3) G Q1 Q2).  It is the direct (Clebsch-Gordan
 * style) form of the product, used as the O(L^6) comparator of the benchmark and
 * for inspection; the forward path never uses it.  Same argument rules as
 * spingtp_plan_create.  Writes min(capacity, NC1 NC2 NCO) doubles to `tensor`
 * (may be NULL when capacity is 0) and the full count to *count.
 */
spingtp_status spingtp_dense_tensor_host(int L1, int L2, int Lout, const int* spins, int n_spins,
                                         unsigned flags, double* tensor, size_t capacity, size_t* count);

/*
 * Host-only inspection of the matrix-core operand tables of the kernel for
 * L1 = L2 = Lout = L and spins {-1, 0, +1} (family 4 below), exactly as
 * spingtp_plan_create uploads them.  Needs no GPU.  Words are packed fp16
 * pairs (element 2w in the low half of word w); layout, per 64 lanes x 8 words
 * (4 words hi, 4 words lo):
 *   [0, 512)                 the step-(B) trig operand, lane l = row l % 32
 *                            (phi point), K elements 8 (l / 32) + e;
 *   [512 + 512 (type NB + b), ...)  the step-(D) operand of table type 0 (R0, P1)
 *                            or 1 (P2) and K block b, NB = ceil((3L + 1) / 16);
 *   [512 (1 + 2 NB), + 1024) (L = 8 only) the second K block of step (B), once
 *                            for input 1 (cos(8 phi) at kappa 16 only) and once
 *                            for input 2 (cos(8 phi) at kappa 24 only).
 * At L = 8 the first block holds sin(8 phi) at kappa 8, which sin 0 leaves free.
 * 1 <= L <= 8, else SPINGTP_ERR_INVALID_ARG.  Writes min(capacity, total) words
 * to `words` (may be NULL when capacity is 0) and the total to *count.
 */
spingtp_status spingtp_mfma_operands_host(int L, uint32_t* words, size_t capacity, size_t* count);

/*
 * Host-only inspection of the tensor table of the precontracted kernel of
 * spingtp_forward_v1 (family 5 below), exactly as spingtp_plan_create uploads it.
 * Needs no GPU.  Same argument rules as spingtp_plan_create; shapes the kernel does
 * not cover (a degree above 6 with spins {-1, 0, +1}, above 7 with spin {0}) give
 * SPINGTP_ERR_UNSUPPORTED.
 * Word layout, with P = 256 (threads of one workgroup):
 *   [0, 16)                NC1, NC2, NCO, BLK1 = (L1+1)^2, KS = ceil(NC1/16),
 *                          NT = ceil(NCO/16), IPT, KST = 16 KS + 4, NB3, RB,
 *                          STRIDE, n_spins, NC1, 0, 0, 0: the k3 rows of the
 *                          edge kernel come in NB3 blocks of RB rows (one block of
 *                          16 NT rows when KS, NT <= 5, else blocks of 48 rows);
 *                          each block holds STRIDE items per thread, IPT of them
 *                          used (STRIDE = IPT, a multiple of 8, for one block;
 *                          else IPT is a multiple of 16 and STRIDE = IPT + 16);
 *   [16, 16 + 2 NB3 STRIDE P)  per block b, items [item][thread], two words each:
 *                          dst | k2 << 16 | last << 24, then the fp32 value (bits).
 * Thread t adds value * x2[k2] for the items of a block in order to a running
 * sum; an item with `last` set stores the sum as the edge kernel entry K[k1][k3]
 * with dst = (k3 - RB b) KST + k1, and restarts the sum at 0.  Padding items are
 * all-zero words.
 * With SPINGTP_TABLES_BACKWARD in `flags` (L1 = L2 = Lout only): the table of
 * spingtp_backward_v1, whose items use J x2 (k2 replaced by J's source slot, the
 * value by J's sign times the value; see spingtp_conj_map_host).
 * With SPINGTP_CHANNEL_WEIGHTS: the table of spingtp_forward_v1_weighted.  Word 0
 * is then the number of path slots Q (the contraction length; KS covers it, from
 * the kernel's instantiations), word 13 the number of paths and word 14 the
 * offset of Q words after the items: path slot q = x1 slot | path << 16, listed
 * path by path; an item's kernel position is dst = k3 KST + q.
 * With both flags: the entry lists of the per-channel weighted kernels
 * (spingtp_backward_v1_weighted, spingtp_forward_weighted, spingtp_backward_weighted):
 * words [0, 11) NC1, NC2, NCO, NP (paths), NNZ (nonzeros of T), the word offsets of
 * SEG1, SEG2, SEGP (NC1 + 1, NC2 + 1, NP + 1 list boundaries, counted in entries)
 * and of LIST1, LIST2, LISTP.  An entry is two words, a | b << 10 | c << 20
 * and an fp32 value: LIST1 holds per k1 (path, k2, k3), LIST2 per k2 (path, k1, k3),
 * LISTP per path (k1, k2, k3); words 11, 12 the offsets of SEG3 (NCO + 1) and
 * LIST3, per k3 (path, k1, k2), the list of spingtp_forward_weighted; words [16, 36)
 * five key boundaries per list (LIST1, LIST2, LISTP, LIST3) splitting it among the
 * kernel's four waves; each segment is padded to a multiple of 8 entries
 * of value 0 whose fields are the row lengths (NP, NC1, NC2 or NCO: the zero
 * columns), and each list ends with 96 more such entries.
 * SPINGTP_ERR_UNSUPPORTED where the kernel does not take the shape.
 * Writes min(capacity, total) words to `words` (may be NULL when capacity is 0)
 * and the total to *count.
 */
spingtp_status spingtp_pre_table_host(int L1, int L2, int Lout, const int* spins, int n_spins, unsigned flags,
                                      uint32_t* words, size_t capacity, size_t* count);

/*
 * Host-only inspection of the entry table of the direct kernel (family 6) for one
 * role of the tensor T[k1][k2][k3] of spingtp_dense_tensor_host, exactly as
 * spingtp_plan_create uploads it.  Needs no GPU.  Same argument rules as
 * spingtp_plan_create; role 0 = forward (out[k3] from A = x1 at a = k1, B = x2
 * at b = k2), 1 = gradient w.r.t. x1 (out[k1] from A = grad_out at a = k3,
 * B = x2 at b = k2), 2 = gradient w.r.t. x2 (out[k2] from A = grad_out at
 * a = k3, B = x1 at b = k1); another role gives SPINGTP_ERR_INVALID_ARG, a
 * shape whose tile does not fit the kernel's LDS SPINGTP_ERR_UNSUPPORTED.
 * Word layout:
 *   [0, 8)         NCA, NCB, NCO (widths of A, B, out), STA, STB, STO (odd LDS
 *                  row strides, each above its width: column NCA of A and NCB
 *                  of B hold 0), NBATCH, 16 (entries per batch);
 *   [8, 13)        output-slot boundaries o_0 = 0 <= ... <= o_4 = NCO of the four
 *                  waves of a workgroup (wave w computes slots [o_w, o_(w+1)));
 *   [13, 18)       the first batch of each wave's range, and NBATCH;
 *   [18, 18 + NCO) batches per output slot, in output order;
 *   then NBATCH batches of 24 words: 8 index words (entry 2i in the low 16 bits
 *   of word i, entry 2i + 1 in the high 16 bits, each a | b << 8), then the 16
 *   fp32 values (bits); and 48 zero words.  out[o] = sum over the entries of
 *   slot o of value * A[a] * B[b]; entries are the nonzeros of T in ascending
 *   (a, b) order, padded with (NCA, NCB, 0) entries.  Rows longer than 254
 *   (8-bit indices) give SPINGTP_ERR_UNSUPPORTED.
 * Writes min(capacity, total) words to `words` (may be NULL when capacity is 0)
 * and the total to *count.
 */
spingtp_status spingtp_direct_table_host(int L1, int L2, int Lout, const int* spins, int n_spins, unsigned flags,
                                         int role, uint32_t* words, size_t capacity, size_t* count);

/*
 * Describe the kernel a plan launches: writes the waves per workgroup, units per
 * workgroup, LDS bytes per workgroup and a kernel-family id to the 4 ints of
 * `info`.  Families: 1 = one lane per unit, one wave per quadrature node (L <= 6
 * and the mixed-degree shapes); 2 = lane pairs per unit (L = 7, 8); 3 = lane
 * pairs with the nodes processed in rounds (L = 9..16, fp32 only); 4 = the
 * matrix-core kernel (L1 = L2 = Lout = 5, 6, and 4 for bf16; spins {-1, 0, +1};
 * the default there unless SPINGTP_KERNEL_VALU is given); 6 = the direct
 * sparse-tensor kernel (one wave per 64 units; shapes without a Fourier kernel,
 * spins {-2..2}).
 */
spingtp_status spingtp_plan_kernel_info(spingtp_plan plan, int* info);

/* The same four ints for the kernel of spingtp_forward_v1.  Family 5 = the
 * precontracted kernel: one workgroup per edge, `units` = 1 (edge). */
spingtp_status spingtp_plan_kernel_info_v1(spingtp_plan plan, int* info);

#ifdef __cplusplus
}
#endif

#endif /* SPINGTP_H */
