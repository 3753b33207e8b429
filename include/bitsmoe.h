/*
 * bitsmoe.h -- C ABI of the MI355X (gfx950) BitsMoE spectral quantizer.
 *
 * BitsMoE (arXiv 2606.00079) quantizes the experts of an MoE projection
 * through a shared basis: the E expert weights of one projection type share
 * an output space (Sec. 3.2), so the left singular vectors of the
 * concatenation W_cat = [W_1 ... W_E] (App. B.1, Eqs. app_down_w_cat and
 * app_down_cat_svd_absorbed) are kept unquantized, and each expert keeps its
 * coordinates in that basis, C_e = U^T W_e, whose rows ("spectral units") are
 * quantized at a width chosen per unit.  The width comes from an integer
 * program over an activation-aware loss (Sec. 3.3, Eq.
 * ilp_piecewise_projection), here the exact loss
 * delta H delta^T of App. B.2 (Eq. app_down_exact_metric).
 *
 * One projection runs, in order:
 *   bitsmoe_gram          H = X^T X / n                      (device)
 *   bitsmoe_gram_experts  M = sum_e W_e W_e^T                (device)
 *   bitsmoe_shared_basis  U = top-r eigenvectors of M        (host LAPACK)
 *     or bitsmoe_shared_basis_gpu (tridiagonal reduction on the device)
 *   bitsmoe_project       C_e = U^T W_e                      (device)
 *   bitsmoe_score         L[u][j] = delta H delta^T          (device)
 *   bitsmoe_allocate      widths per unit under a budget     (host, exact)
 *   bitsmoe_pack_layout   word offsets of the packed units   (host)
 *   bitsmoe_pack          bit-plane codes + fp16 params      (device)
 *
 * The paper's own allocation prices widths by a closed-form surrogate
 * instead of a measured loss (App. B.3-B.5); the library offers it too:
 *   bitsmoe_surrogate         L[u][j] = alpha^2 beta^gamma E(b_j),
 *                             widths {0,1,2,3,4,6,8,16}       (device)
 *   bitsmoe_surrogate_budget  equivalent-bit budget           (host)
 * and bitsmoe_allocate accepts those widths (0 = evicted, 16 = fp16).
 *
 * The paper builds the gate/up bases in the shared *input* space instead
 * (Sec. 3.2); that construction is available as well:
 *   bitsmoe_gram_experts_in   M_in = sum_e W_e^T W_e               (device)
 *   bitsmoe_project_in        C_e = Phi_r^T W_e^T (units W_e phi_k) (device)
 *   bitsmoe_basis_importance  beta_k = phi_k^T H phi_k             (device)
 *   bitsmoe_score_diag        L = beta_k ||c - Q_b(c)||^2          (device)
 * and the paper's per-expert, routing-weighted calibration Grams:
 *   bitsmoe_gram_routed       H_e = (1/n) sum_t g_te x_t x_t^T     (device)
 *   bitsmoe_score_routed      L = delta H_e delta^T                (device)
 * and serving a projection from its packed factors:
 *   bitsmoe_moe_decode        y = U sum_j g_j C^_{e_j} x           (device)
 *   bitsmoe_moe_decode_topk   the same from a device top-k table   (device)
 *   bitsmoe_moe_decode_topk_noalloc  the same, allocating nothing   (device)
 *   bitsmoe_moe_decode_in     y = sum_j g_j C^_{e_j}^T Phi^T x      (device)
 *
 * Conventions shared by every call:
 *  - Pointers named *_dev are device memory on the current HIP device;
 *    *_host are host memory.  The caller allocates and owns every input and
 *    output; the library never frees caller memory.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Device calls only enqueue work on it and return without waiting, unless
 *    stated otherwise.  The library keeps per-device scratch memory that is
 *    reused by every call on that device, so calls on one device must be
 *    ordered (one stream, or synchronized by the caller); calls that overlap
 *    on one device race on the scratch.
 *  - Every call returns a status.  Arguments are checked before any work is
 *    enqueued; on a non-OK status nothing has been enqueued unless the status
 *    is BITSMOE_ERR_DEVICE, and the outputs are unspecified.
 *    bitsmoe_last_error() gives a text for the last non-OK status of the
 *    calling thread.
 *  - Device pointers must be 16-byte aligned (hipMalloc and the usual
 *    framework allocators give 256 bytes); a misaligned one gives
 *    BITSMOE_ERR_ARG.
 *  - Matrices are row-major and densely packed unless a stride is given.
 *  - Shape rules that are not met give BITSMOE_ERR_SHAPE; null pointers and
 *    non-positive sizes give BITSMOE_ERR_ARG.
 */
#ifndef BITSMOE_H
#define BITSMOE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BITSMOE_OK = 0,
  BITSMOE_ERR_ARG = 1,          /* null pointer, non-positive size, bad enum   */
  BITSMOE_ERR_SHAPE = 2,        /* size outside the supported shape rules       */
  BITSMOE_ERR_DTYPE = 3,        /* unsupported element type                     */
  BITSMOE_ERR_DEVICE = 4,       /* a HIP call or kernel launch failed           */
  BITSMOE_ERR_NOMEM = 5,        /* scratch or host memory could not be had      */
  BITSMOE_ERR_NUMERIC = 6,      /* non-finite input, or the eigensolver failed  */
  BITSMOE_ERR_INFEASIBLE = 7,   /* budget below min(bits) * units               */
  BITSMOE_ERR_UNAVAILABLE = 8   /* no LAPACK library could be loaded            */
} bitsmoe_status;

/* The two sentinels are not element types: they make every int a valid
 * value of the enum (in C++ an enum otherwise only spans its enumerators'
 * bit range), so an unsupported code from a caller is rejected with
 * BITSMOE_ERR_DTYPE instead of being undefined behaviour. */
typedef enum {
  BITSMOE_F32 = 0,   /* IEEE fp32                                   */
  BITSMOE_BF16 = 1,  /* bfloat16, read as exact values              */
  BITSMOE_DTYPE_RANGE_MIN_ = -2147483647 - 1,
  BITSMOE_DTYPE_RANGE_MAX_ = 2147483647
} bitsmoe_dtype;

/* Largest candidate width and group sizes accepted by score and pack. */
#define BITSMOE_MAX_BITS 8
#define BITSMOE_MAX_NBITS 8
/* Widths bitsmoe_allocate accepts: 0 (evicted) .. 16 (fp16). */
#define BITSMOE_ALLOC_MAX_BITS 16
/* Columns of the surrogate table: widths 0, 1, 2, 3, 4, 6, 8, 16. */
#define BITSMOE_SURROGATE_NWIDTHS 8

/*
 * Step 1a -- calibration Gram.
 * H = X^T X / n, the token-averaged outer product of the calibration rows.
 * The paper weights tokens by routing affinity, H = X Diag(g) X^T
 * (App. B.2, Eq. app_affinity_gram); this call uses g_t = 1/n for every row.
 *   X_dev  [n][d] of type xt (bf16, or fp32 which is split into two bf16
 *          terms so that the result keeps fp32 accuracy)
 *   H_dev  [d][d] fp32 output, full symmetric matrix.
 * Shape rules: n >= 1, d >= 64 and d % 64 == 0.
 */
bitsmoe_status bitsmoe_gram(const void* X_dev, bitsmoe_dtype xt, int64_t n, int64_t d,
                            float* H_dev, void* stream);

/*
 * Step 1b -- cross-expert Gram.
 * M = sum_e W_e W_e^T = W_cat W_cat^T, whose eigenvectors are the left
 * singular vectors of W_cat = [W_1 ... W_E] (App. B.1, Eqs. app_down_w_cat,
 * app_down_cat_svd_absorbed).  Partial sums over K chunks of at most 4096
 * terms are formed in fp32 and added in fp64 in a fixed order, so the result
 * is deterministic.
 *   W_dev  [E][d_out][d_in] of type wt
 *   M_dev  [d_out][d_out] fp64 output, full symmetric.
 * Shape rules: E >= 1, d_out % 64 == 0, d_in % 64 == 0.
 */
bitsmoe_status bitsmoe_gram_experts(const void* W_dev, bitsmoe_dtype wt, int64_t E,
                                    int64_t d_out, int64_t d_in, double* M_dev, void* stream);

/*
 * Step 2 -- shared basis (host).
 * Copies M to the host, computes its eigendecomposition with LAPACK (dsyevd)
 * and keeps the r eigenvectors of largest eigenvalue: the retained left
 * singular vectors Phi of W_cat (App. B.1).  Eigenvalues are returned in
 * descending order and each eigenvector is signed so that its entry of
 * largest magnitude is positive (lowest index on ties).
 *   M_dev         [d_out][d_out] fp64 symmetric (read)
 *   Ut_dev        [r][d_out] fp32 output; row k = eigenvector k
 *   eigvals_host  [r] fp64 output (may be NULL)
 *   host_ms       wall time of the whole call in ms (may be NULL)
 * Synchronous: waits for `stream`, and returns after Ut_dev is written.
 * 1 <= r <= d_out.  ERR_UNAVAILABLE if no LAPACK can be loaded (see
 * bitsmoe_set_lapack), ERR_NUMERIC if M is not finite or LAPACK fails.
 */
bitsmoe_status bitsmoe_shared_basis(const double* M_dev, int64_t d_out, int64_t r,
                                    float* Ut_dev, double* eigvals_host, double* host_ms,
                                    void* stream);

/*
 * Step 2 on the GPU: the same outputs and conventions as
 * bitsmoe_shared_basis (eigenvalues descending, each eigenvector's entry of
 * largest magnitude positive), computed on the device:
 *   1. a blocked Householder reduction of M to tridiagonal form Q^T M Q
 *      (fp64, panels of 32 columns);
 *   2. eigenvalues d_out-r+1..d_out of the tridiagonal matrix by bisection,
 *      eigenvectors by inverse iteration (tridiagonal LU with partial
 *      pivoting), eigenvectors of eigenvalues closer than 1e-7 ||T|| made
 *      orthonormal by modified Gram-Schmidt;
 *   3. the back-transformation U = Q Z.
 * Only the two diagonals (for bounds and the finiteness check) and the r
 * eigenvalues cross PCIe.  Inside clusters of (nearly) equal eigenvalues
 * the eigenvectors are a valid orthonormal basis of the cluster but need not
 * equal bitsmoe_shared_basis's.
 *   Arguments as bitsmoe_shared_basis; host_ms is the wall time of the
 *   whole call.
 * Shape rules: 1 <= r <= d_out <= 65536.  Device scratch: (d_out + 6 r)
 * d_out doubles.  The call waits for the stream.  A non-finite M gives
 * BITSMOE_ERR_NUMERIC.
 */
bitsmoe_status bitsmoe_shared_basis_gpu(const double* M_dev, int64_t d_out, int64_t r,
                                        float* Ut_dev, double* eigvals_host, double* host_ms,
                                        void* stream);

/*
 * Step 3 -- expert spectral factors.
 * C_e = U^T W_e for every expert: with W_e = Phi P~_e^T and Phi orthonormal
 * (App. B.1, Eq. app_down_p_tilde_partition), row k of C_e is the spectral
 * component of expert e along basis vector k.  U is split into two bf16
 * terms (and fp32 W into two as well) so the product keeps fp32 accuracy.
 *   Ut_dev  [r][d_out] fp32
 *   W_dev   [E][d_out][d_in] of type wt
 *   C_dev   [E][r][d_in] fp32 output; unit u = e*r + k is row u.
 * Shape rules: d_out % 64 == 0, d_in % 64 == 0, 1 <= r <= d_out.
 */
bitsmoe_status bitsmoe_project(const float* Ut_dev, const void* W_dev, bitsmoe_dtype wt,
                               int64_t E, int64_t d_out, int64_t d_in, int64_t r,
                               float* C_dev, void* stream);

/*
 * Step 4 -- activation-aware loss table.
 * For every unit row c (length d) and every candidate width b = bits[j]:
 * the row is fake-quantized group-wise (groups of `group` consecutive
 * entries, asymmetric min/max round-to-nearest: s = fp16(fl32(max-min) /
 * (2^b-1)), m = fp16(min), q = clamp(rint((c-m)/s), 0, 2^b-1), x = m + q s),
 * delta = c - x, and
 *     L[u][j] = delta H delta^T,
 * the per-component term of the exact output-space loss
 * sum_k alpha_k^2 eps_k^T H eps_k (App. B.2, Eq. app_down_exact_metric).
 *   C_dev      [units][d] fp32
 *   H_dev      [d][d] fp32 symmetric positive semidefinite (as bitsmoe_gram
 *              writes it); the call relies on the symmetry and reads the
 *              upper triangle of 256 x 256 blocks and the diagonal
 *   bits_host  [nbits] widths, strictly ascending, each in 1..8
 *   L_dev      [units][nbits] fp32 output
 * Shape rules: d % 64 == 0, d < 2^22, group in {32, 64, 128, 256},
 * d % group == 0, 1 <= nbits <= 8.
 * Accuracy: the off-diagonal part of H enters through fp16 matrix-core
 * products of operands scaled by exact powers of two (per row for the
 * errors, per call for H), with fp32 accumulation; the diagonal part is
 * added in fp32.  Per-entry relative error is typically ~1e-4.
 */
bitsmoe_status bitsmoe_score(const float* C_dev, int64_t units, int64_t d, const float* H_dev,
                             const int* bits_host, int nbits, int group, float* L_dev,
                             void* stream);

/*
 * ILP (host) -- per-projection bit allocation (Sec. 3.3, Eq.
 * ilp_piecewise_projection; App. B.4, Eq. ilp_piecewise_eps):
 *     minimize sum_u L[u][j_u]  subject to  sum_u bits[j_u] <= budget_bits.
 * Solved exactly: costs are first mapped to int64 as
 * rint(L * 2^K / max|L|), K = 62 - ceil(log2(units + 1)), so every sum is
 * exact; among all optima the lexicographically smallest width vector (in
 * unit order) is returned.
 *   L_host         [units][nbits] fp32 (finite)
 *   bits_host      [nbits] strictly ascending widths, each in
 *                  0..BITSMOE_ALLOC_MAX_BITS (0 = the unit is evicted)
 *   bits_out_host  [units] output: the chosen width of each unit
 *   objective_out  sum of the chosen L in fp64 (may be NULL)
 * ERR_INFEASIBLE if budget_bits < bits[0] * units; ERR_NUMERIC for a
 * non-finite cost; ERR_NOMEM if the exact search does not fit in memory.
 */
bitsmoe_status bitsmoe_allocate(const float* L_host, int64_t units, const int* bits_host,
                                int nbits, int64_t budget_bits, uint8_t* bits_out_host,
                                double* objective_out);

/*
 * Same as bitsmoe_allocate, with solver controls for testing and reporting:
 *   full_dp_limit  instances with units * (capacity + 1) <= this use a plain
 *                  dynamic program over all units; larger ones first fix
 *                  every unit whose reduced cost at the LP-relaxation
 *                  multiplier exceeds the LP gap (such a unit takes the same
 *                  width in every optimum) and run the exact program on the
 *                  rest.  < 0 selects the default (2^26).
 *   core_units_out number of units left to the exact program (may be NULL).
 */
bitsmoe_status bitsmoe_allocate_ex(const float* L_host, int64_t units, const int* bits_host,
                                   int nbits, int64_t budget_bits, uint8_t* bits_out_host,
                                   double* objective_out, int64_t full_dp_limit,
                                   int64_t* core_units_out);

/*
 * Input-space basis of a gate/up projection (Sec. 3.2, Eq.
 * shared_basis_input_proj): the experts are stacked along their output
 * channels, W_cat = [W_1; ...; W_E] = P~_cat Phi^T, so Phi holds the
 * eigenvectors of
 *     M_in = W_cat^T W_cat = sum_e W_e^T W_e,
 * computed here in fp64 (same engine and fixed-order reduction as
 * bitsmoe_gram, over the E * d_out stacked rows).  The basis itself comes
 * from bitsmoe_shared_basis(M_in, d_in, r).
 *   W_dev  [E][d_out][d_in] of type wt
 *   M_dev  [d_in][d_in] fp64 output, full symmetric
 * Shape rules: d_out % 64 == 0, d_in % 64 == 0.
 */
bitsmoe_status bitsmoe_gram_experts_in(const void* W_dev, bitsmoe_dtype wt, int64_t E,
                                       int64_t d_out, int64_t d_in, double* M_dev, void* stream);

/*
 * Input-space spectral units: C_e = Phi_r^T W_e^T, so row k of C_e is the
 * column p~_{e,k} = W_e phi_k of P~_e = W_e Phi (Definitions
 * spectral_energy_matrix and spectral_matrix); unit u = e*r + k, length d_out.
 * As in bitsmoe_project, the fp32 basis is split into bf16 hi + lo terms.
 *   Vt_dev  [r][d_in] fp32 (row k = phi_k, e.g. from bitsmoe_shared_basis)
 *   W_dev   [E][d_out][d_in] of type wt
 *   C_dev   [E][r][d_out] fp32 output
 * Shape rules: d_out % 64 == 0, d_in % 64 == 0, 1 <= r <= d_in.
 */
bitsmoe_status bitsmoe_project_in(const float* Vt_dev, const void* W_dev, bitsmoe_dtype wt,
                                  int64_t E, int64_t d_out, int64_t d_in, int64_t r,
                                  float* C_dev, void* stream);

/*
 * Activation-aware importance of each input-space basis vector (Eq.
 * beta_def): beta[k] = phi_k^T H phi_k for the rows phi_k of Vt, through the
 * same fp16 matrix-core form as bitsmoe_score (relative error ~1e-4).
 *   Vt_dev    [r][d] fp32;  H_dev [d][d] fp32 symmetric (as bitsmoe_score)
 *   beta_dev  [r] fp32 output
 * Shape rules: d % 64 == 0, d < 2^22.
 */
bitsmoe_status bitsmoe_basis_importance(const float* Vt_dev, int64_t r, int64_t d,
                                        const float* H_dev, float* beta_dev, void* stream);

/*
 * Loss table of the input-space units under the paper's diagonal
 * approximation (the cross terms phi_k^T H phi_l, k != l, of Lemma
 * spectrum_wise_error_decomp dropped; Corollary additive_spectrum_wise_loss):
 *     L[u][j] = beta[u % r] * ||c_u - Q_{bits[j]}(c_u)||^2
 * with the group-wise quantizer of bitsmoe_score (so widths and codes match
 * bitsmoe_pack).  The error norms are summed in fp32.
 *   C_dev     [units][d] fp32 (from bitsmoe_project_in)
 *   beta_dev  [r] fp32 (from bitsmoe_basis_importance)
 *   L_dev     [units][nbits] fp32 output
 * Shape rules as bitsmoe_score.
 */
bitsmoe_status bitsmoe_score_diag(const float* C_dev, int64_t units, int64_t d,
                                  const float* beta_dev, int64_t r, const int* bits_host, int nbits,
                                  int group, float* L_dev, void* stream);

/*
 * Routing-affinity-weighted calibration Gram of every expert (App. B.2, Eq.
 * app_affinity_gram: H = X Diag(g) X^T over the tokens routed to the expert):
 *     H_e = (1/n) sum_{i in [offsets[e], offsets[e+1])} w_i x_{rows[i]} x_{rows[i]}^T
 * with the same 1/n as bitsmoe_gram (so, with every token's weights summing
 * to 1, sum_e H_e is the shared Gram).  The routed rows are gathered on the
 * device (the weighted side split into bf16 hi + lo) and all experts' Grams
 * run in one batched symmetric matrix-core launch, reduced in fp64 in a
 * fixed order.
 *   X_dev         [n][d] of type xt (calibration rows)
 *   offsets_host  [E + 1] non-decreasing, offsets[0] = 0 (host)
 *   rows_host     [offsets[E]] row of X of each routed entry, in [0, n) (host)
 *   weights_host  [offsets[E]] routing weight of each entry, finite, >= 0 (host)
 *   H_dev         [E][d][d] fp32 output, full symmetric
 * The host tables are copied to the device before the call returns (the
 * call synchronizes `stream` for that).  Shape rules: d % 64 == 0,
 * 1 <= E <= 65535.
 */
bitsmoe_status bitsmoe_gram_routed(const void* X_dev, bitsmoe_dtype xt, int64_t n, int64_t d,
                                   int64_t E, const int64_t* offsets_host, const int32_t* rows_host,
                                   const float* weights_host, float* H_dev, void* stream);

/*
 * bitsmoe_score with one H per expert: the units are grouped by expert,
 * units_per_h consecutive units per H, and unit u is scored against
 * H_dev[u / units_per_h] (the routed Grams of bitsmoe_gram_routed).
 *   H_dev  [units / units_per_h][d][d] fp32 symmetric
 * Shape rules as bitsmoe_score, plus units % units_per_h == 0 and
 * units_per_h * nbits % 256 == 0 (every 256-row tile of error rows belongs
 * to one expert).
 */
bitsmoe_status bitsmoe_score_routed(const float* C_dev, int64_t units, int64_t d, const float* H_dev,
                                    int64_t units_per_h, const int* bits_host, int nbits, int group,
                                    float* L_dev, void* stream);

/*
 * Stage-3 inference of one projection from its packed factors (Sec. 4.4:
 * the packed expert-specific factors are dequantized inside the expert
 * kernels).  With the output-space basis W_e ~ U C^_e, every token b gets
 *     y_b = U z_b,   z_b = sum over token b's routing entries i of
 *                          weights[i] C^_{e(i)} x_b,
 * where e(i) is the expert whose range [offsets[e], offsets[e+1]) holds i and
 * C^_e is expert e's r packed units decoded exactly as bitsmoe_unpack does
 * (widths 0..8 and 16).  Each unit row is decoded once per chunk of its
 * expert's tokens (below 16 tokens, or when d_in is not a multiple of 128,
 * chunks of two on the vector units; otherwise chunks of 8, or 16 when the
 * experts average more than 8 tokens, on the matrix cores: the codes as
 * exact fp16 integers times the tokens as fp16 hi + lo, per group
 * s sum q x + m sum x in fp32, and y = U z as an fp32 matrix product); the
 * basis is applied once per token.
 *   codes_dev, params_dev, bits_dev, word_offsets_dev, total_words
 *               the packed units of all E * r units (as from bitsmoe_pack;
 *               bits and offsets must cover E * r units)
 *   Ut_dev      [r][d_out] fp32 shared basis (bitsmoe_shared_basis)
 *   X_dev       [B][d_in] fp32 tokens
 *   offsets_host, tokens_host, weights_host
 *               the routing, grouped by expert as for bitsmoe_gram_routed
 *               (tokens in [0, B), finite weights); copied to the device
 *               before the call returns
 *   Y_dev       [B][d_out] fp32 output (a token without entries gets 0)
 * Shape rules: d_in % 64 == 0, d_in <= 2^20, group in {32, 64, 128, 256},
 * d_in % group == 0, r <= 8192, E and B <= 65535, and at most 65535 chunks
 * of four routing entries of one expert.  A unit whose width or offsets are
 * inconsistent contributes nothing.  The call waits for the stream once
 * (after copying the routing tables) before it enqueues the kernels.
 */
bitsmoe_status bitsmoe_moe_decode(const uint64_t* codes_dev, const uint16_t* params_dev,
                                  const uint8_t* bits_dev, const int64_t* word_offsets_dev,
                                  int64_t total_words, int64_t E, int64_t r, int64_t d_in, int group,
                                  const float* Ut_dev, int64_t d_out, const float* X_dev, int64_t B,
                                  const int64_t* offsets_host, const int32_t* tokens_host,
                                  const float* weights_host, float* Y_dev, void* stream);

/*
 * Stage-3 inference of a gate/up projection built in input space
 * (bitsmoe_gram_experts_in, bitsmoe_project_in; Sec. 3.2 and Sec. 4.4): the
 * units of C^_e are the columns W_e phi_k (length d_out), so the basis is
 * applied once per token before the experts,
 *     z_b = Phi_r^T x_b,   y_b = sum over token b's routing entries i of
 *                                 weights[i] C^_{e(i)}^T z_b.
 *   codes_dev .. total_words   the packed units of all E * r units, of
 *               length d_out (as from bitsmoe_pack)
 *   Vt_dev      [r][d_in] fp32 basis rows phi_k^T
 *   X_dev       [B][d_in] fp32 tokens
 *   offsets_host, tokens_host, weights_host   as bitsmoe_moe_decode
 *   Y_dev       [B][d_out] fp32 output (a token without entries gets 0)
 * Shape rules: d_out % 64 == 0, d_out % group == 0, group in {32, 64, 128,
 * 256}, d_out and d_in <= 2^20, r <= 8192, E and B <= 65535, at most 65535
 * chunks of four routing entries of one expert.  Units with inconsistent
 * widths or offsets contribute nothing.  The call waits for the stream once
 * (after copying the routing tables).
 */
bitsmoe_status bitsmoe_moe_decode_in(const uint64_t* codes_dev, const uint16_t* params_dev,
                                     const uint8_t* bits_dev, const int64_t* word_offsets_dev,
                                     int64_t total_words, int64_t E, int64_t r, int64_t d_out,
                                     int group, const float* Vt_dev, int64_t d_in,
                                     const float* X_dev, int64_t B, const int64_t* offsets_host,
                                     const int32_t* tokens_host, const float* weights_host,
                                     float* Y_dev, void* stream);

/*
 * bitsmoe_moe_decode with the router's top-k table on the device, for
 * decode loops: token b's routing entries are the k slots
 * topk_experts_dev[b][0..k) with weights topk_weights_dev[b][0..k), summed
 * in slot order.  Nothing is read back to the host and the call does not
 * wait for the stream (after the first call on a device, which allocates
 * the partial sums).  Each slot's expert row is decoded for that token
 * alone below 16 tokens (or when d_in is not a multiple of 128); otherwise
 * the slots are grouped by expert on the device (E <= 4096) and each
 * expert's rows are decoded once per chunk of its tokens on the matrix
 * cores (as in bitsmoe_moe_decode).
 *   topk_experts_dev  [B][k] int32; a slot whose expert is outside [0, E)
 *                     contributes nothing
 *   topk_weights_dev  [B][k] fp32, used as given
 * Shape rules as bitsmoe_moe_decode, plus 1 <= k <= E and B * k <= 65535.
 */
bitsmoe_status bitsmoe_moe_decode_topk(const uint64_t* codes_dev, const uint16_t* params_dev,
                                       const uint8_t* bits_dev, const int64_t* word_offsets_dev,
                                       int64_t total_words, int64_t E, int64_t r, int64_t d_in,
                                       int group, const float* Ut_dev, int64_t d_out,
                                       const float* X_dev, int64_t B, int64_t k,
                                       const int32_t* topk_experts_dev,
                                       const float* topk_weights_dev, float* Y_dev, void* stream);

/*
 * bitsmoe_moe_decode_topk for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, results and shape rules as
 * bitsmoe_moe_decode_topk; it calls no hipMalloc, hipFree or other
 * allocating routine, creates no events and does not wait.
 * Its scratch (the partial sums, [B * k][r] fp32; on the matrix-core path
 * also the tokens as fp16, their block sums, the routing tables and the
 * token sums [B rounded up to 64][r], about 4 B d_in + 16 B k + 4 B r bytes
 * more) lives in a fixed 16 MiB device
 * array that every GPU the library runs on holds until the process ends; a
 * call that needs more (B * k * r near 4194304 floats or above) gives
 * BITSMOE_ERR_SHAPE.  The array's address on a device is looked up on the
 * first call on that device.  Every call on one GPU shares that GPU's
 * array: calls that overlap on one GPU (different streams, or several host
 * threads) race on it and must be ordered by the caller.  Nothing in the
 * array needs clearing between calls: each call writes every value it
 * reads.
 */
bitsmoe_status bitsmoe_moe_decode_topk_noalloc(const uint64_t* codes_dev,
                                               const uint16_t* params_dev, const uint8_t* bits_dev,
                                               const int64_t* word_offsets_dev,
                                               int64_t total_words, int64_t E, int64_t r,
                                               int64_t d_in, int group, const float* Ut_dev,
                                               int64_t d_out, const float* X_dev, int64_t B,
                                               int64_t k, const int32_t* topk_experts_dev,
                                               const float* topk_weights_dev, float* Y_dev,
                                               void* stream);

/*
 * The paper's surrogate cost table (App. B.3-B.4, Theorem
 * app_spectrum_loss; candidate widths of Eq. piecewise_error_surrogate).
 * For unit row c (length d): alpha^2 = ||c||^2, p = c / alpha,
 * beta = p^T H p (the output-space importance of Eq. app_down_beta_approx),
 * rho = ||p||_inf, cos theta = ||p||_1 / sqrt(d), and
 *     L[u][j] = alpha^2 beta^gamma E(b_j),  b = 0, 1, 2, 3, 4, 6, 8, 16:
 *     E(0) = 1 (eviction), E(1) = sin^2 theta (sign quantizer),
 *     E(2|3|4) = kappa_host[0|1|2], E(6|8|16) = (d rho^2 / 3) 4^-b.
 * A zero row costs 0 at every width.
 *   C_dev       [units][d] fp32
 *   H_dev       [d][d] fp32 symmetric positive semidefinite (upper triangle
 *               of 256 x 256 blocks and the diagonal are read)
 *   gamma       smoothing exponent in [0, 1] (the paper: 0.7 for
 *               Qwen3-30B-A3B, 0.5 for Mixtral-8x7B, 0.2 for DeepSeek-V2-Lite)
 *   kappa_host  [3] low-bit coefficients for widths 2, 3, 4 (the paper's
 *               Table kappa_values: 0.14949200, 0.04067890, 0.01184786)
 *   L_dev       [units][BITSMOE_SURROGATE_NWIDTHS] fp32 output
 *   stats_dev   [units][4] fp32 output {alpha^2, beta, rho, cos theta}, or NULL
 * Shape rules: d % 64 == 0, d < 2^22.  beta comes from the same fp16
 * matrix-core form as bitsmoe_score (relative error ~1e-4).
 */
bitsmoe_status bitsmoe_surrogate(const float* C_dev, int64_t units, int64_t d, const float* H_dev,
                                 double gamma, const double* kappa_host, float* L_dev,
                                 float* stats_dev, void* stream);

/*
 * ILP budget of one projection under the paper's equivalent bit-width
 * (App. B.5, Eqs. app_projection_bit_budget, app_projection_normalized_budget):
 * E experts of n_out x m weights at b_eq bits per weight, minus the fp16
 * shared basis (n_out x r), divided by the spectral-vector length m:
 *     budget = floor((E n_out m b_eq - 16 n_out r) / m)
 * (the paper's floor(E n b_eq - 16 n^2 / m) at r = n_out).
 * ERR_INFEASIBLE if the basis alone exceeds the storage.
 */
bitsmoe_status bitsmoe_surrogate_budget(int64_t E, int64_t n_out, int64_t m, int64_t r,
                                        double b_eq, int64_t* budget_out);

/*
 * Packed layout (host): unit u occupies bits[u] * d/64 uint64 words starting
 * at word_offsets_host[u]; word_offsets_host has units + 1 entries and the
 * last one is the total.  d % 64 == 0; each width is 1..8, or one of the
 * surrogate's extra candidates 0 (evicted, no words) and 16 (fp16 row).
 */
bitsmoe_status bitsmoe_pack_layout(const uint8_t* bits_host, int64_t units, int64_t d,
                                   int64_t* word_offsets_host);

/*
 * Step 5 -- pack the factors at the chosen widths.
 * Each unit row is quantized by the same group rule as bitsmoe_score, with
 * the quotient (c - m)/s taken in fp64, and stored as bit planes: plane t
 * (0 = least significant) of unit u is the word range
 * [off[u] + t*d/64, off[u] + (t+1)*d/64), and bit j of word w of a plane is
 * bit t of the code of entry 64*w + j.  params_dev[u][g] holds the fp16 bit
 * patterns {scale, min} of group g.  The surrogate's extra widths: 16 stores
 * the row in fp16 (round to nearest even), entry k in bits 16 (k % 4) of word
 * k / 4 of the unit; 0 (eviction) stores no words.  Both get zero params.
 *   C_dev             [units][d] fp32
 *   bits_dev          [units] widths (device)
 *   word_offsets_dev  [units + 1] from bitsmoe_pack_layout (device)
 *   codes_dev         [total_words] uint64 output
 *   params_dev        [units][d/group][2] uint16 output
 * A unit whose width is not 0, 1..8 or 16, or whose offsets do not match its
 * width or exceed total_words, is left unwritten.
 */
bitsmoe_status bitsmoe_pack(const float* C_dev, int64_t units, int64_t d, int group,
                            const uint8_t* bits_dev, const int64_t* word_offsets_dev,
                            int64_t total_words, uint64_t* codes_dev, uint16_t* params_dev,
                            void* stream);

/*
 * Inverse of bitsmoe_pack: x = m + q * s per entry, fp32 [units][d].  This
 * is the dequantized factor a decoder would use; it equals the fake-quant
 * value of bitsmoe_score's rule (the stored fp16 row at width 16, zeros at
 * width 0).
 */
bitsmoe_status bitsmoe_unpack(const uint64_t* codes_dev, const uint16_t* params_dev,
                              const uint8_t* bits_dev, const int64_t* word_offsets_dev,
                              int64_t total_words, int64_t units, int64_t d, int group,
                              float* Chat_dev, void* stream);

/* Path of a LAPACK shared library for bitsmoe_shared_basis (LP64 or ILP64
 * dsyevd; both plain and "64_"-suffixed symbol names are tried).  When never
 * set, the environment variable BITSMOE_LAPACK is used, then liblapack.so.3. */
bitsmoe_status bitsmoe_set_lapack(const char* path);

/* Kernel timing for measurement.  While enabled, every device call records a
 * pair of HIP events on its stream around each of its main kernels, under
 * the names "gram", "gram_experts", "project", "score_dgen", "score_gemm",
 * "pack".  bitsmoe_kernel_time waits for the recorded events of `name`,
 * returns their summed duration in ms and the number of launches, and
 * forgets them.  Enabling costs two event records per kernel and no
 * synchronization; each record also holds the stream for a few microseconds
 * between kernels.  bitsmoe_timing_only(name) restricts the records to the
 * kernels timed under `name` (NULL or "": all of them), so that one kernel
 * can be timed inside a measured region without the others' records. */
bitsmoe_status bitsmoe_timing(int enable);
bitsmoe_status bitsmoe_timing_only(const char* name);
bitsmoe_status bitsmoe_kernel_time(const char* name, double* total_ms, int64_t* launches);

/* Text of the last non-OK status on the calling thread ("" if none). */
const char* bitsmoe_last_error(void);

/* Frees the scratch memory the library holds on every device.  Must not
 * race with calls in flight. */
void bitsmoe_release(void);

/* Library version string. */
const char* bitsmoe_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BITSMOE_H */
