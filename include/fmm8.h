/*
 * fmm8 -- Strassen-type rank-7 bilinear matrix multiplication under a
 * block-scaled e4m3 model, with an fp64 error measurement, on AMD MI355X
 * (gfx950).
 *
 * The operation (Section 2.1 and Section 2.2 of "Fast Matrix Multiplication
 * in fp8: Certified Coefficient Optimization and Measured Error"):
 *
 *   A (M x K) and B (K x N) are split into a 2^l x 2^l grid of sub-blocks.
 *   For every term r of the depth-l flattened realization (U, V, w)
 *     x_r = sum_b U[r,b] A_b   (fp32)          -- encoded combinations,
 *     y_r = sum_b V[r,b] B_b   (fp32)
 *   are formed from the unquantized operands, quantized to e4m3 with one
 *   scale per block of `block` consecutive elements along the contracted
 *   axis (Assumption 1; Appendix E.2), multiplied with fp32 accumulation,
 *   and decoded:  C_(I,K) = sum_r w[r, K 2^l + I] P_r.
 *
 * Coefficient conventions (Appendix A, eq. A.1): rv(A) = (a11,a12,a21,a22);
 * U_r is indexed by 2i+j for A-block (i,j), V_r by 2j+k, and the third factor
 * is cyclic, w_r = rv(W_r^T), indexed by 2k+i.  A depth-l table (Section 3.2,
 * Kronecker powers; Section 4.3, flattened realizations) has T = R^l terms
 * r = sum_t r_t R^(l-t) and 4^l columns, sub-block (P,Q) at column P 2^l + Q;
 * each entry is the product of the l base coefficients, multiplied left to
 * right in binary64 and rounded once to binary32.
 *
 * Memory and ownership.  Every device buffer is allocated and owned by the
 * caller; matrices are row-major and contiguous, batch-major.  Opaque host
 * handles (fmm_real, fmm_plan) are owned by the library and released with
 * their _destroy call.  fmm_encode, fmm_multiply and fmm_matmul never
 * allocate; fmm_plan_create uploads the plan's coefficient tables to the
 * device that is current at the time of the call, and the plan may only be
 * used with that device.
 *
 * Execution.  Device calls are asynchronous on `stream` (a hipStream_t
 * passed as void*; NULL is the null stream) and never synchronize the host.
 * A plan is immutable: one plan may be used concurrently on several streams
 * with distinct workspaces.
 *
 * Errors.  Every call returns an int status: FMM_OK (0) or a negative code.
 * No exception crosses the boundary.  Device-side problems (a failed launch)
 * are reported as FMM_ERR_HIP; fmm_status_string() names any code, and
 * fmm_last_error_detail() returns the last HIP error string of the calling
 * thread.  Non-finite inputs are undefined behaviour.
 */
#ifndef FMM8_H
#define FMM8_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
enum {
  FMM_OK = 0,
  FMM_ERR_ARG = -1,          /* null pointer, out-of-range enum, bad tolerance */
  FMM_ERR_SHAPE = -2,        /* dimensions not divisible as required */
  FMM_ERR_UNSUPPORTED = -3,  /* a shape/rule/block/depth the library does not run */
  FMM_ERR_NOT_EXACT = -4,    /* Brent residual above the tolerance */
  FMM_ERR_SINGULAR = -5,     /* a basis change with |det| < 1e-12 */
  FMM_ERR_HIP = -6,          /* a HIP runtime call or a kernel launch failed */
  FMM_ERR_DEVICE = -7,       /* the device is not gfx950 */
  FMM_ERR_WORKSPACE = -8,    /* workspace too small or misaligned */
  FMM_ERR_NOMEM = -9         /* host allocation failed */
};

/* ---- named realizations ------------------------------------------------ */
enum {
  FMM_CUBIC8 = 0,            /* the cubic <2,2,2;8> algorithm, Phi = 8 (Section 3.2) */
  FMM_STRASSEN = 1,          /* Strassen 1969, M1..M7 in classical order, Phi = 32 */
  FMM_WINOGRAD = 2,          /* Strassen-Winograd variant, raw gauge, Phi = 56 (Table E.2) */
  FMM_TSTAR = 3              /* the Phi-optimal T*, Phi = 200/9 (Theorem 1; eq. A.2) */
};

/* ---- block-scale rules (Appendix E.2; power-of-two variants) ------------ */
enum {
  FMM_RULE_FP32_AMAX = 0,    /* s = fl32(max(amax, fl32(1e-12)) / 448), stored as fp32 */
  FMM_RULE_POW2_CEIL = 1,    /* s = 2^e, e the least integer with a <= 448 2^e; E8M0 byte */
  FMM_RULE_POW2_OCP = 2      /* s = 2^(floor(log2 a) - 8) (OCP MX rule, clips to 448); E8M0 */
};

/* ---- plan flags ---------------------------------------------------------- */
enum {
  /* Sum the products of the dequantized operands at fp32 precision.  The
   * default sub-product path feeds the e4m3 codes and E8M0 scales to the
   * fp8 matrix cores, whose dot product aligns each group of eight products
   * to the group's largest and keeps 13 bits below it (measured on gfx950);
   * with this flag the operands go to the bf16 matrix cores (23 retained
   * bits) exactly: with E8M0 scales each code is converted to bf16 together
   * with its block's power of two (the dequantized value itself, exact for
   * every scale the rules produce), with fp32 scales each block's partial
   * sum of codes is scaled and accumulated in fp32.  Half the peak rate of
   * the default path.  FP32_AMAX scales and block 16 always take this path;
   * tile-aligned plans (FMM_LAYOUT_TILE256x64) on it run on 256 x 128 tiles
   * whatever K. */
  FMM_FLAG_EXACT_DOT = 1,
  /* Weight-side deployment granularity (Appendix E, weight-scale
   * granularity; the real kernel's 128 x 128 weight blocks): one B-side scale
   * covers 128 consecutive columns of B (rows of y_r^T) x `block` positions
   * of the contracted axis, its maximum taken over the encoded combination;
   * the last block of a ragged N / 2 is short.  The stored scales stay one per
   * (row, block), replicated over each 128-row block.  Depth 1 only
   * (FMM_ERR_UNSUPPORTED otherwise).  The encoder reads B twice. */
  FMM_FLAG_B_BLOCK128 = 2,
  /* Round each encoded B combination to bfloat16 (nearest, ties to even)
   * before its scale and cast (Appendix E: the real path's pre-round of the
   * encoded weights).  Depth 1 only. */
  FMM_FLAG_B_BF16 = 4,
  /* Take the large-tile sub-product path (FMM_LAYOUT_TILE256x64) whenever
   * the shape allows it.  Without the flag, plans on the fp8 matrix cores
   * take that path only where K / 2^l >= 1024: it writes every fp32 P_r to
   * the workspace and reads it back, which costs more than it saves on short
   * contractions (exact-dot plans take it whenever the shape allows).  No
   * effect on the result's definition; shapes the path cannot take ignore
   * the flag. */
  FMM_FLAG_LARGE_TILE = 8
};

typedef struct fmm_real fmm_real;   /* a base realization (U, V, w) of <m,k,n;R>, binary64 */
typedef struct fmm_plan fmm_plan;   /* one problem shape bound to a realization */

typedef struct {
  int64_t batch;   /* number of independent products, >= 0 */
  int64_t M, K, N; /* each >= 0 and divisible by 2^depth (by m, k, n for a realization of
                    * another shape <m,k,n;R>); K / 2^depth (K / k) divisible by block */
  int32_t depth;   /* recursion (Kronecker) depth l: 1, 2 or 3 */
  int32_t block;   /* e4m3 block length along the contracted axis: 16, 32 or 128 */
  int32_t rule;    /* FMM_RULE_* */
  int32_t flags;   /* FMM_FLAG_* bits; others must be 0 */
} fmm_plan_desc;

/* Layouts of the quantized operands in a workspace (fmm_view.code_layout). */
enum {
  /* codes [batch][terms][rows][kdim], scales [batch][terms][rows][kblocks] */
  FMM_LAYOUT_ROWS = 0,
  /* codes [batch][terms][rows / 256][kdim / 64][256][64]: 256-row x 64-byte
   * tiles, each contiguous; inside a tile, 16-byte chunk c of tile row t sits
   * at chunk c ^ ((t >> 2) & 3) of that row.
   * scales [batch][terms][kblocks][rows]: for each block of the contracted
   * axis, one scale per row.  E8M0 bytes have the rows of every 256-row tile
   * permuted so that tile row 128 h + 32 i + j (h < 2, i < 4, j < 32) sits at
   * byte 4 (32 h + j) + i; fp32 scales (FMM_RULE_FP32_AMAX) are in row order.
   * Used by plans whose sub-products run on 256-row tiles: depth 1 or 2,
   * M / 2^l and N / 2^l multiples of 256, K / 2^l a multiple of 64 (of 128
   * at block 128), and either fp32 scales (the exact-dot path) or E8M0
   * scales with K / 2^l >= 1024 or FMM_FLAG_LARGE_TILE (the fp8 matrix cores
   * at blocks 32 and 128, the exact-dot path at block 16 or with
   * FMM_FLAG_EXACT_DOT); and every plan of a
   * realization of another shape (rows M / m and N / n, kdim K / k).  The B
   * side is read as 128-row halves of these tiles. */
  FMM_LAYOUT_TILE256x64 = 1,
  /* codes [batch][terms][rows / 128][kdim / 128][128][128]: 128-row x 128-byte
   * tiles, each contiguous; inside a tile, 16-byte chunk c of tile row t sits
   * at chunk c ^ (t & 7) ^ ((t >> 3) & 1) of that row.
   * scales [batch][terms][rows / 128][kdim / 128][128][4 or 8]: for each tile
   * row and 128-byte step, 4 E8M0 bytes: at block 32 the step's blocks 0, 2,
   * 1, 3 in that order, at block 128 the step's one block repeated 4 times;
   * at block 16, 8 bytes: the step's blocks 0, 2, 4, 6, then 1, 3, 5, 7.
   * Used by the other plans with E8M0 scales (blocks 16, 32 and 128) whose
   * M / 2^l and N / 2^l are multiples of 128 and K / 2^l a multiple of 128. */
  FMM_LAYOUT_TILE128x128 = 2
};

/* Where the quantized operands of one side sit inside a workspace, in layout
 * code_layout (A side: rows = M / 2^l; B side: rows = N / 2^l, i.e. y_r
 * transposed; the contracted axis has kdim = K / 2^l codes in kblocks blocks).
 * codes : uint8 e4m3 codes
 * scales: one per block; uint8 E8M0 (e + 127) when scale_bytes == 1, IEEE
 *         binary32 when scale_bytes == 4. */
typedef struct {
  void *codes;
  void *scales;
  int64_t batch, terms, rows, kdim, kblocks;
  int32_t scale_bytes;
  int32_t code_layout; /* FMM_LAYOUT_* */
} fmm_view;

/* ---- realizations (host only; no device needed) ------------------------ */

/* A named realization.  *out receives a new handle. */
int fmm_realization_builtin(int which, fmm_real **out);

/* A realization of <m,k,n;R> (Section 2.1: R rank-one terms of the matrix
 * multiplication tensor of an m x k by k x n product) from caller arrays U, V,
 * w, each R x (m k), R x (k n), R x (n m) row-major binary64: A is split into
 * an m x k grid of sub-blocks, block (i, j) at index i k + j; B into a k x n
 * grid, block (j, l) at j n + l; C block (i, l) takes w's index l m + i (the
 * cyclic third factor of Appendix A; at <2,2,2> the conventions above).
 * Exact means sum_r U_r[i k + j] V_r[j' n + l] w_r[l' m + i'] =
 * [j = j'][l = l'][i = i'] (the Brent equations); if the largest deviation
 * exceeds tol the call fails with FMM_ERR_NOT_EXACT (tol < 0 is FMM_ERR_ARG).
 * <2,2,2;R> takes 1 <= R <= 8 and runs at depths 1 to 3.  Other shapes (the
 * rows of Table E.1 beyond <2,2,2>) take m k, k n, n m <= 64 and
 * 1 <= R <= 4096 (FMM_ERR_UNSUPPORTED for larger grids; m, k or n < 1 or R
 * out of range: FMM_ERR_ARG) and run at depth 1 only, on the large-tile plans
 * (FMM_LAYOUT_TILE256x64). */
int fmm_realization_create(int m, int k, int n, int R, const double *U, const double *V,
                           const double *w, double tol, fmm_real **out);

/* D . g for g = (X, Y, Z) in GL(2)^3 (eq. A.1):
 *   u -> u (X (x) Y^-T), v -> v (Y (x) Z^-T), w -> w (Z (x) X^-T),
 * each 2x2 factor given row-major (4 doubles).  Evaluated in binary64 in
 * this order: the inverse by the adjugate (det = a d - b c, entries divided
 * by det), then the Kronecker matrix, then u K with each entry summed in
 * ascending index; no fused multiply-add.  |det| < 1e-12 gives
 * FMM_ERR_SINGULAR.
 * Another shape <m,k,n> takes g in GL(m) x GL(k) x GL(n): X m x m, Y k x k,
 * Z n x n row-major, the same formulas (u indexed i k + j, so
 * X (x) Y^-T has entry [i k + j][i' k + j'] = X[i][i'] (Y^-T)[j][j'];
 * likewise v, w), i.e. U_r -> X^T U_r Y^-T, V_r -> Y^T V_r Z^-T,
 * W_r -> Z^T W_r X^-T as matrices; the inverses by Gauss-Jordan elimination
 * with partial pivoting. */
int fmm_realization_transform(const fmm_real *d, const double X[4], const double Y[4],
                              const double Z[4], fmm_real **out);

/* The canonical rebalanced gauge (Appendix E.2):
 * (U_r, V_r, W_r) -> (U_r / s_r, s_r V_r, W_r), s_r = sqrt(|U_r| / |V_r|)
 * (terms with a zero U_r or V_r unchanged); any shape. */
int fmm_realization_rebalance(const fmm_real *d, fmm_real **out);

/* Re-basing (Section 3.1; the protocol of Appendix E.2): minimize Phi over
 * the change-of-basis orbit D . g, g = (X, Y, Z) in GL(2)^3 (eq. A.1), or in
 * GL(m) x GL(k) x GL(n) for another shape (fmm_realization_transform's
 * action; P = m^2 + k^2 + n^2 entries, 12 at <2,2,2>).
 * Starts: g = (I, I, I) (the realization itself) and, for s < nstarts, the
 * caller's triple starts[P s .. P s + P - 1] = (X, Y, Z), each row-major
 * (the paper draws X, Y, Z as I + 0.45 N(0,1) and rejects |det| < 1e-3; the
 * caller does the drawing).  Each start runs limited-memory BFGS (memory 10)
 * with a strong-Wolfe line search (c1 = 1e-4, c2 = 0.9) in binary64 over the
 * P entries of g, with the exact gradient, until the largest gradient entry
 * is at most gtol * max(1, Phi), progress falls below rounding, or max_iter
 * iterations.  The terminal g gives D . g by fmm_realization_transform's
 * arithmetic; among the terminal realizations with a finite Phi and a Brent
 * residual <= tol, the one with the least Phi (the earliest start on ties)
 * is returned in *out (a new handle), its Phi in *phi (may be NULL).
 * start_phi (may be NULL; 1 + nstarts entries) receives each start's terminal
 * Phi, NaN where it was singular or failed the exactness check.
 * Errors: FMM_ERR_ARG (null d or out; nstarts < 0; starts NULL while
 * nstarts > 0; max_iter < 1; gtol <= 0; tol < 0 or NaN); FMM_ERR_NOT_EXACT
 * if no start ends exact within tol.  Host only. */
int fmm_realization_optimize(const fmm_real *d, int nstarts, const double *starts, int max_iter,
                             double gtol, double tol, fmm_real **out, double *phi, double *start_phi);

/* Phi(D . g) for g = (X, Y, Z) = g[0..3], g[4..7], g[8..11] (row-major 2x2
 * each; eq. A.1) and its gradient with respect to those 12 entries, the
 * objective fmm_realization_optimize minimizes (another shape: X, Y, Z of
 * m^2, k^2, n^2 entries in that order, P in all, and grad of P entries).
 * phi may be NULL.  Errors: FMM_ERR_ARG (null d, g or grad).  A singular g
 * gives non-finite values. */
int fmm_realization_phi_gradient(const fmm_real *d, const double *g, double *phi, double *grad);

/* Phi = sum_r |U_r|^2 |V_r|^2 |W_r|^2 and Gamma = sum_r |U_r||V_r||W_r|
 * (Section 2.1) of the depth-l flattening (Phi^l, Gamma^l), and the Brent
 * residual of the base realization.  Any output pointer may be NULL.  Other
 * shapes than <2,2,2>: depth 1 only (FMM_ERR_UNSUPPORTED otherwise). */
int fmm_realization_metrics(const fmm_real *d, int depth, double *phi, double *gamma,
                            double *brent_resid);

/* R (base rank) and T = R^depth (other shapes: depth 1 only, as above). */
int fmm_realization_terms(const fmm_real *d, int depth, int64_t *rank, int64_t *terms);

/* The shape <m,k,n> and rank R of a realization (any pointer may be NULL). */
int fmm_realization_shape(const fmm_real *d, int *m, int *k, int *n, int *R);

/* The base coefficients, R x (m k), R x (k n), R x (n m) binary64 (R x 4 each
 * at <2,2,2>; any pointer may be NULL). */
int fmm_realization_coefficients(const fmm_real *d, double *U, double *V, double *w);

/* The exact fp32 depth-l tables the kernels use, T x 4^l each (other shapes:
 * depth 1, R x (m k), R x (k n), R x (n m), each entry rounded once). */
int fmm_realization_tables(const fmm_real *d, int depth, float *U, float *V, float *w);

void fmm_realization_destroy(fmm_real *d);

/* ---- plans and the product --------------------------------------------- */

/* Validates desc (FMM_ERR_ARG / FMM_ERR_SHAPE / FMM_ERR_UNSUPPORTED are
 * returned before any device call), then uploads the coefficient tables to
 * the current device (FMM_ERR_DEVICE if it is not gfx950).
 * A realization of another shape <m,k,n;R> splits A into m x k sub-blocks of
 * M / m x K / k, B into k x n of K / k x N / n, and runs at depth 1 on the
 * large-tile path only: M / m and N / n multiples of 256 and K / k a multiple
 * of 64 (of 128 at block 128), with no flags but FMM_FLAG_EXACT_DOT and
 * FMM_FLAG_LARGE_TILE; anything else is FMM_ERR_UNSUPPORTED (dimensions not
 * divisible by m, k, n or K / k by block: FMM_ERR_SHAPE).  Such plans have
 * no operand-noise or cross-term pass (FMM_ERR_UNSUPPORTED). */
int fmm_plan_create(const fmm_real *d, const fmm_plan_desc *desc, fmm_plan **out);

/* Bytes of device workspace fmm_encode/fmm_multiply/fmm_matmul need: the
 * codes and scales of both operands, plus, for large-tile plans the fp32
 * sub-products P_r, for the others at depth >= 2 the inner-level partial
 * products, and with FMM_FLAG_B_BLOCK128 the B side's 2-D block maxima.
 * The workspace must be 256-byte aligned. */
int fmm_plan_workspace_size(const fmm_plan *p, size_t *bytes);

/* Steps "encode + quantize" of both operands (device pointers dA: batch x M x K,
 * dB: batch x K x N, fp32, each 16-byte aligned) into the workspace. */
int fmm_encode(const fmm_plan *p, const float *dA, const float *dB, void *dWs, void *stream);

/* Pointers and extents of the quantized operands inside dWs (host call). */
int fmm_operand_views(const fmm_plan *p, void *dWs, fmm_view *a, fmm_view *b);

/* Steps "fp8 sub-products + W-combine" (Algorithm 1, the products P_r of the
 * quantized operands and C = sum_r w_r (x) P_r): reads the encoded workspace
 * and writes C (batch x M x N fp32, 4-byte aligned).  Equal to fmm_products
 * followed by fmm_combine on the same stream. */
int fmm_multiply(const fmm_plan *p, void *dWs, float *dC, void *stream);

/* The first half of fmm_multiply: the T block-scaled fp8 sub-products with
 * fp32 accumulation.  Plans with the large-tile layout (fmm_view.code_layout
 * == FMM_LAYOUT_TILE256x64) write every P_r, fp32, to the workspace (and
 * fmm_combine forms C = sum_r w_r (x) P_r over all T terms in one pass, in
 * ascending r with one fused multiply-add per nonzero weight); the others
 * fold the base-level w into the sub-product kernel and write C (depth 1) or
 * the per-outer-term partial sums (depth >= 2, workspace). */
int fmm_products(const fmm_plan *p, void *dWs, float *dC, void *stream);

/* The second half of fmm_multiply: what remains of the W-combine after
 * fmm_products (reads the workspace, writes C); nothing for the plans that
 * fold it into the sub-product kernel at depth 1. */
int fmm_combine(const fmm_plan *p, void *dWs, float *dC, void *stream);

/* fmm_encode followed by fmm_multiply. */
int fmm_matmul(const fmm_plan *p, const float *dA, const float *dB, float *dC, void *dWs,
               void *stream);

void fmm_plan_destroy(fmm_plan *p);

/* ---- error measurement (Appendix E.2: relative error against an fp64 product) */

/* dCref = A B in binary64 (batch x M x N), from the fp32 operands. */
int fmm_reference_f64(int64_t batch, int64_t M, int64_t K, int64_t N, const float *dA,
                      const float *dB, double *dCref, void *stream);

/* Device scratch the reduction below needs (bytes; the scratch passed must
 * hold at least that many and be 8-byte aligned, else FMM_ERR_WORKSPACE). */
int fmm_error_stats_scratch_size(int64_t batch, int64_t M, int64_t N, size_t *bytes);

/* Per product b: dOut[2b] = sum (C - Cref)^2, dOut[2b+1] = sum Cref^2, binary64,
 * by a fixed-order two-pass reduction (identical results run to run).
 * dOut is a device pointer to 2*batch doubles. */
int fmm_error_stats(int64_t batch, int64_t M, int64_t N, const float *dC, const double *dCref,
                    double *dOut, void *dScratch, size_t scratch_bytes, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * fmm_error_stats without the scratch argument.  The reduction's partials
 * live in a static device array of the library (8 MiB on every device the
 * library runs on, held until the process ends), so at most
 * FMM_ERROR_STATS_NOALLOC_MAX_BATCH products per call; a larger batch fails
 * with FMM_ERR_WORKSPACE (fmm_last_error_detail() says why) before any device
 * call.  Same kernels, same fixed order and results as fmm_error_stats.  The
 * call itself allocates nothing; its first call on a device looks up the
 * array's device address there.  Calls on one device share the array: calls
 * that overlap in time on one device (other streams, other threads) race and
 * must be serialized by the caller.  Every partial is written before it is
 * read, so a call does not depend on what an earlier call left there. */
#define FMM_ERROR_STATS_NOALLOC_MAX_BATCH 1024
int fmm_error_stats_noalloc(int64_t batch, int64_t M, int64_t N, const float *dC, const double *dCref,
                            double *dOut, void *stream);

/* ---- the codec alone --------------------------------------------------- */

/* Operand-side rounding energy of the encoding in dWs (Appendix D,
 * eq. D.1: the noise coefficient s^2 = sum (xhat - x)^2 / sum x^2 of the
 * model of Section 2.2).  Call after fmm_encode with the same dA, dB and
 * workspace: the combinations x_r are formed again with the encoder's
 * arithmetic, the stored codes and scales are decoded to xhat_r (exact in
 * binary64), and dOut (device, [batch][2][T][2] binary64; side 0 = A, 1 = B)
 * receives, for every batch element, side and flattened term, the sums of
 * (xhat - x)^2 and of x^2 over the term's positions (binary64, a fixed
 * summation order, so repeated calls agree bit for bit).  With
 * FMM_FLAG_B_BF16, x is the combination before the bfloat16 rounding.
 * dScratch: device, 8-byte aligned, at least fmm_encode_noise_scratch_size
 * bytes (FMM_ERR_WORKSPACE otherwise).  Depths 1 and 2 (FMM_ERR_UNSUPPORTED
 * at depth 3).  Asynchronous on stream. */
int fmm_encode_noise_scratch_size(const fmm_plan *p, size_t *bytes);
int fmm_encode_noise(const fmm_plan *p, const float *dA, const float *dB, const void *dWs, double *dOut,
                     void *dScratch, size_t scratch_bytes, void *stream);

/* The cross-term diagnostic of the error model (Appendix D: the share of
 * the error's linear part that the diagonal sum defining Phi leaves out).
 * Call after fmm_encode with the same dA, dB and workspace; depth-1 plans
 * only (FMM_ERR_UNSUPPORTED otherwise), any layout, rule and block.  With
 * X_r, Y_r the fp32 combinations (the encoder's arithmetic), dX_r, dY_r their
 * rounding residuals against the stored codes times their scales, t_r =
 * dX_r Y_r + X_r dY_r (m' x n', binary64) and L_q = sum_r w[r, q] t_r, dOut
 * (device, [batch][2] binary64) receives for every batch element
 * |L|^2 = sum_q |L_q|^2 and diag = sum_{r, q} w[r, q]^2 |t_r|^2, each by a
 * fixed summation order (repeated calls agree bit for bit); the residual
 * fraction is (|L|^2 - diag) / |L|^2.  dScratch: device, 256-byte aligned, at
 * least fmm_cross_terms_scratch_size bytes (16 (M + N) K / 2 + 8 M N / 4
 * bytes per term and product, FMM_ERR_WORKSPACE otherwise).  With
 * FMM_FLAG_B_BF16, Y_r is the combination before the bfloat16 rounding.
 * Asynchronous on stream; measurement, not on the timed path. */
int fmm_cross_terms_scratch_size(const fmm_plan *p, size_t *bytes);
int fmm_cross_terms(const fmm_plan *p, const float *dA, const float *dB, const void *dWs, double *dOut,
                    void *dScratch, size_t scratch_bytes, void *stream);

/* dOut[i] = e4m3 code of dIn[i] at unit scale: round to nearest, ties to the
 * even mantissa field, saturate to +-448, keep the sign (the cast the
 * quantizer applies after dividing by the block scale).  n >= 0; dIn must be
 * 16-byte and dOut 4-byte aligned. */
int fmm_e4m3_quantize(const float *dIn, uint8_t *dOut, int64_t n, void *stream);

/* dOut[i] = e4m3 code of dIn[i] / 2^e: the cast the power-of-two scale rules
 * (FMM_RULE_POW2_CEIL, FMM_RULE_POW2_OCP; E8M0 byte e + 127) apply to every
 * element of a block, through the same device routine as the encoder.  The
 * quotient is the binary32 value fl32(x / 2^e), then cast as above: round to
 * nearest, ties to the even mantissa field, saturate to +-448 (a quotient
 * beyond the binary32 range included), keep the sign.  e in [-126, 127] (the
 * rules produce -48 .. 120; FMM_ERR_ARG otherwise); n >= 0; dIn 16-byte and
 * dOut 4-byte aligned.  Asynchronous on stream. */
int fmm_e4m3_quantize_pow2(const float *dIn, uint8_t *dOut, int64_t n, int32_t e, void *stream);

/* ---- misc ---------------------------------------------------------------- */

const char *fmm_status_string(int status);
const char *fmm_last_error_detail(void);
/* FMM_OK if device `device` is a gfx950, FMM_ERR_DEVICE if not, FMM_ERR_HIP
 * if it cannot be queried. */
int fmm_device_check(int device);

#ifdef __cplusplus
}
#endif

#endif /* FMM8_H */
