// Internal declarations shared by the host library and the kernel launchers.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include "../../include/fmm8.h"

namespace fmm {

constexpr int kMaxRank = 8;    // <2,2,2;R>, R <= 8 (cubic has 8 terms)
constexpr int kMaxRankShape = 4096;  // other shapes <m,k,n;R>: R <= 4096
constexpr int kMaxGridBlocks = 64;   // other shapes: mk, kn, nm <= 64 (the encoder's and combine's widest grid)
constexpr int kMaxDepth = 3;
constexpr int kSplitTile = 256;  // A rows per tile of the large-tile sub-product path (and code image rows)
constexpr int kSplitTileN = 128; // B rows per tile of that path (half a code image)
constexpr int64_t kSplitMinK = 1024;  // smallest K / 2^l the large-tile path takes by default

struct Realization {
  int R;
  double U[kMaxRank][4];
  double V[kMaxRank][4];
  double W[kMaxRank][4];
};

int realization_builtin(int which, Realization &d);
double brent_residual(const Realization &d);
int realization_transform(const Realization &d, const double X[4], const double Y[4],
                          const double Z[4], Realization &out);
void realization_rebalance(const Realization &d, Realization &out);
void realization_phi_gamma(const Realization &d, double &phi, double &gamma);
int64_t ipow(int64_t b, int e);
// Phi(D . g) and its gradient over the 12 entries of g = (X, Y, Z)
double rebase_phi_grad(const Realization &D, const double g[12], double grad[12]);
// re-basing from the identity and nstarts caller starts (fmm_realization_optimize)
int realization_optimize(const Realization &D, int nstarts, const double *starts, int max_iter,
                         double gtol, double tol, Realization &best, double &best_phi, double *start_phi);
void flatten(const double (*base)[4], int R, int depth, float *out);

// A realization of another shape <m,k,n;R>: U R x mk (block i k + j), V R x kn
// (block j n + l), W R x nm (block l m + i), row-major binary64.
struct Shaped {
  int m, k, n, R;
  const double *U, *V, *W;
};
double brent_residual_shape(const Shaped &s);
void phi_gamma_shape(const Shaped &s, double &phi, double &gamma);
// inverse of the n x n row-major G by Gauss-Jordan elimination with partial
// pivoting in binary64; returns the determinant (0 when a pivot vanishes)
double inverse_gj(const double *G, int n, double *inv);
// D . g for X (m x m), Y (k x k), Z (n x n), row-major: U' rows = u (X (x) Y^-T)
// etc.; FMM_ERR_SINGULAR if some |det| < 1e-12
int transform_shape(const Shaped &s, const double *X, const double *Y, const double *Z, std::vector<double> &U,
                    std::vector<double> &V, std::vector<double> &W);
double rebase_phi_grad_shape(const Shaped &S, const double *g, double *grad);
int realization_optimize_shape(const Shaped &S, int nstarts, const double *starts, int max_iter, double gtol,
                               double tol, std::vector<double> &U, std::vector<double> &V, std::vector<double> &W,
                               double &best_phi, double *start_phi);

// ---- device-side coefficient tables -------------------------------------
// For one operand side: the nonzero coefficients of each flattened term in
// ascending sub-block order.  offsets[r] .. offsets[r+1] index entries.
struct CoefEntry {
  int32_t block;   // sub-block index P 2^l + Q
  float coef;      // fp32 flattened coefficient (nonzero)
};

// Everything a launch needs, in one struct passed by value.
struct Problem {
  int64_t batch, M, K, N;
  int64_t mp, kp, np;      // M / 2^l, K / 2^l, N / 2^l
  int depth, nsplit;       // nsplit = 2^l
  int block, rule;
  int R;                   // base rank
  int64_t T;               // R^l
  int64_t To;              // R^(l-1): number of outer terms
  int64_t kblocks;         // kp / block
  int scale_bytes;         // 1 (E8M0) or 4 (fp32)
  int exact_dot;           // FMM_FLAG_EXACT_DOT requested
  int split;               // large-tile sub-products + separate W-combine (depth <= 2, tile-aligned MX)
  int layout;              // FMM_LAYOUT_* of the workspace's codes and scales
  int b_rows;              // rows of y_r^T per B scale block: 1, or 128 (FMM_FLAG_B_BLOCK128)
  int b_bf16;              // round encoded B combinations to bfloat16 first (FMM_FLAG_B_BF16)
  // the sub-block grid: A gm x gk, B gk x gn, C gm x gn (2^l each for
  // <2,2,2> plans; m, k, n for a realization of another shape, whose plans
  // set `shaped` and run at one level on the large-tile path)
  int gm, gk, gn;
  int shaped;
};

// The dense coefficient rows of a plan of another shape are padded with zeros
// to 16 or 64 entries (the encoder's and the W-combine's grid capacities).
inline int grid_capacity(int blocks) { return blocks <= 16 ? 16 : 64; }

// Large-tile plans whose sub-products take an exact-dot kernel (fp32 scales,
// block 16, or the exact-dot flag): the promote kernel for fp32 scales, the
// folded-scale kernel for E8M0 scales.
inline bool exact_split(const Problem &pb) { return pb.exact_dot || pb.scale_bytes == 4 || pb.block == 16; }

// Bytes of one (batch, term) plane of scales for `rows` rows.
inline int64_t scale_plane_bytes(const Problem &pb, int64_t rows) {
  if (pb.layout == FMM_LAYOUT_TILE128x128) return rows * (pb.kp / 128) * (pb.block == 16 ? 8 : 4);
  return rows * pb.kblocks * pb.scale_bytes;
}

// Layout of a workspace: byte offsets from its base.
struct Workspace {
  size_t a_codes, b_codes, a_scales, b_scales, partial, total;
  size_t products;   // split plans only: the fp32 sub-products P_r
  size_t b_amax;     // FMM_FLAG_B_BLOCK128 plans: 2-D block maxima [batch][T][ceil(n'/128)][kblocks] u32
};

// Device copies of the plan's tables (one allocation).
struct DeviceTables {
  const int32_t *a_off;        // T + 1
  const CoefEntry *a_ent;
  const int32_t *b_off;
  const CoefEntry *b_ent;
  const float *w_inner;        // R x 4 fp32 base w (the inner-level decoder), zero-padded to kMaxRank x 4
  const float *w_outer;        // To x 4^(l-1) fp32 flattened depth-(l-1) w (depth >= 2)
  const float *w_full;         // T x 16 fp32 flattened depth-2 w (large-tile plans at depth 2);
                               // other shapes: T x grid_capacity(gm gn), w index l gm + i
  const float *u_dense;        // T x 4^l fp32 flattened U, zeros included (other shapes:
                               // T x grid_capacity(gm gk))
  const float *v_dense;        // T x 4^l fp32 flattened V, zeros included (other shapes:
                               // T x grid_capacity(gk gn))
};

// ---- launchers (kernels_*.hip); return a hipError_t as int ---------------
int launch_encode(const Problem &pb, const DeviceTables &tab, const float *A, const float *B,
                  uint8_t *ws, const Workspace &wl, void *stream);
// sub-products (split plans: into the product region; otherwise with the fused
// inner W-combine, into C at depth 1 or the partial region at depth >= 2)
int launch_products(const Problem &pb, const DeviceTables &tab, const uint8_t *ws, const Workspace &wl,
                    float *C, void *stream);
// what remains of the W-combine after launch_products (nothing for fused depth-1 plans)
int launch_combine(const Problem &pb, const DeviceTables &tab, const uint8_t *ws, const Workspace &wl,
                   float *C, void *stream);
int launch_products_split(const Problem &pb, const uint8_t *ws, const Workspace &wl, void *stream);
int launch_combine_split(const Problem &pb, const DeviceTables &tab, const uint8_t *ws, const Workspace &wl,
                         float *C, void *stream);
// operand-side rounding energy of the encoding in the workspace (depths 1, 2):
// out [batch][2 sides][T][2] binary64 = (sum (xhat - x)^2, sum x^2)
size_t encode_noise_scratch_bytes(const Problem &pb);
int launch_encode_noise(const Problem &pb, const DeviceTables &tab, const float *A, const float *B,
                        const uint8_t *ws, const Workspace &wl, double *out, void *scratch, void *stream);
// the cross-term diagnostic (depth 1): out [batch][2] binary64 = (|L|^2, diag)
size_t cross_terms_scratch_bytes(const Problem &pb);
int launch_cross_terms(const Problem &pb, const DeviceTables &tab, const float *A, const float *B,
                       const uint8_t *ws, const Workspace &wl, double *out, void *scratch, void *stream);
int launch_reference_f64(int64_t batch, int64_t M, int64_t K, int64_t N, const float *A,
                         const float *B, double *Cref, void *stream);
size_t error_stats_scratch_bytes(int64_t batch, int64_t M, int64_t N);
int launch_error_stats(int64_t batch, int64_t M, int64_t N, const float *C, const double *Cref,
                       double *out, void *scratch, void *stream);
// the allocation-free reduction: products per call, and the device address of
// its static scratch on the current device (a hipError_t)
constexpr int64_t kStaticErrorBatch = 1024;
int static_error_scratch(void **ptr);
int launch_e4m3_quantize(const float *in, uint8_t *out, int64_t n, void *stream);
int launch_e4m3_quantize_pow2(const float *in, uint8_t *out, int64_t n, int e, void *stream);

}  // namespace fmm
