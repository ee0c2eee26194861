// Realizations of <2,2,2;R>: the named tables, the change-of-basis action,
// the canonical gauge, Phi/Gamma/Brent, and the depth-l flattening into the
// fp32 tables the kernels consume; and realizations of other shapes
// <m,k,n;R> (Section 2.1), with the shape-independent parts of the same
// (Brent residual, Phi/Gamma, the gauge, fp32 tables at one level).  Host
// code only; compiled with -ffp-contract=off so every binary64 expression
// rounds once per operation.
#include "internal.h"

#include <cmath>
#include <initializer_list>
#include <cstring>
#include <new>
#include <utility>
#include <vector>

namespace fmm {

namespace {

// Correctly rounded binary64 values of the irrational entries of T* (eq. A.2).
constexpr double kXi = 0x1.279a74590331cp-1;    // 1 / sqrt(3)
constexpr double kEta = 0x1.bb67ae8584caap-1;   // sqrt(3) / 2
constexpr double kZeta = 0x1.279a74590331cp-2;  // 1 / (2 sqrt(3)) = xi / 2 exactly

void set_rows(Realization &d, int R, const double (*U)[4], const double (*V)[4],
              const double (*W)[4]) {
  d.R = R;
  for (int r = 0; r < R; ++r)
    for (int c = 0; c < 4; ++c) {
      d.U[r][c] = U[r][c];
      d.V[r][c] = V[r][c];
      d.W[r][c] = W[r][c];
    }
}

// Cubic algorithm: term (i,j,k) in lexicographic order with u = e_{2i+j},
// v = e_{2j+k}, w = e_{2k+i} (cyclic third factor).
void make_cubic(Realization &d) {
  d.R = 8;
  std::memset(d.U, 0, sizeof(d.U));
  std::memset(d.V, 0, sizeof(d.V));
  std::memset(d.W, 0, sizeof(d.W));
  int r = 0;
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j)
      for (int k = 0; k < 2; ++k, ++r) {
        d.U[r][2 * i + j] = 1.0;
        d.V[r][2 * j + k] = 1.0;
        d.W[r][2 * k + i] = 1.0;
      }
}

// Strassen 1969: M1 = (A11+A22)(B11+B22), M2 = (A21+A22)B11, M3 = A11(B12-B22),
// M4 = A22(B21-B11), M5 = (A11+A12)B22, M6 = (A21-A11)(B11+B12),
// M7 = (A12-A22)(B21+B22); C11 = M1+M4-M5+M7, C12 = M3+M5, C21 = M2+M4,
// C22 = M1-M2+M3+M6.  w columns are (C11, C21, C12, C22).
void make_strassen(Realization &d) {
  static const double U[7][4] = {{1, 0, 0, 1}, {0, 0, 1, 1}, {1, 0, 0, 0}, {0, 0, 0, 1},
                                 {1, 1, 0, 0}, {-1, 0, 1, 0}, {0, 1, 0, -1}};
  static const double V[7][4] = {{1, 0, 0, 1}, {1, 0, 0, 0}, {0, 1, 0, -1}, {-1, 0, 1, 0},
                                 {0, 0, 0, 1}, {1, 1, 0, 0}, {0, 0, 1, 1}};
  static const double W[7][4] = {{1, 0, 0, 1}, {0, 1, 0, -1}, {0, 0, 1, 1}, {1, 1, 0, 0},
                                 {-1, 0, 1, 0}, {0, 0, 0, 1}, {1, 0, 0, 0}};
  set_rows(d, 7, U, V, W);
}

// Strassen-Winograd, raw gauge: M1 = A11 B11, M2 = A12 B21,
// M3 = (A11+A12-A21-A22) B22, M4 = A22 (B11-B12-B21+B22),
// M5 = (A21+A22)(B12-B11), M6 = (A21+A22-A11)(B11-B12+B22),
// M7 = (A11-A21)(B22-B12); C11 = M1+M2, C12 = M1+M3+M5+M6,
// C21 = M1-M4+M6+M7, C22 = M1+M5+M6+M7.
void make_winograd(Realization &d) {
  static const double U[7][4] = {{1, 0, 0, 0}, {0, 1, 0, 0}, {1, 1, -1, -1}, {0, 0, 0, 1},
                                 {0, 0, 1, 1}, {-1, 0, 1, 1}, {1, 0, -1, 0}};
  static const double V[7][4] = {{1, 0, 0, 0}, {0, 0, 1, 0}, {0, 0, 0, 1}, {1, -1, -1, 1},
                                 {-1, 1, 0, 0}, {1, -1, 0, 1}, {0, -1, 0, 1}};
  static const double W[7][4] = {{1, 1, 1, 1}, {1, 0, 0, 0}, {0, 0, 1, 0}, {0, -1, 0, 0},
                                 {0, 0, 1, 1}, {0, 1, 1, 1}, {0, 1, 0, 1}};
  set_rows(d, 7, U, V, W);
}

// T* (eq. A.2): the rows of U*, with V*_r = U*_{pi_V(r)} and w*_r = U*_{pi_W(r)},
// pi_V = (1,3,7,6,4,5,2), pi_W = (1,7,2,5,6,4,3) (1-based).
void make_tstar(Realization &d) {
  const double Us[7][4] = {{1, 0, 0, 1},
                           {0, 0, kXi, 1},
                           {1, 0, kXi, 0},
                           {0, 0, -kXi, 1},
                           {0.5, kEta, kZeta, 0.5},
                           {-1, 0, kXi, 0},
                           {-0.5, kEta, kZeta, -0.5}};
  static const int piV[7] = {1, 3, 7, 6, 4, 5, 2};
  static const int piW[7] = {1, 7, 2, 5, 6, 4, 3};
  d.R = 7;
  for (int r = 0; r < 7; ++r)
    for (int c = 0; c < 4; ++c) {
      d.U[r][c] = Us[r][c];
      d.V[r][c] = Us[piV[r] - 1][c];
      d.W[r][c] = Us[piW[r] - 1][c];
    }
}

// 2x2 inverse by the adjugate: det = a d - b c, entries divided by det.
void inverse2(const double g[4], double inv[4]) {
  const double det = g[0] * g[3] - g[1] * g[2];
  inv[0] = g[3] / det;
  inv[1] = (-g[1]) / det;
  inv[2] = (-g[2]) / det;
  inv[3] = g[0] / det;
}

// K = X (x) M with M = (Y^-1)^T: K[2i+j][2i'+j'] = X[i][i'] * M[j][j'].
void kron_inverse_transpose(const double X[4], const double Y[4], double K[4][4]) {
  double Yi[4];
  inverse2(Y, Yi);
  const double M[4] = {Yi[0], Yi[2], Yi[1], Yi[3]};  // transpose
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j)
      for (int ip = 0; ip < 2; ++ip)
        for (int jp = 0; jp < 2; ++jp)
          K[2 * i + j][2 * ip + jp] = X[2 * i + ip] * M[2 * j + jp];
}

// row <- row K, each output summed over the input index in ascending order.
void row_times(double row[4], const double K[4][4]) {
  double out[4];
  for (int c = 0; c < 4; ++c) {
    double s = row[0] * K[0][c];
    for (int a = 1; a < 4; ++a) s = s + row[a] * K[a][c];
    out[c] = s;
  }
  for (int c = 0; c < 4; ++c) row[c] = out[c];
}

double sq_norm(const double v[4]) {
  double s = 0.0;
  for (int c = 0; c < 4; ++c) s = s + v[c] * v[c];
  return s;
}

}  // namespace

int realization_builtin(int which, Realization &d) {
  std::memset(&d, 0, sizeof(d));
  switch (which) {
    case FMM_CUBIC8: make_cubic(d); return FMM_OK;
    case FMM_STRASSEN: make_strassen(d); return FMM_OK;
    case FMM_WINOGRAD: make_winograd(d); return FMM_OK;
    case FMM_TSTAR: make_tstar(d); return FMM_OK;
    default: return FMM_ERR_ARG;
  }
}

double brent_residual(const Realization &d) {
  // <2,2,2> in the cyclic convention: entry [(2i+j)][(2j'+k)][(2k'+i')] is
  // 1 iff j = j', k = k', i = i'.
  double worst = 0.0;
  for (int a = 0; a < 4; ++a)
    for (int b = 0; b < 4; ++b)
      for (int c = 0; c < 4; ++c) {
        double s = 0.0;
        for (int r = 0; r < d.R; ++r) s = s + d.U[r][a] * d.V[r][b] * d.W[r][c];
        const int i = a >> 1, j = a & 1, jp = b >> 1, k = b & 1, kp = c >> 1, ip = c & 1;
        const double want = (j == jp && k == kp && i == ip) ? 1.0 : 0.0;
        const double e = std::fabs(s - want);
        if (!(e <= worst)) worst = e;  // propagates NaN
      }
  return worst;
}

int realization_transform(const Realization &d, const double X[4], const double Y[4],
                          const double Z[4], Realization &out) {
  for (const double *g : {X, Y, Z}) {
    const double det = g[0] * g[3] - g[1] * g[2];
    if (!(std::fabs(det) >= 1e-12)) return FMM_ERR_SINGULAR;
  }
  double KU[4][4], KV[4][4], KW[4][4];
  kron_inverse_transpose(X, Y, KU);
  kron_inverse_transpose(Y, Z, KV);
  kron_inverse_transpose(Z, X, KW);
  out = d;
  for (int r = 0; r < d.R; ++r) {
    row_times(out.U[r], KU);
    row_times(out.V[r], KV);
    row_times(out.W[r], KW);
  }
  return FMM_OK;
}

void realization_rebalance(const Realization &d, Realization &out) {
  out = d;
  for (int r = 0; r < d.R; ++r) {
    const double nu = std::sqrt(sq_norm(d.U[r]));
    const double nv = std::sqrt(sq_norm(d.V[r]));
    if (nu == 0.0 || nv == 0.0) continue;
    const double s = std::sqrt(nu / nv);
    for (int c = 0; c < 4; ++c) {
      out.U[r][c] = d.U[r][c] / s;
      out.V[r][c] = d.V[r][c] * s;
    }
  }
}

void realization_phi_gamma(const Realization &d, double &phi, double &gamma) {
  phi = 0.0;
  gamma = 0.0;
  for (int r = 0; r < d.R; ++r) {
    const double t = sq_norm(d.U[r]) * sq_norm(d.V[r]) * sq_norm(d.W[r]);
    phi = phi + t;
    gamma = gamma + std::sqrt(t);
  }
}

int64_t ipow(int64_t b, int e) {
  int64_t r = 1;
  for (int i = 0; i < e; ++i) r *= b;
  return r;
}

// Depth-l flattening: term r = sum_t r_t R^(l-t) (level 1 most significant);
// column P 2^l + Q of the 2^l x 2^l block grid with P = sum_t p_t 2^(l-t);
// the entry is prod_t base[r_t][2 p_t + q_t], multiplied left to right in
// binary64 and rounded once to binary32.
void flatten(const double (*base)[4], int R, int depth, float *out) {
  const int n = 1 << depth;
  const int64_t T = ipow(R, depth);
  for (int64_t r = 0; r < T; ++r) {
    int digit[8];
    int64_t rr = r;
    for (int t = depth - 1; t >= 0; --t) {
      digit[t] = static_cast<int>(rr % R);
      rr /= R;
    }
    for (int P = 0; P < n; ++P)
      for (int Q = 0; Q < n; ++Q) {
        double c = 0.0;
        for (int t = 0; t < depth; ++t) {
          const int p = (P >> (depth - 1 - t)) & 1;
          const int q = (Q >> (depth - 1 - t)) & 1;
          const double f = base[digit[t]][2 * p + q];
          c = (t == 0) ? f : c * f;
        }
        out[r * n * n + P * n + Q] = static_cast<float>(c);
      }
  }
}

// ---- other shapes <m,k,n;R> ------------------------------------------------
// U_r indexed i k + j (A block (i, j)), V_r j n + l (B block (j, l)), W_r
// l m + i (C block (i, l), the cyclic third factor of the <2,2,2> case).

double brent_residual_shape(const Shaped &s) {
  const int a_n = s.m * s.k, b_n = s.k * s.n, c_n = s.n * s.m;
  double worst = 0.0;
  for (int a = 0; a < a_n; ++a)
    for (int b = 0; b < b_n; ++b)
      for (int c = 0; c < c_n; ++c) {
        double acc = 0.0;
        for (int r = 0; r < s.R; ++r)
          acc = acc + s.U[(size_t)r * a_n + a] * s.V[(size_t)r * b_n + b] * s.W[(size_t)r * c_n + c];
        const int i = a / s.k, j = a % s.k, jp = b / s.n, l = b % s.n, lp = c / s.m, ip = c % s.m;
        const double want = (j == jp && l == lp && i == ip) ? 1.0 : 0.0;
        const double e = std::fabs(acc - want);
        if (!(e <= worst)) worst = e;  // propagates NaN
      }
  return worst;
}

namespace {
double sq_norm_n(const double *v, int len) {
  double s = 0.0;
  for (int c = 0; c < len; ++c) s = s + v[c] * v[c];
  return s;
}
}  // namespace

double inverse_gj(const double *G, int n, double *inv) {
  std::vector<double> A(G, G + (size_t)n * n);
  for (int i = 0; i < n * n; ++i) inv[i] = 0.0;
  for (int i = 0; i < n; ++i) inv[i * n + i] = 1.0;
  double det = 1.0;
  for (int c = 0; c < n; ++c) {
    int piv = c;
    for (int r = c + 1; r < n; ++r)
      if (std::fabs(A[r * n + c]) > std::fabs(A[piv * n + c])) piv = r;
    const double pv = A[piv * n + c];
    if (pv == 0.0 || !std::isfinite(pv)) return 0.0;
    if (piv != c) {
      for (int j = 0; j < n; ++j) {
        std::swap(A[piv * n + j], A[c * n + j]);
        std::swap(inv[piv * n + j], inv[c * n + j]);
      }
      det = -det;
    }
    det = det * pv;
    for (int j = 0; j < n; ++j) {
      A[c * n + j] = A[c * n + j] / pv;
      inv[c * n + j] = inv[c * n + j] / pv;
    }
    for (int r = 0; r < n; ++r) {
      if (r == c) continue;
      const double f = A[r * n + c];
      if (f == 0.0) continue;
      for (int j = 0; j < n; ++j) {
        A[r * n + j] = A[r * n + j] - f * A[c * n + j];
        inv[r * n + j] = inv[r * n + j] - f * inv[c * n + j];
      }
    }
  }
  return det;
}

namespace {
// rows of M (R x p q) times K = P (x) Qinv^T (K[a q + b][a' q + b'] = P[a][a'] Qinv[b'][b]),
// each output entry summed over the input index in ascending order
void rows_times_kron(const double *M, int R, const double *P, int p, const double *Qinv, int q,
                     std::vector<double> &out) {
  const int w = p * q;
  std::vector<double> K((size_t)w * w);
  for (int a = 0; a < p; ++a)
    for (int b = 0; b < q; ++b)
      for (int a2 = 0; a2 < p; ++a2)
        for (int b2 = 0; b2 < q; ++b2) K[(size_t)(a * q + b) * w + a2 * q + b2] = P[a * p + a2] * Qinv[b2 * q + b];
  out.assign((size_t)R * w, 0.0);
  for (int r = 0; r < R; ++r)
    for (int c = 0; c < w; ++c) {
      double s = M[(size_t)r * w] * K[c];
      for (int a = 1; a < w; ++a) s = s + M[(size_t)r * w + a] * K[(size_t)a * w + c];
      out[(size_t)r * w + c] = s;
    }
}
}  // namespace

int transform_shape(const Shaped &s, const double *X, const double *Y, const double *Z, std::vector<double> &U,
                    std::vector<double> &V, std::vector<double> &W) {
  std::vector<double> Xi((size_t)s.m * s.m), Yi((size_t)s.k * s.k), Zi((size_t)s.n * s.n);
  const double dets[3] = {inverse_gj(X, s.m, Xi.data()), inverse_gj(Y, s.k, Yi.data()), inverse_gj(Z, s.n, Zi.data())};
  for (double d : dets)
    if (!(std::fabs(d) >= 1e-12)) return FMM_ERR_SINGULAR;
  rows_times_kron(s.U, s.R, X, s.m, Yi.data(), s.k, U);     // u (X (x) Y^-T)
  rows_times_kron(s.V, s.R, Y, s.k, Zi.data(), s.n, V);     // v (Y (x) Z^-T)
  rows_times_kron(s.W, s.R, Z, s.n, Xi.data(), s.m, W);     // w (Z (x) X^-T)
  return FMM_OK;
}

void phi_gamma_shape(const Shaped &s, double &phi, double &gamma) {
  phi = 0.0;
  gamma = 0.0;
  const int a_n = s.m * s.k, b_n = s.k * s.n, c_n = s.n * s.m;
  for (int r = 0; r < s.R; ++r) {
    const double t = sq_norm_n(s.U + (size_t)r * a_n, a_n) * sq_norm_n(s.V + (size_t)r * b_n, b_n) *
                     sq_norm_n(s.W + (size_t)r * c_n, c_n);
    phi = phi + t;
    gamma = gamma + std::sqrt(t);
  }
}

}  // namespace fmm

// ---------------------------------------------------------------------------
// C-ABI
// ---------------------------------------------------------------------------
using fmm::Realization;

struct fmm_real {
  int m = 2, k = 2, n = 2;
  Realization d;                   // <2,2,2>: the coefficients; other shapes: d.R only
  std::vector<double> U, V, W;     // other shapes: R x mk, R x kn, R x nm
  bool is222() const { return m == 2 && k == 2 && n == 2; }
  fmm::Shaped shaped() const { return {m, k, n, d.R, U.data(), V.data(), W.data()}; }
};

extern "C" {

int fmm_realization_builtin(int which, fmm_real **out) {
  if (!out) return FMM_ERR_ARG;
  *out = nullptr;
  fmm_real *h = new (std::nothrow) fmm_real;
  if (!h) return FMM_ERR_NOMEM;
  const int st = fmm::realization_builtin(which, h->d);
  if (st != FMM_OK) {
    delete h;
    return st;
  }
  *out = h;
  return FMM_OK;
}

int fmm_realization_create(int m, int k, int n, int R, const double *U, const double *V, const double *w,
                           double tol, fmm_real **out) {
  if (!out) return FMM_ERR_ARG;
  *out = nullptr;
  if (m < 1 || k < 1 || n < 1) return FMM_ERR_ARG;
  if (int64_t(m) * k > fmm::kMaxGridBlocks || int64_t(k) * n > fmm::kMaxGridBlocks || int64_t(n) * m > fmm::kMaxGridBlocks)
    return FMM_ERR_UNSUPPORTED;
  const bool is222 = m == 2 && k == 2 && n == 2;
  if (!U || !V || !w || R < 1 || R > (is222 ? fmm::kMaxRank : fmm::kMaxRankShape) || !(tol >= 0.0))
    return FMM_ERR_ARG;
  fmm_real *h = new (std::nothrow) fmm_real;
  if (!h) return FMM_ERR_NOMEM;
  std::memset(&h->d, 0, sizeof(h->d));
  if (!is222) {
    h->m = m; h->k = k; h->n = n;
    h->d.R = R;
    try {
      h->U.assign(U, U + (size_t)R * m * k);
      h->V.assign(V, V + (size_t)R * k * n);
      h->W.assign(w, w + (size_t)R * n * m);
    } catch (...) {
      delete h;
      return FMM_ERR_NOMEM;
    }
    const double res = fmm::brent_residual_shape(h->shaped());
    if (!(res <= tol)) {
      delete h;
      return FMM_ERR_NOT_EXACT;
    }
    *out = h;
    return FMM_OK;
  }
  h->d.R = R;
  for (int r = 0; r < R; ++r)
    for (int c = 0; c < 4; ++c) {
      h->d.U[r][c] = U[4 * r + c];
      h->d.V[r][c] = V[4 * r + c];
      h->d.W[r][c] = w[4 * r + c];
    }
  const double res = fmm::brent_residual(h->d);
  if (!(res <= tol)) {
    delete h;
    return FMM_ERR_NOT_EXACT;
  }
  *out = h;
  return FMM_OK;
}

int fmm_realization_transform(const fmm_real *d, const double X[4], const double Y[4],
                              const double Z[4], fmm_real **out) {
  if (!out) return FMM_ERR_ARG;
  *out = nullptr;
  if (!d || !X || !Y || !Z) return FMM_ERR_ARG;
  if (!d->is222()) {
    fmm_real *h = new (std::nothrow) fmm_real;
    if (!h) return FMM_ERR_NOMEM;
    int st;
    try {
      h->m = d->m; h->k = d->k; h->n = d->n;
      std::memset(&h->d, 0, sizeof(h->d));
      h->d.R = d->d.R;
      st = fmm::transform_shape(d->shaped(), X, Y, Z, h->U, h->V, h->W);
    } catch (...) {
      st = FMM_ERR_NOMEM;
    }
    if (st != FMM_OK) {
      delete h;
      return st;
    }
    *out = h;
    return FMM_OK;
  }
  fmm_real *h = new (std::nothrow) fmm_real;
  if (!h) return FMM_ERR_NOMEM;
  const int st = fmm::realization_transform(d->d, X, Y, Z, h->d);
  if (st != FMM_OK) {
    delete h;
    return st;
  }
  *out = h;
  return FMM_OK;
}

int fmm_realization_rebalance(const fmm_real *d, fmm_real **out) {
  if (!out) return FMM_ERR_ARG;
  *out = nullptr;
  if (!d) return FMM_ERR_ARG;
  fmm_real *h = new (std::nothrow) fmm_real;
  if (!h) return FMM_ERR_NOMEM;
  if (d->is222()) {
    fmm::realization_rebalance(d->d, h->d);
    *out = h;
    return FMM_OK;
  }
  // other shapes: the same gauge on rows of length mk and kn
  try {
    *h = *d;
  } catch (...) {
    delete h;
    return FMM_ERR_NOMEM;
  }
  const int a_n = d->m * d->k, b_n = d->k * d->n;
  for (int r = 0; r < d->d.R; ++r) {
    const double *u = d->U.data() + (size_t)r * a_n, *v = d->V.data() + (size_t)r * b_n;
    double nu = 0.0, nv = 0.0;
    for (int c = 0; c < a_n; ++c) nu = nu + u[c] * u[c];
    for (int c = 0; c < b_n; ++c) nv = nv + v[c] * v[c];
    nu = std::sqrt(nu);
    nv = std::sqrt(nv);
    if (nu == 0.0 || nv == 0.0) continue;
    const double s = std::sqrt(nu / nv);
    for (int c = 0; c < a_n; ++c) h->U[(size_t)r * a_n + c] = u[c] / s;
    for (int c = 0; c < b_n; ++c) h->V[(size_t)r * b_n + c] = v[c] * s;
  }
  *out = h;
  return FMM_OK;
}

int fmm_realization_metrics(const fmm_real *d, int depth, double *phi, double *gamma,
                            double *brent_resid) {
  if (!d || depth < 1 || depth > fmm::kMaxDepth) return FMM_ERR_ARG;
  if (!d->is222() && depth != 1) return FMM_ERR_UNSUPPORTED;
  double p, g;
  if (d->is222())
    fmm::realization_phi_gamma(d->d, p, g);
  else
    fmm::phi_gamma_shape(d->shaped(), p, g);
  if (phi) *phi = std::pow(p, depth);
  if (gamma) *gamma = std::pow(g, depth);
  if (brent_resid) *brent_resid = d->is222() ? fmm::brent_residual(d->d) : fmm::brent_residual_shape(d->shaped());
  return FMM_OK;
}

int fmm_realization_terms(const fmm_real *d, int depth, int64_t *rank, int64_t *terms) {
  if (!d || depth < 1 || depth > fmm::kMaxDepth) return FMM_ERR_ARG;
  if (!d->is222() && depth != 1) return FMM_ERR_UNSUPPORTED;
  if (rank) *rank = d->d.R;
  if (terms) *terms = fmm::ipow(d->d.R, depth);
  return FMM_OK;
}

int fmm_realization_shape(const fmm_real *d, int *m, int *k, int *n, int *R) {
  if (!d) return FMM_ERR_ARG;
  if (m) *m = d->m;
  if (k) *k = d->k;
  if (n) *n = d->n;
  if (R) *R = d->d.R;
  return FMM_OK;
}

int fmm_realization_coefficients(const fmm_real *d, double *U, double *V, double *w) {
  if (!d) return FMM_ERR_ARG;
  if (!d->is222()) {
    if (U) std::memcpy(U, d->U.data(), d->U.size() * sizeof(double));
    if (V) std::memcpy(V, d->V.data(), d->V.size() * sizeof(double));
    if (w) std::memcpy(w, d->W.data(), d->W.size() * sizeof(double));
    return FMM_OK;
  }
  for (int r = 0; r < d->d.R; ++r)
    for (int c = 0; c < 4; ++c) {
      if (U) U[4 * r + c] = d->d.U[r][c];
      if (V) V[4 * r + c] = d->d.V[r][c];
      if (w) w[4 * r + c] = d->d.W[r][c];
    }
  return FMM_OK;
}

int fmm_realization_tables(const fmm_real *d, int depth, float *U, float *V, float *w) {
  if (!d || depth < 1 || depth > fmm::kMaxDepth) return FMM_ERR_ARG;
  if (!d->is222()) {
    if (depth != 1) return FMM_ERR_UNSUPPORTED;
    for (size_t i = 0; i < d->U.size(); ++i)
      if (U) U[i] = static_cast<float>(d->U[i]);
    for (size_t i = 0; i < d->V.size(); ++i)
      if (V) V[i] = static_cast<float>(d->V[i]);
    for (size_t i = 0; i < d->W.size(); ++i)
      if (w) w[i] = static_cast<float>(d->W[i]);
    return FMM_OK;
  }
  if (U) fmm::flatten(d->d.U, d->d.R, depth, U);
  if (V) fmm::flatten(d->d.V, d->d.R, depth, V);
  if (w) fmm::flatten(d->d.W, d->d.R, depth, w);
  return FMM_OK;
}

void fmm_realization_destroy(fmm_real *d) { delete d; }

}  // extern "C"
