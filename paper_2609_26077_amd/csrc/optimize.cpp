// Re-basing: minimization of Phi over a realization's change-of-basis orbit
// (Section 3.1; the re-basing protocol of Appendix E.2).
//
// The orbit is D . g for g = (X, Y, Z) in GL(2)^3 under the right action of
// eq. A.1; Phi(D . g) = sum_r |u_r K_U|^2 |v_r K_V|^2 |w_r K_W|^2 with
// K_U = X (x) Y^-T, K_V = Y (x) Z^-T, K_W = Z (x) X^-T.  Each start is driven
// by limited-memory BFGS over the 12 entries of (X, Y, Z) with a line search
// that enforces the strong Wolfe conditions; the gradient is exact, carried
// by forward-mode dual numbers through the same expression.  Realizations of
// other shapes <m,k,n> take the same protocol over GL(m) x GL(k) x GL(n)
// (m^2 + k^2 + n^2 entries) with the gradient in closed form.
#include "internal.h"

#include <cmath>
#include <cstring>
#include <limits>
#include <new>
#include <algorithm>
#include <vector>

namespace fmm {

namespace {

constexpr int kN = 12;   // entries of (X, Y, Z)

// A value with its 12 partial derivatives.
struct Dual {
  double v;
  double d[kN];
};

Dual constant(double c) {
  Dual r;
  r.v = c;
  for (int i = 0; i < kN; ++i) r.d[i] = 0.0;
  return r;
}
Dual add(const Dual &a, const Dual &b) {
  Dual r;
  r.v = a.v + b.v;
  for (int i = 0; i < kN; ++i) r.d[i] = a.d[i] + b.d[i];
  return r;
}
Dual sub(const Dual &a, const Dual &b) {
  Dual r;
  r.v = a.v - b.v;
  for (int i = 0; i < kN; ++i) r.d[i] = a.d[i] - b.d[i];
  return r;
}
Dual mul(const Dual &a, const Dual &b) {
  Dual r;
  r.v = a.v * b.v;
  for (int i = 0; i < kN; ++i) r.d[i] = a.d[i] * b.v + a.v * b.d[i];
  return r;
}
Dual scale(const Dual &a, double c) {
  Dual r;
  r.v = a.v * c;
  for (int i = 0; i < kN; ++i) r.d[i] = a.d[i] * c;
  return r;
}
Dual divide(const Dual &a, const Dual &b) {
  Dual r;
  r.v = a.v / b.v;
  for (int i = 0; i < kN; ++i) r.d[i] = (a.d[i] * b.v - a.v * b.d[i]) / (b.v * b.v);
  return r;
}

// K = P (x) Q^-T for 2x2 P, Q (row-major): K[2i+j][2i'+j'] = P[i][i'] (Q^-T)[j][j'].
void kron_inv_t(const Dual P[4], const Dual Q[4], Dual K[4][4]) {
  const Dual det = sub(mul(Q[0], Q[3]), mul(Q[1], Q[2]));
  // Q^-1 = adj(Q) / det; its transpose
  Dual M[4];
  M[0] = divide(Q[3], det);
  M[1] = divide(scale(Q[2], -1.0), det);
  M[2] = divide(scale(Q[1], -1.0), det);
  M[3] = divide(Q[0], det);
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j)
      for (int ip = 0; ip < 2; ++ip)
        for (int jp = 0; jp < 2; ++jp) K[2 * i + j][2 * ip + jp] = mul(P[2 * i + ip], M[2 * j + jp]);
}

// |row K|^2
Dual sq_image(const double row[4], const Dual K[4][4]) {
  Dual s = constant(0.0);
  for (int c = 0; c < 4; ++c) {
    Dual e = constant(0.0);
    for (int a = 0; a < 4; ++a)
      if (row[a] != 0.0) e = add(e, scale(K[a][c], row[a]));
    s = add(s, mul(e, e));
  }
  return s;
}

// Phi(D . g) and its gradient with respect to the 12 entries of g.
double phi_grad(const Realization &D, const double g[kN], double grad[kN]) {
  Dual x[kN];
  for (int i = 0; i < kN; ++i) {
    x[i] = constant(g[i]);
    x[i].d[i] = 1.0;
  }
  const Dual *X = x, *Y = x + 4, *Z = x + 8;
  Dual KU[4][4], KV[4][4], KW[4][4];
  kron_inv_t(X, Y, KU);
  kron_inv_t(Y, Z, KV);
  kron_inv_t(Z, X, KW);
  Dual phi = constant(0.0);
  for (int r = 0; r < D.R; ++r)
    phi = add(phi, mul(mul(sq_image(D.U[r], KU), sq_image(D.V[r], KV)), sq_image(D.W[r], KW)));
  for (int i = 0; i < kN; ++i) grad[i] = phi.d[i];
  return phi.v;
}

// ---- the objective over a general orbit GL(m) x GL(k) x GL(n) ----------------
//
// For another shape <m,k,n> (U_r an m x k matrix, V_r k x n, W_r n x m; the
// flattened indices i k + j, j n + l, l m + i) the action is
//   U_r -> X^T U_r Y^-T,   V_r -> Y^T V_r Z^-T,   W_r -> Z^T W_r X^-T,
// the matrix form of u -> u (X (x) Y^-T) and its cyclic companions (eq. A.1
// at <2,2,2>).  It keeps a realization exact: <U', A> = <U, X A Y^-1>, so the
// trilinear form becomes tr(X A B C X^-1) = tr(A B C).  With a_r = |U'_r|^2,
// b_r = |V'_r|^2, c_r = |W'_r|^2 and Phi = sum_r a_r b_r c_r, differentiating
// |X^T U Y^-T|^2 etc. (d(Y^-T) = -Y^-T dY^T Y^-T) gives
//   dPhi/dX = 2 X^-T sum_r (b_r c_r U'_r U'_r^T - a_r b_r W'_r^T W'_r),
//   dPhi/dY = 2 Y^-T sum_r (a_r c_r V'_r V'_r^T - b_r c_r U'_r^T U'_r),
//   dPhi/dZ = 2 Z^-T sum_r (a_r b_r W'_r W'_r^T - a_r c_r V'_r^T V'_r).

// C (p x q) = op(A) B with op(A) = A^T (A is r x p) or A (p x r); B r x q.
void matmul_t(const double *A, bool transA, const double *B, int p, int r, int q, double *C) {
  for (int i = 0; i < p; ++i)
    for (int j = 0; j < q; ++j) {
      double s = 0.0;
      for (int t = 0; t < r; ++t) s = s + (transA ? A[t * p + i] : A[i * r + t]) * B[t * q + j];
      C[i * q + j] = s;
    }
}

// C (p x q) = A B^T with A p x r, B q x r.
void matmul_bt(const double *A, const double *B, int p, int r, int q, double *C) {
  for (int i = 0; i < p; ++i)
    for (int j = 0; j < q; ++j) {
      double s = 0.0;
      for (int t = 0; t < r; ++t) s = s + A[i * r + t] * B[j * r + t];
      C[i * q + j] = s;
    }
}

// M' = P^T M Qinv^T for M (p x q), P (p x p), Qinv (q x q); returns |M'|^2.
double image(const double *M, const double *P, const double *Qinv, int p, int q, double *T, double *out) {
  matmul_t(P, true, M, p, p, q, T);          // P^T M
  matmul_bt(T, Qinv, p, q, q, out);          // (P^T M) Qinv^T
  double s = 0.0;
  for (int i = 0; i < p * q; ++i) s = s + out[i] * out[i];
  return s;
}

double phi_grad_shape(const Shaped &S, const double *x, double *grad) {
  const int m = S.m, k = S.k, n = S.n;
  const int nx = m * m, ny = k * k, nz = n * n;
  const double *X = x, *Y = x + nx, *Z = x + nx + ny;
  std::vector<double> Xi(nx), Yi(ny), Zi(nz);
  const double dx = inverse_gj(X, m, Xi.data()), dy = inverse_gj(Y, k, Yi.data()), dz = inverse_gj(Z, n, Zi.data());
  if (dx == 0.0 || dy == 0.0 || dz == 0.0) {
    const double nan = std::numeric_limits<double>::quiet_NaN();
    for (int i = 0; i < nx + ny + nz; ++i) grad[i] = nan;
    return nan;
  }
  std::vector<double> AX(nx, 0.0), AY(ny, 0.0), AZ(nz, 0.0);
  std::vector<double> Up(m * k), Vp(k * n), Wp(n * m), T(64 * 64), G(64 * 64);
  double phi = 0.0;
  for (int r = 0; r < S.R; ++r) {
    const double a = image(S.U + (size_t)r * m * k, X, Yi.data(), m, k, T.data(), Up.data());
    const double b = image(S.V + (size_t)r * k * n, Y, Zi.data(), k, n, T.data(), Vp.data());
    const double c = image(S.W + (size_t)r * n * m, Z, Xi.data(), n, m, T.data(), Wp.data());
    phi = phi + a * b * c;
    // AX += b c U' U'^T - a b W'^T W'
    matmul_bt(Up.data(), Up.data(), m, k, m, G.data());
    for (int i = 0; i < nx; ++i) AX[i] = AX[i] + b * c * G[i];
    matmul_t(Wp.data(), true, Wp.data(), m, n, m, G.data());
    for (int i = 0; i < nx; ++i) AX[i] = AX[i] - a * b * G[i];
    // AY += a c V' V'^T - b c U'^T U'
    matmul_bt(Vp.data(), Vp.data(), k, n, k, G.data());
    for (int i = 0; i < ny; ++i) AY[i] = AY[i] + a * c * G[i];
    matmul_t(Up.data(), true, Up.data(), k, m, k, G.data());
    for (int i = 0; i < ny; ++i) AY[i] = AY[i] - b * c * G[i];
    // AZ += a b W' W'^T - a c V'^T V'
    matmul_bt(Wp.data(), Wp.data(), n, m, n, G.data());
    for (int i = 0; i < nz; ++i) AZ[i] = AZ[i] + a * b * G[i];
    matmul_t(Vp.data(), true, Vp.data(), n, k, n, G.data());
    for (int i = 0; i < nz; ++i) AZ[i] = AZ[i] - a * c * G[i];
  }
  // grad = 2 P^-T A for each factor P
  matmul_t(Xi.data(), true, AX.data(), m, m, m, grad);
  matmul_t(Yi.data(), true, AY.data(), k, k, k, grad + nx);
  matmul_t(Zi.data(), true, AZ.data(), n, n, n, grad + nx + ny);
  for (int i = 0; i < nx + ny + nz; ++i) grad[i] = 2.0 * grad[i];
  return phi;
}

// ---- limited-memory BFGS with a strong-Wolfe line search -------------------

// An objective over n parameters: its value and gradient at x.
struct Objective {
  int n;
  const Realization *D;    // <2,2,2> (12 parameters) ...
  const Shaped *S;         // ... or another shape (m^2 + k^2 + n^2)
  double operator()(const double *x, double *g) const { return D ? phi_grad(*D, x, g) : phi_grad_shape(*S, x, g); }
};

double dot(const double *a, const double *b, int n) {
  double s = 0.0;
  for (int i = 0; i < n; ++i) s += a[i] * b[i];
  return s;
}
double max_abs(const double *a, int n) {
  double m = 0.0;
  for (int i = 0; i < n; ++i) m = std::fmax(m, std::fabs(a[i]));
  return m;
}

// A trial point of the line search x + t p.
struct Trial {
  double t = 0.0, f = 0.0, dphi = 0.0;     // step, value, directional derivative
  std::vector<double> x, g;
};

bool evaluate(const Objective &F, const double *x0, const double *p, double t, Trial &tr) {
  const int n = F.n;
  tr.t = t;
  tr.x.resize(n);
  tr.g.resize(n);
  for (int i = 0; i < n; ++i) tr.x[i] = x0[i] + t * p[i];
  tr.f = F(tr.x.data(), tr.g.data());
  tr.dphi = dot(tr.g.data(), p, n);
  return std::isfinite(tr.f) && std::isfinite(tr.dphi);
}

// Minimizer of the cubic interpolating (a, fa, da) and (b, fb, db), kept
// inside the middle 80% of [a, b]; bisection where the cubic has no minimum.
double interpolate(const Trial &a, const Trial &b) {
  const double lo = std::fmin(a.t, b.t), hi = std::fmax(a.t, b.t);
  const double d1 = a.dphi + b.dphi - 3.0 * (a.f - b.f) / (a.t - b.t);
  const double rad = d1 * d1 - a.dphi * b.dphi;
  double t = 0.5 * (a.t + b.t);
  if (rad >= 0.0) {
    const double d2 = std::copysign(std::sqrt(rad), b.t - a.t);
    const double den = b.dphi - a.dphi + 2.0 * d2;
    if (den != 0.0) {
      const double c = b.t - (b.t - a.t) * (b.dphi + d2 - d1) / den;
      if (std::isfinite(c)) t = c;
    }
  }
  const double w = hi - lo;
  return std::fmin(std::fmax(t, lo + 0.1 * w), hi - 0.1 * w);
}

// Line search for the strong Wolfe conditions along p from (x0, f0, g0):
//   f(t) <= f0 + c1 t f'(0)   and   |f'(t)| <= c2 |f'(0)|
// by bracketing (the step doubles while the conditions fail without a
// bracket) and then zooming with safeguarded cubic interpolation.  Trial
// points that are singular or non-finite count as too long.  Returns false
// if no acceptable step was found.
bool strong_wolfe(const Objective &F, const double *x0, double f0, const double *g0, const double *p,
                  Trial &out) {
  constexpr double c1 = 1e-4, c2 = 0.9;
  const int n = F.n;
  const double d0 = dot(g0, p, n);
  if (!(d0 < 0.0)) return false;
  Trial prev;
  prev.t = 0.0; prev.f = f0; prev.dphi = d0;
  prev.x.assign(x0, x0 + n);
  prev.g.assign(g0, g0 + n);
  Trial lo, hi, cur;
  bool bracket = false;
  double t = 1.0;
  for (int it = 0; it < 60; ++it) {
    const bool ok = evaluate(F, x0, p, t, cur);
    if (!ok || cur.f > f0 + c1 * t * d0 || (it > 0 && cur.f >= prev.f)) {
      if (!ok) {            // too far: shrink towards the last good point
        t = prev.t + 0.5 * (t - prev.t);
        if (t - prev.t < 1e-16) return false;
        continue;
      }
      lo = prev; hi = cur; bracket = true;
      break;
    }
    if (std::fabs(cur.dphi) <= -c2 * d0) {
      out = cur;
      return true;
    }
    if (cur.dphi >= 0.0) {
      lo = cur; hi = prev; bracket = true;
      break;
    }
    prev = cur;
    t *= 2.0;
  }
  if (!bracket) return false;
  for (int it = 0; it < 80; ++it) {
    const double tj = interpolate(lo, hi);
    Trial tr;
    const bool ok = evaluate(F, x0, p, tj, tr);
    if (!ok || tr.f > f0 + c1 * tj * d0 || tr.f >= lo.f) {
      hi = tr;
      if (!ok) { hi.f = std::numeric_limits<double>::infinity(); hi.dphi = 0.0; }
    } else {
      if (std::fabs(tr.dphi) <= -c2 * d0) {
        out = tr;
        return true;
      }
      if (tr.dphi * (hi.t - lo.t) >= 0.0) hi = lo;
      lo = tr;
    }
    if (std::fabs(hi.t - lo.t) <= 1e-16 * std::fmax(1.0, std::fabs(lo.t))) break;
  }
  // no point met both conditions: accept the best sufficient-decrease point
  if (lo.t > 0.0 && lo.f < f0) {
    out = lo;
    return true;
  }
  return false;
}

// L-BFGS from x (F.n entries); returns the terminal value, x updated.
double lbfgs(const Objective &F, double *x, int max_iter, double gtol) {
  constexpr int kMem = 10;
  const int n = F.n;
  std::vector<double> S((size_t)kMem * n), Yv((size_t)kMem * n), g(n), q(n), p(n), s(n), y(n);
  double rho[kMem], alpha[kMem];
  int count = 0, head = 0;
  double f = F(x, g.data());
  if (!std::isfinite(f)) return f;
  for (int it = 0; it < max_iter; ++it) {
    if (max_abs(g.data(), n) <= gtol * std::fmax(1.0, f)) break;
    // two-loop recursion: p = -H g
    for (int i = 0; i < n; ++i) q[i] = g[i];
    for (int k = 0; k < count; ++k) {
      const int j = (head - 1 - k + kMem) % kMem;
      alpha[j] = rho[j] * dot(&S[(size_t)j * n], q.data(), n);
      for (int i = 0; i < n; ++i) q[i] -= alpha[j] * Yv[(size_t)j * n + i];
    }
    double gamma = 1.0;
    if (count > 0) {
      const int j = (head - 1 + kMem) % kMem;
      gamma = dot(&S[(size_t)j * n], &Yv[(size_t)j * n], n) / dot(&Yv[(size_t)j * n], &Yv[(size_t)j * n], n);
    } else {
      gamma = 1.0 / std::fmax(max_abs(g.data(), n), 1e-300);   // first step of length ~1 in the largest entry
    }
    for (int i = 0; i < n; ++i) q[i] *= gamma;
    for (int k = count - 1; k >= 0; --k) {
      const int j = (head - 1 - k + kMem) % kMem;
      const double beta = rho[j] * dot(&Yv[(size_t)j * n], q.data(), n);
      for (int i = 0; i < n; ++i) q[i] += S[(size_t)j * n + i] * (alpha[j] - beta);
    }
    for (int i = 0; i < n; ++i) p[i] = -q[i];
    if (!(dot(p.data(), g.data(), n) < 0.0)) {   // not a descent direction: restart from steepest descent
      count = 0;
      for (int i = 0; i < n; ++i) p[i] = -g[i] / std::fmax(max_abs(g.data(), n), 1e-300);
    }
    Trial tr;
    if (!strong_wolfe(F, x, f, g.data(), p.data(), tr)) {
      if (count == 0) break;             // steepest descent failed too: stationary to rounding
      count = 0;
      continue;
    }
    for (int i = 0; i < n; ++i) {
      s[i] = tr.x[i] - x[i];
      y[i] = tr.g[i] - g[i];
    }
    const double sy = dot(s.data(), y.data(), n);
    const double fold = f;
    for (int i = 0; i < n; ++i) {
      x[i] = tr.x[i];
      g[i] = tr.g[i];
    }
    f = tr.f;
    if (sy > 1e-300) {
      std::copy(s.begin(), s.end(), S.begin() + (size_t)head * n);
      std::copy(y.begin(), y.end(), Yv.begin() + (size_t)head * n);
      rho[head] = 1.0 / sy;
      head = (head + 1) % kMem;
      if (count < kMem) ++count;
    }
    if (fold - f <= 1e-16 * std::fabs(f)) break;   // no progress above rounding
  }
  return f;
}

}  // namespace

double rebase_phi_grad(const Realization &D, const double g[12], double grad[12]) {
  return phi_grad(D, g, grad);
}

double rebase_phi_grad_shape(const Shaped &S, const double *g, double *grad) {
  return phi_grad_shape(S, g, grad);
}

int realization_optimize(const Realization &D, int nstarts, const double *starts, int max_iter,
                         double gtol, double tol, Realization &best, double &best_phi,
                         double *start_phi) {
  static const double kIdentity[kN] = {1, 0, 0, 1, 1, 0, 0, 1, 1, 0, 0, 1};
  const Objective F{kN, &D, nullptr};
  bool found = false;
  best_phi = std::numeric_limits<double>::infinity();
  for (int s = 0; s <= nstarts; ++s) {
    double x[kN];
    std::memcpy(x, s == 0 ? kIdentity : starts + (size_t)kN * (s - 1), sizeof(x));
    double phi_end = lbfgs(F, x, max_iter, gtol);
    Realization cand;
    double terminal = std::numeric_limits<double>::quiet_NaN();
    if (std::isfinite(phi_end) && realization_transform(D, x, x + 4, x + 8, cand) == FMM_OK) {
      double phi = 0.0, gamma = 0.0;
      realization_phi_gamma(cand, phi, gamma);
      if (std::isfinite(phi) && brent_residual(cand) <= tol) {
        terminal = phi;
        if (phi < best_phi) {
          best_phi = phi;
          best = cand;
          found = true;
        }
      }
    }
    if (start_phi) start_phi[s] = terminal;
  }
  return found ? FMM_OK : FMM_ERR_NOT_EXACT;
}

int realization_optimize_shape(const Shaped &S, int nstarts, const double *starts, int max_iter, double gtol,
                               double tol, std::vector<double> &bU, std::vector<double> &bV,
                               std::vector<double> &bW, double &best_phi, double *start_phi) {
  const int np = S.m * S.m + S.k * S.k + S.n * S.n;
  const Objective F{np, nullptr, &S};
  std::vector<double> x(np), ident(np, 0.0);
  for (int i = 0; i < S.m; ++i) ident[i * S.m + i] = 1.0;
  for (int i = 0; i < S.k; ++i) ident[S.m * S.m + i * S.k + i] = 1.0;
  for (int i = 0; i < S.n; ++i) ident[S.m * S.m + S.k * S.k + i * S.n + i] = 1.0;
  bool found = false;
  best_phi = std::numeric_limits<double>::infinity();
  std::vector<double> U, V, W;
  for (int s = 0; s <= nstarts; ++s) {
    const double *x0 = s == 0 ? ident.data() : starts + (size_t)np * (s - 1);
    std::copy(x0, x0 + np, x.begin());
    const double phi_end = lbfgs(F, x.data(), max_iter, gtol);
    double terminal = std::numeric_limits<double>::quiet_NaN();
    if (std::isfinite(phi_end) &&
        transform_shape(S, x.data(), x.data() + S.m * S.m, x.data() + S.m * S.m + S.k * S.k, U, V, W) == FMM_OK) {
      const Shaped C{S.m, S.k, S.n, S.R, U.data(), V.data(), W.data()};
      double phi = 0.0, gamma = 0.0;
      phi_gamma_shape(C, phi, gamma);
      if (std::isfinite(phi) && brent_residual_shape(C) <= tol) {
        terminal = phi;
        if (phi < best_phi) {
          best_phi = phi;
          bU = U; bV = V; bW = W;
          found = true;
        }
      }
    }
    if (start_phi) start_phi[s] = terminal;
  }
  return found ? FMM_OK : FMM_ERR_NOT_EXACT;
}

}  // namespace fmm

namespace {

// the base realization behind a handle, read through the C-ABI: <2,2,2>
// into D; another shape into the vectors and S
struct Base {
  int m = 2, k = 2, n = 2;
  fmm::Realization D;
  std::vector<double> U, V, W;
  fmm::Shaped S;
  bool is222() const { return m == 2 && k == 2 && n == 2; }
  int params() const { return m * m + k * k + n * n; }
};

int base_of(const fmm_real *d, Base &b) {
  int R = 0;
  int st = fmm_realization_shape(d, &b.m, &b.k, &b.n, &R);
  if (st != FMM_OK) return st;
  if (b.is222()) {
    std::memset(&b.D, 0, sizeof(b.D));
    b.D.R = R;
    return fmm_realization_coefficients(d, &b.D.U[0][0], &b.D.V[0][0], &b.D.W[0][0]);
  }
  try {
    b.U.resize((size_t)R * b.m * b.k);
    b.V.resize((size_t)R * b.k * b.n);
    b.W.resize((size_t)R * b.n * b.m);
  } catch (...) {
    return FMM_ERR_NOMEM;
  }
  b.S = {b.m, b.k, b.n, R, b.U.data(), b.V.data(), b.W.data()};
  return fmm_realization_coefficients(d, b.U.data(), b.V.data(), b.W.data());
}

}  // namespace

extern "C" {

int fmm_realization_optimize(const fmm_real *d, int nstarts, const double *starts, int max_iter,
                             double gtol, double tol, fmm_real **out, double *phi, double *start_phi) {
  if (!out) return FMM_ERR_ARG;
  *out = nullptr;
  if (!d || nstarts < 0 || (nstarts > 0 && !starts) || max_iter < 1 || !(gtol > 0.0) || !(tol >= 0.0))
    return FMM_ERR_ARG;
  Base b;
  int st = base_of(d, b);
  if (st != FMM_OK) return st;
  double best_phi = 0.0;
  // exactness is checked against tol inside; the handle takes the coefficients as they are
  const double inf = std::numeric_limits<double>::infinity();
  if (b.is222()) {
    fmm::Realization best;
    st = fmm::realization_optimize(b.D, nstarts, starts, max_iter, gtol, tol, best, best_phi, start_phi);
    if (st != FMM_OK) return st;
    st = fmm_realization_create(2, 2, 2, best.R, &best.U[0][0], &best.V[0][0], &best.W[0][0], inf, out);
  } else {
    std::vector<double> U, V, W;
    try {
      st = fmm::realization_optimize_shape(b.S, nstarts, starts, max_iter, gtol, tol, U, V, W, best_phi, start_phi);
    } catch (...) {
      return FMM_ERR_NOMEM;
    }
    if (st != FMM_OK) return st;
    st = fmm_realization_create(b.m, b.k, b.n, b.S.R, U.data(), V.data(), W.data(), inf, out);
  }
  if (st == FMM_OK && phi) *phi = best_phi;
  return st;
}

int fmm_realization_phi_gradient(const fmm_real *d, const double *g, double *phi, double *grad) {
  if (!d || !g || !grad) return FMM_ERR_ARG;
  Base b;
  const int st = base_of(d, b);
  if (st != FMM_OK) return st;
  double v;
  try {
    v = b.is222() ? fmm::rebase_phi_grad(b.D, g, grad) : fmm::rebase_phi_grad_shape(b.S, g, grad);
  } catch (...) {
    return FMM_ERR_NOMEM;
  }
  if (phi) *phi = v;
  return FMM_OK;
}

}  // extern "C"
