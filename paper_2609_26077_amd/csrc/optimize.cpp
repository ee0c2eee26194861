// Re-basing: minimization of Phi over a realization's change-of-basis orbit
// (Section 3.1; the re-basing protocol of Appendix E.2).
//
// The orbit is D . g for g = (X, Y, Z) in GL(2)^3 under the right action of
// eq. A.1; Phi(D . g) = sum_r |u_r K_U|^2 |v_r K_V|^2 |w_r K_W|^2 with
// K_U = X (x) Y^-T, K_V = Y (x) Z^-T, K_W = Z (x) X^-T.  Each start is driven
// by limited-memory BFGS over the 12 entries of (X, Y, Z) with a line search
// that enforces the strong Wolfe conditions; the gradient is exact, carried
// by forward-mode dual numbers through the same expression.
#include "internal.h"

#include <cmath>
#include <cstring>
#include <limits>
#include <new>
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

double dot(const double *a, const double *b) {
  double s = 0.0;
  for (int i = 0; i < kN; ++i) s += a[i] * b[i];
  return s;
}
double max_abs(const double *a) {
  double m = 0.0;
  for (int i = 0; i < kN; ++i) m = std::fmax(m, std::fabs(a[i]));
  return m;
}

// A trial point of the line search x + t p.
struct Trial {
  double t, f, dphi;     // step, value, directional derivative
  double x[kN], g[kN];
};

bool evaluate(const Realization &D, const double *x0, const double *p, double t, Trial &tr) {
  tr.t = t;
  for (int i = 0; i < kN; ++i) tr.x[i] = x0[i] + t * p[i];
  tr.f = phi_grad(D, tr.x, tr.g);
  tr.dphi = dot(tr.g, p);
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
bool strong_wolfe(const Realization &D, const double *x0, double f0, const double *g0, const double *p,
                  Trial &out) {
  constexpr double c1 = 1e-4, c2 = 0.9;
  const double d0 = dot(g0, p);
  if (!(d0 < 0.0)) return false;
  Trial prev;
  prev.t = 0.0; prev.f = f0; prev.dphi = d0;
  std::memcpy(prev.x, x0, sizeof(prev.x));
  std::memcpy(prev.g, g0, sizeof(prev.g));
  Trial lo, hi, cur;
  bool bracket = false;
  double t = 1.0;
  for (int it = 0; it < 60; ++it) {
    const bool ok = evaluate(D, x0, p, t, cur);
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
    const bool ok = evaluate(D, x0, p, tj, tr);
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

// L-BFGS from x (12 entries of g); returns the terminal Phi, x updated.
double lbfgs(const Realization &D, double x[kN], int max_iter, double gtol) {
  constexpr int kMem = 10;
  double S[kMem][kN], Yv[kMem][kN], rho[kMem];
  int count = 0, head = 0;
  double g[kN];
  double f = phi_grad(D, x, g);
  if (!std::isfinite(f)) return f;
  for (int it = 0; it < max_iter; ++it) {
    if (max_abs(g) <= gtol * std::fmax(1.0, f)) break;
    // two-loop recursion: p = -H g
    double q[kN], alpha[kMem];
    for (int i = 0; i < kN; ++i) q[i] = g[i];
    for (int k = 0; k < count; ++k) {
      const int j = (head - 1 - k + kMem) % kMem;
      alpha[j] = rho[j] * dot(S[j], q);
      for (int i = 0; i < kN; ++i) q[i] -= alpha[j] * Yv[j][i];
    }
    double gamma = 1.0;
    if (count > 0) {
      const int j = (head - 1 + kMem) % kMem;
      gamma = dot(S[j], Yv[j]) / dot(Yv[j], Yv[j]);
    } else {
      gamma = 1.0 / std::fmax(max_abs(g), 1e-300);   // first step of length ~1 in the largest entry
    }
    for (int i = 0; i < kN; ++i) q[i] *= gamma;
    for (int k = count - 1; k >= 0; --k) {
      const int j = (head - 1 - k + kMem) % kMem;
      const double beta = rho[j] * dot(Yv[j], q);
      for (int i = 0; i < kN; ++i) q[i] += S[j][i] * (alpha[j] - beta);
    }
    double p[kN];
    for (int i = 0; i < kN; ++i) p[i] = -q[i];
    if (!(dot(p, g) < 0.0)) {            // not a descent direction: restart from steepest descent
      count = 0;
      for (int i = 0; i < kN; ++i) p[i] = -g[i] / std::fmax(max_abs(g), 1e-300);
    }
    Trial tr;
    if (!strong_wolfe(D, x, f, g, p, tr)) {
      if (count == 0) break;             // steepest descent failed too: stationary to rounding
      count = 0;
      continue;
    }
    double s[kN], y[kN];
    for (int i = 0; i < kN; ++i) {
      s[i] = tr.x[i] - x[i];
      y[i] = tr.g[i] - g[i];
    }
    const double sy = dot(s, y);
    const double fold = f;
    std::memcpy(x, tr.x, sizeof(tr.x));
    std::memcpy(g, tr.g, sizeof(tr.g));
    f = tr.f;
    if (sy > 1e-300) {
      std::memcpy(S[head], s, sizeof(s));
      std::memcpy(Yv[head], y, sizeof(y));
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

int realization_optimize(const Realization &D, int nstarts, const double *starts, int max_iter,
                         double gtol, double tol, Realization &best, double &best_phi,
                         double *start_phi) {
  static const double kIdentity[kN] = {1, 0, 0, 1, 1, 0, 0, 1, 1, 0, 0, 1};
  bool found = false;
  best_phi = std::numeric_limits<double>::infinity();
  for (int s = 0; s <= nstarts; ++s) {
    double x[kN];
    std::memcpy(x, s == 0 ? kIdentity : starts + (size_t)kN * (s - 1), sizeof(x));
    double phi_end = lbfgs(D, x, max_iter, gtol);
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

}  // namespace fmm

namespace {

// the base realization behind a handle, read through the C-ABI
int realization_of(const fmm_real *d, fmm::Realization &D) {
  int m = 0, k = 0, n = 0, Rs = 0;
  int st = fmm_realization_shape(d, &m, &k, &n, &Rs);
  if (st != FMM_OK) return st;
  if (m != 2 || k != 2 || n != 2) return FMM_ERR_UNSUPPORTED;   // the orbit under GL(2)^3 is <2,2,2>'s
  int64_t R = 0, T = 0;
  st = fmm_realization_terms(d, 1, &R, &T);
  if (st != FMM_OK) return st;
  std::memset(&D, 0, sizeof(D));
  D.R = (int)R;
  return fmm_realization_coefficients(d, &D.U[0][0], &D.V[0][0], &D.W[0][0]);
}

}  // namespace

extern "C" {

int fmm_realization_optimize(const fmm_real *d, int nstarts, const double *starts, int max_iter,
                             double gtol, double tol, fmm_real **out, double *phi, double *start_phi) {
  if (!out) return FMM_ERR_ARG;
  *out = nullptr;
  if (!d || nstarts < 0 || (nstarts > 0 && !starts) || max_iter < 1 || !(gtol > 0.0) || !(tol >= 0.0))
    return FMM_ERR_ARG;
  fmm::Realization D, best;
  int st = realization_of(d, D);
  if (st != FMM_OK) return st;
  double best_phi = 0.0;
  st = fmm::realization_optimize(D, nstarts, starts, max_iter, gtol, tol, best, best_phi, start_phi);
  if (st != FMM_OK) return st;
  // exactness was checked against tol above; the handle takes the coefficients as they are
  st = fmm_realization_create(2, 2, 2, best.R, &best.U[0][0], &best.V[0][0], &best.W[0][0],
                              std::numeric_limits<double>::infinity(), out);
  if (st == FMM_OK && phi) *phi = best_phi;
  return st;
}

int fmm_realization_phi_gradient(const fmm_real *d, const double g[12], double *phi, double grad[12]) {
  if (!d || !g || !grad) return FMM_ERR_ARG;
  fmm::Realization D;
  const int st = realization_of(d, D);
  if (st != FMM_OK) return st;
  const double v = fmm::rebase_phi_grad(D, g, grad);
  if (phi) *phi = v;
  return FMM_OK;
}

}  // extern "C"
