// Host check of the SHAC adjoint (paper_2512_13359_amd/csrc/shac_adjoint.hpp) in double
// precision: every vector-Jacobian product against central differences of the forward it
// differentiates, on seeded random inputs (non-unit stage quaternions, attitude errors
// with either sign of the scalar part, small and large angles).  Prints one line per
// product with the largest error relative to the product's scale and exits non-zero if
// any exceeds the bound.
#include <cmath>
#include <cstdio>
#include <random>

#include "shac_adjoint.hpp"

using namespace auv::adj;
typedef double T;

static std::mt19937_64 gen(12345);
static T U(T lo, T hi) { return std::uniform_real_distribution<T>(lo, hi)(gen); }

static Model<T> model() {
  Model<T> M;
  const T m = 11.5, I = 0.16, A[6] = {5.5, 12.7, 14.6, 0.12, 0.12, 0.12};
  const T DL[6] = {4.0, 6.2, 5.2, 0.07, 0.07, 0.07}, DQ[6] = {18.2, 21.7, 37.0, 1.5, 1.5, 1.5};
  for (int i = 0; i < 3; ++i) {
    M.Mlin[i] = m + A[i];
    M.Mang[i] = I + A[3 + i];
    M.iMlin[i] = 1.0 / M.Mlin[i];
    M.iMang[i] = 1.0 / M.Mang[i];
    M.A1[i] = A[i];
  }
  for (int i = 0; i < 6; ++i) { M.DL[i] = DL[i]; M.DQ[i] = DQ[i]; }
  M.BmW = 114.8 - U(0.95, 1.05) * 112.8;
  return M;
}

static T* slot(X13<T>& x, int k) {   // component k of the 13 in the order p, q, v, w
  return k < 3 ? &x.p[k] : (k < 7 ? &x.q[k - 3] : (k < 10 ? &x.v[k - 7] : &x.w[k - 10]));
}

static X13<T> rand_state(bool unit_q, T vs = 1.0) {
  X13<T> x;
  for (int i = 0; i < 3; ++i) { x.p[i] = U(-2, 2); x.v[i] = U(-vs, vs); x.w[i] = U(-vs, vs); }
  T n = 0;
  for (int i = 0; i < 4; ++i) { x.q[i] = U(-1, 1); n += x.q[i] * x.q[i]; }
  n = std::sqrt(n) * (unit_q ? 1.0 : U(0.9, 1.1));
  for (int i = 0; i < 4; ++i) x.q[i] /= n;
  return x;
}

static T dot13(const X13<T>& a, const X13<T>& b) {
  T s = 0;
  for (int i = 0; i < 3; ++i) s += a.p[i] * b.p[i] + a.v[i] * b.v[i] + a.w[i] * b.w[i];
  for (int i = 0; i < 4; ++i) s += a.q[i] * b.q[i];
  return s;
}

static double worst = 0.0;
static bool report(const char* what, double err, double scale, double bound) {
  const double rel = err / (scale > 0 ? scale : 1.0);
  std::printf("%-28s max rel err %.3e (bound %.1e)\n", what, rel, bound);
  if (rel > worst) worst = rel;
  return rel <= bound;
}

int main() {
  bool ok = true;
  const T eps = 1e-6;
  // ---- rhs ------------------------------------------------------------------------
  {
    double err = 0, scale = 0;
    for (int trial = 0; trial < 50; ++trial) {
      Model<T> M = model();
      X13<T> x = rand_state(false, 1.5), gd = rand_state(false, 3.0), gx;
      T tau[6], gtau[6] = {0, 0, 0, 0, 0, 0};
      for (int i = 0; i < 6; ++i) tau[i] = U(-40, 40);
      zero(gx);
      rhs_vjp(M, x, gd, gx, gtau);
      for (int k = 0; k < 19; ++k) {
        X13<T> xp = x, xm = x, dp, dm;
        T tp[6], tm[6];
        for (int i = 0; i < 6; ++i) tp[i] = tm[i] = tau[i];
        if (k < 13) { *slot(xp, k) += eps; *slot(xm, k) -= eps; } else { tp[k - 13] += eps; tm[k - 13] -= eps; }
        rhs(M, tp, xp, dp);
        rhs(M, tm, xm, dm);
        const T fd = (dot13(gd, dp) - dot13(gd, dm)) / (2 * eps);
        const T an = k < 13 ? *slot(gx, k) : gtau[k - 13];
        err = std::fmax(err, std::fabs(fd - an));
        scale = std::fmax(scale, std::fabs(an));
      }
    }
    ok &= report("rhs_vjp", err, scale, 1e-7);
  }
  // ---- RK4 substep with renormalisation ---------------------------------------------
  {
    double err = 0, scale = 0;
    for (int trial = 0; trial < 50; ++trial) {
      Model<T> M = model();
      X13<T> x = rand_state(true, 1.5), g = rand_state(false, 1.0), g0 = g;
      T tau[6], gtau[6] = {0, 0, 0, 0, 0, 0};
      for (int i = 0; i < 6; ++i) tau[i] = U(-40, 40);
      const T h = 0.025;
      substep_vjp(M, tau, h, x, g, gtau);
      for (int k = 0; k < 19; ++k) {
        X13<T> xp = x, xm = x;
        T tp[6], tm[6];
        for (int i = 0; i < 6; ++i) tp[i] = tm[i] = tau[i];
        if (k < 13) { *slot(xp, k) += eps; *slot(xm, k) -= eps; } else { tp[k - 13] += eps; tm[k - 13] -= eps; }
        substep(M, tp, h, xp);
        substep(M, tm, h, xm);
        const T fd = (dot13(g0, xp) - dot13(g0, xm)) / (2 * eps);
        const T an = k < 13 ? *slot(g, k) : gtau[k - 13];
        err = std::fmax(err, std::fabs(fd - an));
        scale = std::fmax(scale, std::fabs(an));
      }
    }
    ok &= report("substep_vjp", err, scale, 1e-7);
  }
  // ---- observation: general, small-angle (series branch) and negative scalar part ----
  for (int kind = 0; kind < 3; ++kind) {
    double err = 0, scale = 0;
    for (int trial = 0; trial < 60; ++trial) {
      X13<T> x = rand_state(true, 1.0), gx;
      T pg[3] = {U(-2, 2), U(-2, 2), U(-2, 2)}, qg[4];
      if (kind == 1) {   // goal within a few degrees of the attitude
        T n = 0;
        for (int i = 0; i < 4; ++i) { qg[i] = x.q[i] + U(-0.01, 0.01); n += qg[i] * qg[i]; }
        for (int i = 0; i < 4; ++i) qg[i] /= std::sqrt(n);
      } else {
        X13<T> y = rand_state(true);
        for (int i = 0; i < 4; ++i) qg[i] = y.q[i];
      }
      T ew = 0;
      for (int i = 0; i < 4; ++i) ew += x.q[i] * qg[i];
      if ((kind == 2) != (ew < 0))
        for (int i = 0; i < 4; ++i) qg[i] = -qg[i];
      T go[12];
      for (int i = 0; i < 12; ++i) go[i] = U(-1, 1);
      zero(gx);
      observe_vjp(x, pg, qg, go, gx);
      for (int k = 0; k < 13; ++k) {
        X13<T> xp = x, xm = x;
        *slot(xp, k) += eps;
        *slot(xm, k) -= eps;
        T op[12], om[12];
        observe(xp, pg, qg, op);
        observe(xm, pg, qg, om);
        T fd = 0;
        for (int i = 0; i < 12; ++i) fd += go[i] * (op[i] - om[i]) / (2 * eps);
        err = std::fmax(err, std::fabs(fd - *slot(gx, k)));
        scale = std::fmax(scale, std::fabs(*slot(gx, k)));
      }
    }
    const char* names[3] = {"observe_vjp", "observe_vjp small angle", "observe_vjp scalar < 0"};
    ok &= report(names[kind], err, scale, 1e-7);
  }
  // ---- reward ------------------------------------------------------------------------
  {
    Task<T> K{60.0, 10.0, 1.0, {1.0, 1.0, 1.5}, 0.5, 0.01, 0.05, 0.1, 0.8};
    double err = 0, scale = 0;
    for (int trial = 0; trial < 50; ++trial) {
      T o[12], u[6], ab[6], go[12], gu[6] = {0, 0, 0, 0, 0, 0}, gab[6] = {0, 0, 0, 0, 0, 0};
      for (int i = 0; i < 12; ++i) o[i] = U(-2, 2);
      for (int i = 0; i < 6; ++i) { u[i] = U(-1, 1); ab[i] = U(-1, 1); }
      const T c = U(-2, 2);
      reward_grad(K, c, o, u, ab, go, gu, gab);
      for (int k = 0; k < 24; ++k) {
        T* v = k < 12 ? &o[k] : (k < 18 ? &u[k - 12] : &ab[k - 18]);
        const T keep = *v;
        *v = keep + eps;
        const T rp = reward(K, o, u, ab);
        *v = keep - eps;
        const T rm = reward(K, o, u, ab);
        *v = keep;
        const T fd = c * (rp - rm) / (2 * eps);
        const T an = k < 12 ? go[k] : (k < 18 ? gu[k - 12] : gab[k - 18]);
        err = std::fmax(err, std::fabs(fd - an));
        scale = std::fmax(scale, std::fabs(an));
      }
    }
    ok &= report("reward_grad", err, scale, 1e-7);
  }
  std::printf("worst %.3e %s\n", worst, ok ? "OK" : "FAIL");
  return ok ? 0 : 1;
}
