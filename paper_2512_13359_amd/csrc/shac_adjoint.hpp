// The paper task's control step for one environment in scalar form (one lane per
// environment), and its reverse-mode derivative: vector-Jacobian products of the Fossen
// right-hand side, of one RK4 substep with quaternion renormalisation, of the observation
// (body-frame position error, rotation vector of the attitude error, velocities) and the
// gradient of the five-term reward.  These carry the SHAC state adjoint back through a
// window (the differentiable-simulation learner, paper Sec. III-A3).
//
// Model (paper task): no current, centre of buoyancy at the centre of gravity, weight
// gamma W per environment, diagonal mass matrix (body origin at the CoG):
//   dv = (tau_f - w x (Mlin v) - (DL + DQ |v|) v - (B - gamma W) k) / Mlin,   k = R^T e3
//   dw = (tau_m - w x (Mang w) - v x (A1 v) - (DLa + DQa |w|) w) / Mang
//   dp = R v,   dq = 1/2 q (x) (0, w)
// Derivative conventions: d|x|/dx = sign(x) (0 at 0); the clip of the action is handled
// by the caller.
//
// Every function is a template on the real type T: the SHAC kernel uses float, a host
// check instantiates double and compares each product with central differences of the
// forward.  No HIP header is needed (AUV_HD marks host + device functions under hipcc).
#pragma once

#include <math.h>

#if defined(__HIPCC__)
#define AUV_HD __host__ __device__ __forceinline__
#else
#define AUV_HD inline
#endif

namespace auv {
namespace adj {

AUV_HD float r_sqrt(float x) { return sqrtf(x); }
AUV_HD double r_sqrt(double x) { return sqrt(x); }
AUV_HD float r_atan2(float y, float x) { return atan2f(y, x); }
AUV_HD double r_atan2(double y, double x) { return atan2(y, x); }
template <class T> AUV_HD T r_abs(T x) { return x < T(0) ? -x : x; }
template <class T> AUV_HD T r_sign(T x) { return x > T(0) ? T(1) : (x < T(0) ? T(-1) : T(0)); }

// Per-environment model constants.
template <class T>
struct Model {
  T Mlin[3], Mang[3], iMlin[3], iMang[3], A1[3], DL[6], DQ[6], BmW;
};

// State (p, q = (w, x, y, z), v, omega); also used for its time derivative and cotangents.
template <class T>
struct X13 {
  T p[3], q[4], v[3], w[3];
};

template <class T>
AUV_HD void zero(X13<T>& x) {
  for (int i = 0; i < 3; ++i) x.p[i] = x.v[i] = x.w[i] = T(0);
  for (int i = 0; i < 4; ++i) x.q[i] = T(0);
}

// x + c d (p, q, v, w)
template <class T>
AUV_HD X13<T> axpy(const X13<T>& x, T c, const X13<T>& d) {
  X13<T> y;
  for (int i = 0; i < 3; ++i) {
    y.p[i] = x.p[i] + c * d.p[i];
    y.v[i] = x.v[i] + c * d.v[i];
    y.w[i] = x.w[i] + c * d.w[i];
  }
  for (int i = 0; i < 4; ++i) y.q[i] = x.q[i] + c * d.q[i];
  return y;
}

template <class T>
AUV_HD void add_to(X13<T>& y, T c, const X13<T>& d) {
  for (int i = 0; i < 3; ++i) {
    y.p[i] += c * d.p[i];
    y.v[i] += c * d.v[i];
    y.w[i] += c * d.w[i];
  }
  for (int i = 0; i < 4; ++i) y.q[i] += c * d.q[i];
}

// ---------------------------------------------------------------- rotation ------------
// R(q) = I + 2 w S(e) + 2 S(e)^2 written out (also for non-unit stage quaternions).
template <class T>
AUV_HD void rot(const T q[4], T R[3][3]) {
  const T w = q[0], x = q[1], y = q[2], z = q[3];
  R[0][0] = T(1) - T(2) * (y * y + z * z); R[0][1] = T(2) * (x * y - w * z); R[0][2] = T(2) * (x * z + w * y);
  R[1][0] = T(2) * (x * y + w * z); R[1][1] = T(1) - T(2) * (x * x + z * z); R[1][2] = T(2) * (y * z - w * x);
  R[2][0] = T(2) * (x * z - w * y); R[2][1] = T(2) * (y * z + w * x); R[2][2] = T(1) - T(2) * (x * x + y * y);
}

// gq += dR/dq^T gR (entry by entry of the formula above)
template <class T>
AUV_HD void rot_vjp(const T q[4], const T gR[3][3], T gq[4]) {
  const T w = q[0], x = q[1], y = q[2], z = q[3];
  T gw = T(0), gx = T(0), gy = T(0), gz = T(0);
  gy += T(-4) * y * gR[0][0]; gz += T(-4) * z * gR[0][0];
  gx += T(2) * y * gR[0][1]; gy += T(2) * x * gR[0][1]; gw += T(-2) * z * gR[0][1]; gz += T(-2) * w * gR[0][1];
  gx += T(2) * z * gR[0][2]; gz += T(2) * x * gR[0][2]; gw += T(2) * y * gR[0][2]; gy += T(2) * w * gR[0][2];
  gx += T(2) * y * gR[1][0]; gy += T(2) * x * gR[1][0]; gw += T(2) * z * gR[1][0]; gz += T(2) * w * gR[1][0];
  gx += T(-4) * x * gR[1][1]; gz += T(-4) * z * gR[1][1];
  gy += T(2) * z * gR[1][2]; gz += T(2) * y * gR[1][2]; gw += T(-2) * x * gR[1][2]; gx += T(-2) * w * gR[1][2];
  gx += T(2) * z * gR[2][0]; gz += T(2) * x * gR[2][0]; gw += T(-2) * y * gR[2][0]; gy += T(-2) * w * gR[2][0];
  gy += T(2) * z * gR[2][1]; gz += T(2) * y * gR[2][1]; gw += T(2) * x * gR[2][1]; gx += T(2) * w * gR[2][1];
  gx += T(-4) * x * gR[2][2]; gy += T(-4) * y * gR[2][2];
  gq[0] += gw; gq[1] += gx; gq[2] += gy; gq[3] += gz;
}

// a x b
template <class T>
AUV_HD void cross(const T a[3], const T b[3], T c[3]) {
  c[0] = a[1] * b[2] - a[2] * b[1];
  c[1] = a[2] * b[0] - a[0] * b[2];
  c[2] = a[0] * b[1] - a[1] * b[0];
}

// --------------------------------------------------------------- right side -----------
template <class T>
AUV_HD void rhs(const Model<T>& M, const T tau[6], const X13<T>& x, X13<T>& d) {
  T R[3][3];
  rot(x.q, R);
  for (int i = 0; i < 3; ++i) d.p[i] = R[i][0] * x.v[0] + R[i][1] * x.v[1] + R[i][2] * x.v[2];
  T a[3], b[3], c[3], wa[3], wb[3], vc[3];
  for (int i = 0; i < 3; ++i) {
    a[i] = M.Mlin[i] * x.v[i];
    b[i] = M.Mang[i] * x.w[i];
    c[i] = M.A1[i] * x.v[i];
  }
  cross(x.w, a, wa);
  cross(x.w, b, wb);
  cross(x.v, c, vc);
  for (int i = 0; i < 3; ++i) {
    const T F = tau[i] - wa[i] - (M.DL[i] + M.DQ[i] * r_abs(x.v[i])) * x.v[i] - M.BmW * R[2][i];
    const T G = tau[3 + i] - wb[i] - vc[i] - (M.DL[3 + i] + M.DQ[3 + i] * r_abs(x.w[i])) * x.w[i];
    d.v[i] = F * M.iMlin[i];
    d.w[i] = G * M.iMang[i];
  }
  const T h0 = T(0.5) * x.w[0], h1 = T(0.5) * x.w[1], h2 = T(0.5) * x.w[2];
  d.q[0] = -(x.q[1] * h0 + x.q[2] * h1 + x.q[3] * h2);
  d.q[1] = x.q[0] * h0 + x.q[2] * h2 - x.q[3] * h1;
  d.q[2] = x.q[0] * h1 + x.q[3] * h0 - x.q[1] * h2;
  d.q[3] = x.q[0] * h2 + x.q[1] * h1 - x.q[2] * h0;
}

// Cotangent gd of the derivative d = rhs(x) -> gx (q, v, w components; accumulated) and
// gtau (accumulated).  The position does not enter the right side.
template <class T>
AUV_HD void rhs_vjp(const Model<T>& M, const X13<T>& x, const X13<T>& gd, X13<T>& gx, T gtau[6]) {
  T R[3][3], gR[3][3];
  rot(x.q, R);
  for (int i = 0; i < 3; ++i)
    for (int j = 0; j < 3; ++j) gR[i][j] = T(0);
  T gF[3], gG[3], a[3], b[3], c[3];
  for (int i = 0; i < 3; ++i) {
    gF[i] = gd.v[i] * M.iMlin[i];
    gG[i] = gd.w[i] * M.iMang[i];
    gtau[i] += gF[i];
    gtau[3 + i] += gG[i];
    a[i] = M.Mlin[i] * x.v[i];
    b[i] = M.Mang[i] * x.w[i];
    c[i] = M.A1[i] * x.v[i];
  }
  // F = ... - w x a: cotangent of (w x a) is -gF; d(w x a) -> w: a x g, a: g x w
  T nF[3], nG[3], t[3], ga[3], gb[3], gc[3];
  for (int i = 0; i < 3; ++i) { nF[i] = -gF[i]; nG[i] = -gG[i]; }
  cross(a, nF, t);
  for (int i = 0; i < 3; ++i) gx.w[i] += t[i];
  cross(nF, x.w, ga);
  // G = ... - w x b - v x c
  cross(b, nG, t);
  for (int i = 0; i < 3; ++i) gx.w[i] += t[i];
  cross(nG, x.w, gb);
  cross(c, nG, t);
  for (int i = 0; i < 3; ++i) gx.v[i] += t[i];
  cross(nG, x.v, gc);
  for (int i = 0; i < 3; ++i) {
    gx.v[i] += M.Mlin[i] * ga[i] + M.A1[i] * gc[i];
    gx.w[i] += M.Mang[i] * gb[i];
    // damping (DL + DQ |x|) x has derivative DL + 2 DQ |x|
    gx.v[i] -= gF[i] * (M.DL[i] + T(2) * M.DQ[i] * r_abs(x.v[i]));
    gx.w[i] -= gG[i] * (M.DL[3 + i] + T(2) * M.DQ[3 + i] * r_abs(x.w[i]));
    // restoring force -(B - gamma W) R[2][i]
    gR[2][i] -= M.BmW * gF[i];
  }
  // dp = R v
  for (int i = 0; i < 3; ++i)
    for (int j = 0; j < 3; ++j) {
      gx.v[j] += R[i][j] * gd.p[i];
      gR[i][j] += gd.p[i] * x.v[j];
    }
  rot_vjp(x.q, gR, gx.q);
  // dq = 1/2 q (x) (0, w)
  const T* q = x.q;
  const T* w = x.w;
  const T* g = gd.q;
  gx.q[0] += T(0.5) * (g[1] * w[0] + g[2] * w[1] + g[3] * w[2]);
  gx.q[1] += T(0.5) * (-g[0] * w[0] - g[2] * w[2] + g[3] * w[1]);
  gx.q[2] += T(0.5) * (-g[0] * w[1] + g[1] * w[2] - g[3] * w[0]);
  gx.q[3] += T(0.5) * (-g[0] * w[2] - g[1] * w[1] + g[2] * w[0]);
  gx.w[0] += T(0.5) * (-g[0] * q[1] + g[1] * q[0] + g[2] * q[3] - g[3] * q[2]);
  gx.w[1] += T(0.5) * (-g[0] * q[2] - g[1] * q[3] + g[2] * q[0] + g[3] * q[1]);
  gx.w[2] += T(0.5) * (-g[0] * q[3] + g[1] * q[2] - g[2] * q[1] + g[3] * q[0]);
}

// --------------------------------------------------------------- RK4 substep ----------
// Classic RK4 of length h with tau held, then the quaternion divided by its norm.
template <class T>
AUV_HD void substep(const Model<T>& M, const T tau[6], T h, X13<T>& x) {
  X13<T> k1, k2, k3, k4;
  rhs(M, tau, x, k1);
  rhs(M, tau, axpy(x, T(0.5) * h, k1), k2);
  rhs(M, tau, axpy(x, T(0.5) * h, k2), k3);
  rhs(M, tau, axpy(x, h, k3), k4);
  const T h6 = h / T(6);
  X13<T> y = x;
  add_to(y, h6, k1);
  add_to(y, T(2) * h6, k2);
  add_to(y, T(2) * h6, k3);
  add_to(y, h6, k4);
  const T inv = T(1) / r_sqrt(y.q[0] * y.q[0] + y.q[1] * y.q[1] + y.q[2] * y.q[2] + y.q[3] * y.q[3]);
  for (int i = 0; i < 4; ++i) y.q[i] *= inv;
  x = y;
}

// g: cotangent of the substep's output on entry, of its input x0 on return; gtau accumulated.
template <class T>
AUV_HD void substep_vjp(const Model<T>& M, const T tau[6], T h, const X13<T>& x0, X13<T>& g, T gtau[6]) {
  // forward recompute: stage inputs and the unnormalised result
  X13<T> k1, k2, k3, k4, s2, s3, s4;
  rhs(M, tau, x0, k1);
  s2 = axpy(x0, T(0.5) * h, k1);
  rhs(M, tau, s2, k2);
  s3 = axpy(x0, T(0.5) * h, k2);
  rhs(M, tau, s3, k3);
  s4 = axpy(x0, h, k3);
  rhs(M, tau, s4, k4);
  const T h6 = h / T(6);
  T y[4];
  for (int i = 0; i < 4; ++i) y[i] = x0.q[i] + h6 * (k1.q[i] + T(2) * k2.q[i] + T(2) * k3.q[i] + k4.q[i]);
  const T nrm = r_sqrt(y[0] * y[0] + y[1] * y[1] + y[2] * y[2] + y[3] * y[3]);
  const T inv = T(1) / nrm;
  // normalisation: q_out = y / |y|  ->  gy = (g - q_out (q_out . g)) / |y|
  T dot = T(0);
  for (int i = 0; i < 4; ++i) dot += y[i] * inv * g.q[i];
  for (int i = 0; i < 4; ++i) g.q[i] = (g.q[i] - y[i] * inv * dot) * inv;
  // y = x0 + h/6 (k1 + 2 k2 + 2 k3 + k4)
  X13<T> gk, gs;
  gk = g;
  for (int i = 0; i < 3; ++i) { gk.p[i] *= h6; gk.v[i] *= h6; gk.w[i] *= h6; }
  for (int i = 0; i < 4; ++i) gk.q[i] *= h6;
  // stage 4: k4 = f(x0 + h k3), weight 1
  zero(gs);
  rhs_vjp(M, s4, gk, gs, gtau);
  add_to(g, T(1), gs);
  X13<T> g3 = gk;                       // cotangent of k3: 2 h6 g + h gs4
  add_to(g3, T(1), gk);
  add_to(g3, h, gs);
  zero(gs);
  rhs_vjp(M, s3, g3, gs, gtau);
  add_to(g, T(1), gs);
  X13<T> g2 = gk;                       // cotangent of k2: 2 h6 g + h/2 gs3
  add_to(g2, T(1), gk);
  add_to(g2, T(0.5) * h, gs);
  zero(gs);
  rhs_vjp(M, s2, g2, gs, gtau);
  add_to(g, T(1), gs);
  X13<T> g1 = gk;                       // cotangent of k1: h6 g + h/2 gs2
  add_to(g1, T(0.5) * h, gs);
  zero(gs);
  rhs_vjp(M, x0, g1, gs, gtau);
  add_to(g, T(1), gs);
}

// ----------------------------------------------------------- observation, reward -----
// o = [R^T (p_goal - p), rotation vector of q^* (x) q_goal (non-negative scalar part), v, w]
template <class T>
AUV_HD void observe(const X13<T>& x, const T pg[3], const T qg[4], T o[12]) {
  T R[3][3];
  rot(x.q, R);
  T d[3];
  for (int j = 0; j < 3; ++j) d[j] = pg[j] - x.p[j];
  for (int i = 0; i < 3; ++i) o[i] = R[0][i] * d[0] + R[1][i] * d[1] + R[2][i] * d[2];
  const T* q = x.q;
  const T ew = q[0] * qg[0] + q[1] * qg[1] + q[2] * qg[2] + q[3] * qg[3];
  T c[3];
  cross(q + 1, qg + 1, c);
  T ev[3];
  for (int i = 0; i < 3; ++i) ev[i] = q[0] * qg[1 + i] - qg[0] * q[1 + i] - c[i];
  const T n = r_sqrt(ev[0] * ev[0] + ev[1] * ev[1] + ev[2] * ev[2]), aw = r_abs(ew);
  const T k = n > T(0) ? T(2) * r_atan2(n, aw) / n : T(2) / aw;
  const T sk = ew < T(0) ? -k : k;
  for (int i = 0; i < 3; ++i) {
    o[3 + i] = sk * ev[i];
    o[6 + i] = x.v[i];
    o[9 + i] = x.w[i];
  }
}

// gx += (do/dx)^T go
template <class T>
AUV_HD void observe_vjp(const X13<T>& x, const T pg[3], const T qg[4], const T go[12], X13<T>& gx) {
  T R[3][3], gR[3][3];
  rot(x.q, R);
  T d[3];
  for (int j = 0; j < 3; ++j) d[j] = pg[j] - x.p[j];
  for (int j = 0; j < 3; ++j) {
    const T gd = R[j][0] * go[0] + R[j][1] * go[1] + R[j][2] * go[2];
    gx.p[j] -= gd;
    for (int i = 0; i < 3; ++i) gR[j][i] = d[j] * go[i];
  }
  rot_vjp(x.q, gR, gx.q);
  // rotation vector s k(n, aw) ev with aw = |ew|, n = |ev|, k = 2 atan2(n, aw) / n
  const T* q = x.q;
  const T ew = q[0] * qg[0] + q[1] * qg[1] + q[2] * qg[2] + q[3] * qg[3];
  T c[3], ev[3];
  cross(q + 1, qg + 1, c);
  for (int i = 0; i < 3; ++i) ev[i] = q[0] * qg[1 + i] - qg[0] * q[1 + i] - c[i];
  const T n2 = ev[0] * ev[0] + ev[1] * ev[1] + ev[2] * ev[2];
  const T n = r_sqrt(n2), aw = r_abs(ew);
  const T s = ew < T(0) ? T(-1) : T(1);
  const T k = n > T(0) ? T(2) * r_atan2(n, aw) / n : T(2) / aw;
  const T r2 = n2 + aw * aw;
  // kn = (dk/dn) / n = (n dtheta/dn - theta) / n^3, by its series in t = n / aw for small t
  T kn;
  if (n < T(0.1) * aw) {
    const T t2 = n2 / (aw * aw);
    kn = T(2) / (aw * aw * aw) * (T(-2.0 / 3.0) + t2 * (T(0.8) + t2 * (T(-6.0 / 7.0) + t2 * T(8.0 / 9.0))));
  } else {
    kn = (T(2) * aw * n / r2 - T(2) * r_atan2(n, aw)) / (n2 * n);
  }
  const T ka = T(-2) / r2;            // dk/daw
  const T* gt = go + 3;
  const T dot = gt[0] * ev[0] + gt[1] * ev[1] + gt[2] * ev[2];
  T gev[3];
  for (int i = 0; i < 3; ++i) gev[i] = s * (k * gt[i] + dot * kn * ev[i]);
  const T gew = dot * ka;             // s^2 = 1
  // ew = q . qg;  ev = q_w qg_v - qg_w q_v - q_v x qg_v
  for (int i = 0; i < 4; ++i) gx.q[i] += gew * qg[i];
  gx.q[0] += gev[0] * qg[1] + gev[1] * qg[2] + gev[2] * qg[3];
  T t[3];
  cross(gev, qg + 1, t);
  for (int i = 0; i < 3; ++i) {
    gx.q[1 + i] += -qg[0] * gev[i] + t[i];
    gx.v[i] += go[6 + i];
    gx.w[i] += go[9 + i];
  }
}

// Reward weights of the paper task.
template <class T>
struct Task {
  T f_max, tau_max, w_pos, d_pos[3], w_att, w_act, w_vel, w_mavg, beta;
};

// r = -w_pos |D dp|^2 - w_att |theta|^2 - w_act |u_3:6|^2 - w_vel |w|^2 - w_mavg |u - abar|^2
template <class T>
AUV_HD T reward(const Task<T>& K, const T o[12], const T u[6], const T ab[6]) {
  T pos = T(0), att = T(0), act = T(0), vel = T(0), mavg = T(0);
  for (int i = 0; i < 3; ++i) {
    const T dp = K.d_pos[i] * o[i];
    pos += dp * dp;
    att += o[3 + i] * o[3 + i];
    act += u[3 + i] * u[3 + i];
    vel += o[9 + i] * o[9 + i];
  }
  for (int j = 0; j < 6; ++j) mavg += (u[j] - ab[j]) * (u[j] - ab[j]);
  return -K.w_pos * pos - K.w_att * att - K.w_act * act - K.w_vel * vel - K.w_mavg * mavg;
}

// c times the gradient of the reward: go (set), gu (added), gab (added).
template <class T>
AUV_HD void reward_grad(const Task<T>& K, T c, const T o[12], const T u[6], const T ab[6], T go[12], T gu[6],
                        T gab[6]) {
  for (int i = 0; i < 3; ++i) {
    go[i] = c * T(-2) * K.w_pos * K.d_pos[i] * K.d_pos[i] * o[i];
    go[3 + i] = c * T(-2) * K.w_att * o[3 + i];
    go[6 + i] = T(0);
    go[9 + i] = c * T(-2) * K.w_vel * o[9 + i];
  }
  for (int j = 0; j < 6; ++j) {
    const T m = c * T(2) * K.w_mavg * (u[j] - ab[j]);
    gu[j] -= m + (j >= 3 ? c * T(2) * K.w_act * u[j] : T(0));
    gab[j] += m;
  }
}

// Body wrench of the clipped action u: tau = (f_max u_0:3, tau_max u_3:6).
template <class T>
AUV_HD void wrench(const Task<T>& K, const T u[6], T tau[6]) {
  for (int i = 0; i < 3; ++i) {
    tau[i] = K.f_max * u[i];
    tau[3 + i] = K.tau_max * u[3 + i];
  }
}

}  // namespace adj
}  // namespace auv
