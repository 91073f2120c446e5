// Environment step with four lanes per environment ("quad" layout) for the fused policy
// rollout, so that a workgroup's four waves share the physics of its 64 environments.
//
// Lane l serves environment slot l / 4 of its wave and component c = l % 4: lanes c = 0,
// 1, 2 hold the x, y, z components of every 3-vector (p, v, omega, and derived vectors)
// and the vector part of the quaternion; lane 3 holds the quaternion's scalar part and
// zero in every 3-vector.  Cross products and dot products across the four lanes use DPP
// quad permutations (no LDS, no waits).  The arithmetic is the same as the one-lane-per-
// environment form in auv_device.hpp; only its distribution over lanes differs.
#pragma once

#include "auv_device.hpp"

namespace auv {
namespace quad {

constexpr int QP(int a, int b, int c, int d) { return a | (b << 2) | (c << 4) | (d << 6); }
constexpr int P1 = QP(1, 2, 0, 3);    // lane c reads component c+1 (mod 3)
constexpr int P2 = QP(2, 0, 1, 3);    // lane c reads component c+2 (mod 3)
constexpr int SW1 = QP(1, 0, 3, 2), SW2 = QP(2, 3, 0, 1);
constexpr int BC0 = QP(0, 0, 0, 0), BC1 = QP(1, 1, 1, 1), BC2 = QP(2, 2, 2, 2), BC3 = QP(3, 3, 3, 3);
constexpr int XE1 = QP(0, 2, 1, 3);   // (e x e1) = (0, e_z, -e_y)
constexpr int XE2 = QP(2, 1, 0, 3);   // (e x e2) = (-e_z, 0, e_x)

template <int C>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), C, 0xF, 0xF, true));
}

// sum over the four lanes of a quad, every lane gets it.  Not contracted with the product
// that usually feeds it: an fma would need the swapped value as its own moved operand.
__device__ __forceinline__ float qsum(float x) {
#pragma clang fp contract(off)
  x += dpp<SW1>(x);
  return x + dpp<SW2>(x);
}

struct Perm { float p1, p2; };
__device__ __forceinline__ Perm perm(float x) { return Perm{dpp<P1>(x), dpp<P2>(x)}; }
// (a x b)_c = a_{c+1} b_{c+2} - a_{c+2} b_{c+1}, b given by its two rotations
__device__ __forceinline__ float cross(float a, const Perm& b) { return dpp<P1>(a) * b.p2 - dpp<P2>(a) * b.p1; }

// Per-lane constants of the layout.
struct QK {
  int c;
  float m3;    // 1 in vector lanes, 0 in lane 3
  float m3x2;  // 2 m3
  float d2;    // e3 (1 in lane 2)
  float sx1;   // sign pattern of e x e1: (0, +1, -1, 0)
  float sx2;   // sign pattern of e x e2: (-1, 0, +1, 0)
  float e1, e2;
  float hm3;   // 1/2 in vector lanes
  float hs3;   // -1/2 in lane 3
};

__device__ __forceinline__ QK make_qk(int lane) {
  QK K;
  K.c = lane & 3;
  K.m3 = K.c < 3 ? 1.0f : 0.0f;
  K.m3x2 = 2.0f * K.m3;
  K.d2 = K.c == 2 ? 1.0f : 0.0f;
  K.e1 = K.c == 0 ? 1.0f : 0.0f;
  K.e2 = K.c == 1 ? 1.0f : 0.0f;
  K.sx1 = K.c == 1 ? 1.0f : (K.c == 2 ? -1.0f : 0.0f);
  K.sx2 = K.c == 0 ? -1.0f : (K.c == 2 ? 1.0f : 0.0f);
  K.hm3 = 0.5f * K.m3;
  K.hs3 = K.c == 3 ? -0.5f : 0.0f;
  return K;
}

// Per-lane (component c) model constants of one environment; zero in lane 3.  Indices of
// the neighbouring components are taken mod 3 (c+1, c+2).
struct QModel {
  float iMlin;                       // 1 / (m + added mass), linear DOF c
  float KA1, KA2n;                   // Mlin_c / Mlin_{c+2}, -Mlin_c / Mlin_{c+1}
  float DLi, DQi, BmWi;              // linear damping and (B - W), divided by Mlin_c
  float Mang, iMang, A1, DLa, DQa;   // angular DOF c; A1 = linear added mass (Munk term)
  float cw, cw1, cw2;                // world current, its components c+1 and c+2
  float Brb1, Brb2n;                 // (B r_b)_{c+1}, -(B r_b)_{c+2}
};

// Per-lane reference data: lanes 0-2 the Lissajous position component (in turns), lane 3
// the yaw ramp (psi / 4 pi, in turns); goal pose in quad layout.
struct QRef {
  float pg, amp, fr, ph;   // p_goal_c, A_c, f_c [turns / s], phase_c / 2 pi  (lane 3: 0, 0, yaw rate / 4 pi, yaw0 / 4 pi)
  float qg;                // goal quaternion, quad layout
};

// Component c of (x0, x1, x2) with x3 in lane 3, by 0/1 weights (arithmetic rather than an
// index, which would put the source arrays in scratch memory).
__device__ __forceinline__ float pick(const QK& K, float x0, float x1, float x2, float x3) {
  const float w0 = K.c == 0 ? 1.0f : 0.0f, w1 = K.c == 1 ? 1.0f : 0.0f, w2 = K.c == 2 ? 1.0f : 0.0f;
  return __builtin_fmaf(w0, x0, __builtin_fmaf(w1, x1, __builtin_fmaf(w2, x2, (1.0f - K.m3) * x3)));
}

// Scalar (one-lane) parameters -> this lane's model and reference constants.  PAPER: the
// paper task's weight gamma W (gamma in parameter row 13) and the buoyancy centre at the
// centre of gravity (no restoring moment).
template <bool PAPER = false>
__device__ __forceinline__ void make_lane_consts(const VehArgs& V, const QK& K, const Params& P, QModel& M,
                                                 QRef& F) {
  Model S;
  make_model(V, P, S);
  // component c, c+1 and c+2 (mod 3) of a 3-vector given by its three entries
  auto c0 = [&](const float* x) { return pick(K, x[0], x[1], x[2], 0.0f); };
  auto c1 = [&](const float* x) { return pick(K, x[1], x[2], x[0], 0.0f); };
  auto c2 = [&](const float* x) { return pick(K, x[2], x[0], x[1], 0.0f); };
  M.iMlin = c0(S.iMlin);
  M.KA1 = c0(S.Mlin) * c2(S.iMlin);
  M.KA2n = -(c0(S.Mlin) * c1(S.iMlin));
  M.DLi = c0(S.DL) * M.iMlin;
  M.DQi = c0(S.DQ) * M.iMlin;
  M.BmWi = (PAPER ? __builtin_fmaf(-P.amp[0], V.W, V.B) : V.BmW) * M.iMlin;
  M.Mang = c0(S.Mang);
  M.iMang = c0(S.iMang);
  M.A1 = c0(S.A1);
  M.DLa = c0(S.DL + 3);
  M.DQa = c0(S.DQ + 3);
  M.cw = c0(P.cw);
  M.cw1 = c1(P.cw);
  M.cw2 = c2(P.cw);
  M.Brb1 = PAPER ? 0.0f : c1(V.Brb);
  M.Brb2n = PAPER ? 0.0f : -c2(V.Brb);
  constexpr float INV_2PI = 0.159154943091895336f, INV_4PI = 0.0795774715459476679f;
  F.pg = pick(K, P.pg[0], P.pg[1], P.pg[2], 0.0f);
  F.amp = pick(K, P.amp[0], P.amp[1], P.amp[2], 0.0f);
  F.fr = pick(K, P.freq[0], P.freq[1], P.freq[2], P.yaw_rate * INV_4PI);
  F.ph = pick(K, P.phase[0] * INV_2PI, P.phase[1] * INV_2PI, P.phase[2] * INV_2PI, P.yaw0 * INV_4PI);
  F.qg = pick(K, P.qg[1], P.qg[2], P.qg[3], P.qg[0]);
}

// ------------------------------------------------------------ Fossen right side ----
// Same equations as auv::rhs, one component per lane.  Rotation by the stage quaternion
// (w, e), not renormalised: R x = s x + 2 (e.x) e + 2 w (e x x) and R^T x = s x +
// 2 (e.x) e - 2 w (e x x) with s = 1 - 2 e.e (the Euler-Rodrigues matrix I + 2 w S(e) +
// 2 S(e)^2 applied to a vector).
//
// Cross products cost no lane moves of their own: with P1, P2 the quad permutations that
// read component c+1, c+2,  x x y = P1(x . P1 y) - P2(x . P2 y)  (elementwise products);
// the permutations are linear, and a per-component factor f moves inside them as
// f . P1(z) = P1(z . P2 f), f . P2(z) = P2(z . P1 f).  So each output that is a sum of
// cross products (scaled or not) takes one P1 and one P2, fused into its final adds.  The
// force equation is divided by the mass first (tfi = tau_f / Mlin and the constants of
// QModel), so that its cross product and the current's c_b x w share those two moves.
__device__ __forceinline__ void rhs(const QK& K, const QModel& M, float tfi, float tm, float q, float v,
                                    float om, float& dp, float& dq, float& dv, float& dw) {
  const float e = q * K.m3;
  const float E2 = q * K.m3x2;                        // 2 e
  const float wb = dpp<BC3>(q);                       // w in every lane
  const float e1 = dpp<P1>(e), e2 = dpp<P2>(e);       // e_{c+1}, e_{c+2}
  const float wb2 = wb + wb;
  const float g1 = wb2 * e1, g2 = wb2 * e2;
  const float s = __builtin_fmaf(-2.0f, qsum(e * e), 1.0f);
  // dp = R v, with 2 w (e x v) = P2(g2 v) - P1(g1 v)
  dp = __builtin_fmaf(qsum(E2 * v), e, s * v) + dpp<P2>(g2 * v) + dpp<P1>(-(g1 * v));
  // c_b = R^T c_w, with e x c_w = e1 cw2 - e2 cw1
  float cb = __builtin_fmaf(qsum(E2 * M.cw), e, s * M.cw);
  cb = __builtin_fmaf(-g1, M.cw2, cb);
  cb = __builtin_fmaf(g2, M.cw1, cb);
  // k = R^T e3, with e x e3 = (e_y, -e_x, 0) = e1 [c = 0] - e2 [c = 1]
  float k = __builtin_fmaf(dpp<BC2>(E2), e, s * K.d2);
  k = __builtin_fmaf(-g1, K.e1, k);
  k = __builtin_fmaf(g2, K.e2, k);
  const float vr = v - cb;
  const float w1 = dpp<P1>(om), w2 = dpp<P2>(om);
  const float r1 = dpp<P1>(vr), r2 = dpp<P2>(vr);
  // dv = (tau_f + (Mlin vr) x w - (DL + DQ |vr|) vr - (B - W) k) / Mlin + c_b x w
  const float al = w1 * __builtin_fmaf(vr, M.KA1, cb);
  const float be = w2 * __builtin_fmaf(vr, M.KA2n, -cb);
  float fb = __builtin_fmaf(-__builtin_fmaf(M.DQi, fabsf(vr), M.DLi), vr, tfi);
  fb = __builtin_fmaf(-M.BmWi, k, fb);
  dv = fb + dpp<P1>(al) + dpp<P2>(be);
  // dw = (tau_m + (Mang w) x w + (A1 vr) x vr + k x (B r_b) - (DL + DQ |w|) w) / Mang
  const float b = M.Mang * om;
  const float a1 = M.A1 * vr;
  const float ga = __builtin_fmaf(k, M.Brb1, __builtin_fmaf(a1, r1, b * w1));
  const float gb = __builtin_fmaf(k, M.Brb2n, __builtin_fmaf(-a1, r2, -(b * w2)));
  const float G = __builtin_fmaf(-__builtin_fmaf(M.DQa, fabsf(om), M.DLa), om, tm);
  dw = (G + dpp<P1>(ga) + dpp<P2>(gb)) * M.iMang;
  // dq = 1/2 q (x) (0, w): vector part 1/2 (w om + e x om), scalar part -1/2 e.om
  const float exo = __builtin_fmaf(e1, w2, -(e2 * w1));
  dq = __builtin_fmaf(K.hs3, qsum(e * om), K.hm3 * __builtin_fmaf(wb, om, exo));
}

// One RK4 substep of length h with the wrench held (tfi = tau_f / Mlin), given the
// derivative (dp, dq, dv, dw) at the substep's start.
__device__ __forceinline__ void rk4_from(const QK& K, const QModel& M, float tfi, float tm, float h, float& p,
                                         float& q, float& v, float& om, float dp, float dq, float dv, float dw) {
  float ap = dp, aq = dq, av = dv, aw = dw;
#pragma unroll
  for (int stage = 1; stage < 4; ++stage) {
    const float cs = (stage == 3) ? h : 0.5f * h;
    rhs(K, M, tfi, tm, __builtin_fmaf(cs, dq, q), __builtin_fmaf(cs, dv, v), __builtin_fmaf(cs, dw, om), dp, dq, dv,
        dw);
    const float wgt = (stage == 3) ? 1.0f : 2.0f;
    ap = __builtin_fmaf(wgt, dp, ap);
    aq = __builtin_fmaf(wgt, dq, aq);
    av = __builtin_fmaf(wgt, dv, av);
    aw = __builtin_fmaf(wgt, dw, aw);
  }
  const float h6 = h * (1.0f / 6.0f);
  p = __builtin_fmaf(h6, ap, p);
  q = __builtin_fmaf(h6, aq, q);
  v = __builtin_fmaf(h6, av, v);
  om = __builtin_fmaf(h6, aw, om);
  q *= rsqrtf(qsum(q * q));
}

__device__ __forceinline__ void rk4(const QK& K, const QModel& M, float tfi, float tm, float h, float& p, float& q,
                                    float& v, float& om) {
  float dp, dq, dv, dw;
  rhs(K, M, tfi, tm, q, v, om, dp, dq, dv, dw);
  rk4_from(K, M, tfi, tm, h, p, q, v, om, dp, dq, dv, dw);
}

// --------------------------------------------------- reference, observation ----------
__device__ __forceinline__ void reference(const EnvArgs& E, const QK& K, const QRef& F, int ep_step, float& pr,
                                          float& qr) {
  if (E.flags & F_LISSAJOUS) {
    const float t = (float)ep_step * E.dt;
    float s, c;
    sincos_turns(__builtin_fmaf(F.fr, t, F.ph), &s, &c);
    pr = K.m3 * __builtin_fmaf(F.amp, s, F.pg);
    const float sy = dpp<BC3>(s), cy = dpp<BC3>(c);
    qr = K.c == 3 ? cy : (K.c == 2 ? sy : 0.0f);
  } else {
    pr = F.pg;
    qr = F.qg;
  }
}

// Rotation helpers for a quaternion in quad layout.
struct QRot { float e, wb, s; Perm eP; };
__device__ __forceinline__ QRot qrot(const QK& K, float q) {
  QRot r;
  r.e = q * K.m3;
  r.wb = dpp<BC3>(q);
  r.s = __builtin_fmaf(-2.0f, qsum(r.e * r.e), 1.0f);
  r.eP = perm(r.e);
  return r;
}
__device__ __forceinline__ float rot_T(const QRot& r, float x) {   // R^T x
  const float ex = qsum(r.e * x);
  return __builtin_fmaf(r.s, x, 2.0f * __builtin_fmaf(ex, r.e, r.wb * cross(x, r.eP)));
}

// Columns 0 and 1 of the reference rotation R(q_ref), this lane's component:
// R_ref e1 = s e1 + 2 e_x e + 2 w (e x e1), likewise for e2.  Depends only on the reference.
struct QRefCols { float r0, r1; };
__device__ __forceinline__ QRefCols ref_columns(const QK& K, float qr) {
  const QRot Rr = qrot(K, qr);
  QRefCols o;
  o.r0 = __builtin_fmaf(Rr.s, K.e1, 2.0f * __builtin_fmaf(dpp<BC0>(Rr.e), Rr.e, Rr.wb * dpp<XE1>(Rr.e) * K.sx1));
  o.r1 = __builtin_fmaf(Rr.s, K.e2, 2.0f * __builtin_fmaf(dpp<BC1>(Rr.e), Rr.e, Rr.wb * dpp<XE2>(Rr.e) * K.sx2));
  return o;
}

// Observation components of this lane (body-frame position error and the body-frame
// reference columns) and |dp|.
struct QObs { float dpb, c0, c1; };
__device__ __forceinline__ void observe(const QK& K, float p, float q, float pr, const QRefCols& rc, QObs& o,
                                        float& dist) {
  const QRot R = qrot(K, q);
  o.dpb = rot_T(R, pr - p);
  o.c0 = rot_T(R, rc.r0);
  o.c1 = rot_T(R, rc.r1);
  dist = sqrtf(qsum(o.dpb * o.dpb));
}

// Attitude-error angle 2 atan2(|vec(q_err)|, |scalar(q_err)|) of q_err = q^* (x) q_ref:
// scalar w wr + e.er, vector w er - wr e - e x er.
__device__ __forceinline__ float attitude_error(const QK& K, float q, float qr) {
  const float e = q * K.m3, er = qr * K.m3;
  const float wb = dpp<BC3>(q), wr = dpp<BC3>(qr);
  const float ew = qsum(q * qr);
  const float vec = __builtin_fmaf(wb, er, -wr * e) - cross(e, perm(er));
  return 2.0f * atan2f(sqrtf(qsum(vec * vec)), fabsf(ew));
}

// Observation of the paper task: body-frame position error and the rotation vector of
// q_err = q^* (x) q_ref (shortest rotation: the sign of the scalar part folded in), this
// lane's components in o.dpb and o.c0; |dp| in dist.
__device__ __forceinline__ void observe_paper(const QK& K, float p, float q, float pr, float qr, QObs& o,
                                              float& dist) {
  const QRot R = qrot(K, q);
  o.dpb = rot_T(R, pr - p);
  const float e = R.e, er = qr * K.m3;
  const float wr = dpp<BC3>(qr);
  const float ew = qsum(q * qr);                                   // scalar part of q_err
  const float vec = __builtin_fmaf(R.wb, er, -wr * e) - cross(e, perm(er));
  const float n = sqrtf(qsum(vec * vec)), aw = fabsf(ew);
  const float k = n > 0.0f ? 2.0f * atan2f(n, aw) / n : 2.0f / aw;
  o.c0 = (ew < 0.0f ? -k : k) * vec;
  o.c1 = 0.0f;
  dist = sqrtf(qsum(o.dpb * o.dpb));
}

// Reward of the paper task from the post-step observation (dp_b, rotation vector, omega),
// this lane's clipped force / torque commands (uf, ut: components c and 3 + c) and their
// moving averages before this step (af, at); lane 3 holds zeros.  dc = D_c.
__device__ __forceinline__ float paper_reward(const TaskArgs& T, float dc, const QObs& o, float om, float uf,
                                              float ut, float af, float at) {
  const float dpw = dc * o.dpb, df = uf - af, dt = ut - at;
  const float pos = qsum(dpw * dpw), att = qsum(o.c0 * o.c0), act = qsum(ut * ut), vel = qsum(om * om);
  const float mavg = qsum(__builtin_fmaf(df, df, dt * dt));
  return -T.w_pos * pos - T.w_att * att - T.w_act * act - T.w_vel * vel - T.w_mavg * mavg;
}

// Clip this lane's two actions, broadcast all eight across the quad, body wrench with
// this lane's force and moment rows Tf, Tm of the allocation table (f_max folded in).
__device__ __forceinline__ void wrench(const float Tf[8], const float Tm[8], float a0, float a1, float& u0,
                                       float& u1, float& tf, float& tm, float& usq) {
  u0 = fminf(fmaxf(a0, -1.0f), 1.0f);
  u1 = fminf(fmaxf(a1, -1.0f), 1.0f);
  const float u[8] = {dpp<BC0>(u0), dpp<BC0>(u1), dpp<BC1>(u0), dpp<BC1>(u1),
                      dpp<BC2>(u0), dpp<BC2>(u1), dpp<BC3>(u0), dpp<BC3>(u1)};
  float f = 0.0f, m = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    f = __builtin_fmaf(Tf[j], u[j], f);
    m = __builtin_fmaf(Tm[j], u[j], m);
  }
  tf = f;
  tm = m;
  usq = qsum(__builtin_fmaf(u0, u0, u1 * u1));
}


// ------------------------------------------------------ allocation table in LDS ----
// Rows c = 0..2: force row c, rows 4 + c: moment row c, each x f_max; rows 3 and 7 zero
// (lane 3 of a quad reads them).  Written by the first 64 threads of the block.
__device__ __forceinline__ void stage_alloc(const VehArgs& V, float (*alloc)[8], int tid) {
  if (tid < 64) {
    const int row = tid >> 3, j = tid & 7;
    const int src = row < 3 ? row : (row >= 4 && row < 7 ? row - 1 : -1);
    alloc[row][j] = src >= 0 ? V.alloc[src * 8 + j] * V.f_max : 0.0f;
  }
}

__device__ __forceinline__ void alloc_rows(const float (*alloc)[8], int c, float Tf[8], float Tm[8]) {
  typedef float f4 __attribute__((ext_vector_type(4)));
  *reinterpret_cast<f4*>(&Tf[0]) = *reinterpret_cast<const f4*>(&alloc[c][0]);
  *reinterpret_cast<f4*>(&Tf[4]) = *reinterpret_cast<const f4*>(&alloc[c][4]);
  *reinterpret_cast<f4*>(&Tm[0]) = *reinterpret_cast<const f4*>(&alloc[4 + c][0]);
  *reinterpret_cast<f4*>(&Tm[4]) = *reinterpret_cast<const f4*>(&alloc[4 + c][4]);
}

// ------------------------------------------------- one environment, quad layout ----
// What a lane holds of its environment between control steps.  Observation rows of the
// environment: 0-2 dp_b, 3-5 and 6-8 the two reference columns, 9-11 v, 12-14 omega,
// 15-22 the previous clipped action (lane c: rows 15 + 2c, 16 + 2c).
struct QEnv {
  float p, q, v, om;   // position, quaternion (lane 3: scalar part), body velocities
  float u0, u1;        // this lane's two components of the previous clipped action
  int ep;              // control steps into the episode
  uint32_t episode;
  QObs ob;
};

// Buffers of environment i -> lane; an idle environment (i >= n) gets a harmless dummy
// vehicle at rest that is stepped but never stored.  PAPER: observation rows 0-2 dp_b, 3-5
// rotation vector, 6-8 v, 9-11 omega, 12-14 / 15-17 the moving averages of the force /
// torque commands (state, kept in u0 / u1 of lanes 0-2).
template <bool PAPER = false>
__device__ __forceinline__ void load_env(const VehArgs& V, const EnvArgs& E, const QK& K, int i, bool valid,
                                         QEnv& X, QModel& M, QRef& F) {
  const int c = K.c, cv = c < 3 ? c : 0;   // cv: a valid row for lane 3's loads
  const size_t N = (size_t)E.n;
  Params P;
  if (valid) {
    X.p = c < 3 ? E.state[cv * N + i] : 0.0f;
    X.q = E.state[(c < 3 ? 4 + c : 3) * N + i];
    X.v = c < 3 ? E.state[(7 + cv) * N + i] : 0.0f;
    X.om = c < 3 ? E.state[(10 + cv) * N + i] : 0.0f;
    load_params(E.params, E.n, i, P);
    X.ep = E.ep_step[i];
    X.episode = E.episode[i];
    X.ob.dpb = c < 3 ? E.obs[cv * N + i] : 0.0f;
    X.ob.c0 = c < 3 ? E.obs[(3 + cv) * N + i] : 0.0f;
    if (PAPER) {
      X.ob.c1 = 0.0f;
      X.u0 = c < 3 ? E.obs[(12 + cv) * N + i] : 0.0f;
      X.u1 = c < 3 ? E.obs[(15 + cv) * N + i] : 0.0f;
    } else {
      X.ob.c1 = c < 3 ? E.obs[(6 + cv) * N + i] : 0.0f;
      X.u0 = E.obs[(15 + 2 * c) * N + i];
      X.u1 = E.obs[(16 + 2 * c) * N + i];
    }
  } else {
    X.p = X.v = X.om = X.u0 = X.u1 = 0.0f;
    X.q = c == 3 ? 1.0f : 0.0f;
    X.ep = 0;
    X.episode = 0;
    P = Params{{1, 1, 1}, {0, 0, 0}, {0, 0, 0}, {1, 0, 0, 0}, {0, 0, 0}, {0, 0, 0}, {0, 0, 0}, 0, 0};
    X.ob = QObs{0, 0, 0};
  }
  make_lane_consts<PAPER>(V, K, P, M, F);
}

// The observation of X into rows k of obs[k * stride + at].  PAPER: the 12 observation
// rows, then with `state` the moving-average rows 12-17, else zeros in rows 12-22.
template <bool PAPER = false>
__device__ __forceinline__ void store_obs(float* __restrict__ obs, size_t stride, size_t at, int c, const QEnv& X,
                                          bool state = true) {
  if (PAPER) {   // a record (state false) gets zeros in rows 12-22
    if (c < 3) {
      obs[c * stride + at] = X.ob.dpb;
      obs[(3 + c) * stride + at] = X.ob.c0;
      obs[(6 + c) * stride + at] = X.v;
      obs[(9 + c) * stride + at] = X.om;
      obs[(12 + c) * stride + at] = state ? X.u0 : 0.0f;
      obs[(15 + c) * stride + at] = state ? X.u1 : 0.0f;
      if (!state) obs[(18 + c) * stride + at] = 0.0f;
    } else if (!state) {
      obs[21 * stride + at] = 0.0f;
      obs[22 * stride + at] = 0.0f;
    }
    return;
  }
  if (c < 3) {
    obs[c * stride + at] = X.ob.dpb;
    obs[(3 + c) * stride + at] = X.ob.c0;
    obs[(6 + c) * stride + at] = X.ob.c1;
    obs[(9 + c) * stride + at] = X.v;
    obs[(12 + c) * stride + at] = X.om;
  }
  obs[(15 + 2 * c) * stride + at] = X.u0;
  obs[(16 + 2 * c) * stride + at] = X.u1;
}

// Non-finite state components of the quad's environment held by this lane: p, v, omega
// components in lanes 0-2, the quaternion component in every lane (13 per environment).
__device__ __forceinline__ uint32_t nonfinite_quad(int c, const QEnv& X) {
  const uint32_t vec = nonfinite(X.p) + nonfinite(X.v) + nonfinite(X.om);
  return (c < 3 ? vec : 0u) + nonfinite(X.q);
}

// The 13 state rows of X into s[k * stride + at] (p, q = (w, x, y, z), v, omega).
__device__ __forceinline__ void store_state(float* __restrict__ s, size_t stride, size_t at, int c, const QEnv& X) {
  if (c < 3) {
    s[c * stride + at] = X.p;
    s[(7 + c) * stride + at] = X.v;
    s[(10 + c) * stride + at] = X.om;
  }
  s[(c < 3 ? 4 + c : 3) * stride + at] = X.q;
}

// Lane -> buffers of environment i (state, current observation, counters).
template <bool PAPER = false>
__device__ __forceinline__ void store_env(const EnvArgs& E, int c, int i, const QEnv& X) {
  const size_t N = (size_t)E.n;
  store_state(E.state, N, (size_t)i, c, X);
  store_obs<PAPER>(E.obs, N, (size_t)i, c, X);
  if (c == 0) {
    E.ep_step[i] = X.ep;
    E.episode[i] = X.episode;
  }
}

// Auto-reset of a finished episode (the whole quad calls it): fresh draws for the next
// episode, step 0, previous action 0, and the observation of the new initial state
// (pr, qr, rc: its reference).  The new parameters are stored at once.
template <bool PAPER = false>
__device__ __forceinline__ void new_episode(const VehArgs& V, const EnvArgs& E, const QK& K, uint32_t gid, int i,
                                            bool valid, QEnv& X, QModel& M, QRef& F, float& pr, float& qr,
                                            QRefCols& rc, float& dist) {
  X.episode += 1u;
  State xs;
  Params P;
  if (PAPER)
    paper_reset_draws(E, gid, X.episode, xs, P);
  else
    reset_draws(E, gid, X.episode, xs, P);
  make_lane_consts<PAPER>(V, K, P, M, F);
  if (valid && K.c == 0) store_params(E.params, E.n, i, P);
  X.ep = 0;
  X.p = pick(K, xs.p[0], xs.p[1], xs.p[2], 0.0f);
  X.q = pick(K, xs.q[1], xs.q[2], xs.q[3], xs.q[0]);
  X.v = X.om = 0.0f;
  X.u0 = X.u1 = 0.0f;
  reference(E, K, F, 0, pr, qr);
  if (PAPER) {
    observe_paper(K, X.p, X.q, pr, qr, X.ob, dist);
  } else {
    rc = ref_columns(K, qr);
    observe(K, X.p, X.q, pr, rc, X.ob, dist);
  }
}

}  // namespace quad
}  // namespace auv
