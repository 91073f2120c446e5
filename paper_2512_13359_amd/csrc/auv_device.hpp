// Device-side building blocks of the rollout step, one lane per environment, fp32,
// everything in registers: Philox draws, reset / domain randomisation, the Fossen
// right-hand side in expanded cross-product form, RK4, reference, observation, reward.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace auv {

// ---------------------------------------------------------------- launch arguments --
struct VehArgs {
  float m, inertia[3], added_mass[6], lin_damp[6], quad_damp[6];
  float BmW;     // B - W
  float Brb[3];  // B * r_b
  float B, W;    // buoyancy and weight (the paper task scales W per environment)
  float f_max;
  float alloc[48];
};

// The paper's own training task (selected by EnvArgs::task): normalised 6-D body wrench,
// five-term reward with an exponential moving average of past actions, gravity factor
// per environment, goal attitude from Euler angles.
struct TaskArgs {
  float f_max, tau_max;                 // wrench at |u| = 1 (N, N m)
  float w_pos, d_pos[3], w_att, w_act, w_vel, w_mavg;
  float beta;                           // moving average: abar <- beta abar + (1 - beta) u
  float g_lo, g_span;                   // gravity factor U[g_lo, g_lo + g_span]
  float eul_lo, eul_span;               // goal roll, pitch, yaw U[eul_lo, eul_lo + eul_span]
};
constexpr uint32_t TASK_WORKLOAD = 0, TASK_PAPER = 1;

struct EnvArgs {
  float* state;
  float* params;
  int32_t* ep_step;
  uint32_t* episode;
  float* obs;
  int32_t n, substeps, H;
  float dt, h;
  uint32_t key0, key1, flags, env_offset;
  uint32_t sync_polls;   // bound on the polls of one inter-wave wait (fused policy rollout)
  uint32_t task;         // TASK_WORKLOAD or TASK_PAPER
  TaskArgs tk;
  uint32_t* status;      // [2] or null: non-finite state components seen, abandoned waits
};

// Per-step output pointers of the environment loops; any may be null.
struct StepOut {
  float* obs;          // [23][T][N] observation each action was chosen on
  float* act;          // [8][T][N] action before clipping (input in external mode)
  float* logp;         // [T][N] log-prob of the sampled action
  float* reward;       // [T][N]
  float* done;         // [T][N] as 0 / 1
  uint8_t* done_u8;    // [N] (single-step form)
  float* traj;         // [13][T+1][N]
  float* stats_work;   // [3][G][T] per-group partial sums
};

constexpr uint32_t F_DR = 1, F_CURRENT = 2, F_LISSAJOUS = 4, F_STAGGER = 8;
constexpr int OBS = 23, ACT = 8, NS = 13, NP = 24;

// ------------------------------------------------------------------------ Philox ----
// Philox4x32-10 (Salmon et al., SC'11): ten rounds of two 32x32->64 products, key
// bumped by the Weyl constants between rounds.
struct U4 { uint32_t x, y, z, w; };

__device__ __forceinline__ U4 philox(U4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    const uint32_t lo0 = 0xD2511F53u * c.x, hi0 = __umulhi(0xD2511F53u, c.x);
    const uint32_t lo1 = 0xCD9E8D57u * c.z, hi1 = __umulhi(0xCD9E8D57u, c.z);
    c = U4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
  }
  return c;
}

// top 24 bits -> [0, 1), exact
__device__ __forceinline__ float u01(uint32_t w) { return (float)(w >> 8) * 0x1p-24f; }
// top 24 bits + 1 -> (0, 1], exact
__device__ __forceinline__ float u01_open0(uint32_t w) { return (float)((w >> 8) + 1u) * 0x1p-24f; }
// lo + span * u rounded once
__device__ __forceinline__ float affine(float lo, float span, float u) { return __builtin_fmaf(span, u, lo); }

// -------------------------------------------------------------- per-env data -------
struct State { float p[3], q[4], v[3], w[3]; };

struct Params {
  float s[3];       // mass, added-mass, damping scales
  float cw[3];      // world current
  float pg[3], qg[4];
  float amp[3], freq[3], phase[3];
  float yaw_rate, yaw0;
};

// Derived per-env model constants (recomputed whenever params change).
struct Model {
  float Mlin[3], Mang[3];    // m' + A_lin, I' + A_ang
  float iMlin[3], iMang[3];  // reciprocals
  float A1[3];               // linear added mass
  float DL[6], DQ[6];
};

// Every product is rounded before it is added (no contraction): the constants are built at
// more than one place in a kernel (load and in-kernel reset), and a fused multiply-add
// chosen differently at each would make a resumed run differ from an uninterrupted one.
__device__ __forceinline__ void make_model(const VehArgs& V, const Params& P, Model& M) {
#pragma clang fp contract(off)
  const float m = P.s[0] * V.m;
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    M.A1[i] = P.s[1] * V.added_mass[i];
    M.Mlin[i] = m + M.A1[i];
    M.Mang[i] = P.s[0] * V.inertia[i] + P.s[1] * V.added_mass[3 + i];
    M.iMlin[i] = 1.0f / M.Mlin[i];
    M.iMang[i] = 1.0f / M.Mang[i];
  }
#pragma unroll
  for (int i = 0; i < 6; ++i) {
    M.DL[i] = P.s[2] * V.lin_damp[i];
    M.DQ[i] = P.s[2] * V.quad_damp[i];
  }
}

// ------------------------------------------------------------------ rotations ------
struct Rot { float r[3][3]; };

// R(q) = I + 2 eta S(eps) + 2 S(eps)^2 written out (also applied to stage quaternions)
__device__ __forceinline__ Rot rot_of(const float q[4]) {
  const float w = q[0], x = q[1], y = q[2], z = q[3];
  const float xx = x * x, yy = y * y, zz = z * z;
  const float xy = x * y, xz = x * z, yz = y * z, wx = w * x, wy = w * y, wz = w * z;
  Rot R;
  R.r[0][0] = 1.0f - 2.0f * (yy + zz); R.r[0][1] = 2.0f * (xy - wz); R.r[0][2] = 2.0f * (xz + wy);
  R.r[1][0] = 2.0f * (xy + wz); R.r[1][1] = 1.0f - 2.0f * (xx + zz); R.r[1][2] = 2.0f * (yz - wx);
  R.r[2][0] = 2.0f * (xz - wy); R.r[2][1] = 2.0f * (yz + wx); R.r[2][2] = 1.0f - 2.0f * (xx + yy);
  return R;
}

// ------------------------------------------------------------ Fossen right side ----
// d/dt of (p, q, v, omega) for wrench tau (body), world current cw.  Relative-velocity
// form: v_r = v - R^T cw;
//   (M_RB + M_A) dnu_r = tau - [m' w x v_r + w x (A1 v_r) ; w x (I' w) + v_r x (A1 v_r)
//                        + w x (A2 w)] - D(nu_r) nu_r - g(q)
//   dv = dv_r + (R^T cw) x w,  dp = R v,  dq = 1/2 q (x) (0, w).
struct Deriv { float p[3], q[4], v[3], w[3]; };

__device__ __forceinline__ void rhs(const VehArgs& V, const Model& M, const float cw[3],
                                    const float tau[6], const float q[4], const float v[3],
                                    const float w[3], Deriv& d) {
  const Rot R = rot_of(q);
  d.p[0] = R.r[0][0] * v[0] + R.r[0][1] * v[1] + R.r[0][2] * v[2];
  d.p[1] = R.r[1][0] * v[0] + R.r[1][1] * v[1] + R.r[1][2] * v[2];
  d.p[2] = R.r[2][0] * v[0] + R.r[2][1] * v[1] + R.r[2][2] * v[2];
  float cb[3];
#pragma unroll
  for (int i = 0; i < 3; ++i) cb[i] = R.r[0][i] * cw[0] + R.r[1][i] * cw[1] + R.r[2][i] * cw[2];
  const float k[3] = {R.r[2][0], R.r[2][1], R.r[2][2]};   // R^T e3
  float vr[3];
#pragma unroll
  for (int i = 0; i < 3; ++i) vr[i] = v[i] - cb[i];
  // linear: tau_f - w x (Mlin vr) - (DL + DQ|vr|) vr - (B - W) k
  float a[3];
#pragma unroll
  for (int i = 0; i < 3; ++i) a[i] = M.Mlin[i] * vr[i];
  float F[3];
  F[0] = tau[0] - (w[1] * a[2] - w[2] * a[1]);
  F[1] = tau[1] - (w[2] * a[0] - w[0] * a[2]);
  F[2] = tau[2] - (w[0] * a[1] - w[1] * a[0]);
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    F[i] -= (M.DL[i] + M.DQ[i] * fabsf(vr[i])) * vr[i];
    F[i] -= V.BmW * k[i];
  }
  // angular: tau_m - w x (Mang w) - vr x (A1 vr) - (DL + DQ|w|) w - B r_b x k
  float b[3], c[3];
#pragma unroll
  for (int i = 0; i < 3; ++i) { b[i] = M.Mang[i] * w[i]; c[i] = M.A1[i] * vr[i]; }
  float G[3];
  G[0] = tau[3] - (w[1] * b[2] - w[2] * b[1]) - (vr[1] * c[2] - vr[2] * c[1]);
  G[1] = tau[4] - (w[2] * b[0] - w[0] * b[2]) - (vr[2] * c[0] - vr[0] * c[2]);
  G[2] = tau[5] - (w[0] * b[1] - w[1] * b[0]) - (vr[0] * c[1] - vr[1] * c[0]);
  G[0] -= V.Brb[1] * k[2] - V.Brb[2] * k[1];
  G[1] -= V.Brb[2] * k[0] - V.Brb[0] * k[2];
  G[2] -= V.Brb[0] * k[1] - V.Brb[1] * k[0];
#pragma unroll
  for (int i = 0; i < 3; ++i) G[i] -= (M.DL[3 + i] + M.DQ[3 + i] * fabsf(w[i])) * w[i];
  // accelerations; current term (R^T cw) x w
  d.v[0] = F[0] * M.iMlin[0] + (cb[1] * w[2] - cb[2] * w[1]);
  d.v[1] = F[1] * M.iMlin[1] + (cb[2] * w[0] - cb[0] * w[2]);
  d.v[2] = F[2] * M.iMlin[2] + (cb[0] * w[1] - cb[1] * w[0]);
#pragma unroll
  for (int i = 0; i < 3; ++i) d.w[i] = G[i] * M.iMang[i];
  // quaternion kinematics
  const float hw0 = 0.5f * w[0], hw1 = 0.5f * w[1], hw2 = 0.5f * w[2];
  d.q[0] = -(q[1] * hw0 + q[2] * hw1 + q[3] * hw2);
  d.q[1] = q[0] * hw0 + q[2] * hw2 - q[3] * hw1;
  d.q[2] = q[0] * hw1 + q[3] * hw0 - q[1] * hw2;
  d.q[3] = q[0] * hw2 + q[1] * hw1 - q[2] * hw0;
}

// One classic RK4 substep of size h with tau held, then quaternion renormalisation.
__device__ __forceinline__ void rk4(const VehArgs& V, const Model& M, const float cw[3],
                                    const float tau[6], float h, State& x) {
  Deriv k, acc;
  float qs[4], vs[3], ws[3];
  rhs(V, M, cw, tau, x.q, x.v, x.w, k);
#pragma unroll
  for (int i = 0; i < 3; ++i) { acc.p[i] = k.p[i]; acc.v[i] = k.v[i]; acc.w[i] = k.w[i]; }
#pragma unroll
  for (int i = 0; i < 4; ++i) acc.q[i] = k.q[i];
#pragma unroll
  for (int stage = 1; stage < 4; ++stage) {
    const float c = (stage == 3) ? h : 0.5f * h;
#pragma unroll
    for (int i = 0; i < 4; ++i) qs[i] = x.q[i] + c * k.q[i];
#pragma unroll
    for (int i = 0; i < 3; ++i) { vs[i] = x.v[i] + c * k.v[i]; ws[i] = x.w[i] + c * k.w[i]; }
    rhs(V, M, cw, tau, qs, vs, ws, k);
    const float wgt = (stage == 3) ? 1.0f : 2.0f;
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      acc.p[i] += wgt * k.p[i]; acc.v[i] += wgt * k.v[i]; acc.w[i] += wgt * k.w[i];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) acc.q[i] += wgt * k.q[i];
  }
  const float h6 = h * (1.0f / 6.0f);
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    x.p[i] += h6 * acc.p[i]; x.v[i] += h6 * acc.v[i]; x.w[i] += h6 * acc.w[i];
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) x.q[i] += h6 * acc.q[i];
  const float inv = rsqrtf(x.q[0] * x.q[0] + x.q[1] * x.q[1] + x.q[2] * x.q[2] + x.q[3] * x.q[3]);
#pragma unroll
  for (int i = 0; i < 4; ++i) x.q[i] *= inv;
}

// ------------------------------------------------------- thrust -> body wrench ------
__device__ __forceinline__ void wrench(const VehArgs& V, const float u[8], float tau[6]) {
#pragma unroll
  for (int r = 0; r < 6; ++r) {
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) s += V.alloc[r * 8 + j] * (V.f_max * u[j]);
    tau[r] = s;
  }
}

// ------------------------------------------------------ sine and cosine in turns --
// sin(2 pi f) for |f| <= 1/4 turn: Taylor series of sin y, y = 2 pi f in [-pi/2, pi/2],
// through y^13 (truncation below 7e-10, under fp32 rounding).
__device__ __forceinline__ float sin_quarter(float f) {
  const float y = 6.28318530717958648f * f;
  const float y2 = y * y;
  float p = 1.0f / 6227020800.0f;
  p = __builtin_fmaf(p, y2, -1.0f / 39916800.0f);
  p = __builtin_fmaf(p, y2, 1.0f / 362880.0f);
  p = __builtin_fmaf(p, y2, -1.0f / 5040.0f);
  p = __builtin_fmaf(p, y2, 1.0f / 120.0f);
  p = __builtin_fmaf(p, y2, -1.0f / 6.0f);
  return __builtin_fmaf(p * y2, y, y);
}

// sin and cos of 2 pi x for x in turns: exact reduction to r = x - rint(x) in
// [-1/2, 1/2], then sin(2 pi r) = sin_quarter(r) or sin_quarter(+-1/2 - r) and
// cos(2 pi r) = sin_quarter(1/4 - |r|).
__device__ __forceinline__ void sincos_turns(float x, float* s, float* c) {
  const float r = x - rintf(x);
  const float a = fabsf(r);
  *s = sin_quarter(a > 0.25f ? copysignf(0.5f, r) - r : r);
  *c = sin_quarter(0.25f - a);
}

// --------------------------------------------------------------- reset draws --------
// 32 words from blocks (gid, episode, 0, 0..7).  Word map: 0-2 scales, 3-5 current,
// 6-8 p0, 9-11 q0 (Shoemake), 12-14 p_goal, 15-17 q_goal, 18-20 amplitude,
// 21-23 frequency, 24-26 phase, 27 yaw rate, 28 yaw0, 29-31 unused.
__device__ __forceinline__ void shoemake(float u1, float u2, float u3, float q[4]) {
  const float r1 = sqrtf(1.0f - u1), r2 = sqrtf(u1);
  float s1, c1, s2, c2;
  sincospif(2.0f * u2, &s1, &c1);
  sincospif(2.0f * u3, &s2, &c2);
  q[0] = r2 * c2; q[1] = r1 * s1; q[2] = r1 * c1; q[3] = r2 * s2;
}

__device__ __forceinline__ void reset_draws(const EnvArgs& E, uint32_t gid, uint32_t episode,
                                            State& x, Params& P) {
  uint32_t wd[32];
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const U4 r = philox(U4{gid, episode, 0u, (uint32_t)b}, E.key0, E.key1);
    wd[4 * b] = r.x; wd[4 * b + 1] = r.y; wd[4 * b + 2] = r.z; wd[4 * b + 3] = r.w;
  }
  const bool dr = E.flags & F_DR, cur = E.flags & F_CURRENT;
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    P.s[i] = dr ? affine(0.8f, 0.4f, u01(wd[i])) : 1.0f;
    P.cw[i] = cur ? affine(-0.3f, 0.6f, u01(wd[3 + i])) : 0.0f;
    x.p[i] = affine(-2.0f, 4.0f, u01(wd[6 + i]));
    P.pg[i] = affine(-2.0f, 4.0f, u01(wd[12 + i]));
    P.amp[i] = affine(0.5f, 1.5f, u01(wd[18 + i]));
    P.freq[i] = affine(0.02f, 0.08f, u01(wd[21 + i]));
    P.phase[i] = affine(0.0f, 6.28318548f, u01(wd[24 + i]));
    x.v[i] = 0.0f;
    x.w[i] = 0.0f;
  }
  shoemake(u01(wd[9]), u01(wd[10]), u01(wd[11]), x.q);
  shoemake(u01(wd[15]), u01(wd[16]), u01(wd[17]), P.qg);
  P.yaw_rate = affine(-0.1f, 0.2f, u01(wd[27]));
  P.yaw0 = affine(-3.14159274f, 6.28318548f, u01(wd[28]));
}

// Reset of the paper task: the vehicle at rest at the origin, level; goal position
// U[-2, 2]^3 (words 12-14), goal attitude q_z(yaw) q_y(pitch) q_x(roll) from Euler angles
// (words 15-17), gravity factor (word 0, kept in parameter row 13); no other
// randomisation.  Same counters as reset_draws (only blocks 0, 3 and 4 are needed).
__device__ __forceinline__ void paper_reset_draws(const EnvArgs& E, uint32_t gid, uint32_t episode, State& x,
                                                  Params& P) {
  const U4 b0 = philox(U4{gid, episode, 0u, 0u}, E.key0, E.key1);
  const U4 b3 = philox(U4{gid, episode, 0u, 3u}, E.key0, E.key1);
  const U4 b4 = philox(U4{gid, episode, 0u, 4u}, E.key0, E.key1);
  const uint32_t pw[3] = {b3.x, b3.y, b3.z};          // words 12, 13, 14
  const uint32_t ew[3] = {b3.w, b4.x, b4.y};          // words 15, 16, 17: roll, pitch, yaw
  float half[3];
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    P.s[i] = 1.0f;
    P.cw[i] = 0.0f;
    P.pg[i] = affine(-2.0f, 4.0f, u01(pw[i]));
    P.amp[i] = 0.0f;
    P.freq[i] = 0.0f;
    P.phase[i] = 0.0f;
    half[i] = 0.5f * affine(E.tk.eul_lo, E.tk.eul_span, u01(ew[i]));
    x.p[i] = 0.0f;
    x.v[i] = 0.0f;
    x.w[i] = 0.0f;
  }
  P.amp[0] = affine(E.tk.g_lo, E.tk.g_span, u01(b0.x));
  P.yaw_rate = 0.0f;
  P.yaw0 = 0.0f;
  float sr, cr, sp, cp, sy, cy;
  sincosf(half[0], &sr, &cr);
  sincosf(half[1], &sp, &cp);
  sincosf(half[2], &sy, &cy);
  P.qg[0] = cy * cp * cr + sy * sp * sr;
  P.qg[1] = cy * cp * sr - sy * sp * cr;
  P.qg[2] = cy * sp * cr + sy * cp * sr;
  P.qg[3] = sy * cp * cr - cy * sp * sr;
  x.q[0] = 1.0f;
  x.q[1] = x.q[2] = x.q[3] = 0.0f;
}

// ---------------------------------------------------- reference / obs / reward ------
// Lissajous: p_goal + A sin(2 pi f t + phase), yaw psi0 + psi_dot t, evaluated in turns
// (f t + phase / 2 pi and psi / 4 pi).
__device__ __forceinline__ void reference(const EnvArgs& E, const Params& P, int ep_step,
                                          float pr[3], float qr[4]) {
  if (E.flags & F_LISSAJOUS) {
    const float t = (float)ep_step * E.dt;
    constexpr float INV_2PI = 0.159154943091895336f, INV_4PI = 0.0795774715459476679f;
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      float s, c;
      sincos_turns(__builtin_fmaf(P.freq[i], t, P.phase[i] * INV_2PI), &s, &c);
      pr[i] = __builtin_fmaf(P.amp[i], s, P.pg[i]);
    }
    float s, c;
    sincos_turns(__builtin_fmaf(P.yaw_rate, t, P.yaw0) * INV_4PI, &s, &c);
    qr[0] = c; qr[1] = 0.0f; qr[2] = 0.0f; qr[3] = s;
  } else {
#pragma unroll
    for (int i = 0; i < 3; ++i) pr[i] = P.pg[i];
#pragma unroll
    for (int i = 0; i < 4; ++i) qr[i] = P.qg[i];
  }
}

// Observation (first 15 rows; rows 15..22 are the previous action) plus |dp| and the
// attitude-error angle 2 atan2(|vec(q^* (x) q_ref)|, |scalar(q^* (x) q_ref)|).
__device__ __forceinline__ void observe(const State& x, const float pr[3], const float qr[4],
                                        float o[15], float& dist, float& theta) {
  const Rot R = rot_of(x.q);
  const Rot Rr = rot_of(qr);
  float dw[3];
#pragma unroll
  for (int i = 0; i < 3; ++i) dw[i] = pr[i] - x.p[i];
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    o[i] = R.r[0][i] * dw[0] + R.r[1][i] * dw[1] + R.r[2][i] * dw[2];
    o[3 + i] = R.r[0][i] * Rr.r[0][0] + R.r[1][i] * Rr.r[1][0] + R.r[2][i] * Rr.r[2][0];
    o[6 + i] = R.r[0][i] * Rr.r[0][1] + R.r[1][i] * Rr.r[1][1] + R.r[2][i] * Rr.r[2][1];
    o[9 + i] = x.v[i];
    o[12 + i] = x.w[i];
  }
  dist = sqrtf(o[0] * o[0] + o[1] * o[1] + o[2] * o[2]);
  // q_err = q^* (x) q_ref
  const float ew = x.q[0] * qr[0] + x.q[1] * qr[1] + x.q[2] * qr[2] + x.q[3] * qr[3];
  const float ex = x.q[0] * qr[1] - qr[0] * x.q[1] - (x.q[2] * qr[3] - x.q[3] * qr[2]);
  const float ey = x.q[0] * qr[2] - qr[0] * x.q[2] - (x.q[3] * qr[1] - x.q[1] * qr[3]);
  const float ez = x.q[0] * qr[3] - qr[0] * x.q[3] - (x.q[1] * qr[2] - x.q[2] * qr[1]);
  theta = 2.0f * atan2f(sqrtf(ex * ex + ey * ey + ez * ez), fabsf(ew));
}

// ------------------------------------------------------------- buffer access -------
__device__ __forceinline__ void load_state(const float* __restrict__ s, int n, int i, State& x) {
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    x.p[k] = s[k * n + i]; x.v[k] = s[(7 + k) * n + i]; x.w[k] = s[(10 + k) * n + i];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) x.q[k] = s[(3 + k) * n + i];
}

__device__ __forceinline__ void store_state(float* __restrict__ s, size_t stride, size_t i, const State& x) {
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    s[k * stride + i] = x.p[k]; s[(7 + k) * stride + i] = x.v[k]; s[(10 + k) * stride + i] = x.w[k];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) s[(3 + k) * stride + i] = x.q[k];
}

__device__ __forceinline__ void load_params(const float* __restrict__ s, int n, int i, Params& P) {
  float v[NP];
#pragma unroll
  for (int k = 0; k < NP; ++k) v[k] = s[k * n + i];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    P.s[k] = v[k]; P.cw[k] = v[3 + k]; P.pg[k] = v[6 + k];
    P.amp[k] = v[13 + k]; P.freq[k] = v[16 + k]; P.phase[k] = v[19 + k];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) P.qg[k] = v[9 + k];
  P.yaw_rate = v[22];
  P.yaw0 = v[23];
}

__device__ __forceinline__ void store_params(float* __restrict__ s, int n, int i, const Params& P) {
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    s[k * n + i] = P.s[k]; s[(3 + k) * n + i] = P.cw[k]; s[(6 + k) * n + i] = P.pg[k];
    s[(13 + k) * n + i] = P.amp[k]; s[(16 + k) * n + i] = P.freq[k]; s[(19 + k) * n + i] = P.phase[k];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) s[(9 + k) * n + i] = P.qg[k];
  s[22 * n + i] = P.yaw_rate;
  s[23 * n + i] = P.yaw0;
}

// ------------------------------------------------------------ failure detection ----
// Non-finite state components of one environment, counted where an episode ends (before
// its reset overwrites the state) and where a launch ends, and added to status[0].  Lanes
// with nothing to report issue no atomic, so the count costs nothing while all is finite.
__device__ __forceinline__ uint32_t nonfinite(float x) { return __builtin_isfinite(x) ? 0u : 1u; }

__device__ __forceinline__ uint32_t nonfinite_state(const State& x) {
  uint32_t n = 0;
#pragma unroll
  for (int k = 0; k < 3; ++k) n += nonfinite(x.p[k]) + nonfinite(x.v[k]) + nonfinite(x.w[k]);
#pragma unroll
  for (int k = 0; k < 4; ++k) n += nonfinite(x.q[k]);
  return n;
}

__device__ __forceinline__ void report_status(uint32_t* status, uint32_t nonfinite_count, uint32_t abandoned) {
  if (status && nonfinite_count) atomicAdd(&status[0], nonfinite_count);
  if (status && abandoned) atomicAdd(&status[1], abandoned);
}

// Sum over the 64 lanes of a wave in a fixed butterfly order (every lane gets the sum).
// DPP lane moves for reductions (GCN row = 16 lanes): rotate right within each row, and
// broadcast lane 15 / 31 into the following row(s) (rows outside row_mask read zero).
constexpr int DPP_ROW_ROR4 = 0x124, DPP_ROW_ROR8 = 0x128, DPP_ROW_BCAST15 = 0x142, DPP_ROW_BCAST31 = 0x143;
constexpr int DPP_QUAD_SWAP1 = 0xB1, DPP_QUAD_SWAP2 = 0x4E;   // quad_perm [1,0,3,2], [2,3,0,1]

template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ float dpp_move(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, ROW_MASK, 0xF,
                                                               ROW_MASK == 0xF));
}

// Sum of one value per row position over the four rows of a wave, with every lane of a row
// holding its row's total on entry: the total lands in lane 63 and is returned wave-uniform.
__device__ __forceinline__ float rows_sum(float v) {
  v += dpp_move<DPP_ROW_BCAST15, 0xA>(v);   // rows 1, 3 += rows 0, 2
  v += dpp_move<DPP_ROW_BCAST31, 0xC>(v);   // rows 2, 3 += row 1
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// Sum over the 64 lanes of a wave (wave-uniform result).
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_move<DPP_QUAD_SWAP1>(v);
  v += dpp_move<DPP_QUAD_SWAP2>(v);
  v += dpp_move<DPP_ROW_ROR4>(v);
  v += dpp_move<DPP_ROW_ROR8>(v);
  return rows_sum(v);
}

// Sum over the quads of a wave of a value that is the same in the four lanes of each quad.
__device__ __forceinline__ float wave_sum_quads(float v) {
  v += dpp_move<DPP_ROW_ROR4>(v);
  v += dpp_move<DPP_ROW_ROR8>(v);
  return rows_sum(v);
}

}  // namespace auv
