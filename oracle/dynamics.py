"""Fossen 6-DOF equations of motion and RK4 (oracle side, float64).

The paper's MPC baseline steps the nonlinear 6-DOF equations of motion of Fossen
(Sec. IV-D, Eq. 8, "Model Predictive Controller Baseline"); the rollout uses the same model
with added mass, Coriolis and centripetal terms, linear and quadratic damping,
restoring forces from weight and buoyancy with the centre of buoyancy offset from the
centre of gravity (the offset the paper names as its main sim-to-real gap, Sec. VI-A),
and a constant irrotational ocean current.

Conventions: world frame NED (z down), body frame forward-right-down with its origin at
the centre of gravity, Hamilton quaternion q = (w, x, y, z) rotating body -> world.
State x = (p[3] world, q[4], v[3] body, omega[3] body), absolute velocities.

Equations (relative-velocity form, exact for a constant irrotational current when the
rigid-body Coriolis matrix is written independently of linear velocity):
    (M_RB + M_A) dnu_r/dt + C_RB(nu_r) nu_r + C_A(nu_r) nu_r + D(nu_r) nu_r + g(q) = tau
    nu_r = nu - (R^T c_w, 0),   dnu/dt = dnu_r/dt + (-S(omega) R^T c_w, 0)
    dp/dt = R(q) v,             dq/dt = 1/2 [-eps^T ; eta I + S(eps)] omega
All matrices are built explicitly and the mass matrix is solved with numpy.linalg.solve.

The same model has a second textbook form, selected by rhs(..., form=FORM_MIXED): the
rigid-body terms act on the absolute velocity and only the hydrodynamic terms on the
relative one,
    M_RB dnu/dt + C_RB(nu) nu + M_A dnu_r/dt + C_A(nu_r) nu_r + D(nu_r) nu_r + g(q) = tau,
with dnu_r/dt = dnu/dt - dnu_c/dt and dnu_c/dt = d(R^T c_w)/dt = -omega x R^T c_w.  For a
constant irrotational current and this C_RB the two forms are the same equations (the
difference M_RB dnu_c/dt + C_RB(nu) nu - C_RB(nu_r) nu_r vanishes), so they agree to
rounding for every current and bit for bit at c_w = 0.  FORM_NO_CURRENT_RATE is the
relative form without the dnu_c/dt term, the simplification many simulators make; it is
kept only so that tests can show which pins reject it.

Arrays are batched over environments along the LAST axis for states ([13, n]) and along
the FIRST axis for matrices ([n, 6, 6]).
"""
from __future__ import annotations

import numpy as np


def skew(a: np.ndarray) -> np.ndarray:
    """S(a) with S(a) b = a x b; a [n, 3] -> [n, 3, 3]."""
    n = a.shape[0]
    s = np.zeros((n, 3, 3))
    s[:, 0, 1], s[:, 0, 2] = -a[:, 2], a[:, 1]
    s[:, 1, 0], s[:, 1, 2] = a[:, 2], -a[:, 0]
    s[:, 2, 0], s[:, 2, 1] = -a[:, 1], a[:, 0]
    return s


def rotation(q: np.ndarray) -> np.ndarray:
    """R(q) = I + 2 eta S(eps) + 2 S(eps)^2 (Euler-Rodrigues form); q [4, n] -> [n, 3, 3].

    This is the rotation matrix of a unit quaternion; the same formula is applied to the
    (slightly non-unit) RK4 stage quaternions."""
    eta = q[0]
    s = skew(q[1:4].T)
    return np.eye(3)[None] + 2.0 * eta[:, None, None] * s + 2.0 * s @ s


def quat_rate_matrix(q: np.ndarray) -> np.ndarray:
    """T(q) with dq/dt = T(q) omega: T = 1/2 [-eps^T ; eta I + S(eps)]; q [4, n] -> [n, 4, 3]."""
    n = q.shape[1]
    t = np.zeros((n, 4, 3))
    t[:, 0, :] = -q[1:4].T
    t[:, 1:4, :] = q[0][:, None, None] * np.eye(3)[None] + skew(q[1:4].T)
    return 0.5 * t


class Vehicle:
    """Per-environment model constants, float64.

    Domain randomisation multiplies the rigid-body mass and inertia by s_m, the added
    mass by s_a and both damping matrices by s_d; weight, buoyancy and the buoyancy
    offset are not randomised."""

    def __init__(self, veh: dict, n: int, s_m=None, s_a=None, s_d=None):
        one = np.ones(n)
        s_m = one if s_m is None else np.asarray(s_m, np.float64)
        s_a = one if s_a is None else np.asarray(s_a, np.float64)
        s_d = one if s_d is None else np.asarray(s_d, np.float64)
        f64 = lambda x: np.asarray(x, np.float32).astype(np.float64)  # noqa: E731
        m = f64(veh["m"]) * s_m                                       # [n]
        inertia = f64(veh["inertia"])[None, :] * s_m[:, None]        # [n, 3]
        self.M_RB = np.zeros((n, 6, 6))
        for i in range(3):
            self.M_RB[:, i, i] = m
            self.M_RB[:, 3 + i, 3 + i] = inertia[:, i]
        self.M_A = np.zeros((n, 6, 6))
        ma = f64(veh["added_mass"])[None, :] * s_a[:, None]
        for i in range(6):
            self.M_A[:, i, i] = ma[:, i]
        self.D_L = f64(veh["lin_damp"])[None, :] * s_d[:, None]       # [n, 6]
        self.D_Q = f64(veh["quad_damp"])[None, :] * s_d[:, None]      # [n, 6]
        self.m = m
        self.inertia = inertia
        self.W = float(f64(veh["W"]))
        self.B = float(f64(veh["B"]))
        self.r_b = f64(veh["r_b"])
        self.M = self.M_RB + self.M_A

    def C_RB(self, nu: np.ndarray) -> np.ndarray:
        """Rigid-body Coriolis-centripetal matrix, linear-velocity-independent form
        (origin at the CoG): [[m S(omega), 0], [0, -S(I omega)]]; nu [n, 6]."""
        n = nu.shape[0]
        c = np.zeros((n, 6, 6))
        c[:, 0:3, 0:3] = self.m[:, None, None] * skew(nu[:, 3:6])
        c[:, 3:6, 3:6] = -skew(self.inertia * nu[:, 3:6])
        return c

    def C_A(self, nu: np.ndarray) -> np.ndarray:
        """Added-mass Coriolis-centripetal matrix for a diagonal M_A:
        [[0, -S(A11 v)], [-S(A11 v), -S(A22 omega)]]; nu [n, 6]."""
        a = np.einsum("nij,nj->ni", self.M_A, nu)
        n = nu.shape[0]
        c = np.zeros((n, 6, 6))
        c[:, 0:3, 3:6] = -skew(a[:, 0:3])
        c[:, 3:6, 0:3] = -skew(a[:, 0:3])
        c[:, 3:6, 3:6] = -skew(a[:, 3:6])
        return c

    def D(self, nu: np.ndarray) -> np.ndarray:
        """Damping matrix D_L + diag(D_Q |nu|); nu [n, 6]."""
        d = self.D_L + self.D_Q * np.abs(nu)
        n = nu.shape[0]
        out = np.zeros((n, 6, 6))
        for i in range(6):
            out[:, i, i] = d[:, i]
        return out

    def g(self, R: np.ndarray) -> np.ndarray:
        """Restoring vector g(q) = [(B - W) k ; B r_b x k], k = R^T e_3 (the world down
        direction in body axes); it sits on the left-hand side of the equations."""
        k = R[:, 2, :]                                                 # row 3 of R = R^T e3
        f = np.reshape(self.B - self.W, (-1, 1)) * k                   # W: one value or one per env
        mom = self.B * np.cross(np.broadcast_to(self.r_b, k.shape), k)
        return np.concatenate([f, mom], axis=1)


FORM_RELATIVE, FORM_MIXED, FORM_NO_CURRENT_RATE = "relative", "mixed", "no_current_rate"


def rhs(x: np.ndarray, tau: np.ndarray, veh: Vehicle, c_w: np.ndarray, form: str = FORM_RELATIVE) -> np.ndarray:
    """dx/dt for states x [13, n], body wrench tau [6, n], world current c_w [3, n]; `form`
    selects one of the two equivalent forms of the equations (module docstring)."""
    p, q, v, w = x[0:3], x[3:7], x[7:10], x[10:13]
    R = rotation(q)                                                    # [n, 3, 3]
    c_b = np.einsum("nji,jn->ni", R, c_w)                              # R^T c_w, [n, 3]
    nu = np.concatenate([v.T, w.T], axis=1)                            # [n, 6]
    nu_r = nu - np.concatenate([c_b, np.zeros_like(c_b)], axis=1)
    nu_c_dot = np.concatenate([-np.cross(w.T, c_b), np.zeros_like(c_b)], axis=1)
    ca = np.einsum("nij,nj->ni", veh.C_A(nu_r), nu_r)
    dm = np.einsum("nij,nj->ni", veh.D(nu_r), nu_r)
    gr = veh.g(R)
    if form == FORM_MIXED:
        # (M_RB + M_A) dnu/dt = tau - C_RB(nu) nu - C_A(nu_r) nu_r - D(nu_r) nu_r - g + M_A dnu_c/dt
        lhs_terms = np.einsum("nij,nj->ni", veh.C_RB(nu), nu) + ca + dm + gr
        f = (tau.T - lhs_terms) + np.einsum("nij,nj->ni", veh.M_A, nu_c_dot)
        nu_dot = np.linalg.solve(veh.M, f[..., None])[..., 0]
    elif form in (FORM_RELATIVE, FORM_NO_CURRENT_RATE):
        lhs_terms = np.einsum("nij,nj->ni", veh.C_RB(nu_r), nu_r) + ca + dm + gr
        nu_r_dot = np.linalg.solve(veh.M, (tau.T - lhs_terms)[..., None])[..., 0]   # [n, 6]
        nu_dot = nu_r_dot + nu_c_dot if form == FORM_RELATIVE else nu_r_dot
    else:
        raise ValueError(f"unknown form {form!r}")
    p_dot = np.einsum("nij,jn->in", R, v)
    q_dot = np.einsum("nij,jn->in", quat_rate_matrix(q), w)
    return np.concatenate([p_dot, q_dot, nu_dot.T], axis=0)


def rk4_substep(x, tau, veh, c_w, h, form=FORM_RELATIVE):
    """Classic four-stage Runge-Kutta step of size h with the wrench held constant,
    followed by renormalisation of the quaternion (stage quaternions are not normalised)."""
    k1 = rhs(x, tau, veh, c_w, form)
    k2 = rhs(x + 0.5 * h * k1, tau, veh, c_w, form)
    k3 = rhs(x + 0.5 * h * k2, tau, veh, c_w, form)
    k4 = rhs(x + h * k3, tau, veh, c_w, form)
    xn = x + (h / 6.0) * (k1 + 2.0 * k2 + 2.0 * k3 + k4)
    xn[3:7] /= np.linalg.norm(xn[3:7], axis=0, keepdims=True)
    return xn


def integrate(x, tau, veh, c_w, dt, substeps):
    """One control interval dt: `substeps` RK4 substeps of dt/substeps, wrench held."""
    h = dt / substeps
    for _ in range(substeps):
        x = rk4_substep(x, tau, veh, c_w, h)
    return x


def kinetic_energy(x: np.ndarray, veh: Vehicle) -> np.ndarray:
    """T = 1/2 nu^T M nu per env (used by the energy invariant)."""
    nu = np.concatenate([x[7:10].T, x[10:13].T], axis=1)
    return 0.5 * np.einsum("ni,nij,nj->n", nu, veh.M, nu)
