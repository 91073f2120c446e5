"""Inertia-box fluid model (oracle side, float64): the hydrodynamics of the paper's MJX
simulation (Sec. IV-B, Environment Specifications).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper passage: the vehicle is one free body driven by forces and torques on its free joint;
hydrodynamic forces come from MuJoCo's inertia-based fluid model with water's density and
viscosity, in which the body is replaced by the solid box that has its mass and principal
inertia, and the forces and torques are quadratic drag and viscous resistance on that box;
buoyancy is folded into the effective gravity with the centres of gravity and buoyancy
aligned.  The model's own definition is not in this repository; it is restated here from its
physics, and every term is pinned by a test against what that physics fixes (box inertia,
drag integrated over the box faces, Stokes' laws, closed-form terminal velocity and spin-down).

Model, body frame (the principal axes; the body origin at the centre of gravity):
  equivalent box  s_i = sqrt(6 (I_j + I_k - I_i) / m)      ({i, j, k} = {x, y, z})
                  (a uniform solid box of mass m and sides s has I_i = m (s_j^2 + s_k^2) / 12)
  viscous         f = -3 pi mu d v,  g = -pi mu d^3 w,  d = (s_x + s_y + s_z) / 3
                  (Stokes drag and torque of the sphere of diameter d)
  quadratic       f_i = -1/2 rho s_j s_k |v_i| v_i          (the face normal to axis i)
                  g_i = -rho s_i (s_j^4 + s_k^4) / 64 |w_i| w_i (faces normal to j and k, swept
                                                             at w_i times their distance)
  no added mass, rigid-body Coriolis terms only, restoring force (B - gamma W) k as in the
  paper task (effective gravity), no restoring moment.
Readings: water at about 20 C, rho = 1000 kg/m^3, mu = 1.0e-3 Pa s (the paper says "water");
the medium is at rest (no current).

In the Fossen form used by dynamics.py this is M = M_RB, D(nu) = D_L + D_Q |nu| with
D_L = (3 pi mu d, 3 pi mu d, 3 pi mu d, pi mu d^3, pi mu d^3, pi mu d^3) and D_Q = the
quadratic coefficients above; InertiaBoxVehicle builds exactly those matrices.
"""
from __future__ import annotations

import math

import numpy as np

from . import dynamics as dyn

RHO_WATER = 1000.0
MU_WATER = 1.0e-3


def _f64(x):
    return np.asarray(x, np.float32).astype(np.float64)


def equivalent_box(m: float, inertia) -> np.ndarray:
    """Sides (s_x, s_y, s_z) of the uniform solid box with mass m and principal inertia I."""
    I = np.asarray(inertia, np.float64)
    arg = 6.0 * (np.roll(I, -1) + np.roll(I, -2) - I) / m
    if np.any(arg <= 0.0):
        raise ValueError("inertia violates the triangle inequality of a solid body")
    return np.sqrt(arg)


def drag_coefficients(m: float, inertia, rho: float, mu: float) -> dict:
    """Linear (viscous) and quadratic coefficients per body axis (surge, sway, heave, roll,
    pitch, yaw): force_i = -(lin_i + quad_i |nu_i|) nu_i."""
    s = equivalent_box(m, inertia)
    d = float(np.mean(s))
    sx, sy, sz = s
    lin = np.array([3.0 * math.pi * mu * d] * 3 + [math.pi * mu * d ** 3] * 3)
    quad = np.array([0.5 * rho * sy * sz, 0.5 * rho * sx * sz, 0.5 * rho * sx * sy,
                     rho * sx * (sy ** 4 + sz ** 4) / 64.0, rho * sy * (sx ** 4 + sz ** 4) / 64.0,
                     rho * sz * (sx ** 4 + sy ** 4) / 64.0])
    return dict(box=s, d=d, lin=lin, quad=quad)


class InertiaBoxVehicle(dyn.Vehicle):
    """dynamics.Vehicle with the inertia-box fluid model: no added mass (so no added-mass
    Coriolis terms) and the box's viscous + quadratic drag as its damping."""

    def __init__(self, veh: dict, n: int, rho: float = RHO_WATER, mu: float = MU_WATER):
        v = dict(veh)
        v["added_mass"] = np.zeros(6, np.float32)
        super().__init__(v, n)
        c = drag_coefficients(float(_f64(veh["m"])), _f64(veh["inertia"]), rho, mu)
        self.D_L = np.broadcast_to(c["lin"], (n, 6)).copy()
        self.D_Q = np.broadcast_to(c["quad"], (n, 6)).copy()
        self.fluid = c


def terminal_speed(F: float, lin: float, quad: float) -> float:
    """Steady speed under a constant force F along one axis: quad v^2 + lin v = F."""
    return (-lin + math.sqrt(lin * lin + 4.0 * quad * F)) / (2.0 * quad)


def speed_from_rest(F: float, t, mass: float, lin: float, quad: float):
    """Speed along one axis of mass dv/dt = F - lin v - quad |v| v from v(0) = 0 (closed form):
    with the roots v+ > 0 > v- of quad v^2 + lin v - |F| = 0 and k = quad (v+ - v-) / mass,
    v = sign(F) (v+ - r v-) / (1 - r),  r = (v+ / v-) exp(-k t)."""
    t = np.asarray(t, np.float64)
    a = abs(F)
    disc = math.sqrt(lin * lin + 4.0 * quad * a)
    vp, vm = (-lin + disc) / (2.0 * quad), (-lin - disc) / (2.0 * quad)
    r = (vp / vm) * np.exp(-quad * (vp - vm) * t / mass)
    return math.copysign(1.0, F) * (vp - r * vm) / (1.0 - r)


def spin_down(w0: float, t, inertia: float, lin: float, quad: float):
    """Angular rate of I dw/dt = -(lin + quad |w|) w from w0 > 0 (closed form):
    w(t) = lin / (quad ((1 + lin / (quad w0)) exp(lin t / I) - 1))."""
    t = np.asarray(t, np.float64)
    return lin / (quad * ((1.0 + lin / (quad * w0)) * np.exp(lin * t / inertia) - 1.0))
