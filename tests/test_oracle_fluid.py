"""Pins of the inertia-box fluid model (oracle/fluid.py) against what its physics fixes:
the box has the body's mass and inertia; the quadratic drag torque is the pressure drag
integrated over the box's mid-plane plates (midpoint quadrature); the rigid body integrated
with the model reaches the closed-form terminal speed, spins down along the closed-form
solution of I dw/dt = -(lin + quad |w|) w, and starts from rest with acceleration F / m (no
added mass); the paper task's oracle runs it when the task asks for it."""
import math

import numpy as np

import workloads as W
from oracle import dynamics as dyn
from oracle import fluid as fl
from oracle import paper_task as P


def test_equivalent_box_has_the_body_mass_and_inertia():
    r = np.random.default_rng(0)
    for _ in range(20):
        m = r.uniform(1, 50)
        s = r.uniform(0.1, 1.0, 3)
        I = m * (np.roll(s, -1) ** 2 + np.roll(s, -2) ** 2) / 12.0       # a solid box's inertia
        assert np.allclose(fl.equivalent_box(m, I), s, rtol=1e-12)
    s = fl.equivalent_box(11.5, [0.16, 0.16, 0.16])
    assert np.allclose(s, math.sqrt(6 * 0.16 / 11.5))


def test_quadratic_drag_torque_is_the_plate_pressure_integral():
    """Rotation about x at rate w: the plates through the centre normal to y and to z, each
    element moving at w times its distance from the axis, pressure drag rho/2 u |u| per
    area; midpoint quadrature against rho s_x (s_y^4 + s_z^4) / 64."""
    rho, w = 1000.0, 1.7
    box = np.array([0.3, 0.5, 0.2])
    inertia = (np.roll(box, -1) ** 2 + np.roll(box, -2) ** 2) / 12.0          # unit mass
    c = fl.drag_coefficients(1.0, inertia, rho, 1e-3)
    assert np.allclose(c["box"], box, rtol=1e-12)
    n = 200000
    torque = 0.0
    for side, other in ((box[2], box[0]), (box[1], box[0])):   # plate normal to y spans z; normal to z spans y
        z = (np.arange(n) + 0.5) / n * side - side / 2
        torque += np.sum(z * 0.5 * rho * (w * z) * np.abs(w * z)) * (side / n) * other
    assert abs(torque - c["quad"][3] * w * w) <= 1e-8 * torque
    # translation along x: the face normal to x, pressure drag over its area
    assert np.isclose(c["quad"][0], 0.5 * rho * box[1] * box[2])


def _level_body(n=1):
    veh = dict(W.VEHICLE)
    veh["r_b"] = np.zeros(3, np.float32)
    v = fl.InertiaBoxVehicle(veh, n)
    v.W = v.B                                       # neutrally buoyant: no vertical force
    x = np.zeros((13, n))
    x[3] = 1.0
    return v, x


def test_terminal_speed_and_start_without_added_mass():
    v, x = _level_body()
    F = 30.0
    tau = np.array([[F], [0], [0], [0], [0], [0]], np.float64)
    d0 = dyn.rhs(x, tau, v, np.zeros((3, 1)))
    assert np.isclose(d0[7, 0], F / float(np.float32(11.5)), rtol=1e-14)          # no added mass
    c = v.fluid
    m = float(np.float32(11.5))
    for k in range(2000):                                                          # 20 s
        x = dyn.rk4_substep(x, tau, v, np.zeros((3, 1)), 0.01)
        if k % 200 == 199:
            t = (k + 1) * 0.01
            assert abs(x[7, 0] - fl.speed_from_rest(F, t, m, c["lin"][0], c["quad"][0])) <= 1e-9
    assert abs(x[7, 0] - fl.terminal_speed(F, c["lin"][0], c["quad"][0])) <= 1e-9
    assert np.allclose(x[8:13, 0], 0.0, atol=1e-12) and np.allclose(x[3:7, 0], [1, 0, 0, 0], atol=1e-12)


def test_spin_down_follows_the_closed_form():
    v, x = _level_body()
    w0 = 2.0
    x[10] = w0
    t, h = 0.0, 0.002
    c = v.fluid
    I = float(np.float32(0.16))
    errs = []
    for k in range(1500):                                                          # 3 s
        x = dyn.rk4_substep(x, np.zeros((6, 1)), v, np.zeros((3, 1)), h)
        t += h
        if k % 100 == 99:
            errs.append(abs(x[10, 0] - fl.spin_down(w0, t, I, c["lin"][3], c["quad"][3])))
    assert max(errs) <= 1e-9
    assert x[10, 0] < 0.6 * w0                                                     # it did slow down


def test_paper_task_oracle_selects_the_fluid_model():
    cfg = dict(n_envs=8, seed=6, flags=0, episode_len=512, substeps=2, dt_control=0.05)
    e = P.PaperEnv(cfg, W.VEHICLE, W.PAPER_TASK_BOX)
    e.reset()
    assert isinstance(e.veh, fl.InertiaBoxVehicle)
    assert np.all(e.veh.M_A == 0) and np.allclose(e.veh.W, float(np.float32(112.8)) * e.gfac)
    f = P.PaperEnv(cfg, W.VEHICLE, W.PAPER_TASK)
    f.reset()
    assert not isinstance(f.veh, fl.InertiaBoxVehicle)
    a = np.full((6, 8), 0.5)
    e.step(a)
    f.step(a)
    assert not np.allclose(e.x, f.x)                                               # different hydrodynamics
