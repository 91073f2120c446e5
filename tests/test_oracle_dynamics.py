"""Pins for the oracle's Fossen dynamics and RK4 (CPU only): closed forms, invariants,
library special cases and convergence order."""
import math

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st
from scipy.spatial.transform import Rotation

import workloads as W
from oracle import dynamics as dyn


def _state(n=1, p=(0, 0, 0), q=(1, 0, 0, 0), v=(0, 0, 0), w=(0, 0, 0)):
    x = np.zeros((13, n))
    x[0:3] = np.asarray(p, float).reshape(3, -1)
    x[3:7] = np.asarray(q, float).reshape(4, -1)
    x[7:10] = np.asarray(v, float).reshape(3, -1)
    x[10:13] = np.asarray(w, float).reshape(3, -1)
    return x


def _run(x, veh, n_steps, h, tau=None, c_w=None):
    n = x.shape[1]
    tau = np.zeros((6, n)) if tau is None else tau
    c_w = np.zeros((3, n)) if c_w is None else c_w
    traj = [x]
    for _ in range(n_steps):
        x = dyn.rk4_substep(x, tau, veh, c_w, h)
        traj.append(x)
    return np.stack(traj)           # [n_steps+1, 13, n]


def _p4(z):
    return 1 + z + z * z / 2 + z ** 3 / 6 + z ** 4 / 24


NEUTRAL = dict(W=114.8, B=114.8, r_b=[0.0, 0.0, 0.0], quad_damp=[0.0] * 6)


@pytest.mark.parametrize("axis", range(6))
def test_linear_damping_decay_discrete_closed_form(axis):
    """1-DOF decay under linear damping: RK4 multiplies the speed by P4(-k h) per step,
    k = d / (m + m_a), and moves the position by (1 - P4^n) u0 / k."""
    vd = W.vehicle_variant(**NEUTRAL)
    veh = dyn.Vehicle(vd, 1)
    h, n_steps, s0 = 0.02, 1000, 0.7
    nu0 = np.zeros(6)
    nu0[axis] = s0
    x0 = _state(v=nu0[:3], w=nu0[3:])
    traj = _run(x0, veh, n_steps, h)
    if axis < 3:
        M = float(np.float32(vd["m"])) + float(np.float32(vd["added_mass"][axis]))
    else:
        M = float(np.float32(vd["inertia"][axis - 3])) + float(np.float32(vd["added_mass"][axis]))
    k = float(np.float32(vd["lin_damp"][axis])) / M
    fac = _p4(-k * h)
    n = np.arange(n_steps + 1)
    speed = traj[:, 7 + axis, 0]
    assert np.allclose(speed, s0 * fac ** n, rtol=1e-12, atol=1e-15)
    # the discrete factor approximates exp(-k h) to RK4's local error
    assert abs(fac - math.exp(-k * h)) < (k * h) ** 5 / 100
    if axis < 3:
        pos = traj[:, axis, 0]
        assert np.allclose(pos, s0 * (1 - fac ** n) / k, rtol=1e-12, atol=1e-14)
        # other components stay exactly at rest
        others = [i for i in range(13) if i not in (axis, 7 + axis, 3)]
        assert np.all(traj[:, others, 0] == 0.0)
    if axis == 5:
        # yaw: q = (cos psi/2, 0, 0, sin psi/2) with psi -> s0 (1 - fac^n)/k to RK4 accuracy
        psi = s0 * (1 - fac ** n) / k
        assert np.allclose(traj[:, 3, 0], np.cos(psi / 2), atol=1e-9)
        assert np.allclose(traj[:, 6, 0], np.sin(psi / 2), atol=1e-9)
    # numeric values named in the design: surge 4/17, sway, heave, rotations 0.25
    want = {0: 4.0 / 17.0, 1: 6.2 / 24.2, 2: 5.2 / 26.1, 3: 0.25, 4: 0.25, 5: 0.25}[axis]
    assert k == pytest.approx(want, rel=1e-6)


def test_quadratic_damping_bernoulli_closed_form():
    """u' = -(d_l u + d_q u|u|)/M has u(t) = d_l u0 e^{-kt} / (d_l + d_q u0 (1 - e^{-kt}))
    for u0 > 0; RK4 error shrinks 16x when h halves."""
    vd = W.vehicle_variant(W=114.8, B=114.8, r_b=[0.0, 0.0, 0.0])
    veh = dyn.Vehicle(vd, 1)
    dl, dq = float(np.float32(4.0)), float(np.float32(18.2))
    M = float(np.float32(11.5)) + float(np.float32(5.5))
    u0, t_end = 2.0, 2.0
    k = dl / M
    exact = dl * u0 * math.exp(-k * t_end) / (dl + dq * u0 * (1 - math.exp(-k * t_end)))
    errs = []
    for h in (0.04, 0.02, 0.01):
        traj = _run(_state(v=(u0, 0, 0)), veh, int(round(t_end / h)), h)
        errs.append(abs(traj[-1, 7, 0] - exact))
    assert errs[1] < 1e-7
    assert 12 < errs[0] / errs[1] < 20 and 12 < errs[1] / errs[2] < 20


def test_steady_state_surge_full_thrust():
    """Constant full surge command (thrusters 0-3 at +1) against linear + quadratic
    damping: u_ss = (-d_l + sqrt(d_l^2 + 4 d_q F)) / (2 d_q) = 2.3858 m/s, F = 160 cos 45."""
    vd = W.vehicle_variant(W=114.8, B=114.8, r_b=[0.0, 0.0, 0.0])
    veh = dyn.Vehicle(vd, 1)
    f = 40.0 * np.array([1, 1, 1, 1, 0, 0, 0, 0], float)
    tau = (W.ALLOC.astype(np.float64) @ f)[:, None]
    F = tau[0, 0]
    assert F == pytest.approx(160 * math.cos(math.pi / 4), rel=1e-7)
    assert np.all(np.abs(tau[1:, 0]) < 1e-6)
    x = _state()
    for _ in range(3000):
        x = dyn.rk4_substep(x, tau, veh, np.zeros((3, 1)), 0.02)
    dl, dq = float(np.float32(4.0)), float(np.float32(18.2))
    u_ss = (-dl + math.sqrt(dl * dl + 4 * dq * F)) / (2 * dq)
    assert u_ss == pytest.approx(2.3858, abs=1e-4)
    assert x[7, 0] == pytest.approx(u_ss, abs=1e-9)


def test_neutral_buoyancy_rest_is_exactly_at_rest():
    vd = W.vehicle_variant(W=114.8, B=114.8)        # default CoB offset, upright
    veh = dyn.Vehicle(vd, 3)
    x0 = np.repeat(_state(p=(0.5, -1.0, 2.0)), 3, axis=1)
    traj = _run(x0, veh, 500, 0.02)
    assert np.all(traj == x0[None])


def test_terminal_rise_speed():
    """Default W < B, upright: heave settles where B - W = d_l w + d_q w^2, w = -0.1726."""
    veh = dyn.Vehicle(W.vehicle_variant(), 1)
    traj = _run(_state(), veh, 1500, 0.02)
    dl, dq = float(np.float32(5.2)), float(np.float32(37.0))
    dBW = float(np.float32(114.8)) - float(np.float32(112.8))
    w_ss = (-dl + math.sqrt(dl * dl + 4 * dq * dBW)) / (2 * dq)
    assert w_ss == pytest.approx(0.1726, abs=1e-4)
    assert traj[-1, 9, 0] == pytest.approx(-w_ss, abs=1e-8)
    assert np.all(np.abs(traj[-1, [7, 8, 10, 11, 12], 0]) < 1e-12)


def test_restoring_moment_small_roll_oscillation():
    """Small roll with W = B: phi'' (I + A) + d phi' + B z_b phi = 0, omega_n = 2.864 rad/s
    and zeta ~ 0.044 (small-angle approximation, weak pin at the 1 % level)."""
    vd = W.vehicle_variant(W=114.8, B=114.8, quad_damp=[0.0] * 6)
    veh = dyn.Vehicle(vd, 1)
    phi0 = 0.02
    q0 = (math.cos(phi0 / 2), math.sin(phi0 / 2), 0, 0)
    h = 0.002
    traj = _run(_state(q=q0), veh, 5000, h)
    roll = 2 * np.arctan2(traj[:, 4, 0], traj[:, 3, 0])
    Ieff = float(np.float32(0.16)) + float(np.float32(0.12))
    wn = math.sqrt(float(np.float32(114.8)) * 0.02 / Ieff)
    zeta = float(np.float32(0.07)) / (2 * Ieff * wn)
    assert wn == pytest.approx(2.864, abs=1e-3) and zeta == pytest.approx(0.0436, abs=1e-3)
    wd = wn * math.sqrt(1 - zeta ** 2)
    # zero crossings from above: spacing is the damped period
    s = np.sign(roll)
    idx = np.nonzero((s[:-1] > 0) & (s[1:] <= 0))[0]
    period = np.mean(np.diff(idx)) * h
    assert period == pytest.approx(2 * math.pi / wd, rel=1e-2)


def test_current_drift():
    """W = B, r_b = 0, no thrust, body velocity equal to the current: no relative flow,
    so the vehicle drifts with the current: p(t) = p0 + c_w t, q and nu constant."""
    vd = W.vehicle_variant(W=114.8, B=114.8, r_b=[0.0, 0.0, 0.0])
    n = 8
    veh = dyn.Vehicle(vd, n)
    r = np.random.Generator(np.random.PCG64(2))
    q = r.standard_normal((4, n))
    q /= np.linalg.norm(q, axis=0)
    c_w = r.uniform(-0.3, 0.3, (3, n))
    R = dyn.rotation(q)
    v = np.einsum("nji,jn->in", R, c_w)
    x0 = _state(n=n, p=r.uniform(-2, 2, (3, n)), q=q, v=v)
    traj = _run(x0, veh, 500, 0.02, c_w=c_w)
    t = 500 * 0.02
    assert np.allclose(traj[-1, 0:3], x0[0:3] + c_w * t, atol=1e-12)
    assert np.allclose(traj[-1, 3:13], x0[3:13], atol=1e-13)


def test_current_relative_flow_damps_to_current():
    """With a current, zero thrust and W = B, r_b = 0, the relative flow decays: the body
    velocity relaxes to the current expressed in body axes, R^T c_w, and the rotation
    stops (the vehicle may have turned on the way, through the Munk moment)."""
    vd = W.vehicle_variant(W=114.8, B=114.8, r_b=[0.0, 0.0, 0.0])
    veh = dyn.Vehicle(vd, 1)
    c_w = np.array([[0.3], [-0.2], [0.1]])
    traj = _run(_state(), veh, 4000, 0.02, c_w=c_w)
    R = dyn.rotation(traj[-1, 3:7])[0]
    assert np.allclose(traj[-1, 7:10, 0], R.T @ c_w[:, 0], atol=1e-6)
    assert np.all(np.abs(traj[-1, 10:13, 0]) < 1e-6)


@settings(max_examples=40, deadline=None)
@given(st.lists(st.floats(-1.5, 1.5), min_size=6, max_size=6),
       st.lists(st.floats(-1, 1), min_size=4, max_size=4).filter(lambda a: np.linalg.norm(a) > 0.1))
def test_energy_non_increasing_without_restoring_and_current(nu0, q0):
    """c = 0, tau = 0, g = 0: C_RB and C_A do no work, damping only removes energy, so
    T = 1/2 nu^T M nu never increases (up to rounding)."""
    veh = dyn.Vehicle(W.vehicle_variant(W=114.8, B=114.8, r_b=[0.0, 0.0, 0.0]), 1)
    q0 = np.asarray(q0) / np.linalg.norm(q0)
    traj = _run(_state(q=q0, v=nu0[:3], w=nu0[3:]), veh, 200, 0.02)
    T = np.array([dyn.kinetic_energy(x, veh)[0] for x in traj])
    assert np.all(T[1:] <= T[:-1] * (1 + 1e-12) + 1e-300)


def test_energy_conserved_without_damping():
    """Same with zero damping: the Coriolis terms are workless, so T is conserved up to
    RK4's O(h^4) drift (a sign error in C_RB or C_A breaks this by orders of magnitude)."""
    vd = W.vehicle_variant(W=114.8, B=114.8, r_b=[0.0, 0.0, 0.0], lin_damp=[0.0] * 6,
                           quad_damp=[0.0] * 6)
    n = 16
    veh = dyn.Vehicle(vd, n)
    r = np.random.Generator(np.random.PCG64(9))
    x0 = _state(n=n, v=r.uniform(-1, 1, (3, n)), w=r.uniform(-2, 2, (3, n)))
    traj = _run(x0, veh, 500, 0.005)
    T = np.stack([dyn.kinetic_energy(x, veh) for x in traj])
    assert np.max(np.abs(T / T[0] - 1)) < 1e-7
    # angular momentum-like check: the motion really is non-trivial
    assert np.max(np.abs(traj[-1, 10:13] - x0[10:13])) > 0.05


def test_quaternion_unit_norm_invariant():
    veh = dyn.Vehicle(W.vehicle_variant(), 4)
    r = np.random.Generator(np.random.PCG64(4))
    q = r.standard_normal((4, 4))
    q /= np.linalg.norm(q, axis=0)
    x = _state(n=4, q=q, v=r.uniform(-1, 1, (3, 4)), w=r.uniform(-3, 3, (3, 4)))
    tau = r.uniform(-50, 50, (6, 4))
    for _ in range(300):
        x = dyn.rk4_substep(x, tau, veh, np.full((3, 4), 0.2), 0.02)
        assert np.all(np.abs(np.linalg.norm(x[3:7], axis=0) - 1) <= 1e-12)


def test_rk4_fourth_order_on_full_model():
    """Error against an h/64 reference over 1 s shrinks by ~16 per halving of h.  The
    quadratic damping |nu| nu has a kink at nu = 0 that lowers the order wherever a
    velocity component changes sign, so it is switched off here (the Bernoulli case pins
    it on its own)."""
    n = 6
    r = np.random.Generator(np.random.PCG64(12))
    s = r.uniform(0.8, 1.2, (3, n))
    veh = dyn.Vehicle(W.vehicle_variant(quad_damp=[0.0] * 6), n, *s)
    q = r.standard_normal((4, n))
    q /= np.linalg.norm(q, axis=0)
    x0 = _state(n=n, p=r.uniform(-2, 2, (3, n)), q=q, v=r.uniform(-1, 1, (3, n)),
                w=r.uniform(-1.5, 1.5, (3, n)))
    tau = r.uniform(-60, 60, (6, n))
    tau[3:] *= 0.01
    c_w = r.uniform(-0.3, 0.3, (3, n))

    def run(h):
        x = x0.copy()
        for _ in range(int(round(1.0 / h))):
            x = dyn.rk4_substep(x, tau, veh, c_w, h)
        return x

    ref = run(0.04 / 64)
    e = [np.max(np.abs(run(h) - ref)) for h in (0.04, 0.02, 0.01, 0.005)]
    ratios = [e[0] / e[1], e[1] / e[2], e[2] / e[3]]
    assert all(14 < rr < 18 for rr in ratios), (e, ratios)


def test_rotation_matches_scipy():
    r = np.random.Generator(np.random.PCG64(6))
    q = r.standard_normal((4, 50))
    q /= np.linalg.norm(q, axis=0)
    mine = dyn.rotation(q)
    ref = Rotation.from_quat(np.stack([q[1], q[2], q[3], q[0]], axis=1)).as_matrix()
    assert np.allclose(mine, ref, atol=1e-14)


def test_quaternion_rate_matches_body_rate_rotation():
    """q(t) = q0 (x) exp(omega t / 2) for a constant body rate: the derivative at t = 0
    equals T(q0) omega (central difference, scipy's rotation-vector map)."""
    r = np.random.Generator(np.random.PCG64(8))
    for _ in range(10):
        q0 = r.standard_normal(4)
        q0 /= np.linalg.norm(q0)
        om = r.uniform(-2, 2, 3)
        R0 = Rotation.from_quat([q0[1], q0[2], q0[3], q0[0]])
        eps = 1e-6

        def q_at(t):
            qs = (R0 * Rotation.from_rotvec(om * t)).as_quat()
            qs = np.array([qs[3], qs[0], qs[1], qs[2]])
            return qs if np.dot(qs, q0) > 0 else -qs

        fd = (q_at(eps) - q_at(-eps)) / (2 * eps)
        mine = dyn.quat_rate_matrix(q0[:, None])[0] @ om
        assert np.allclose(mine, fd, atol=1e-8)


def test_position_rate_is_world_frame_velocity():
    """dp/dt = R v: a body-x velocity with a 90 degree yaw moves the vehicle along world y."""
    veh = dyn.Vehicle(W.vehicle_variant(W=114.8, B=114.8, r_b=[0, 0, 0]), 1)
    c = math.cos(math.pi / 4)
    xdot = dyn.rhs(_state(q=(c, 0, 0, c), v=(1.0, 0, 0)), np.zeros((6, 1)), veh, np.zeros((3, 1)))
    assert np.allclose(xdot[0:3, 0], [0, 1, 0], atol=1e-15)


def test_allocation_table_matches_geometry():
    Tm = W.ALLOC.astype(np.float64)
    for i in range(8):
        d, rpos = W.THRUSTER_DIR[i], W.THRUSTER_POS[i]
        col = np.concatenate([d, np.cross(rpos, d)])
        assert np.allclose(Tm[:, i], col, atol=5e-8)
    assert np.linalg.matrix_rank(Tm) == 6
    wrench_max = 40.0 * np.abs(Tm).sum(axis=1)
    assert np.allclose(wrench_max, [113.137, 113.137, 160.0, 34.88, 19.2, 30.207], atol=2e-3)


def _rand_states(n, seed):
    r = np.random.Generator(np.random.PCG64(seed))
    q = r.standard_normal((4, n))
    q /= np.linalg.norm(q, axis=0)
    return _state(n=n, p=r.uniform(-2, 2, (3, n)), q=q, v=r.uniform(-1.5, 1.5, (3, n)),
                  w=r.uniform(-1.5, 1.5, (3, n))), r


def test_current_forms_coincide():
    """The relative-velocity form and the mixed form (rigid-body terms on the absolute
    velocity, hydrodynamic terms on the relative one, added-mass inertia on dnu_r/dt) are
    the same equations for a constant irrotational current: bit-identical at c_w = 0,
    equal to rounding for any current, with domain-randomised constants and the default
    W != B and buoyancy offset."""
    n = 64
    x, r = _rand_states(n, 11)
    veh = dyn.Vehicle(W.VEHICLE, n, s_m=r.uniform(0.8, 1.2, n), s_a=r.uniform(0.8, 1.2, n), s_d=r.uniform(0.8, 1.2, n))
    tau = r.uniform(-50, 50, (6, n))
    zero = np.zeros((3, n))
    a = dyn.rhs(x, tau, veh, zero, dyn.FORM_RELATIVE)
    b = dyn.rhs(x, tau, veh, zero, dyn.FORM_MIXED)
    assert np.array_equal(a, b)
    c_w = r.uniform(-0.3, 0.3, (3, n))
    a = dyn.rhs(x, tau, veh, c_w, dyn.FORM_RELATIVE)
    b = dyn.rhs(x, tau, veh, c_w, dyn.FORM_MIXED)
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12)
    # and the forms are not trivially equal: without dnu_c/dt the result moves
    c = dyn.rhs(x, tau, veh, c_w, dyn.FORM_NO_CURRENT_RATE)
    assert np.abs(c[7:10] - a[7:10]).max() > 1e-2
    xa, xb = x.copy(), x.copy()
    for _ in range(200):
        xa = dyn.rk4_substep(xa, tau * 0, veh, c_w, 0.02, dyn.FORM_RELATIVE)
        xb = dyn.rk4_substep(xb, tau * 0, veh, c_w, 0.02, dyn.FORM_MIXED)
    assert np.allclose(xa, xb, rtol=1e-10, atol=1e-10)


def test_current_rate_term_by_finite_difference():
    """dnu/dt(x, c_w) - dnu/dt(x with v -> v - R^T c_w, no current) is the rate of the body-
    frame current, d/dt R(q(t))^T c_w along dq/dt = 1/2 q (x) (0, omega): for a constant body
    rate the attitude is q(t) = q0 (x) (cos(|w| t / 2), sin(|w| t / 2) w / |w|), rotated here
    with scipy and differenced centrally."""
    n = 16
    x, r = _rand_states(n, 12)
    veh = dyn.Vehicle(W.VEHICLE, n)
    c_w = r.uniform(-0.3, 0.3, (3, n))
    tau = r.uniform(-50, 50, (6, n))
    R0 = Rotation.from_quat(np.stack([x[4], x[5], x[6], x[3]], axis=1))
    c_b = R0.inv().apply(c_w.T).T
    xr = x.copy()
    xr[7:10] -= c_b
    diff = dyn.rhs(x, tau, veh, c_w)[7:13] - dyn.rhs(xr, tau, veh, np.zeros((3, n)))[7:13]
    dt = 1e-4
    w = x[10:13].T
    fd = []
    for s in (dt, -dt):
        Rt = R0 * Rotation.from_rotvec(w * s)          # body-frame rate: q0 (x) exp(w t / 2)
        fd.append(Rt.inv().apply(c_w.T).T)
    rate = (fd[0] - fd[1]) / (2 * dt)
    assert np.allclose(diff[0:3], rate, atol=1e-7)
    assert np.allclose(diff[3:6], 0.0, atol=1e-12)
    assert np.abs(rate).max() > 0.05                   # the term is exercised


def test_current_coupling_spinning_drift_closed_form():
    """W = B, r_b = 0, no thrust, a current, body velocity equal to the current in body axes
    (no relative flow) and a spin.  With the isotropic inertia and rotational added mass no
    Coriolis or Munk term arises, so the relative flow stays zero while the vehicle turns:
    the vehicle drifts with the current, p(t) = p0 + c_w t, and each body rate decays by its
    1-DOF linear + quadratic damping closed form
        w(t) = d_l w0 e^{-kt} / (d_l + d_q |w0| (1 - e^{-kt})),  k = d_l / (I + A),
    with the yaw angle of a spin about the body z axis
        psi(t) = (I + A) / d_q ln(1 + d_q w0 (1 - e^{-kt}) / d_l).
    The drift needs the body-frame current's rate: dropping it lets p leave the line by
    O(|c_w| psi)."""
    vd = W.vehicle_variant(W=114.8, B=114.8, r_b=[0.0, 0.0, 0.0])
    f = lambda v: float(np.float32(v))  # noqa: E731
    Mrot = f(vd["inertia"][2]) + f(vd["added_mass"][5])
    dl, dq = f(vd["lin_damp"][5]), f(vd["quad_damp"][5])
    assert f(vd["inertia"][0]) == f(vd["inertia"][2]) and f(vd["added_mass"][3]) == f(vd["added_mass"][5])
    r = np.random.Generator(np.random.PCG64(13))
    n = 8
    q0 = r.standard_normal((4, n))
    q0 /= np.linalg.norm(q0, axis=0)
    c_w = r.uniform(-0.3, 0.3, (3, n))
    R0 = Rotation.from_quat(np.stack([q0[1], q0[2], q0[3], q0[0]], axis=1))
    v0 = R0.inv().apply(c_w.T).T
    w0 = np.zeros((3, n))
    w0[2, :4] = r.uniform(0.5, 1.5, 4) * np.array([1, -1, 1, -1])          # spin about body z
    w0[:, 4:] = r.uniform(-1.2, 1.2, (3, 4))                                # any direction
    p0 = r.uniform(-2, 2, (3, n))
    x0 = _state(n=n, p=p0, q=q0, v=v0, w=w0)
    h, steps = 0.01, 300
    t = h * steps
    veh = dyn.Vehicle(vd, n)
    traj = _run(x0, veh, steps, h, c_w=c_w)
    xe = traj[-1]
    k = dl / Mrot
    e = math.exp(-k * t)
    w_want = dl * w0 * e / (dl + dq * np.abs(w0) * (1 - e))
    assert np.allclose(xe[10:13], w_want, rtol=1e-7, atol=1e-9)
    assert np.allclose(xe[0:3], p0 + c_w * t, atol=1e-7)
    assert np.allclose(xe[7:10], Rotation.from_quat(np.stack([xe[4], xe[5], xe[6], xe[3]], axis=1)).inv()
                       .apply(c_w.T).T, atol=1e-8)
    psi = Mrot / dq * np.log(1 + dq * np.abs(w0[2, :4]) * (1 - e) / dl) * np.sign(w0[2, :4])
    q_want = (R0[:4] * Rotation.from_rotvec(np.stack([0 * psi, 0 * psi, psi], axis=1))).as_quat()
    q_want = np.stack([q_want[:, 3], q_want[:, 0], q_want[:, 1], q_want[:, 2]])
    s = np.sign(np.sum(q_want * xe[3:7, :4], axis=0))
    assert np.allclose(xe[3:7, :4], q_want * s, atol=1e-8)
    # without the body-frame current's rate (or with its sign flipped) the drift fails
    for bad in (dyn.FORM_NO_CURRENT_RATE,):
        xb = x0
        for _ in range(steps):
            xb = dyn.rk4_substep(xb, np.zeros((6, n)), veh, c_w, h, bad)
        assert np.abs(xb[0:3] - (p0 + c_w * t)).max() > 1e-2
