"""fp64 CPU oracle for the batched 6-DOF underwater-vehicle rollout step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and its
Python binding) imports, calls or links anything under this directory; only the tests,
the smoke check and the CPU-baseline leg of the benchmark do.

The oracle is the method written out plainly, step by step, in NumPy float64,
vectorised over environments, with the textbook matrix forms (6x6 mass, Coriolis and
damping matrices, a linear solve) where the GPU path uses hand-expanded cross products.
It shares no code with the HIP path: its only inputs are the seeded data in
``workloads`` and counter-based Philox draws it computes itself.

Modules
  rng       Philox4x32-10, uniform / affine maps, Shoemake rotations, Box-Muller
  dynamics  Fossen 6-DOF equations of motion (paper Sec. IV-D, Eq. 8, the model behind the
            MPC baseline) and classic RK4 with quaternion renormalisation
  env       reset / domain randomisation, references, observation, reward, auto-reset,
            batch statistics, rollouts (paper Sec. IV-A, IV-B, IV-C, V-A)
  mlp       bf16 round-to-nearest-even, policy / value MLP forward, Gaussian log-prob
  gae       generalised advantage estimation (the PPO learner of Sec. III-A1)
  paper_task the paper's own training task: 12-D axis-angle observation, 6-D wrench action,
            five-term reward with an action moving average, gravity randomisation
  ppo       clipped-surrogate PPO objective, its gradient through both MLPs (with the
            bf16 quantisation points of the MFMA path), global-norm clipping, Adam
  fluid     the inertia-box fluid model of the paper's MJX simulation (equivalent box,
            viscous + quadratic drag, no added mass) as an alternate hydrodynamics
  shac      the SHAC actor objective over a short window of the paper task and its
            gradient through the policy, reward, observation, RK4 + Fossen and the
            terminal value (torch autograd on float64 tensors)

Every function is pinned by a ``-m "not gpu"`` test against closed forms, invariants,
special cases or an independent library; see the test files under ``tests/``.
"""
from . import rng, dynamics, fluid, mlp, gae, env, ppo, paper_task, shac  # noqa: F401
