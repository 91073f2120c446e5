"""Batched 6-DOF underwater-vehicle rollout on AMD Instinct MI355X (gfx950).

The compute path is libauv.so (HIP kernels behind the C interface in include/auv.h);
`_abi` binds it with ctypes under the same names; `env.AuvEnv` owns the environment
buffers and `ppo.PpoLearner` those of the PPO update, `shac.ShacLearner` those of the SHAC actor.
Importing this package loads the library and fails if it has not been built.
"""
from . import _abi  # noqa: F401  (loads libauv.so; raises ImportError if missing)
from ._abi import (AUV_ACT_EXTERNAL, AUV_ACT_POLICY_MEAN, AUV_ACT_POLICY_SAMPLE,  # noqa: F401
                   AUV_ACT_RANDOM, AUV_F_CURRENT, AUV_F_DR, AUV_F_LISSAJOUS, AUV_F_STAGGER,
                   AuvError)
from .env import AuvEnv, upload_mlp  # noqa: F401
from .ppo import PpoLearner, PpoNet  # noqa: F401
from .shac import ShacLearner  # noqa: F401
