"""Seeded synthetic inputs for the revisit-consistency hot path.

This package only *synthesises* inputs: camera trajectories, planar metric
depth maps rendered from random planes, Q/K/V tensors and slot tables. It
contains none of the method's arithmetic (no retrieval score, no
reprojection warp, no attention), so the fp64 oracle and the HIP path can
both consume exactly the same arrays without sharing any code.

Every array is produced on the host by ``numpy.random.Generator(PCG64(seed))``
and returned as numpy (fp32 / int32, bf16 tensors as their fp32 values
rounded to nearest-even bf16). See ``workloads.configs`` for the five
workload recipes.
"""

from .configs import (  # noqa: F401
    CONFIG_NAMES,
    Workload,
    make_config,
    make_c1,
    make_c2,
    make_c3,
    make_c4,
    make_c5,
    make_reproj_batch,
    make_rotation_batch,
)
from .synth import bf16_round, bf16_bits, look_pose, perturb_pose  # noqa: F401
