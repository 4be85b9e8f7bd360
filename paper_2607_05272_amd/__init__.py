"""MI355X (gfx950) batched rollout of the inference-serving simulator of "Adaptive
Inference Batching using Policy Gradients": Python binding of libbatchsim.so.

The binding only marshals arguments; all simulation, policy and return computation runs
in the library's HIP kernels. Torch provides device memory and the stream.
"""
from .sim import (Sim, weights_layout, pack_weights, unpack_weights,  # noqa: F401
                  Trajectory)
from ._lib import (SimError, load, ALGO_PPO, ALGO_REINFORCE, FUSE_OFF, FUSE_AUTO,  # noqa: F401
                   FUSE_ON)
