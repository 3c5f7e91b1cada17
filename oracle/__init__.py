"""CPU oracle (test infrastructure only): a plain fp64 NumPy statement of the
layer-parallel ResNet hot path, used to check the GPU library. Only tests, the
smoke check and the benchmark's CPU-baseline leg import it."""
from .lp_oracle import *  # noqa: F401,F403
