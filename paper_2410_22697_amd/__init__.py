"""MI355X-native per-partition sampling + halo prefetch buffer + feature gather
(MassiveGNN, arXiv 2410.22697) behind the C ABI of include/massive.h.

`Massive` is the only entry point; every step runs in libmassive's HIP
kernels. Importing `Massive` raises if libmassive.so has not been built.
"""
from .massive import (EXPORTS, LIB_PATH, MAX_INFLIGHT, TIMING_GROUPS, BatchBuffers, Massive,  # noqa: F401
                      MassiveError, StepResult, load)
