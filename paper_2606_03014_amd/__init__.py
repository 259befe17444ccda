"""MI355X-native ragged mixture-of-agents generation engine.

The computation lives in libmoa.so (hand-written HIP kernels for gfx950 and a
C++ host engine behind the C ABI of include/moa.h); this package is its thin
Python binding (``moa``) and the host feeder (``engine``).
"""
from . import moa
from .engine import Engine, Feeder, run_feeder, run_straggler, engine_cfg, model_cfg

__all__ = ["moa", "Engine", "Feeder", "run_feeder", "run_straggler", "engine_cfg", "model_cfg"]
