"""Seeded synthetic inputs shared by the GPU path's tests and bench and by the CPU oracle.

This package holds the configuration table and random draws only; it computes no
part of any compression method."""
from .configs import CONFIGS, PAPER_GRID, config  # noqa: F401
from .gen import (Workload, make_workload, prompt_kv, prompt_q, step_inputs,  # noqa: F401
                  calib_kv, key_sigma)
