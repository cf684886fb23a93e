"""Seeded synthetic inputs for the candidate-scoring path.

This package produces inputs only: observed configurations and SLO values,
GP hyperparameters, a candidate pool, a trained random forest exported to flat
arrays, Delta, the reference point, the best observed value.  It holds none of
the scoring arithmetic (no GP, acquisition, hypervolume, forest walk or
selection), and both the product path and the oracle read what it produces.
"""
from .synth import (CONFIGS, MASTER_SEED, levels, make_pool, make_workload, sobol_table,  # noqa: F401
                    space_constraints, vllm_decode, vllm_space)
