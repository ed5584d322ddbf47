"""Seeded synthetic inputs shared by the oracle and the GPU library.

This package is the only code both sides use.  It holds the workload shapes
and the random-input recipe, and none of the method's arithmetic.
"""
from .configs import (DONOR_BLANK, DONOR_DIFF, DONOR_ZERO, WORKLOADS, Workload,
                      get)
from .inputs import (cell_lw, cell_steps, derive_seed, make_layer, make_new_rows, make_q, to_numpy,
                     torch_dtype)

__all__ = ["DONOR_BLANK", "DONOR_DIFF", "DONOR_ZERO", "WORKLOADS", "Workload", "get",
           "cell_lw", "cell_steps", "derive_seed", "make_layer", "make_new_rows", "make_q", "to_numpy",
           "torch_dtype"]
