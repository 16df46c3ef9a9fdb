"""Seeded synthetic input generator (shapes, lengths, indices, weights, table
values).  Shared by the CPU oracle and the GPU path; holds none of the pooling
arithmetic."""
from .configs import (ALL, BF16, DLRM, F16, F32, FULL, LARGE, MIXED, SKEWED, TINY,  # noqa: F401
                      TINY_INT, Workload, scaled)
from .gen import Inputs, counter_values, make_inputs, splitmix64, table_seed  # noqa: F401
