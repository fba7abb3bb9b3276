"""Seeded synthetic workloads (graph descriptions + tensors) shared by the
oracle and the library's tests and benchmark.  Holds no operator or
scheduling arithmetic."""
from .configs import (CONFIG_NAMES, NETWORK_NAMES, SPECS, infer_shapes, make, make_tensors,  # noqa: F401
                      param_shapes, unit_ops, with_batch)
