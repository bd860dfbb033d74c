"""fp64 CPU oracle (test infrastructure only; see oracle.py)."""
from .oracle import (all_rows, attention, attention_parallel, attention_rows, build,
                     default_workers, to_f64, weights)

__all__ = ["all_rows", "attention", "attention_parallel", "attention_rows", "build",
           "default_workers", "to_f64", "weights"]
