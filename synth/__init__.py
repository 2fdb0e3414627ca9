"""Seeded synthetic inputs for the M-FAC IHVP workloads.

This package draws random numbers and nothing else: gradient rows, extra query
vectors and weights with the shapes and distributions of the workloads the
library is measured on. It holds none of the method's arithmetic. Both the HIP
path (tests, bench) and the fp64 oracle take their inputs from here; neither
imports the other.
"""

from .workloads import WORKLOADS, Workload, get_workload
from .gen import GradientStream, seed64

__all__ = ["WORKLOADS", "Workload", "get_workload", "GradientStream", "seed64"]
