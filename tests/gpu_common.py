"""Shared helpers for the GPU parity tests (HIP path vs the fp64 oracle)."""

import sys

import numpy as np
import pytest
import torch

# Relative L2 bound for fp32 outputs against the fp64 oracle (the bound the
# dynamic and static paths are held to at every size).
REL_TOL = 1e-4


def rel_l2(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2107_03356_amd import _binding as B
    B.load()  # must not fall back: a missing library is an error where a GPU is present
    return torch.device("cuda:0")


def say(*a):
    """Name the case before a GPU step (flushed, so a fault still shows it)."""
    print("[case]", *a, file=sys.stderr, flush=True)
