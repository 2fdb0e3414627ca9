"""The synthetic workloads, named by what they are.

Each entry fixes the problem shape (d, m, lambda, block size), the gradient
distribution and the run length. The gradient matrices stand in for the
per-sample gradients of the paper's models (ResNet18 ~11.2M and ResNet50
~25.6M parameters, Section 1 and Appendix on NF-ResNet50); no dataset or trained
weight is used anywhere.

Distributions:
  "gauss"      entries N(0, 1/d)
  "lognormal"  per-coordinate scale s_j ~ LogNormal(0, 1), fixed per seed;
               entries s_j * N(0, 1) / sqrt(d)
A fraction ``corr_frac`` of stream rows are made correlated with the previous
stream row: g_r = 0.8 * g_{r-1} + 0.6 * noise_r (computed in fp64, stored fp32).
"""

from dataclasses import dataclass, replace
from typing import Optional


@dataclass(frozen=True)
class Workload:
    name: str
    kind: str            # "dynamic", "static" or "optim"
    d: int
    m: int
    lam: float
    dist: str            # "gauss" or "lognormal"
    steps: int = 0       # sliding steps after the window is full (dynamic)
    queries: int = 0     # extra IHVP queries fused into every step (dynamic)
    corr_frac: float = 0.0
    block: int = 0       # static: block size B (B divides d)
    theta_std: float = 0.0
    fill_by_replace: bool = False   # dynamic: start empty, fill with m replaces
    scale_d: int = 0     # d in the 1/sqrt(d) entry scale (0: the workload's own d);
                         # reduced-size parity cases keep the full-size scale
    batch: int = 0       # optim: mini-batch size of the model's synthetic batches
    model: str = ""      # optim: the network trained
    page_cols: int = 0   # static: G in pinned host memory, paged through the device in pages of this many columns

    def scaled(self, **kw) -> "Workload":
        """Same recipe at another size (parity cases the oracle finishes in seconds)."""
        return replace(self, **kw)


WORKLOADS = {
    # tiny sliding window; every step checked against the oracle
    "dyn_tiny_d4096_m16": Workload(
        "dyn_tiny_d4096_m16", "dynamic", d=4096, m=16, lam=1e-3, dist="gauss",
        steps=32, fill_by_replace=True),
    # mid-size window, coefficient phase comparable to the streaming passes
    "dyn_d1m_m256": Workload(
        "dyn_d1m_m256", "dynamic", d=1_048_576, m=256, lam=1e-4, dist="lognormal",
        steps=100),
    # ResNet18-sized window with 8 extra IHVP queries fused into each step
    "dyn_resnet18_d11.2m_m1024_q8": Workload(
        "dyn_resnet18_d11.2m_m1024_q8", "dynamic", d=11_200_000, m=1024, lam=1e-5,
        dist="lognormal", steps=200, queries=8),
    # ResNet50-sized window (~105 GB fp32 resident in HBM), 10% correlated rows
    "dyn_resnet50_d25.6m_m1024": Workload(
        "dyn_resnet50_d25.6m_m1024", "dynamic", d=25_600_000, m=1024, lam=1e-5,
        dist="lognormal", steps=200, corr_frac=0.1),
    # static block-wise pruning statistics: 2048 blocks of 2048 coordinates
    "static_d4.19m_b2048_m1024": Workload(
        "static_d4.19m_b2048_m1024", "static", d=4_194_304, m=1024, lam=1e-4,
        dist="lognormal", block=2048, theta_std=0.05),
    # the full-d static precompute (Section 3.1, a single block B = d) at the
    # same size
    "static_full_d4.19m_m1024": Workload(
        "static_full_d4.19m_m1024", "static", d=4_194_304, m=1024, lam=1e-4,
        dist="lognormal", block=4_194_304, theta_std=0.05),
    # the two static workloads with G in pinned host memory, paged through the
    # device (Appendix C's host paging): 64 blocks per page, and 8 column pages
    "static_paged_d4.19m_b2048_m1024": Workload(
        "static_paged_d4.19m_b2048_m1024", "static", d=4_194_304, m=1024, lam=1e-4,
        dist="lognormal", block=2048, theta_std=0.05, page_cols=64 * 2048),
    "static_paged_full_d4.19m_m1024": Workload(
        "static_paged_full_d4.19m_m1024", "static", d=4_194_304, m=1024, lam=1e-4,
        dist="lognormal", block=4_194_304, theta_std=0.05, page_cols=524_288),
    # the optimizer loop on a CIFAR-shaped ResNet-20 (269,722 weights), batch 128,
    # window m = 512 (Section 4.2, Table 4 settings); random inputs and labels
    "optim_resnet20_cifar_b128_m512": Workload(
        "optim_resnet20_cifar_b128_m512", "optim", d=269_722, m=512, lam=1e-4,
        dist="gauss", steps=100, batch=128, model="resnet20"),
    # the same loop on a CIFAR-100-shaped WRN-40-2 (2,255,156 weights; Section 4.2,
    # Table 4's wide-ResNet runs)
    "optim_wrn40_2_cifar100_b128_m512": Workload(
        "optim_wrn40_2_cifar100_b128_m512", "optim", d=2_255_156, m=512, lam=1e-4,
        dist="gauss", steps=50, batch=128, model="wrn40_2"),
}

HEADLINE = "dyn_resnet50_d25.6m_m1024"


def get_workload(name: str) -> Workload:
    return WORKLOADS[name]
