"""Host-side checks of bench.py: the one-GPU contract and the workload shapes
its modes rely on (no GPU needed)."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_optimizer_models_have_the_workload_sizes():
    sys.path.insert(0, ROOT)
    import bench
    from synth import WORKLOADS
    for wl in WORKLOADS.values():
        if wl.kind == "optim":
            net = bench.OPTIM_MODELS[wl.model][0]()
            assert sum(p.numel() for p in net.parameters()) == wl.d, wl.name


def test_pass_bytes_match_the_algorithmic_budget():
    """2 m d 4 + 3 d 4 bytes per step at the ResNet50-sized window (210.0 GB)."""
    sys.path.insert(0, ROOT)
    import bench
    b1, b2, bw = bench.pass_bytes(25_600_000, 1024)
    assert b1 + b2 + bw == 2 * 1024 * 25_600_000 * 4 + 4 * 25_600_000 * 4
    assert abs((b1 + b2 + bw) / 1e9 - 210.0) < 0.5


@pytest.mark.parametrize("kernel", ["k_pass1", "k_pass2_rows"])
def test_committed_counters_match_the_current_pass_sources(kernel):
    """The committed HBM counter summary was taken on the current streaming
    kernels (else bench.py reports traffic as null) and on the ResNet50-sized
    window: a workload without its own summary gets no traffic figure."""
    sys.path.insert(0, ROOT)
    import bench
    assert kernel == "k_pass1" or kernel == bench.pass2_kernel(1, 1024)
    assert bench.read_counters("dyn_d1m_m256", kernel) is None
    t = bench.read_counters("dyn_resnet50_d25.6m_m1024", kernel)
    if t is None:
        pytest.skip("the committed HBM counters were taken on other pass sources: retake them")
    b1, b2, _ = bench.pass_bytes(25_600_000, 1024)
    alg = b1 if kernel == "k_pass1" else b2
    assert abs(t / alg - 1.0) < 0.02


@pytest.mark.parametrize("kernel", ["k_pass1", "k_pass2"])
def test_multi_vector_counters_cover_their_algorithmic_bytes(kernel):
    """The 8-query window's own summary: traffic at least its algorithmic
    bytes (4(m + 9)d for pass 1, 4(m + 17)d for pass 2) and within 5%."""
    sys.path.insert(0, ROOT)
    import bench
    t = bench.read_counters("dyn_resnet18_d11.2m_m1024_q8", kernel)
    if t is None:
        pytest.skip("no counters of the 8-query window on the current pass sources: retake them")
    d, m = 11_200_000, 1024
    alg = 4.0 * (m + 9) * d if kernel == "k_pass1" else 4.0 * (m + 17) * d
    assert 0.99 < t / alg < 1.05
