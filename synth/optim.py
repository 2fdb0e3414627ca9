"""Seeded inputs for the optimizer-loop cases: initial weights, loss
coefficients and mini-batches. Random draws only (no optimizer arithmetic).

Two problems:
  linear_problem  loss_t(w) = sum_i <C_{t,i}, w_i> over a list of parameter
                  tensors; its gradient C_t does not depend on w, so both sides
                  of a parity test see the same gradient sequence.
  mlp_problem     a tanh MLP with a squared-error loss on Gaussian inputs and
                  targets (the gradient depends on the weights).
"""

import torch

from .gen import seed64


def _gen(seed, stream):
    g = torch.Generator(device="cpu")
    g.manual_seed(seed64(seed, stream, 0) & ((1 << 63) - 1))
    return g


def linear_problem(seed, shapes, steps, scale=1.0):
    """(w0 list, [C_t list for t < steps]) as float64 CPU tensors."""
    g = _gen(seed, 20)
    w0 = [torch.randn(s, generator=g, dtype=torch.float64) * 0.1 for s in shapes]
    C = [[torch.randn(s, generator=g, dtype=torch.float64) * scale for s in shapes] for _ in range(steps)]
    return w0, C


def mlp_problem(seed, sizes, batch, steps):
    """(weights list [W1, b1, W2, b2, ...], [(x_t, y_t) for t < steps]) as
    float64 CPU tensors; W_l is (sizes[l+1], sizes[l])."""
    g = _gen(seed, 21)
    ws = []
    for a, b in zip(sizes[:-1], sizes[1:]):
        ws.append(torch.randn((b, a), generator=g, dtype=torch.float64) / a ** 0.5)
        ws.append(torch.randn((b,), generator=g, dtype=torch.float64) * 0.1)
    data = [(torch.randn((batch, sizes[0]), generator=g, dtype=torch.float64),
             torch.randn((batch, sizes[-1]), generator=g, dtype=torch.float64)) for _ in range(steps)]
    return ws, data
