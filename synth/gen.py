"""Keyed random draws for the synthetic workloads.

Every draw is keyed by (seed, stream, index) through splitmix64, so a row can be
produced on its own, in any order and in any batch size, and always comes out
the same on the same device type. torch's generator is Philox on the GPU and
Mersenne Twister on the CPU, so the GPU and CPU draws of one key differ: a test
that compares the HIP path with the oracle draws once and hands the same fp32
values to both.

Streams:
  0  per-coordinate scales s_j (fixed per seed)
  1  window rows and step rows (the gradient stream)
  2  extra query vectors
  3  Bernoulli draws deciding which stream rows are correlated
  4  weights theta (static pruning scores)
"""

import math

import torch

_MASK = (1 << 64) - 1


def _splitmix64(x: int) -> int:
    x = (x + 0x9E3779B97F4A7C15) & _MASK
    z = x
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return z ^ (z >> 31)


def seed64(seed: int, stream: int, index: int) -> int:
    """64-bit generator seed for one keyed draw."""
    h = _splitmix64(seed & _MASK)
    h = _splitmix64(h ^ (stream & _MASK))
    h = _splitmix64(h ^ (index & _MASK))
    return h


def _generator(device, seed, stream, index) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed64(seed, stream, index))
    return g


class GradientStream:
    """Rows of the gradient stream, query vectors and weights of one workload.

    Row r < m fills slot r of the window; step t (0-based) inserts row m + t.
    """

    def __init__(self, wl, seed: int = 0, device="cpu"):
        self.wl = wl
        self.seed = seed
        self.device = torch.device(device)
        self._scales = None
        self._last = None  # (r, row) cache for sequential correlated rows

    # -- per-coordinate scales ------------------------------------------------
    def scales(self):
        """fp64 s_j ~ LogNormal(0, 1), or None for the plain Gaussian recipe."""
        if self.wl.dist == "gauss":
            return None
        if self._scales is None:
            g = _generator(self.device, self.seed, 0, 0)
            z = torch.randn(self.wl.d, generator=g, device=self.device, dtype=torch.float64)
            self._scales = torch.exp(z)
        return self._scales

    def _fresh(self, stream: int, index: int) -> torch.Tensor:
        d = self.wl.d
        g = _generator(self.device, self.seed, stream, index)
        z = torch.randn(d, generator=g, device=self.device, dtype=torch.float32)
        s = self.scales()
        z64 = z.to(torch.float64)
        if s is not None:
            z64 *= s
        z64 /= math.sqrt(self.wl.scale_d or d)
        return z64.to(torch.float32)

    def is_correlated(self, r: int) -> bool:
        if self.wl.corr_frac <= 0.0 or r == 0:
            return False
        g = torch.Generator(device="cpu")
        g.manual_seed(seed64(self.seed, 3, r))
        u = torch.rand(1, generator=g, dtype=torch.float64).item()
        return u < self.wl.corr_frac

    # -- gradient stream ------------------------------------------------------
    def row(self, r: int) -> torch.Tensor:
        """Stream row r as an fp32 vector of length d on the stream's device."""
        if self._last is not None and self._last[0] == r:
            return self._last[1].clone()
        if not self.is_correlated(r):
            out = self._fresh(1, r)
        else:
            # walk back to the last uncorrelated row, then forward
            r0 = r
            while self.is_correlated(r0):
                r0 -= 1
            if self._last is not None and r0 <= self._last[0] < r:
                r0, prev = self._last[0], self._last[1]
            else:
                prev = self._fresh(1, r0)
            for rr in range(r0 + 1, r + 1):
                noise = self._fresh(1, rr)
                prev = (0.8 * prev.to(torch.float64) + 0.6 * noise.to(torch.float64)).to(torch.float32)
            out = prev
        self._last = (r, out)
        return out.clone()

    def rows(self, r0: int, n: int) -> torch.Tensor:
        out = torch.empty((n, self.wl.d), dtype=torch.float32, device=self.device)
        for i in range(n):
            out[i] = self.row(r0 + i)
        return out

    def window(self) -> torch.Tensor:
        """The m initial rows (stream rows 0..m-1)."""
        return self.rows(0, self.wl.m)

    def step_row(self, t: int) -> torch.Tensor:
        return self.row(self.wl.m + t)

    # -- queries and weights --------------------------------------------------
    def queries(self, t: int, n: int) -> torch.Tensor:
        """n extra query vectors for step t, same scales as the gradients."""
        out = torch.empty((n, self.wl.d), dtype=torch.float32, device=self.device)
        for q in range(n):
            out[q] = self._fresh(2, t * 1_000_003 + q)
        return out

    def theta(self) -> torch.Tensor:
        """Weights theta ~ N(0, theta_std^2), fp32."""
        g = _generator(self.device, self.seed, 4, 0)
        z = torch.randn(self.wl.d, generator=g, device=self.device, dtype=torch.float32)
        return (z.to(torch.float64) * self.wl.theta_std).to(torch.float32)
