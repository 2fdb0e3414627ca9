"""The oracle's pins are sharp: planted mistakes in the oracle are caught.

Each case loads a copy of one oracle module whose source has one plausible
slip planted in it (a damping scale, a sign, a triangular flag, a block
offset, a ring index, a tie order, a dropped factor or term), runs the pins
of that module against the copy, and requires at least one pin to fail. The
same pins pass on the unmodified module. Everything here runs on the CPU;
the pins compare with dense d x d inverses, Python's sort, closed forms and
the hand-worked fixtures, never with the oracle itself.
"""

import importlib.util
import json
import os

import numpy as np
import pytest

from oracle import bruteforce

HERE = os.path.dirname(__file__)
ORACLE = os.path.join(os.path.dirname(HERE), "oracle")


def _load(name, old=None, new=None):
    """oracle.<name> compiled from its source, with `old` replaced by `new`."""
    src = open(os.path.join(ORACLE, f"{name}.py")).read()
    if old is not None:
        assert src.count(old) == 1, f"mutation site not unique in oracle/{name}.py: {old!r}"
        src = src.replace(old, new)
    spec = importlib.util.spec_from_loader(f"oracle._mutant_{name}", loader=None)
    mod = importlib.util.module_from_spec(spec)
    mod.__package__ = "oracle"
    exec(compile(src, f"<mutant oracle/{name}.py>", "exec"), mod.__dict__)
    return mod


def _rel(a, b):
    return np.linalg.norm(np.asarray(a) - np.asarray(b)) / np.linalg.norm(np.asarray(b))


def _golden():
    with open(os.path.join(HERE, "golden", "handworked.json")) as f:
        return {c["name"]: c for c in json.load(f)["cases"]}


# ------------------------------------------------------------------ pins, by module

def _pins_dynamic(mod):
    """Ring trajectory against dense solves over the explicit last-m window,
    and extra IHVPs at the end."""
    rng = np.random.default_rng(3)
    d, m, lam = 40, 4, 0.3
    rows = (rng.standard_normal((9, d)) / np.sqrt(d)).astype(np.float32)
    orc = mod.WindowOracle(d, m, lam)
    ok = True
    for t in range(len(rows)):
        y = orc.slide(rows[t])
        win = rows[max(0, t - m + 1):t + 1]
        ok &= _rel(y, bruteforce.ihvp(win, lam, rows[t].astype(np.float64), m=m)) < 1e-10
    X = rng.standard_normal((2, d)).astype(np.float32)
    ok &= _rel(orc.ihvp(X), bruteforce.ihvp(rows[-m:], lam, X.astype(np.float64), m=m)) < 1e-10
    return bool(ok)


def _pins_static(mod):
    """Per-block diagonal against the dense inverse, three blocks against the
    blocks one by one, and the hand-worked fixtures."""
    rng = np.random.default_rng(5)
    m, B, lam = 6, 24, 1e-2
    G = (rng.standard_normal((m, 3 * B)) / np.sqrt(B)).astype(np.float32)
    ok = _rel(mod.block_inv_diag(G[:, :B], lam), bruteforce.inv_diag(G[:, :B], lam)) < 1e-11
    dense = np.concatenate([bruteforce.inv_diag(G[:, b * B:(b + 1) * B], lam) for b in range(3)])
    ok &= _rel(mod.inv_diag(G, lam, B), dense) < 1e-11
    gd = _golden()
    for name in ("sherman_morrison_m1_d2", "orthogonal_rows_m2_d2", "coupled_m2_d3"):
        c = gd[name]
        got = mod.block_inv_diag(np.array(c["G"], np.float32), c["lam"], c["m"])
        ok &= bool(np.allclose(got, c["diag"], rtol=1e-13, atol=0))
    return bool(ok)


def _pins_mask(mod):
    """Keep-mask against Python's sort with exact ties; scores and masks of the
    hand-worked fixture."""
    rng = np.random.default_rng(7)
    d = 301
    s = rng.integers(0, 12, d).astype(np.float64) / 7.0
    ok = True
    for keep in (1, 150, 300):
        order = sorted(range(d), key=lambda j: (-s[j], j))
        expect = np.zeros(d, np.uint8)
        expect[order[:keep]] = 1
        ok &= bool(np.array_equal(mod.keep_mask(s, keep), expect))
    c = _golden()["obd_mask_small"]
    sc = mod.scores(c["theta"], c["diag_in"])
    ok &= bool(np.allclose(sc, c["scores"], rtol=1e-15, atol=0))
    ok &= bool(np.array_equal(mod.keep_mask(sc, c["keep"]), c["mask"]))
    return bool(ok)


def _pins_optimizer(mod):
    """Weight trajectory against w <- w - lr * F^-1 (g + wd*w) with F formed
    densely from the explicit last-m list of fp32 vectors."""
    rng = np.random.default_rng(9)
    d, m, lam, lr, wd = 30, 3, 0.2, 0.1, 0.05
    opt = mod.MFACOracle(d, m, lam)
    w = rng.standard_normal(d)
    w_ref = w.copy()
    hist = []
    ok = True
    for _ in range(7):
        g = rng.standard_normal(d) / np.sqrt(d)
        w, _ = opt.step(w, g, lr, wd)
        v = (g + wd * w_ref).astype(np.float32)
        hist.append(v)
        w_ref = w_ref - lr * bruteforce.ihvp(np.array(hist[-m:]), lam, v.astype(np.float64), m=m)
        ok &= _rel(w, w_ref) < 1e-10
    return bool(ok)


def _pins_recursions(mod):
    """The paper's recursions (D, B, q; V, q) against dense inverses."""
    rng = np.random.default_rng(11)
    m, d, lam = 5, 20, 0.1
    G = rng.standard_normal((m, d)) / np.sqrt(d)
    x = rng.standard_normal(d)
    D = mod.dynamic_D(G @ G.T, lam, m)
    B = mod.dynamic_B(D, lam, m)
    ok = _rel(mod.dynamic_ihvp(G, D, B, lam, m, x), bruteforce.ihvp(G, lam, x)) < 1e-10
    V, q = mod.static_precompute(G, lam)
    ok &= _rel(mod.static_ihvp(V, q, lam, x), bruteforce.ihvp(G, lam, x)) < 1e-10
    ok &= _rel(mod.static_inv_diag(V, q, lam), bruteforce.inv_diag(G, lam)) < 1e-10
    return bool(ok)


PINS = {"dynamic": _pins_dynamic, "static": _pins_static, "mask": _pins_mask, "optimizer": _pins_optimizer,
        "recursions": _pins_recursions}


@pytest.mark.parametrize("name", sorted(PINS))
def test_pins_pass_on_the_oracle(name):
    assert PINS[name](_load(name))


MUTANTS = [
    # window oracle (Theorem 1 / Woodbury): damping scale, sign, ring slot, half-updated Gram
    ("dynamic", "A = self.K + self.m * self.lam * np.eye(self.m)", "A = self.K + self.lam * np.eye(self.m)"),
    ("dynamic", "(X[:, j0:j1].astype(np.float64) - U.T @ b) / self.lam",
     "(X[:, j0:j1].astype(np.float64) + U.T @ b) / self.lam"),
    ("dynamic", "slot = self.steps % self.m", "slot = self.steps % (self.m - 1)"),
    ("dynamic", "self.K[:, slot] = p", "pass"),
    # block-wise inverse diagonal: damping scale, sign, transposed factor, block offset
    ("static", "R = np.linalg.cholesky(K + mm * lam * np.eye(Gb.shape[0]))",
     "R = np.linalg.cholesky(K + lam * np.eye(Gb.shape[0]))"),
    ("static", "return (1.0 - np.sum(W * W, axis=0)) / lam", "return (1.0 + np.sum(W * W, axis=0)) / lam"),
    ("static", "W = sla.solve_triangular(R, Gb, lower=True)", "W = sla.solve_triangular(R.T, Gb, lower=False)"),
    ("static", "out.append(block_inv_diag(G[:, b * block:(b + 1) * block], lam, m))",
     "out.append(block_inv_diag(G[:, b:b + block], lam, m))"),
    # OBD scores and keep-mask: tie order, dropped factor 2, ascending instead of descending
    ("mask", "np.lexsort((np.arange(d), -s))", "np.lexsort((-np.arange(d), -s))"),
    ("mask", "return t * t / (2.0 * np.asarray(diag, dtype=np.float64))",
     "return t * t / np.asarray(diag, dtype=np.float64)"),
    ("mask", "np.lexsort((np.arange(d), -s))", "np.lexsort((np.arange(d), s))"),
    # the paper's recursions: dropped m in a pivot, a sign, the printed first
    # denominator of Algorithm 3 (no "m +"), a transposed index
    ("recursions", "D[i:, i:] -= np.outer(r, r) / (m + D[i - 1, i - 1])",
     "D[i:, i:] -= np.outer(r, r) / (D[i - 1, i - 1])"),
    ("recursions", "q[i + 1:] -= q[i] * D[i, i + 1:]", "q[i + 1:] += q[i] * D[i, i + 1:]"),
    ("recursions", "q[i] = mm + v @ g", "q[i] = v @ g if i == 0 else mm + v @ g"),
    ("recursions", "w = -D[:i, i] / piv[:i]", "w = -D[i, :i] / piv[:i]"),
    # optimizer loop: weight decay dropped, wrong step direction
    ("optimizer", "v = np.asarray(g, np.float64) + np.asarray(wd, np.float64) * w",
     "v = np.asarray(g, np.float64)"),
    ("optimizer", "return w - np.asarray(lr, np.float64) * y, y", "return w + np.asarray(lr, np.float64) * y, y"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[f"{n}-{i}" for i, (n, _, _) in enumerate(MUTANTS)])
def test_planted_mistake_is_caught(name, old, new):
    try:
        passed = PINS[name](_load(name, old, new))
    except (AssertionError, ValueError, np.linalg.LinAlgError, IndexError):
        passed = False   # the mutant breaks outright: also caught
    assert not passed, f"oracle/{name}.py with {new!r} for {old!r} still passes its pins"
