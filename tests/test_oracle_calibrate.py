"""The oracle's threshold calibration and P-square streaming quantile against
counting characterisations, an exact identity of the algorithm on linear
data, affine equivariance, convergence to known quantiles, and planted
mistakes. CPU only."""

import math
import os
import types

import numpy as np
import pytest

from oracle import calibrate as ocal

ORACLE_DIR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")


def pin_calibrate(mod):
    """tau is the largest pool value t with #{s >= t} >= k, k = max(1, ceil(q n)),
    NaN excluded (brute force over small pools with ties)."""
    fails = []
    rng = np.random.default_rng(3)
    for trial in range(300):
        n = int(rng.integers(1, 12))
        s = rng.choice([0.1, 0.2, 0.25, 0.5, 0.7, 0.9], size=n).astype(np.float64)
        if trial % 3 == 0:
            s[rng.integers(0, n)] = np.nan
        q = float(rng.choice([0.0, 0.1, 0.3, 0.5, 0.77, 1.0]))
        tau, ns = mod.calibrate_threshold(s, q)
        pool = s[~np.isnan(s)]
        if q == 0.0 or pool.size == 0:
            exp = (math.inf, 0)
        else:
            k = max(1, math.ceil(q * pool.size))
            cands = [t for t in pool if np.count_nonzero(pool >= t) >= k]
            t = max(cands)
            exp = (t, int(np.count_nonzero(pool >= t)))
        if (tau, ns) != exp:
            fails.append(f"pool {s.tolist()} q={q}: {(tau, ns)} != {exp}")
    return fails


def pin_p2_small(mod):
    """Up to 5 observations: the exact nearest-rank quantile."""
    fails = []
    rng = np.random.default_rng(4)
    for _ in range(200):
        n = int(rng.integers(1, 6))
        v = rng.normal(0, 1, n)
        p = float(rng.choice([0.1, 0.5, 0.9]))
        got = mod.p2_quantile(v, p)
        exp = np.sort(v)[max(1, math.ceil(p * n)) - 1]
        if got != exp:
            fails.append(f"{v.tolist()} p={p}: {got} != {exp}")
    return fails


def pin_p2_linear(mod):
    """On the stream 1, 2, .., N the quantile function is the identity, so
    every parabolic or linear prediction is exact: each marker's height
    equals its position after every observation."""
    fails = []
    for p in (0.1, 0.5, 0.9):
        est = mod.P2Quantile(p)
        for t in range(1, 400):
            est.add(float(t))
            if t >= 5 and any(abs(h - n) > 1e-9 for h, n in zip(est.q, est.n)):
                fails.append(f"p={p} after {t}: heights {est.q} positions {est.n}")
                break
    return fails


def pin_p2_affine(mod):
    """a x + b (a > 0) gives a * estimate + b."""
    fails = []
    rng = np.random.default_rng(5)
    for _ in range(20):
        v = rng.exponential(1.0, 300)
        a, b = float(rng.uniform(0.5, 4)), float(rng.uniform(-3, 3))
        e1 = mod.p2_quantile(v, 0.1)
        e2 = mod.p2_quantile(a * v + b, 0.1)
        if not abs(e2 - (a * e1 + b)) <= 1e-9 * (1 + abs(e2)):
            fails.append(f"affine: {e2} vs {a * e1 + b}")
    return fails


def pin_p2_convergence(mod):
    """Long i.i.d. streams: the estimate approaches the distribution's quantile."""
    fails = []
    rng = np.random.default_rng(6)
    u = rng.uniform(0, 1, 100000)
    for p, tol in ((0.1, 0.005), (0.5, 0.005), (0.9, 0.005)):
        e = mod.p2_quantile(u, p)
        if abs(e - p) > tol:
            fails.append(f"uniform p={p}: {e}")
    g = rng.normal(0, 1, 100000)
    if abs(mod.p2_quantile(g, 0.1) - (-1.2815515655446004)) > 0.02:
        fails.append("normal 10th percentile")
    return fails


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "p2_jain_chlamtac_example.txt")


def pin_p2_published_example(mod):
    """The marker heights of the P-square paper's worked example."""
    rows = {}
    for line in open(GOLDEN):
        if line.strip() and not line.startswith("#"):
            key, *vals = line.split()
            rows[key] = [float(v) for v in vals]
    est = mod.P2Quantile(rows["p"][0])
    for x in rows["obs"]:
        est.add(x)
    got = [round(h, 2) for h in est.q]
    fails = [] if got == rows["heights"] else [f"heights {got} != {rows['heights']}"]
    if round(est.estimate(), 2) != rows["heights"][2]:
        fails.append(f"estimate {est.estimate()}")
    return fails


def pin_p2_ties(mod):
    """An observation equal to a marker height belongs to the cell above that
    marker (q_k <= x < q_(k+1)). Worked by hand for p = 0.5 on 1,2,3,4,5,3,3:
    the 6th observation (3) moves positions 4 and 5 to (1,2,3,5,6), whose
    desired positions (1,2.25,3.5,4.75,6) call for no adjustment; the 7th
    gives (1,2,3,6,7) against (1,2.5,4,5.5,7), so the middle marker moves up
    one position to 3 + (2*1/3 + 2*1/1)/4 = 11/3 (parabolic, inside (2, 4))."""
    est = mod.P2Quantile(0.5)
    try:
        for x in (1, 2, 3, 4, 5, 3, 3):
            est.add(float(x))
    except IndexError as e:
        return [f"cell search fell off the markers: {e}"]
    fails = []
    if est.n != [1, 2, 4, 6, 7]:
        fails.append(f"positions {est.n}")
    if abs(est.estimate() - 11.0 / 3.0) > 1e-12:
        fails.append(f"estimate {est.estimate()} != 11/3")
    return fails


def pin_p2_nonfinite(mod):
    """NaN is skipped; an infinite observation makes the estimate NaN."""
    fails = []
    v = list(np.random.default_rng(7).normal(0, 1, 50))
    base = mod.p2_quantile(v, 0.3)
    if mod.p2_quantile(v[:20] + [math.nan] + v[20:], 0.3) != base:
        fails.append("a NaN observation changed the estimate")
    for bad in (math.inf, -math.inf):
        for at in (2, 30):
            e = mod.p2_quantile(v[:at] + [bad] + v[at:], 0.3)
            if not math.isnan(e):
                fails.append(f"{bad} at {at}: estimate {e}")
    if not math.isnan(mod.p2_quantile([], 0.5)) or not math.isnan(mod.p2_quantile([math.nan], 0.5)):
        fails.append("empty stream")
    return fails


ALL = [pin_calibrate, pin_p2_nonfinite, pin_p2_small, pin_p2_linear, pin_p2_affine, pin_p2_convergence,
       pin_p2_published_example, pin_p2_ties]


@pytest.mark.parametrize("pin", ALL, ids=lambda p: p.__name__)
def test_pin(pin):
    fails = pin(ocal)
    assert not fails, "\n".join(fails[:10])


MUTANTS = {
    "k by floor": ("k = max(1, math.ceil(q * s.shape[0]))", "k = max(1, math.floor(q * s.shape[0]))"),
    "NaN in the pool": ("    s = s[~np.isnan(s)]\n    q = float", "    q = float"),
    "strict ship count": ("np.count_nonzero(s >= tau)", "np.count_nonzero(s > tau)"),
    "marker targets": ("self.f = (0.0, self.p / 2.0, self.p, (1.0 + self.p) / 2.0, 1.0)",
                       "self.f = (0.0, self.p, self.p, (1.0 + self.p) / 2.0, 1.0)"),
    "cell boundary": ("while not (q[k] <= x < q[k + 1]):", "while not (q[k] < x <= q[k + 1]):"),
    "infinity fed": ("        if math.isinf(x):\n            self.poisoned = True\n            return\n", ""),
    "parabola sign": ("(n[i] - n[i - 1] + s) * (q[i + 1] - q[i])", "(n[i] - n[i - 1] - s) * (q[i + 1] - q[i])"),
    "linear neighbour": ("qp = q[i] + s * (q[i + s] - q[i]) / (n[i + s] - n[i])",
                         "qp = q[i] + s * (q[i - s] - q[i]) / (n[i - s] - n[i])"),
    "positions above the cell": ("for i in range(k + 1, 5):", "for i in range(k, 5):"),
    "small-sample rank": ("j = max(1, math.ceil(self.p * len(v)))", "j = max(1, math.floor(self.p * len(v)))"),
}


def _mutant(old, new):
    src = open(os.path.join(ORACLE_DIR, "calibrate.py")).read()
    assert src.count(old) == 1, f"mutation site not unique: {old!r}"
    mod = types.ModuleType("calibrate_mutant")
    exec(compile(src.replace(old, new), "mutant:calibrate.py", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    mod = _mutant(*MUTANTS[name])

    def fails(pin):
        try:
            return bool(pin(mod))
        except (IndexError, ValueError, ZeroDivisionError):
            return True

    assert any(fails(pin) for pin in ALL), f"mutant '{name}' passed every pin"
