"""Pins for the oracle's paper feature sequence (top-K entropy and position
fraction): closed forms, special cases and pure-Python brute force.

Each pin takes the functions under test so that the mutation tests can run
the same pins against broken copies of ``oracle/sequence.py``. The brute
force picks the K most probable tokens by enumerating every K-subset of the
nucleus and keeping one of largest mass (no sort), with each probability
computed on its own as 1 / sum_w exp((z_w - z_v) / T).
"""

from __future__ import annotations

import itertools
import math

import numpy as np

from tests.pins import close

F32 = np.float32


def brute_topk_entropy(z, T, P, K):
    """H^{top-K} of a tiny row (V <= 8) by enumeration."""
    V = len(z)
    z = [float(v) for v in z]

    def prob(v):
        if z[v] == -math.inf:
            return 0.0
        return 1.0 / math.fsum(math.exp((z[w] - z[v]) / T) if z[w] != -math.inf else 0.0 for w in range(V))

    p = [prob(v) for v in range(V)]
    total = math.fsum(p)
    if P is None or P >= 1.0:
        N = list(range(V))
    else:
        # the nucleus: the first m tokens of the order (larger logit, then
        # lower index) for the smallest m such that some m-subset reaches P
        order = sorted(range(V), key=lambda v: (-z[v], v))
        m = next(m for m in range(1, V + 1)
                 if any(math.fsum(p[v] for v in sub) >= P * total for sub in itertools.combinations(range(V), m)))
        N = order[:m]
    mass_N = math.fsum(p[v] for v in N)
    q = {v: p[v] / mass_N for v in N}
    kk = min(K, len(N))
    best = max(itertools.combinations(N, kk), key=lambda sub: math.fsum(q[v] for v in sub))
    return -math.fsum(q[v] * math.log(q[v]) for v in best if q[v] > 0)


def _f32(x):
    return np.asarray(x, dtype=F32)


def pin_topk_uniform(tk):
    """V equal logits: each p = 1/V, so H^{top-K} = min(K, V)/V * ln V."""
    fails = []
    for V, K, c, T in [(10, 3, 0.0, 1.0), (10, 10, 2.5, 0.7), (10, 25, -1.0, 1.3), (151936, 20, 0.75, 0.7)]:
        got = tk(np.full(V, c, dtype=F32), "f32", T, None, K)
        exp = min(K, V) / V * math.log(V)
        if not close(got, exp, 1e-11):
            fails.append(f"uniform V={V} K={K}: {got} != {exp}")
    return fails


def pin_topk_one(tk):
    """K = 1: H = -m ln m, m the largest probability computed directly."""
    rng = np.random.default_rng(21)
    fails = []
    for T in (0.4, 1.0, 2.0):
        z = _f32(rng.normal(0, 2, 300))
        zd = z.astype(np.float64)
        m = 1.0 / math.fsum(math.exp((w - zd.max()) / float(F32(T))) for w in zd)
        got = tk(z, "f32", T, None, 1)
        if not close(got, -m * math.log(m), 1e-11):
            fails.append(f"K=1 T={T}: {got} != {-m * math.log(m)}")
    return fails


def pin_topk_full(tk):
    """K >= V (or K >= the number of finite logits): the full Shannon entropy,
    computed from each probability on its own."""
    rng = np.random.default_rng(22)
    fails = []
    for V, K, masked in [(50, 50, 0), (50, 64, 0), (40, 30, 15)]:
        z = rng.normal(0, 1.5, V)
        z[:masked] = -np.inf
        z = _f32(z)
        T = float(F32(0.8))
        fin = [float(w) for w in z if w != -np.inf]
        p = [1.0 / math.fsum(math.exp((w - v) / T) for w in fin) for v in fin]
        H = -math.fsum(x * math.log(x) for x in p)
        got = tk(z, "f32", 0.8, None, K)
        if not close(got, H, 1e-11):
            fails.append(f"full V={V} K={K} masked={masked}: {got} != {H}")
    return fails


def pin_topk_ties(tk):
    """3 logits at 1 and 7 at 0, K = 5: the top 5 are the three at 1 and any
    two of the zeros (every choice gives the same sum)."""
    z = _f32([0, 1, 0, 0, 1, 0, 0, 1, 0, 0])
    S = 3 * math.e + 7
    p1, p0 = math.e / S, 1.0 / S
    exp = -(3 * p1 * math.log(p1) + 2 * p0 * math.log(p0))
    got = tk(z, "f32", 1.0, None, 5)
    return [] if close(got, exp, 1e-12) else [f"ties: {got} != {exp}"]


def pin_topk_nucleus(tk):
    """Top-p: the K terms use the probabilities renormalised on the nucleus;
    with a nucleus of at most K tokens the sum is the nucleus entropy."""
    fails = []
    # dyadic row: logits ln 8, ln 4, ln 2, ln 1 give masses 8:4:2:1 (+ 4 masked)
    z = _f32([math.log(8), math.log(4), math.log(2), 0.0, -np.inf, -np.inf, -np.inf, -np.inf])
    # P = 0.75 of 15 = 11.25: the nucleus is {8, 4} (12 >= 11.25)
    q = [8 / 12, 4 / 12]
    exp = -math.fsum(x * math.log(x) for x in q)
    for K in (2, 3, 20):
        got = tk(z, "f32", 1.0, 0.75, K)
        if not close(got, exp, 1e-6):  # the float32 logits are ln 8 etc. to 6e-8
            fails.append(f"nucleus K={K}: {got} != {exp}")
    got = tk(z, "f32", 1.0, 0.75, 1)
    if not close(got, -q[0] * math.log(q[0]), 1e-6):
        fails.append(f"nucleus K=1: {got}")
    return fails


def pin_topk_brute(tk, n_cases=300, seed=0x50520008):
    """Random tiny rows (V <= 8, ties, masked tokens, top-p, K = 1..V+1) vs brute force."""
    rng = np.random.default_rng(seed)
    fails = []
    for _ in range(n_cases):
        V = int(rng.integers(2, 9))
        z = rng.choice([-2.0, -0.5, 0.0, 1.0, 3.0], size=V) if rng.random() < 0.4 else rng.normal(0, 2.0, V)
        if rng.random() < 0.15:
            z[rng.integers(0, V)] = -np.inf
            if np.isneginf(z).all():
                z[0] = 0.0
        z = _f32(z)
        T = float(rng.uniform(0.3, 1.5))
        P = None if rng.random() < 0.3 else float(rng.uniform(0.05, 0.99))
        K = int(rng.integers(1, V + 2))
        got = tk(z, "f32", T, P, K)
        exp = brute_topk_entropy(z, float(F32(T)), None if P is None else float(F32(P)), K)
        if not close(got, exp, 1e-9):
            fails.append(f"brute V={V} z={z} T={T} P={P} K={K}: {got} != {exp}")
    return fails


def pin_topk_shift(tk):
    """Adding an exact constant to every logit leaves H^{top-K} unchanged."""
    rng = np.random.default_rng(23)
    z = (np.round(rng.normal(0, 4, 3000) * 1024) / 1024).clip(-64, 64).astype(F32)
    fails = []
    for c in (0.5, -7.25):
        zc = (z + F32(c)).astype(F32)
        for P in (None, 0.9):
            a, b = tk(z, "f32", 0.9, P, 20), tk(zc, "f32", 0.9, P, 20)
            if not close(a, b, 1e-11):
                fails.append(f"shift c={c} P={P}: {a} != {b}")
    return fails


def pin_topk_flags(tk):
    """Non-finite rows and bad temperatures give NaN."""
    fails = []
    for z, T, P in [([0.0, np.nan, 1.0], 1.0, None), ([0.0, np.inf], 1.0, None), ([-np.inf, -np.inf], 1.0, None),
                    ([0.0, 1.0], 0.0, None), ([0.0, 1.0], 1.0, 0.0)]:
        got = tk(_f32(z), "f32", T, P, 20)
        if not math.isnan(got):
            fails.append(f"flagged row {z} T={T} P={P}: {got}")
    return fails


ALL_TOPK_PINS = [pin_topk_uniform, pin_topk_one, pin_topk_full, pin_topk_ties, pin_topk_nucleus,
                 pin_topk_brute, pin_topk_shift, pin_topk_flags]


def pin_sequence(mod):
    """rho = t/T per request (empty requests own no rows) and the column
    order (logprob, maxprob, -H^{top-K}, rho)."""
    fails = []
    offsets = np.array([0, 3, 3, 7, 8])
    rho = mod.position_fraction(offsets)
    exp = [1 / 3, 2 / 3, 1.0, 0.25, 0.5, 0.75, 1.0, 1.0]
    if not np.array_equal(rho, np.array(exp)):
        fails.append(f"rho {rho} != {exp}")
    feats = {"logprob": np.arange(8) * -0.5, "maxprob": np.linspace(0.1, 0.8, 8)}
    H = np.linspace(0.0, 2.0, 8)
    X = mod.feature_sequence(feats, H, offsets)
    if X.shape != (8, 4):
        return fails + [f"X shape {X.shape}"]
    for c, col in enumerate([feats["logprob"], feats["maxprob"], -H, np.array(exp)]):
        if not np.array_equal(X[:, c], col):
            fails.append(f"X column {c}: {X[:, c]} != {col}")
    return fails
