"""Pins for the oracle: closed forms, invariants and pure-Python brute force.

Each ``pin_*`` function takes the feature function under test (the oracle's
``token_features``) so that the mutation tests can run the same pins against
deliberately broken copies of the oracle. Nothing here calls the HIP library.

The brute force (``brute_row``) does not reuse the oracle's method: the
order comes from sorting with a key, each probability is computed directly as
1 / sum_w exp((z_w - z_v) / T), and the nucleus is the smallest cardinality
of any token subset whose mass reaches P, found by enumerating all 2^V
subsets.
"""

from __future__ import annotations

import itertools
import math

import numpy as np

F32 = np.float32


def close(a, b, tol=1e-12):
    if isinstance(a, (int, np.integer)) and isinstance(b, (int, np.integer)):
        return a == b
    a, b = float(a), float(b)
    if math.isnan(a) or math.isnan(b):
        return math.isnan(a) and math.isnan(b)
    if math.isinf(a) or math.isinf(b):
        return a == b
    return abs(a - b) <= tol * max(1.0, abs(b))


# ---------------------------------------------------------------------------
# brute force, V <= 8
# ---------------------------------------------------------------------------

def brute_row(z, y, T, P=None):
    """Features of a tiny row by enumeration (Sec. 3.1 definitions)."""
    V = len(z)
    z = [float(v) for v in z]
    order = sorted(range(V), key=lambda v: (-z[v], v))
    rank = order.index(y) + 1
    a = order[0]
    second = z[order[1]]

    def prob(v):  # softmax(z / T)_v without a shared normaliser
        if z[v] == -math.inf:
            return 0.0
        return 1.0 / math.fsum(math.exp((z[w] - z[v]) / T) if z[w] != -math.inf else 0.0 for w in range(V))

    p = [prob(v) for v in range(V)]
    if P is None or P >= 1.0:
        N = set(range(V))
    else:
        best = None
        for m in range(1, V + 1):
            for sub in itertools.combinations(range(V), m):
                if math.fsum(p[v] for v in sub) >= P * math.fsum(p):
                    best = m
                    break
            if best is not None:
                break
        N = set(order[:best])
    mass_N = math.fsum(p[v] for v in N)
    q = {v: p[v] / mass_N for v in N}
    entropy = -math.fsum(q[v] * math.log(q[v]) for v in N if q[v] > 0)
    lse = math.log(math.fsum(math.exp(z[v] / T) for v in N if z[v] != -math.inf))
    logprob = (z[y] / T - lse) if (y in N and z[y] != -math.inf) else -math.inf
    return {
        "max_logit": z[a] / T,
        "lse": lse,
        "entropy": entropy,
        "logprob": logprob,
        "maxprob": max(q.values()),
        "margin": (z[a] - second) / T,
        "rank": rank,
        "argmax": a,
        "cutoff": len(N),
    }


def compare_to_brute(tf, z, y, T, P, tol=1e-9):
    got = tf(np.asarray(z, dtype=F32), "f32", y, T, P)
    ref = brute_row(np.asarray(z, dtype=F32), y, float(F32(T)), None if P is None else float(F32(P)))
    bad = [k for k in ref if not close(got[k], ref[k], tol)]
    return bad, got, ref


# ---------------------------------------------------------------------------
# pins; each returns a list of failure descriptions (empty = pass)
# ---------------------------------------------------------------------------

def pin_uniform(tf):
    """Uniform row: H = ln V, lse = c/T + ln V, p = 1/V, rank = y + 1."""
    fails = []
    for V, c, T, y, dtype in [(1000, 0.75, 0.7, 17, "f32"), (151936, -3.0, 1.0, 151935, "bf16"), (2, 0.0, 2.0, 1, "f32")]:
        raw = np.full(V, c, dtype=F32)
        if dtype == "bf16":
            raw = (raw.view(np.uint32) >> 16).astype(np.uint16)
        T32 = float(F32(T))
        r = tf(raw, dtype, y, T)
        exp = {"entropy": math.log(V), "lse": c / T32 + math.log(V), "maxprob": 1.0 / V,
               "margin": 0.0, "rank": y + 1, "argmax": 0, "logprob": -math.log(V), "max_logit": c / T32,
               "cutoff": V, "flags": 0}
        fails += [f"uniform V={V} {k}: {r[k]} != {v}" for k, v in exp.items() if not close(r[k], v)]
    return fails


def pin_one_hot(tf):
    """All but one token masked with -inf: H = 0, p_max = 1."""
    fails = []
    V, j, T = 64, 9, 0.5
    z = np.full(V, -np.inf, dtype=F32)
    z[j] = 2.5
    for y in (j, 0, 40):
        r = tf(z, "f32", y, T)
        exp = {"entropy": 0.0, "maxprob": 1.0, "lse": 2.5 / T, "max_logit": 2.5 / T, "argmax": j,
               "margin": math.inf, "logprob": 0.0 if y == j else -math.inf,
               # -inf ties break by index; token j outranks every masked token
               "rank": 1 if y == j else 1 + 1 + y - (1 if y > j else 0)}
        fails += [f"one-hot y={y} {k}: {r[k]} != {v}" for k, v in exp.items() if not close(r[k], v)]
    return fails


def pin_two_token(tf):
    """V = 2: a logistic distribution with closed forms in Delta = (a-b)/T."""
    fails = []
    for a, b, T in [(1.0, -0.5, 0.7), (-2.0, 3.0, 1.3), (0.25, 0.25, 1.0), (8.0, -8.0, 0.25)]:
        T32 = float(F32(T))
        d = (a - b) / T32
        ad = abs(d)
        p_hi = 1.0 / (1.0 + math.exp(-ad))
        p_lo = 1.0 - p_hi
        H = -(p_hi * math.log(p_hi) + (p_lo * math.log(p_lo) if p_lo > 0 else 0.0))
        lse = max(a, b) / T32 + math.log1p(math.exp(-ad))
        for y in (0, 1):
            r = tf(np.array([a, b], dtype=F32), "f32", y, T)
            zy = a if y == 0 else b
            exp = {"entropy": H, "maxprob": p_hi, "margin": ad, "lse": lse,
                   "logprob": zy / T32 - lse, "argmax": 0 if a >= b else 1}
            fails += [f"two-token {a},{b},{T} y={y} {k}: {r[k]} != {v}" for k, v in exp.items()
                      if not close(r[k], v, 1e-12)]
    return fails


def pin_dyadic_topp(tf):
    """Uniform V = 8: P = 1/2 keeps 4 tokens, P = 3/4 keeps 6, P -> 0+ keeps 1.

    Hand-derived values are stored in tests/golden/dyadic_topp.txt.
    """
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "dyadic_topp.txt")
    fails = []
    for line in open(path):
        line = line.split("#")[0].strip()
        if not line:
            continue
        kind, V, P, y, k, lp = line.split()
        V, y, k = int(V), int(y), int(k)
        P = float(P)
        if kind == "uniform":
            z = np.zeros(V, dtype=F32)
        else:  # "halving": z_v = -v ln 2 at T = 1, so p_v is proportional to 2^-v
            z = (-np.arange(V) * np.log(2.0)).astype(F32)
        r = tf(z, "f32", y, 1.0, P)
        exp_lp = -math.inf if lp == "-inf" else float(eval(lp, {"ln": math.log}))
        if r["cutoff"] != k:
            fails.append(f"{kind} V={V} P={P}: cutoff {r['cutoff']} != {k}")
        if not close(r["logprob"], exp_lp, 1e-6):
            fails.append(f"{kind} V={V} P={P} y={y}: logprob {r['logprob']} != {exp_lp}")
        if kind == "uniform" and not close(r["entropy"], math.log(k)):
            fails.append(f"uniform V={V} P={P}: entropy {r['entropy']} != ln {k}")
    return fails


def pin_tie_grid(tf, V_max=5):
    """Exhaustive grids z in {-1, 0, 1/2, 1}^V: order-derived integers vs brute force."""
    fails = []
    vals = (-1.0, 0.0, 0.5, 1.0)
    for V in range(2, V_max + 1):
        for z in itertools.product(vals, repeat=V):
            zz = np.asarray(z, dtype=F32)
            order = sorted(range(V), key=lambda v: (-z[v], v))
            for y in range(V):
                r = tf(zz, "f32", y, 1.0)
                if r["rank"] != order.index(y) + 1 or r["argmax"] != order[0]:
                    fails.append(f"ties z={z} y={y}: rank {r['rank']} argmax {r['argmax']}")
                    if len(fails) > 5:
                        return fails
    return fails


def pin_topp_tie_grid(tf):
    """Top-p cutoffs on tie grids vs subset enumeration (V <= 4)."""
    fails = []
    vals = (-1.0, 0.0, 0.5, 1.0)
    for V in (2, 3, 4):
        for z in itertools.product(vals, repeat=V):
            for P in (0.3, 0.55, 0.9):
                for y in range(V):
                    bad, got, ref = compare_to_brute(tf, z, y, 1.0, P)
                    if bad:
                        fails.append(f"topp z={z} P={P} y={y}: {[(k, got[k], ref[k]) for k in bad]}")
                        if len(fails) > 5:
                            return fails
    return fails


def pin_brute_random(tf, n_cases=300, seed=0x50520007):
    """Random tiny rows (V <= 8) with random temperature and top-p vs brute force."""
    rng = np.random.default_rng(seed)
    fails = []
    for _ in range(n_cases):
        V = int(rng.integers(2, 9))
        if rng.random() < 0.3:
            z = rng.choice([-2.0, -0.5, 0.0, 1.0, 3.0], size=V)  # ties
        else:
            z = rng.normal(0, 2.0, size=V)
        if rng.random() < 0.15:
            z[rng.integers(0, V)] = -np.inf
            if np.isneginf(z).all():
                z[0] = 0.0
        T = float(rng.uniform(0.3, 1.5))
        P = None if rng.random() < 0.3 else float(rng.uniform(0.05, 0.99))
        y = int(rng.integers(0, V))
        bad, got, ref = compare_to_brute(tf, z.astype(F32), y, T, P)
        if bad:
            fails.append(f"brute V={V} z={z} T={T} P={P} y={y}: {[(k, got[k], ref[k]) for k in bad]}")
    return fails


def pin_power_of_two_temperature(tf):
    """features(z, T = 2^k) == features(z * 2^-k, T = 1) exactly (scaling is exact)."""
    rng = np.random.default_rng(11)
    fails = []
    z = (rng.normal(0, 3, 4096)).astype(F32)
    for kexp in (-2, -1, 1, 3):
        r1 = tf(z, "f32", 100, 2.0 ** kexp, 0.9)
        r2 = tf((z * F32(2.0 ** -kexp)).astype(F32), "f32", 100, 1.0, 0.9)
        for key in ("max_logit", "lse", "entropy", "logprob", "maxprob", "margin", "rank", "argmax", "cutoff"):
            if not close(r1[key], r2[key], 1e-14):
                fails.append(f"T=2^{kexp} {key}: {r1[key]} != {r2[key]}")
    return fails


def pin_shift(tf):
    """z -> z + c on an exact dyadic grid: max_logit and lse move by c/T, all else is unchanged."""
    rng = np.random.default_rng(12)
    fails = []
    z = (np.round(rng.normal(0, 8, 5000) * 1024) / 1024).clip(-64, 64).astype(F32)
    T = 0.7
    T32 = float(F32(T))
    for c in (0.5, -3.25, 17.0009765625):
        zc = (z + F32(c)).astype(F32)
        assert np.all(zc.astype(np.float64) == z.astype(np.float64) + c), "shift not exact"
        for P in (None, 0.85):
            r1, r2 = tf(z, "f32", 7, T, P), tf(zc, "f32", 7, T, P)
            for key in ("entropy", "logprob", "maxprob", "margin", "rank", "argmax", "cutoff"):
                if not close(r1[key], r2[key], 1e-11):
                    fails.append(f"shift c={c} P={P} {key}: {r1[key]} != {r2[key]}")
            for key in ("max_logit", "lse"):
                if not close(r2[key], r1[key] + c / T32, 1e-11):
                    fails.append(f"shift c={c} P={P} {key}: {r2[key]} != {r1[key]} + c/T")
    return fails


def pin_underflow_logprob(tf):
    """log p(y) stays finite when p(y) underflows float64: (z_y - z_a)/T - log S."""
    z = np.array([0.0, -60.0, -2.0], dtype=F32)
    T = 0.05  # p(1) = exp(-1200) / S underflows
    T32 = float(F32(T))
    S = 1.0 + math.exp(-40.0)  # exp(-1200) is below double's range
    expect = (-60.0) / T32 - math.log(S)
    r = tf(z, "f32", 1, T)
    return [] if close(r["logprob"], expect, 1e-12) else [f"underflow logprob {r['logprob']} != {expect}"]


def pin_permutation(tf):
    """Distinct values: permuting tokens (and y with them) permutes argmax only."""
    rng = np.random.default_rng(13)
    fails = []
    V = 3000
    z = rng.permutation(np.arange(V, dtype=np.float64) * 0.01 - 12).astype(F32)
    perm = rng.permutation(V)
    zp = z[perm]  # new token i is old token perm[i]
    inv = np.argsort(perm)
    for y in (0, 5, 2999):
        for P in (None, 0.7):
            r1, r2 = tf(z, "f32", y, 0.9, P), tf(zp, "f32", int(inv[y]), 0.9, P)
            for key in ("max_logit", "lse", "entropy", "logprob", "maxprob", "margin", "rank", "cutoff"):
                if not close(r1[key], r2[key], 1e-13):
                    fails.append(f"perm y={y} P={P} {key}: {r1[key]} != {r2[key]}")
            if perm[r2["argmax"]] != r1["argmax"]:
                fails.append(f"perm y={y}: argmax does not map")
    return fails


ALL_FEATURE_PINS = [pin_uniform, pin_one_hot, pin_two_token, pin_dyadic_topp, pin_tie_grid,
                    pin_topp_tie_grid, pin_brute_random, pin_power_of_two_temperature, pin_shift,
                    pin_permutation, pin_underflow_logprob]


def pin_bf16_decode(tf):
    """Known bfloat16 bit patterns decode to their exact values (through features)."""
    bits = np.array([0x3F80, 0xC000, 0x4049, 0x0001], dtype=np.uint16)  # 1, -2, 3.140625, 2^-133
    r = tf(bits, "bf16", 2, 1.0)
    fails = []
    if not close(r["max_logit"], 3.140625):
        fails.append(f"bf16 max_logit {r['max_logit']}")
    if not close(r["margin"], 3.140625 - 1.0):
        fails.append(f"bf16 margin {r['margin']}")
    return fails


def pin_aggregate(mod):
    """Aggregation closed forms, run against an aggregation module."""
    fails = []

    def feats(lp, mp, ent, mg):
        return {"logprob": np.asarray(lp, float), "maxprob": np.asarray(mp, float),
                "entropy": np.asarray(ent, float), "margin": np.asarray(mg, float)}

    n = 37
    ar = np.arange(1, n + 1, dtype=float)
    a = mod.request_aggregate(feats(ar, ar, -ar, ar), [0, n], q=0.1)
    j = math.ceil(0.1 * n)
    for stat, v in (("mean", (n + 1) / 2), ("min", 1.0), ("quant", float(j))):
        if not np.array_equal(a[stat][0], [v] * 4):
            fails.append(f"arith {stat}: {a[stat][0]} != {v}")
    s = mod.score_from_aggregates(a)
    if not close(s[0], (n + 1) / 2):
        fails.append(f"default score {s[0]}")
    ship = mod.route(np.array([0.5, 0.4999, np.nan]), 0.5)
    if list(ship) != [1, 0, 0]:
        fails.append(f"route {list(ship)}")
    return fails
