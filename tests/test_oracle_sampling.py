"""The oracle's sampling distribution against closed forms, invariants and
the pinned per-token features, with planted mistakes. CPU only."""

import math
import os
import types

import numpy as np
import pytest

import oracle
from oracle import sampling as osmp

ORACLE_DIR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")


def pin_closed_forms(mod):
    fails = []
    p = mod.token_probabilities(np.full(9, 1.5, np.float32), "f32", 0.7)
    if not np.all(p == 1.0 / 9.0):
        fails.append(f"uniform row: {p}")
    for z0, z1, T in ((0.0, 1.0, 1.0), (2.0, -1.0, 0.5), (3.0, 3.0, 2.0)):
        p = mod.token_probabilities(np.array([z0, z1], np.float32), "f32", T)
        exp = 1.0 / (1.0 + math.exp(-(z0 - z1) / T))
        if abs(p[0] - exp) > 1e-15:
            fails.append(f"logistic {z0} {z1} {T}: {p[0]} vs {exp}")
    p = mod.token_probabilities(np.array([0.0, -np.inf, 0.0, -np.inf], np.float32), "f32", 1.0)
    if not np.array_equal(p, [0.5, 0.0, 0.5, 0.0]):
        fails.append(f"masked: {p}")
    return fails


def pin_invariants(mod):
    fails = []
    rng = np.random.default_rng(8)
    for _ in range(30):
        z = (np.round(rng.normal(0, 3, 50) * 64) / 64).astype(np.float32)  # a 1/64 grid: +4 is exact
        z[rng.random(50) < 0.1] = -np.inf
        z[0] = 1.0  # at least one finite logit
        T = float(np.float32(rng.uniform(0.3, 2.0)))
        p = mod.token_probabilities(z, "f32", T)
        if abs(math.fsum(p) - 1.0) > 1e-14 or (p < 0).any() or (p[np.isneginf(z)] != 0).any():
            fails.append("not a distribution")
        q = mod.token_probabilities(z + np.float32(4.0), "f32", T)
        if np.max(np.abs(p - q)) > 1e-14:
            fails.append("shift")
        bits = (z.view(np.uint32) >> 16).astype(np.uint16)  # bf16 of the truncated values
        zb = (bits.astype(np.uint32) << 16).view(np.float32)
        if np.max(np.abs(mod.token_probabilities(bits, "bf16", T) - mod.token_probabilities(zb, "f32", T))) > 0:
            fails.append("bf16 decoding")
    return fails


def pin_features(mod):
    """log p_y equals the pinned oracle's log-prob of y for every y."""
    fails = []
    rng = np.random.default_rng(9)
    for _ in range(5):
        z = rng.normal(0, 2, 40).astype(np.float32)
        T = 0.8
        p = mod.token_probabilities(z, "f32", T)
        for y in range(40):
            lp = oracle.token_features(z, "f32", y, T)["logprob"]
            if abs(math.log(p[y]) - lp) > 1e-12 * (1 + abs(lp)):
                fails.append(f"y={y}: {math.log(p[y])} vs {lp}")
                break
    return fails


def pin_undefined(mod):
    fails = []
    if mod.token_probabilities(np.array([0.0, np.nan], np.float32), "f32", 1.0) is not None:
        fails.append("NaN row")
    if mod.token_probabilities(np.array([-np.inf, -np.inf], np.float32), "f32", 1.0) is not None:
        fails.append("all masked")
    if mod.token_probabilities(np.array([0.0, 1.0], np.float32), "f32", 0.0) is not None:
        fails.append("T = 0")
    if mod.token_probabilities(np.array([0.0, np.inf], np.float32), "f32", 1.0) is not None:
        fails.append("+inf")
    return fails


ALL = [pin_closed_forms, pin_invariants, pin_features, pin_undefined]


@pytest.mark.parametrize("pin", ALL, ids=lambda p: p.__name__)
def test_pin(pin):
    fails = pin(osmp)
    assert not fails, "\n".join(fails[:10])


MUTANTS = {
    "no temperature": ("    u = z / T\n", "    u = z\n"),
    "normalised by the maximum": ("    return e / math.fsum(e)", "    return e / e.max()"),
    "flags ignored": ("    if f[\"flags\"] & (FLAG_NONFINITE | FLAG_BAD_TP):\n        return None\n", ""),
    "temperature squared": ("    u = z / T\n", "    u = z / (T * T)\n"),
}


@pytest.mark.filterwarnings("ignore::RuntimeWarning")  # a mutant may divide by zero
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    old, new = MUTANTS[name]
    src = open(os.path.join(ORACLE_DIR, "sampling.py")).read()
    assert src.count(old) == 1, f"mutation site not unique: {old!r}"
    mod = types.ModuleType("sampling_mutant")
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), os.path.join(ORACLE_DIR, "sampling.py"), "exec"), mod.__dict__)

    def fails(pin):
        try:
            return bool(pin(mod))
        except (ValueError, ZeroDivisionError, TypeError, FloatingPointError):
            return True

    assert any(fails(pin) for pin in ALL), f"mutant '{name}' passed every pin"
