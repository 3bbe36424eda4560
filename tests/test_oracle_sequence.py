"""The oracle's paper feature sequence (top-K entropy, position fraction)
against its pins, and planted mistakes in copies of it that a pin must catch.
CPU only."""

import os
import types

import pytest

from oracle import sequence
from tests import pins_sequence as ps

ORACLE_DIR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")


@pytest.mark.parametrize("pin", ps.ALL_TOPK_PINS, ids=lambda p: p.__name__)
def test_topk_pin(pin):
    fails = pin(sequence.topk_entropy)
    assert not fails, "\n".join(fails[:10])


def test_sequence_pin():
    fails = ps.pin_sequence(sequence)
    assert not fails, "\n".join(fails)


def test_paper_k():
    assert sequence.PAPER_TOP_K == 20  # Sec. 3.1


MUTANTS = {
    "top-K mass renormalised": ("p = e[live] / S_N", "p = e[live] / math.fsum(e[live])"),
    "K off by one": ("top = order[: min(K, k)]", "top = order[: min(K - 1, k)]"),
    "full distribution under top-p": ("S_N = math.fsum(e[order[:k]])", "S_N = math.fsum(e)"),
    "top-K ignores the nucleus": ("top = order[: min(K, k)]", "top = order[:K]"),
    "entropy sign": ("return float(-math.fsum(p * logp))", "return float(math.fsum(p * logp))"),
    "temperature dropped": ("    u = z / T\n", "    u = z\n"),
    "least probable tokens": ("order = np.lexsort((idx, -z))", "order = np.lexsort((idx, z))"),
    "log of unnormalised mass": ("logp = (u[live] - u[a]) - math.log(S_N)", "logp = u[live] - u[a]"),
    "rho 0-based": ("rho[lo - base + t - 1] = t / n", "rho[lo - base + t - 1] = (t - 1) / n"),
    "h not negated": ("X[:, 2] = -np.asarray(topk_H, dtype=np.float64)", "X[:, 2] = np.asarray(topk_H, dtype=np.float64)"),
}


def _mutant(old, new):
    src = open(os.path.join(ORACLE_DIR, "sequence.py")).read()
    src = src.replace("from .features import", "from oracle.features import")
    assert src.count(old) == 1, f"mutation site not unique: {old!r}"
    src = src.replace(old, new)
    mod = types.ModuleType("sequence_mutant")
    exec(compile(src, "mutant:sequence.py", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_sequence_mutant_is_caught(name):
    mod = _mutant(*MUTANTS[name])
    caught = False
    for pin in ps.ALL_TOPK_PINS:
        try:
            caught = bool(pin(mod.topk_entropy))
        except Exception:  # a crash also counts as caught
            caught = True
        if caught:
            break
    if not caught:
        caught = bool(ps.pin_sequence(mod))
    assert caught, f"no pin catches mutant {name!r}"
