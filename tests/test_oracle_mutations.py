"""Plant plausible mistakes in copies of the oracle; some pin must catch each.

This checks that the pins are strong enough: a dropped term, a wrong sign or
index, a wrong tie-break or a missing temperature in the oracle must fail at
least one of them. The mistakes are planted in in-memory copies of the oracle's
source on the CPU; the real oracle is untouched.
"""

import os
import types

import numpy as np
import pytest

from tests import pins

ORACLE_DIR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")

FEATURE_MUTANTS = {
    "tie-break reversed": ("(idx < y)", "(idx > y)"),
    "rank 0-based": ("rank = 1 + int(", "rank = 0 + int("),
    "argmax last index": ("np.flatnonzero(z == z_max)[0]", "np.flatnonzero(z == z_max)[-1]"),
    "temperature dropped": ("    u = z / T\n", "    u = z\n"),
    "entropy sign": ("entropy = math.log(S_N) - ent_sum / S_N", "entropy = math.log(S_N) + ent_sum / S_N"),
    "entropy in bits": ("entropy = math.log(S_N) - ent_sum / S_N",
                        "entropy = (math.log(S_N) - ent_sum / S_N) / math.log(2)"),
    "lse without max": ("lse = u[a] + math.log(S_N)", "lse = math.log(S_N)"),
    "nucleus not renormalised": ("S_N = math.fsum(e_N)", "S_N = S"),
    "top-p strict inequality": [("side=\"left\"", "side=\"right\""),
                                ("while k > 1 and math.fsum(e[order[: k - 1]]) >= target:",
                                 "while k > 1 and math.fsum(e[order[: k - 1]]) > target:"),
                                ("while k < V and math.fsum(e[order[:k]]) < target:",
                                 "while k < V and math.fsum(e[order[:k]]) <= target:")],
    "top-p off by one": ("nucleus = order[:k]", "nucleus = order[: k + 1]"),
    "margin unscaled": ("margin = (z[a] - z_second) / T", "margin = (z[a] - z_second)"),
    "maxprob from full softmax": ("maxprob = 1.0 / S_N", "maxprob = 1.0 / S"),
    "bf16 decode shift": ("<< np.uint32(16)", "<< np.uint32(15)"),
    "logprob of argmax": ("        logprob = u[y] - lse\n", "        logprob = u[a] - lse\n"),
    "logprob underflow to -inf": ("        logprob = u[y] - lse\n",
                                  "        logprob = u[y] - lse if e[y] > 0.0 else -math.inf\n"),
}


def _mutant(src_name, edits):
    """A module built from the oracle's source with ``edits`` [(old, new), ...] applied."""
    src = open(os.path.join(ORACLE_DIR, src_name)).read()
    for old, new in edits:
        assert src.count(old) == 1, f"mutation site not unique: {old!r}"
        src = src.replace(old, new)
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src, f"mutant:{src_name}", "exec"), mod.__dict__)
    return mod


def _edits(spec):
    return spec if isinstance(spec, list) else [spec]


@pytest.mark.parametrize("name", sorted(FEATURE_MUTANTS))
def test_feature_mutant_is_caught(name):
    mod = _mutant("features.py", _edits(FEATURE_MUTANTS[name]))
    caught = []
    for pin in pins.ALL_FEATURE_PINS + [pins.pin_bf16_decode]:
        try:
            if pin(mod.token_features):
                caught.append(pin.__name__)
        except Exception as exc:  # a crash also counts as caught
            caught.append(f"{pin.__name__} raised {type(exc).__name__}")
        if caught:
            break
    assert caught, f"no pin catches mutant {name!r}"


AGG_MUTANTS = {
    "quantile index +1": ("return float(np.sort(x)[j - 1])", "return float(np.sort(x)[min(j, n - 1)])"),
    "quantile uses floor": ("j = max(1, math.ceil(float(q) * n))", "j = max(1, math.floor(float(q) * n))"),
    "mean over n-1": ("return math.fsum(x) / x.shape[0]", "return math.fsum(x) / max(1, x.shape[0] - 1)"),
    "entropy not negated": ("-np.asarray(feats[\"entropy\"], dtype=np.float64),",
                            "np.asarray(feats[\"entropy\"], dtype=np.float64),"),
    "route strict": ("return (s >= float(tau)).astype(np.uint8)", "return (s > float(tau)).astype(np.uint8)"),
    "min is max": ("out[\"min\"][i, f] = float(seg.min())", "out[\"min\"][i, f] = float(seg.max())"),
}


@pytest.mark.parametrize("name", sorted(AGG_MUTANTS))
def test_aggregate_mutant_is_caught(name):
    mod = _mutant("aggregate.py", _edits(AGG_MUTANTS[name]))
    fails = pins.pin_aggregate(mod)
    assert fails, f"no aggregation pin catches mutant {name!r}"
