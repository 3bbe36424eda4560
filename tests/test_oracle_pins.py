"""The oracle against closed forms, invariants and brute force (CPU only)."""

import math

import numpy as np
import pytest

import oracle
from oracle import aggregate as agg
from tests import pins


@pytest.mark.parametrize("pin", pins.ALL_FEATURE_PINS, ids=lambda p: p.__name__)
def test_feature_pin(pin):
    fails = pin(oracle.token_features)
    assert not fails, "\n".join(fails[:10])


def test_bf16_decode():
    bits = np.array([0x3F80, 0xC000, 0x7F80, 0xFF80, 0x0001, 0x8000, 0x4049], dtype=np.uint16)
    v = oracle.decode_logits(bits, "bf16")
    assert v[0] == 1.0 and v[1] == -2.0
    assert v[2] == math.inf and v[3] == -math.inf
    assert v[4] == 2.0 ** -133  # smallest positive bfloat16 (subnormal)
    assert v[5] == 0.0 and math.copysign(1.0, v[5]) == -1.0
    assert v[6] == 3.140625


def test_flags():
    z = np.zeros(16, dtype=np.float32)
    r = oracle.token_features(z, "f32", 16, 1.0)
    assert r["flags"] == oracle.FLAG_BAD_ID and r["rank"] == -1 and math.isnan(r["logprob"])
    assert r["entropy"] == pytest.approx(math.log(16))
    for T in (0.0, -1.0, math.inf, math.nan, 2.0 ** -101):
        r = oracle.token_features(z, "f32", 1, T)
        assert r["flags"] == oracle.FLAG_BAD_TP and math.isnan(r["entropy"]) and r["argmax"] == -1
    for P in (0.0, -0.5, math.nan):
        assert oracle.token_features(z, "f32", 1, 1.0, P)["flags"] == oracle.FLAG_BAD_TP
    for bad in (math.nan, math.inf):
        zz = z.copy()
        zz[3] = bad
        r = oracle.token_features(zz, "f32", 1, 1.0)
        assert r["flags"] == oracle.FLAG_NONFINITE and math.isnan(r["lse"]) and r["rank"] == -1
    r = oracle.token_features(np.full(4, -np.inf, dtype=np.float32), "f32", 1, 1.0)
    assert r["flags"] == oracle.FLAG_NONFINITE
    zz = z.copy()
    zz[0] = math.nan
    assert oracle.token_features(zz, "f32", -1, 1.0)["flags"] == oracle.FLAG_NONFINITE | oracle.FLAG_BAD_ID
    big = np.array([2.0 ** 101, 0.0], dtype=np.float32)
    assert oracle.token_features(big, "f32", 0, 1.0)["flags"] == oracle.FLAG_BAD_TP
    assert oracle.token_features(big, "f32", 0, 2.0)["flags"] == 0
    assert oracle.token_features(np.zeros(4, dtype=np.float32), "f32", 0, 2.0 ** -100)["flags"] == 0
    zz = z.copy()
    zz[2] = math.nan
    assert oracle.token_features(zz, "f32", 0, 0.0)["flags"] == oracle.FLAG_NONFINITE | oracle.FLAG_BAD_TP


def test_exact_boundary_is_flagged_ambiguous():
    r = oracle.token_features(np.zeros(8, dtype=np.float32), "f32", 0, 1.0, 0.125)
    assert r["cutoff"] == 1 and r["ambiguous"]
    r = oracle.token_features(np.zeros(8, dtype=np.float32), "f32", 0, 1.0, 0.2)
    assert r["cutoff"] == 2 and not r["ambiguous"]


# ---------------------------------------------------------------------------
# aggregation, score, route
# ---------------------------------------------------------------------------

def _feats(lp, mp, ent, mg):
    return {"logprob": np.asarray(lp, float), "maxprob": np.asarray(mp, float),
            "entropy": np.asarray(ent, float), "margin": np.asarray(mg, float)}


def test_aggregate_closed_forms():
    n = 37
    ar = np.arange(1, n + 1, dtype=float)
    const = np.full(n, 0.25)
    f = _feats(ar, const, -ar, ar[::-1])  # -entropy = ar
    a = agg.request_aggregate(f, [0, n], q=0.1)
    j = math.ceil(0.1 * n)  # = 4
    assert a["count"][0] == n
    np.testing.assert_array_equal(a["mean"][0], [(n + 1) / 2, 0.25, (n + 1) / 2, (n + 1) / 2])
    np.testing.assert_array_equal(a["min"][0], [1, 0.25, 1, 1])
    np.testing.assert_array_equal(a["quant"][0], [j, 0.25, j, j])


def test_aggregate_edges():
    f = _feats([1.0, -np.inf, 2.0, np.nan], [0.5, 0.4, 0.3, 0.2], [0, 0, 0, 0], [1, 2, 3, 4])
    a = agg.request_aggregate(f, [0, 1, 1, 3, 4], q=0.5)
    assert list(a["count"]) == [1, 0, 2, 1]
    np.testing.assert_array_equal(a["mean"][0], [1.0, 0.5, 0.0, 1.0])  # n = 1: all stats equal
    assert np.isnan(a["mean"][1]).all()  # empty request
    assert a["mean"][2, 0] == -np.inf and a["min"][2, 0] == -np.inf and a["quant"][2, 0] == -np.inf
    assert a["mean"][2, 1] == pytest.approx(0.35)
    assert np.isnan(a["mean"][3, 0]) and a["mean"][3, 1] == 0.2  # NaN poisons only its feature
    s = agg.score_from_aggregates(a)
    assert s[0] == 0.5 and np.isnan(s[1]) and s[2] == pytest.approx(0.35)
    # a zero weight skips the -inf logprob summaries instead of making NaN
    assert not np.isnan(s[2])


def test_quantile_brute_force():
    """Nearest-rank selection equals the counting characterisation."""
    rng = np.random.default_rng(5)
    for _ in range(200):
        n = int(rng.integers(1, 60))
        x = rng.choice([-1.0, 0.0, 0.5, 2.0, -np.inf], size=n) if rng.random() < 0.5 else rng.normal(size=n)
        q = float(rng.choice([0.0, 0.1, 0.25, 0.5, 0.9, 1.0]))
        a = agg.request_aggregate(_feats(x, x, -x, x), [0, n], q=q)
        j = max(1, math.ceil(q * n))
        # the selected value v satisfies #{x < v} < j <= #{x <= v}
        for col in range(4):
            v = a["quant"][0, col]
            assert np.count_nonzero(x < v) < j <= np.count_nonzero(x <= v)


def test_quantile_rank_rounding():
    """q * n is rounded once in float64: 0.1 * 10 is exactly 1, so j = 1."""
    x = np.arange(10, dtype=float)
    a = agg.request_aggregate(_feats(x, x, -x, x), [0, 10], q=0.1)
    assert a["quant"][0, 0] == 0.0
    a = agg.request_aggregate(_feats(x, x, -x, x), [0, 10], q=0.11)
    assert a["quant"][0, 0] == 1.0


def test_score_and_route():
    f = _feats([-1.0, -3.0], [0.8, 0.6], [0.5, 1.5], [2.0, 0.0])
    a = agg.request_aggregate(f, [0, 2])
    w = np.zeros((3, 4))
    w[0, 0] = 0.5   # mean logprob
    w[1, 2] = -1.0  # min(-entropy)
    w[2, 3] = 2.0   # quantile margin
    s = agg.score_from_aggregates(a, w, bias=0.25, link="identity")
    expect = 0.25 + 0.5 * (-2.0) - 1.0 * (-1.5) + 2.0 * 0.0
    assert s[0] == pytest.approx(expect)
    sg = agg.score_from_aggregates(a, w, bias=0.25, link="sigmoid")
    assert sg[0] == pytest.approx(1 / (1 + math.exp(-expect)))
    ship = agg.route(np.array([0.5, 0.49999, np.nan, 0.7]), 0.5)
    assert list(ship) == [1, 0, 0, 1]
