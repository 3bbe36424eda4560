"""Per-request aggregation, score and routing: HIP path vs the fp64 oracle."""

import numpy as np
import pytest
import torch

import oracle
from oracle import aggregate as oagg
import paper_2608_28726_amd as pr
from paper_2608_28726_amd import workloads as wl
from tests.gpu_common import gpu_features, oracle_features, require_gpu, to_dev
from tests.helpers import assert_floats, assert_ints, decisions_agree

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _synthetic_features(lengths, rng, with_specials=True):
    n = int(np.sum(lengths))
    f = {
        "logprob": rng.normal(-1.0, 1.0, n).astype(np.float32),
        "maxprob": rng.uniform(0, 1, n).astype(np.float32),
        "entropy": rng.uniform(0, 5, n).astype(np.float32),
        "margin": rng.exponential(1.0, n).astype(np.float32),
    }
    # ties: quantise some columns heavily
    f["margin"][: n // 2] = np.round(f["margin"][: n // 2] * 2) / 2
    if with_specials and n > 10:
        f["logprob"][3] = -np.inf
        f["entropy"][7] = np.nan
        f["maxprob"][5] = 0.0
        f["entropy"][9] = 0.0
        f["entropy"][10] = -0.0
    return f


def _to_gpu_feats(f):
    return {k: torch.as_tensor(v).cuda() for k, v in f.items()}


def _gpu_agg(f_gpu, offsets, **kw):
    out = pr.request_aggregate(f_gpu, torch.as_tensor(offsets, dtype=torch.int32).cuda(), **kw)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def _check_agg(g, o, scores_o):
    assert_ints("count", g["count"], o["count"])
    for stat in ("min", "quant"):
        # selections return stored values: exact (with -0 == +0)
        go, oo = g[stat].astype(np.float64), o[stat]
        same = (go == oo) | (np.isnan(go) & np.isnan(oo))
        assert same.all(), f"{stat}: {np.argwhere(~same)[:5].tolist()} gpu {go[~same][:5]} oracle {oo[~same][:5]}"
    assert_floats("mean", g["mean"].ravel(), o["mean"].ravel(), atol=0, rtol=1e-6)
    assert_floats("score", g["score"], scores_o, atol=0, rtol=1e-6)


@pytest.mark.parametrize("q", [0.1, 0.0, 0.5, 1.0, 0.37])
def test_aggregate_synthetic(q):
    rng = np.random.default_rng(int(q * 100) + 1)
    lengths = np.concatenate([[0, 1, 2, 10], rng.integers(0, 600, 40), [5000, 0]])
    offsets = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    f = _synthetic_features(lengths, rng)
    g = _gpu_agg(_to_gpu_feats(f), offsets, q=q)
    o = oagg.request_aggregate({k: v.astype(np.float64) for k, v in f.items()}, offsets, q=q)
    _check_agg(g, o, oagg.score_from_aggregates(o))


def test_score_heads():
    rng = np.random.default_rng(9)
    lengths = rng.integers(1, 300, 30)
    offsets = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    f = _synthetic_features(lengths, rng, with_specials=False)
    w = rng.normal(0, 1, (3, 4))
    w[1, 2] = 0.0
    for link in ("identity", "sigmoid"):
        g = _gpu_agg(_to_gpu_feats(f), offsets, weights=w, bias=0.3, link=link)
        o = oagg.request_aggregate({k: v.astype(np.float64) for k, v in f.items()}, offsets)
        _check_agg(g, o, oagg.score_from_aggregates(o, w, 0.3, link))


def test_route():
    rng = np.random.default_rng(3)
    s = rng.uniform(0, 1, 5000).astype(np.float32)
    s[:4] = [0.5, np.nextafter(np.float32(0.5), np.float32(0)), np.nan, 1.0]
    ship, n_ship = pr.route(torch.as_tensor(s).cuda(), 0.5)
    ship = ship.cpu().numpy()
    expect = oagg.route(s.astype(np.float64), 0.5)
    assert np.array_equal(ship, expect)
    assert int(n_ship.item()) == int(expect.sum())
    e0, n0 = pr.route(torch.empty(0, dtype=torch.float32).cuda(), 0.5)
    assert int(n0.item()) == 0


def test_end_to_end_ragged():
    """Features -> summaries -> score -> route, GPU vs oracle on the ragged row model."""
    w = wl.scaled(wl.WORKLOADS["ragged_64req_v151936_bf16"], n_req=6, len_hi=24)
    b = wl.make_batch(w, device="cpu")
    logits, ids, T = to_dev(b.logits, b.sampled_ids, b.temperature)
    print(f"case e2e rows={b.n_rows}", flush=True)
    feats = pr.token_features(logits, ids, T)
    agg = pr.request_aggregate(feats, torch.as_tensor(b.offsets).cuda(), q=w.q)
    ship, n_ship = pr.route(agg["score"], w.tau)
    torch.cuda.synchronize()
    of = oracle_features(logits, ids, T)
    oa = oagg.request_aggregate(of, b.offsets, q=w.q)
    os_ = oagg.score_from_aggregates(oa)
    assert_floats("score", agg["score"].cpu().numpy(), os_)
    for stat in ("mean", "min", "quant"):
        assert_floats(stat, agg[stat].cpu().numpy().ravel(), oa[stat].ravel())
    assert decisions_agree(ship.cpu().numpy(), os_, w.tau).all()


def test_validate_offsets():
    good = torch.tensor([0, 3, 3, 10], dtype=torch.int32).cuda()
    assert pr.validate_offsets(good, 10)
    assert not pr.validate_offsets(good, 11)
    assert not pr.validate_offsets(torch.tensor([0, 5, 3], dtype=torch.int32).cuda(), 3)
