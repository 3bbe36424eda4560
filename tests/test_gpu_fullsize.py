"""Full-size workloads in the launch configuration bench.py times: the oracle
checks sampled rows and whole requests; properties that hold at any size are
checked on every row."""

import math

import numpy as np
import pytest
import torch

import oracle
from oracle import aggregate as oagg
import paper_2608_28726_amd as pr
from paper_2608_28726_amd import workloads as wl
from tests.gpu_common import compare_features, require_gpu
from tests.helpers import assert_floats, decisions_agree

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _properties(f: dict, V: int, cutoff_is_V=True):
    """Invariants of valid rows: ranges and orderings every feature must obey."""
    flags = f["flags"]
    ok = flags == 0
    assert ok.all(), f"{(~ok).sum()} flagged rows"
    assert (f["rank"] >= 1).all() and (f["rank"] <= V).all()
    assert (f["argmax"] >= 0).all() and (f["argmax"] < V).all()
    assert (f["maxprob"] > 0).all() and (f["maxprob"] <= 1.0 + 1e-6).all()
    assert (f["entropy"] >= -1e-5).all() and (f["entropy"] <= math.log(V) + 1e-4).all()
    assert (f["lse"] >= f["max_logit"] - 1e-5).all()
    assert (f["logprob"] <= 1e-5).all()
    assert (f["margin"] >= 0).all()
    # rank 1 means the sampled token is the most likely one; no token is more
    # likely than the maximum (ties with it may have rank > 1)
    top = f["rank"] == 1
    assert (np.abs(f["logprob"][top] - np.log(f["maxprob"][top])) < 1e-4).all()
    assert (f["logprob"] <= np.log(f["maxprob"]) + 1e-5).all()
    if cutoff_is_V:
        assert (f["cutoff"] == V).all()


def _oracle_rows(b, rows):
    raw = wl.to_host_raw(b.logits[torch.as_tensor(rows, device=b.logits.device)])
    ids = b.sampled_ids.cpu().numpy()[rows]
    T = b.temperature.cpu().numpy()[rows]
    P = None if b.top_p is None else b.top_p.cpu().numpy()[rows]
    return oracle.token_features_batch(raw, "bf16" if b.logits.dtype == torch.bfloat16 else "f32", ids, T, P)


def test_ragged_batch_full_size():
    """64 requests, lengths U{16..512}, V = 151,936 bf16, T = 0.7 (the bench workload)."""
    w = wl.WORKLOADS["ragged_64req_v151936_bf16"]
    b = wl.make_batch(w, device="cuda")
    print(f"case ragged full rows={b.n_rows}", flush=True)
    offsets = torch.as_tensor(b.offsets).cuda()
    feats = pr.token_features(b.logits, b.sampled_ids, b.temperature)
    agg = pr.request_aggregate(feats, offsets, q=w.q)
    scores = agg["score"]
    torch.cuda.synchronize()
    f = {k: v.cpu().numpy() for k, v in feats.items()}
    _properties(f, w.V)
    # two whole requests plus 48 random rows from everywhere
    rng = np.random.default_rng(7)
    reqs = [0, int(rng.integers(1, w.n_req))]
    rows = np.concatenate([np.arange(b.offsets[i], b.offsets[i + 1]) for i in reqs] +
                          [rng.choice(b.n_rows, 48, replace=False)])
    o = _oracle_rows(b, rows)
    compare_features(f, o, rows=rows)
    # summaries and score of the whole requests
    for k, i in enumerate(reqs):
        lo, hi = b.offsets[i], b.offsets[i + 1]
        n = hi - lo
        start = sum(b.offsets[j + 1] - b.offsets[j] for j in reqs[:k])
        seg = {key: o[key][start:start + n] for key in ("logprob", "maxprob", "entropy", "margin")}
        oa = oagg.request_aggregate(seg, [0, n], q=w.q)
        for stat in ("mean", "min", "quant"):
            assert_floats(f"req {i} {stat}", agg[stat][i].cpu().numpy(), oa[stat][0])
        assert_floats(f"req {i} score", scores[i:i + 1].cpu().numpy(), oagg.score_from_aggregates(oa))


def test_offline_512x512_in_chunks():
    """512 requests x 512 tokens of V = 151,936 bf16 (about 80 GB of logits),
    processed as 16 device-resident chunks of 32 whole requests."""
    w = wl.WORKLOADS["offline_512x512_v151936_bf16"]
    n_chunks = 16
    per = w.n_req // n_chunks
    rng = np.random.default_rng(11)
    checked = 0
    for c in range(n_chunks):
        wc = wl.scaled(w, n_req=per, seed=w.seed + c)
        b = wl.make_batch(wc, device="cuda")
        assert b.n_rows == per * 512
        feats = pr.token_features(b.logits, b.sampled_ids, b.temperature)
        agg = pr.request_aggregate(feats, torch.as_tensor(b.offsets).cuda(), q=w.q)
        torch.cuda.synchronize()
        f = {k: v.cpu().numpy() for k, v in feats.items()}
        _properties(f, w.V)
        assert (agg["count"].cpu().numpy() == 512).all()
        if c in (0, n_chunks - 1):
            rows = rng.choice(b.n_rows, 24, replace=False)
            compare_features(f, _oracle_rows(b, rows), rows=rows, what=f"chunk {c} ")
            checked += len(rows)
        del b, feats, agg
        torch.cuda.empty_cache()
    print(f"case offline 512x512: {n_chunks} chunks, {checked} rows checked against the oracle", flush=True)
