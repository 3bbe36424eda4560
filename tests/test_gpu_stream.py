"""Streaming decode: per-step features, device-resident request state and
finish-time verdicts equal the offline path and the oracle."""

import numpy as np
import pytest
import torch

from oracle import aggregate as oagg
import paper_2608_28726_amd as pr
from paper_2608_28726_amd import workloads as wl
from tests.gpu_common import compare_features, oracle_features, require_gpu
from tests.helpers import assert_floats, decisions_agree

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _run_stream(w, n_steps, max_len, check_features=True):
    fin = wl.stream_schedule(w, n_steps)
    st = pr.StreamState(w.n_req, max_len, q=w.q)
    rows_by_slot = {i: [] for i in range(w.n_req)}  # (logits row, id, T) per token, host copies
    results = {}
    for step in range(1, int(fin.max()) + 1):
        active = np.flatnonzero(fin >= step).astype(np.int32)
        logits, ids, T = wl.stream_step_inputs(w, step, active, device="cuda")
        slot_ids = torch.as_tensor(active).cuda()
        out = st.step(logits, slot_ids, ids, T, want_features=check_features)
        raw_ids, raw_T = ids.cpu().numpy(), T.cpu().numpy()
        host = logits.cpu()
        for k, s in enumerate(active):
            rows_by_slot[int(s)].append((host[k], int(raw_ids[k]), float(raw_T[k])))
        if check_features and step % 7 == 1:
            torch.cuda.synchronize()
            compare_features({k: v.cpu().numpy() for k, v in out.items()}, oracle_features(logits, ids, T),
                             what=f"step {step} ")
        ending = active[fin[active] == step]
        if len(ending):
            res = st.finish(torch.as_tensor(ending).cuda(), w.tau)
            torch.cuda.synchronize()
            for k, s in enumerate(ending):
                results[int(s)] = {key: v[k].cpu().numpy() for key, v in res.items()}
    st.close()
    return fin, rows_by_slot, results


def test_stream_matches_offline_and_oracle():
    w = wl.scaled(wl.WORKLOADS["stream_256slots_v151936_bf16"], n_req=12, len_hi=14, V=32000, len_lo=2)
    print("case stream small", flush=True)
    fin, rows_by_slot, results = _run_stream(w, None, max_len=16)
    # offline over the same rows, request = slot
    order = sorted(rows_by_slot)
    logits = torch.stack([r for s in order for r, _, _ in rows_by_slot[s]]).cuda()
    ids = torch.tensor([y for s in order for _, y, _ in rows_by_slot[s]], dtype=torch.int32).cuda()
    T = torch.tensor([t for s in order for _, _, t in rows_by_slot[s]], dtype=torch.float32).cuda()
    offsets = np.concatenate([[0], np.cumsum([len(rows_by_slot[s]) for s in order])]).astype(np.int32)
    feats = pr.token_features(logits, ids, T)
    agg = pr.request_aggregate(feats, torch.as_tensor(offsets).cuda(), q=w.q)
    torch.cuda.synchronize()
    of = oracle_features(logits, ids, T)
    oa = oagg.request_aggregate(of, offsets, q=w.q)
    os_ = oagg.score_from_aggregates(oa)
    for i, s in enumerate(order):
        r = results[s]
        assert int(r["count"]) == fin[s] == offsets[i + 1] - offsets[i]
        for stat in ("min", "quant"):  # streaming == offline exactly for selections
            a, b = r[stat].astype(np.float64), agg[stat][i].cpu().numpy().astype(np.float64)
            assert ((a == b) | (np.isnan(a) & np.isnan(b))).all(), (s, stat, a, b)
        assert_floats("stream mean vs offline", r["mean"], agg["mean"][i].cpu().numpy(), atol=0, rtol=1e-6)
        for stat in ("mean", "min", "quant"):
            assert_floats(f"stream {stat} vs oracle", r[stat], oa[stat][i])
        assert_floats("stream score vs oracle", np.array([r["score"]]), np.array([os_[i]]))
        assert decisions_agree(np.array([r["ship"]]), np.array([os_[i]]), w.tau).all()


def test_stream_overflow_and_reset():
    """Tokens past max_len keep sums and minima but make the quantile NaN; reset clears a slot."""
    w = wl.scaled(wl.WORKLOADS["stream_256slots_v151936_bf16"], n_req=3, len_hi=6, len_lo=6, V=1000)
    st = pr.StreamState(3, 4, q=w.q)
    slots = torch.arange(3, dtype=torch.int32).cuda()
    for step in range(1, 7):
        logits, ids, T = wl.stream_step_inputs(w, step, np.arange(3), device="cuda")
        st.step(logits, slots, ids, T)
    st.reset(slots[2:])
    res = st.finish(slots, 0.5)
    torch.cuda.synchronize()
    cnt = res["count"].cpu().numpy()
    assert list(cnt) == [6, 6, 0]
    q = res["quant"].cpu().numpy()
    assert np.isnan(q).all()
    m = res["mean"].cpu().numpy()
    assert np.isfinite(m[:2]).all() and np.isnan(m[2]).all()
    res2 = st.finish(slots, 0.5)  # finish cleared the slots
    torch.cuda.synchronize()
    assert (res2["count"].cpu().numpy() == 0).all()
    st.close()


def _stream_over_batch(b, max_len, q):
    """Feeds a host-made batch to a stream, request i in slot i, one token per
    step; returns each step's features and every slot's finish result."""
    lengths = np.diff(b.offsets)
    logits, ids, T, P = (t.cuda() for t in (b.logits, b.sampled_ids, b.temperature, b.top_p))
    st = pr.StreamState(len(lengths), max_len, q=q)
    steps = []
    results = {}
    for t in range(int(lengths.max())):
        active = np.flatnonzero(lengths > t).astype(np.int32)
        rows = torch.as_tensor(b.offsets[active] + t, dtype=torch.int64).cuda()
        out = st.step(logits[rows].contiguous(), torch.as_tensor(active).cuda(), ids[rows].contiguous(),
                      T[rows].contiguous(), want_features=True, top_p=P[rows].contiguous())
        torch.cuda.synchronize()
        steps.append((rows.cpu().numpy(), {k: v.cpu().numpy() for k, v in out.items()}))
        ending = active[lengths[active] == t + 1]
        if len(ending):
            res = st.finish(torch.as_tensor(ending).cuda(), 0.5)
            torch.cuda.synchronize()
            for k, s in enumerate(ending):
                results[int(s)] = {key: v[k].cpu().numpy() for key, v in res.items()}
    st.close()
    return steps, results


@pytest.mark.parametrize("V,dtype", [(4096, "f32"), (151936, "bf16")])
def test_stream_with_top_p_matches_offline_and_oracle(V, dtype):
    """Streaming steps with top-p: every step's features equal the oracle's on
    the renormalised nucleus, and each request's verdict at its finish equals
    the offline path's and the oracle's over the same rows."""
    w = wl.scaled(wl.WORKLOADS["topp_128x256_v262144_f32"], n_req=7, len_lo=2, len_hi=9, V=V, dtype=dtype,
                  seed=0x5053)
    b = wl.make_batch(w, device="cpu")
    print(f"case stream top-p V={V} {dtype} rows={b.n_rows}", flush=True)
    steps, results = _stream_over_batch(b, 16, w.q)
    o = oracle_features(b.logits.cuda(), b.sampled_ids.cuda(), b.temperature.cuda(), b.top_p.cuda())
    for k, (rows, f) in enumerate(steps):
        compare_features(f, {key: v[rows] for key, v in o.items()}, what=f"step {k + 1} ")
    oa = oagg.request_aggregate(o, b.offsets, q=w.q)
    os_ = oagg.score_from_aggregates(oa)
    feats = pr.token_features(b.logits.cuda(), b.sampled_ids.cuda(), b.temperature.cuda(), b.top_p.cuda())
    agg = pr.request_aggregate(feats, torch.as_tensor(b.offsets).cuda(), q=w.q)
    torch.cuda.synchronize()
    for i in range(w.n_req):
        r = results[i]
        assert int(r["count"]) == b.offsets[i + 1] - b.offsets[i]
        for stat in ("min", "quant"):  # streaming == offline exactly for selections
            a_, g_ = r[stat].astype(np.float64), agg[stat][i].cpu().numpy().astype(np.float64)
            assert ((a_ == g_) | (np.isnan(a_) & np.isnan(g_))).all(), (i, stat, a_, g_)
        for stat in ("mean", "min", "quant"):
            assert_floats(f"req {i} {stat} vs oracle", r[stat], oa[stat][i])
        assert_floats(f"req {i} score vs oracle", np.array([r["score"]]), np.array([os_[i]]))
        assert decisions_agree(np.array([r["ship"]]), np.array([os_[i]]), 0.5).all()


def test_stream_with_top_p_bounded_memory():
    """The P-square quantile of a streaming run with top-p equals the oracle's
    P-square estimate over the same per-token tuples."""
    import oracle
    w = wl.scaled(wl.WORKLOADS["topp_128x256_v262144_f32"], n_req=4, len_lo=3, len_hi=12, V=2048, seed=0x5054)
    b = wl.make_batch(w, device="cpu")
    steps, results = _stream_over_batch(b, 0, 0.3)
    lengths = np.diff(b.offsets)
    A = {i: [] for i in range(w.n_req)}
    for rows, f in steps:
        for k, row in enumerate(rows):
            i = int(np.searchsorted(b.offsets, row, side="right") - 1)
            A[i].append((f["logprob"][k], f["maxprob"][k], -f["entropy"][k], f["margin"][k]))
    for i in range(w.n_req):
        assert len(A[i]) == lengths[i]
        for c in range(4):
            e = np.float32(oracle.p2_quantile([np.float32(a[c]) for a in A[i]], 0.3))
            got = results[i]["quant"][c]
            assert got == e or (np.isnan(e) and np.isnan(got)), (i, c, got, e)
