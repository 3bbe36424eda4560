"""Threshold calibration (pr_calibrate_threshold) and the bounded-memory
streaming quantile (pr_stream_create with max_len = 0) against the oracle.

Calibration selects one of the scores and counts, so tau and n_ship must be
exact. The P-square markers see the per-token confidence tuples the GPU
computed for each step (returned by the same step call), and the oracle's
P-square is fed the same float32 values, so the estimate must be exact too:
both sides do the same float64 operations in the same order (the library is
built without contraction)."""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_28726_amd as pr
from paper_2608_28726_amd import workloads as wl
from tests.gpu_common import require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _same(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return (a == b) | (np.isnan(a) & np.isnan(b))


# ---------------------------------------------------------------- calibration

def _pool(rng, n, kind):
    if kind == "uniform":
        s = rng.random(n, dtype=np.float32)
    elif kind == "ties":
        s = rng.choice(np.array([0.125, 0.25, 0.5, 0.75, 0.875], dtype=np.float32), size=n)
    elif kind == "sigmoid":  # head-like confidences crowded near 1
        s = (1.0 / (1.0 + np.exp(-rng.normal(3.0, 1.0, n)))).astype(np.float32)
    else:  # "wild": NaN, infinities, signed zeros, negatives
        s = rng.normal(0, 2, n).astype(np.float32)
        m = rng.random(n)
        s[m < 0.1] = np.nan
        s[(m >= 0.1) & (m < 0.15)] = np.inf
        s[(m >= 0.15) & (m < 0.2)] = -np.inf
        s[(m >= 0.2) & (m < 0.3)] = -0.0
        s[(m >= 0.3) & (m < 0.35)] = 0.0
    return s


@pytest.mark.parametrize("n", [0, 1, 2, 7, 1000, 16384, 16385, 100000])
def test_calibrate_matches_oracle(n):
    rng = np.random.default_rng(n + 11)
    for kind in ("uniform", "ties", "sigmoid", "wild"):
        s = _pool(rng, n, kind)
        dev = torch.from_numpy(s).cuda()
        for q in (0.0, 1e-9, 0.05, 0.1, 0.5, 0.77, 1.0):
            print(f"case calibrate n={n} kind={kind} q={q}", flush=True)
            tau, ns = pr.calibrate_threshold(dev, q)
            torch.cuda.synchronize()
            otau, ons = oracle.calibrate_threshold(s.astype(np.float64), q)
            assert float(tau.item()) == otau, (n, kind, q, tau.item(), otau)
            assert int(ns.item()) == ons, (n, kind, q, ns.item(), ons)


def test_calibrate_all_nan_and_large_pool():
    s = np.full(5000, np.nan, dtype=np.float32)
    tau, ns = pr.calibrate_threshold(torch.from_numpy(s).cuda(), 0.3)
    torch.cuda.synchronize()
    assert tau.item() == math.inf and ns.item() == 0
    rng = np.random.default_rng(5)
    s = _pool(rng, 1 << 20, "sigmoid")
    print("case calibrate n=2^20", flush=True)
    tau, ns = pr.calibrate_threshold(torch.from_numpy(s).cuda(), 0.1)
    torch.cuda.synchronize()
    otau, ons = oracle.calibrate_threshold(s.astype(np.float64), 0.1)
    assert tau.item() == otau and ns.item() == ons


def test_calibrated_threshold_routes_the_pool():
    """Routing the pool with its own calibrated tau ships n_ship requests."""
    s = _pool(np.random.default_rng(9), 3000, "sigmoid")
    dev = torch.from_numpy(s).cuda()
    tau, ns = pr.calibrate_threshold(dev, 0.25)
    ship, n_ship = pr.route(dev, float(tau.item()))
    torch.cuda.synchronize()
    assert int(n_ship.item()) == int(ns.item()) >= math.ceil(0.25 * 3000)


# ------------------------------------------------- bounded-memory streaming quantile

def _tuple(out, k):
    """The confidence tuple A = (logprob, maxprob, -entropy, margin) of row k."""
    return (out["logprob"][k], out["maxprob"][k], -out["entropy"][k], out["margin"][k])


def _check_slot(res, k, tokens, q):
    A = np.array(tokens, dtype=np.float32).reshape(-1, 4)
    n = A.shape[0]
    assert int(res["count"][k]) == n
    for f in range(4):
        col = A[:, f].astype(np.float64)
        exp_q = oracle.p2_quantile(col, q)
        got_q = res["quant"][k][f]
        if np.isnan(col).any():
            assert np.isnan(got_q) and np.isnan(res["mean"][k][f]) and np.isnan(res["min"][k][f])
            continue
        assert _same(got_q, np.float32(exp_q)), (k, f, n, got_q, exp_q)
        assert res["min"][k][f] == np.float32(col.min())
        exp_mean = math.fsum(col) / n if np.isfinite(col).all() else col.sum() / n
        m = float(res["mean"][k][f])
        assert _same(m, exp_mean) or abs(m - exp_mean) <= 1e-6 * abs(exp_mean) + 1e-7, (k, f, m, exp_mean)


def _run_p2(w, fin, label):
    st = pr.StreamState(w.n_req, 0, q=w.q)
    tokens = {i: [] for i in range(w.n_req)}
    done = 0
    for step in range(1, int(fin.max()) + 1):
        active = np.flatnonzero(fin >= step).astype(np.int32)
        logits, ids, T = wl.stream_step_inputs(w, step, active, device="cuda")
        out = st.step(logits, torch.as_tensor(active).cuda(), ids, T, want_features=True)
        torch.cuda.synchronize()
        host = {k: v.cpu().numpy() for k, v in out.items()}
        for k, s in enumerate(active):
            tokens[int(s)].append(_tuple(host, k))
        ending = active[fin[active] == step]
        if len(ending):
            res = st.finish(torch.as_tensor(ending).cuda(), w.tau)
            torch.cuda.synchronize()
            res = {key: v.cpu().numpy() for key, v in res.items()}
            for k, s in enumerate(ending):
                _check_slot(res, k, tokens[int(s)], w.q)
                done += 1
    st.close()
    assert done == w.n_req, label


@pytest.mark.parametrize("case", ["split_bf16", "mid_bf16", "wide_f32"])
def test_p2_stream_matches_oracle(case):
    base = wl.WORKLOADS["stream_256slots_v151936_bf16"]
    if case == "split_bf16":  # few rows, full vocabulary: split rows and the merge kernel
        w = wl.scaled(base, n_req=24, len_hi=60, len_lo=1)
    elif case == "mid_bf16":  # 300 rows: one workgroup of 256 threads per row
        w = wl.scaled(base, n_req=300, len_hi=50, len_lo=1, V=8192)
    else:  # float32, up to 256 rows: one workgroup of 1,024 threads per row
        w = wl.scaled(base, n_req=200, len_hi=80, len_lo=3, V=6000, dtype="f32")
    fin = wl.stream_schedule(w)
    print(f"case p2 stream {case}: {w.n_req} slots, up to {int(fin.max())} steps, V={w.V}", flush=True)
    _run_p2(w, fin, case)


def test_p2_stream_nonfinite_reuse_and_reset():
    """+inf margins, -inf log-probs and invalid ids; a slot reused after
    finish starts afresh; reset clears the markers."""
    V, S = 1000, 4
    st = pr.StreamState(S, 0, q=0.3)
    slots = torch.arange(S, dtype=torch.int32).cuda()
    gen = torch.Generator().manual_seed(17)
    tokens = {i: [] for i in range(S)}
    print("case p2 nonfinite", flush=True)
    for rnd in range(2):
        for step in range(1, 13):
            z = torch.randn((S, V), generator=gen) * 3.0
            ids = torch.randint(0, V, (S,), generator=gen, dtype=torch.int32)
            if rnd == 0 and step == 3:  # slot 1: one finite logit: margin +inf
                z[1] = -math.inf
                z[1, 5] = 1.0
                ids[1] = 5
            if rnd == 0 and step == 4:  # slot 2: invalid id: log-prob NaN
                ids[2] = V + 3
            if rnd == 0 and step == 6:  # slot 3: a masked token sampled: log-prob -inf
                z[3, 7] = -math.inf
                ids[3] = 7
            T = torch.full((S,), 0.8)
            out = st.step(z.cuda(), slots, ids.cuda(), T.cuda(), want_features=True)
            torch.cuda.synchronize()
            host = {k: v.cpu().numpy() for k, v in out.items()}
            for k in range(S):
                tokens[k].append(_tuple(host, k))
        res = st.finish(slots, 0.5)
        torch.cuda.synchronize()
        res = {key: v.cpu().numpy() for key, v in res.items()}
        for k in range(S):
            _check_slot(res, k, tokens[k], 0.3)
            tokens[k] = []
        if rnd == 0:
            q = res["quant"]
            assert np.isnan(q[1][3]) and np.isfinite(q[1][:3]).all()  # +inf margin
            assert np.isnan(q[2][0])  # NaN log-prob
            assert np.isnan(q[3][0]) and res["min"][3][0] == -np.inf  # -inf log-prob: min keeps it
    # reset: a slot with tokens is cleared without a verdict
    for step in range(3):
        z = torch.randn((S, V), generator=gen)
        ids = torch.randint(0, V, (S,), generator=gen, dtype=torch.int32)
        st.step(z.cuda(), slots, ids.cuda(), torch.ones(S).cuda())
    st.reset(slots[:2])
    z = torch.randn((S, V), generator=gen)
    ids = torch.randint(0, V, (S,), generator=gen, dtype=torch.int32)
    out = st.step(z.cuda(), slots, ids.cuda(), torch.ones(S).cuda(), want_features=True)
    res = st.finish(slots, 0.5)
    torch.cuda.synchronize()
    host = {k: v.cpu().numpy() for k, v in out.items()}
    res = {key: v.cpu().numpy() for key, v in res.items()}
    assert list(res["count"]) == [1, 1, 4, 4]
    for k in range(2):
        _check_slot(res, k, [_tuple(host, k)], 0.5)
    st.close()


def test_p2_full_schedule():
    """The 256-slot schedule at full size (V = 151,936 bf16, 1,012 steps) in
    bounded-memory mode: every slot's count and a finite score; four
    sampled slots' P-square quantiles equal the oracle's, fed the same
    per-token tuples the steps returned."""
    w = wl.WORKLOADS["stream_256slots_v151936_bf16"]
    fin = wl.stream_schedule(w)
    n_steps = int(fin.max())
    rng = np.random.default_rng(21)
    watch = [int(s) for s in rng.choice(w.n_req, 4, replace=False)]
    tokens = {s: [] for s in watch}
    st = pr.StreamState(w.n_req, 0, q=w.q)
    results = {}
    print(f"case p2 full schedule: {n_steps} steps, watching slots {watch}", flush=True)
    for step in range(1, n_steps + 1):
        active = np.flatnonzero(fin >= step).astype(np.int32)
        logits, ids, T = wl.stream_step_inputs(w, step, active, device="cuda")
        out = st.step(logits, torch.as_tensor(active).cuda(), ids, T, want_features=True)
        rows = [int(np.searchsorted(active, s)) for s in watch if fin[s] >= step]
        if rows:
            sel = torch.as_tensor(rows, device="cuda")
            host = {k: v[sel].cpu().numpy() for k, v in out.items()}
            for j, s in enumerate([s for s in watch if fin[s] >= step]):
                tokens[s].append(_tuple(host, j))
        ending = active[fin[active] == step]
        if len(ending):
            res = st.finish(torch.as_tensor(ending).cuda(), w.tau)
            torch.cuda.synchronize()
            for k, s in enumerate(ending):
                results[int(s)] = {key: v[k].cpu().numpy() for key, v in res.items()}
    st.close()
    assert sorted(results) == list(range(w.n_req))
    for s in range(w.n_req):
        assert int(results[s]["count"]) == fin[s]
        assert np.isfinite(results[s]["score"])
    for s in watch:
        r = {key: np.array([v]) for key, v in results[s].items()}
        _check_slot(r, 0, tokens[s], w.q)


def test_calibrated_head_scores_route_the_batch():
    """Scores from the verifier head, calibrated for a ship fraction, then
    routed with that threshold: exactly the calibrated count ships, and tau
    is the oracle's for the same scores."""
    w = wl.scaled(wl.WORKLOADS["ragged_64req_v151936_bf16"], n_req=40, len_hi=24, len_lo=4, V=4096)
    b = wl.make_batch(w, device="cuda")
    offsets = torch.as_tensor(b.offsets).cuda()
    X = pr.feature_sequence(b.logits, b.sampled_ids, b.temperature, offsets)
    p = pr.verifier_head(X, offsets, torch.tensor(wl.head_weights(), device="cuda"), max_len=w.len_hi)
    tau, ns = pr.calibrate_threshold(p, 0.6)
    ship, n_ship = pr.route(p, float(tau.item()))
    torch.cuda.synchronize()
    otau, ons = oracle.calibrate_threshold(p.cpu().numpy().astype(np.float64), 0.6)
    assert tau.item() == otau and ns.item() == ons == int(n_ship.item()) == int(ship.sum().item())
    assert ons >= math.ceil(0.6 * w.n_req)
