"""Every full-size workload against the float64 oracle: all rows, requests and
decisions (the 512 x 512 offline workload: two whole chunks of 32 requests).

The expected values were computed by the oracle on host-made rows
(tests/golden/make_fullsize.py). Here the same rows are made on the device by
the generator's device twin; per-request (per-step) checksums of the stored
bits must equal the stored ones before anything is compared. The stored
sampled ids are fed as inputs. The launch configuration is the one bench.py
times: the whole batch in one call.
"""

import json
import os

import numpy as np
import pytest
import torch

import paper_2608_28726_amd as pr
from paper_2608_28726_amd import workloads as wl
from tests.helpers import ROOT, assert_floats, assert_ints, decisions_agree, tolerance_ratio
from tests.gpu_common import require_gpu

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(ROOT, "tests", "golden")
FLOATS = ("max_logit", "lse", "entropy", "logprob", "maxprob", "margin")
NUCLEUS_DEPENDENT = ("lse", "entropy", "logprob", "maxprob")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def load(name):
    path = os.path.join(GOLDEN, f"fullsize_{name}.npz")
    assert os.path.exists(path), f"{path} is missing: run tests/golden/make_fullsize.py"
    d = np.load(path, allow_pickle=False)
    g = {k: d[k] for k in d.files}
    g["meta"] = json.loads(bytes(g["meta"]))
    return g


def compare_rows(f: dict, g: dict, what: str, sel=slice(None)):
    """Element-wise parity of per-row outputs f (GPU, numpy) with stored ones."""
    amb = g["ambiguous"][sel]
    ratios = {}
    for k in FLOATS:
        mask = ~amb if k in NUCLEUS_DEPENDENT else None
        ratios[k] = tolerance_ratio(f[k], g[k][sel], mask)
        assert_floats(f"{what} {k}", f[k], g[k][sel], mask=mask)
    print(f"  {what}: worst error / tolerance " + ", ".join(f"{k} {v:.3f}" for k, v in ratios.items()), flush=True)
    for k in ("rank", "argmax"):
        assert_ints(f"{what} {k}", f[k], g[k][sel])
    assert_ints(f"{what} cutoff", f["cutoff"], g["cutoff"][sel], mask=~amb)
    assert_ints(f"{what} flags", f["flags"].astype(np.int64) & 0xFFFFFFFF, g["flags"][sel], mask=~amb)
    return int(amb.sum())


def compare_requests(a: dict, g: dict, prefix: str, tau: float, what: str):
    """Per-request count, summaries, score and decision against stored ones.
    Besides the workload's threshold, the decisions are also compared at the
    median of the oracle's scores, where about half the requests ship."""
    assert_ints(f"{what} count", a["count"], g[prefix + "count"])
    for stat in ("mean", "min", "quant"):
        assert_floats(f"{what} {stat}", a[stat], g[prefix + stat])
    assert_floats(f"{what} score", a["score"], g[prefix + "score"])
    ok = decisions_agree(a["ship"], g[prefix + "score"], tau)
    assert ok.all(), f"{what}: decisions differ for requests {np.flatnonzero(~ok).tolist()}"
    tau_med = float(np.float32(np.nanmedian(g[prefix + "score"])))
    ship_med, n_med = pr.route(torch.as_tensor(np.asarray(a["score"], dtype=np.float32)).cuda(), tau_med)
    ship_med = ship_med.cpu().numpy()
    ok = decisions_agree(ship_med, g[prefix + "score"], tau_med)
    assert ok.all(), f"{what}: decisions at the median differ for requests {np.flatnonzero(~ok).tolist()}"
    print(f"  {what}: {int(a['ship'].sum())} of {len(ok)} ship at tau = {tau}, {int(ship_med.sum())} at the "
          f"median score {tau_med:.6f}", flush=True)


def device_batch(w, g):
    """The workload's batch made on the device with the stored ids; checks the
    plan and the per-request checksums against the stored ones."""
    b = wl.make_batch(w, device="cuda", ids=g["ids"])
    assert np.array_equal(b.offsets, g["offsets"]), "request lengths differ from the stored plan"
    assert np.array_equal(b.temperature.cpu().numpy(), g["T"])
    if "P" in g:
        assert np.array_equal(b.top_p.cpu().numpy(), g["P"])
    ck = wl.row_checksums(b.logits)
    req = np.array([wl.combine_checksums(ck[b.offsets[i]:b.offsets[i + 1]]) for i in range(len(b.offsets) - 1)])
    bad = np.flatnonzero(req != g["checksum_req"])
    assert bad.size == 0, f"device-made rows differ from the host generator's in requests {bad[:8].tolist()}"
    return b


def run_batch(b, w):
    offsets = torch.as_tensor(b.offsets).cuda()
    feats = pr.token_features(b.logits, b.sampled_ids, b.temperature, b.top_p)
    agg = pr.request_aggregate(feats, offsets, q=w.q)
    ship, n_ship = pr.route(agg["score"], w.tau)
    torch.cuda.synchronize()
    f = {k: v.cpu().numpy() for k, v in feats.items()}
    a = {k: v.cpu().numpy() for k, v in agg.items()}
    a["ship"] = ship.cpu().numpy()
    assert int(n_ship.item()) == int(a["ship"].sum())
    return f, a


def check_batch(name, w, label):
    g = load(name)
    b = device_batch(w, g)
    f, a = run_batch(b, w)
    n_amb = compare_rows(f, g, label)
    compare_requests(a, g, "req_", w.tau, label)
    n_band = int((np.abs(g["req_score"] - w.tau) <= 1e-5).sum())
    print(f"case {label}: {b.n_rows} rows and {len(b.offsets) - 1} requests compared "
          f"({n_amb} boundary-ambiguous rows, {n_band} scores in the decision band; "
          f"{int(a['ship'].sum())} ship)", flush=True)
    return b, f, g


def test_pr1_reference_every_row_and_decision():
    """8 requests x 64 tokens, V = 32,000 float32, T = 1, tau = 0.5."""
    w = wl.WORKLOADS["pr1_ref_8x64_v32000_f32"]
    check_batch(w.name, w, "pr1_ref 8x64 V=32000 f32")


def test_ragged_every_row_and_decision():
    """64 requests, lengths U{16..512}, V = 151,936 bf16, T = 0.7 (the bench workload)."""
    w = wl.WORKLOADS["ragged_64req_v151936_bf16"]
    check_batch(w.name, w, "ragged 64req V=151936 bf16")


def test_topp_every_row_and_decision():
    """128 requests x 256 tokens, V = 262,144 float32, per-request T and top-p:
    every row's cutoff, rank and flags (OUTSIDE_NUCLEUS included) exactly."""
    w = wl.WORKLOADS["topp_128x256_v262144_f32"]
    b, f, g = check_batch(w.name, w, "topp 128x256 V=262144 f32")
    outside = (g["flags"] & pr.FLAG_OUTSIDE_NUCLEUS) != 0
    assert np.array_equal((f["flags"] & pr.FLAG_OUTSIDE_NUCLEUS) != 0, outside)
    print(f"case topp: {int(outside.sum())} rows outside the nucleus, cutoff range "
          f"{int(g['cutoff'].min())}..{int(g['cutoff'].max())}", flush=True)


def test_offline_chunks_every_row_and_decision():
    """512 requests x 512 tokens of V = 151,936 bf16 as 16 device-resident
    chunks of 32 whole requests: chunks 0 and 15 (requests 0-31 and 480-511)
    compared row by row and request by request; every chunk's rows checked
    for the invariants of valid rows."""
    w = wl.WORKLOADS["offline_512x512_v151936_bf16"]
    compared = 0
    for c in range(wl.OFFLINE_CHUNKS):
        wc = wl.offline_chunk(w, c)
        name = f"{w.name}_chunk{c:02d}"
        if os.path.exists(os.path.join(GOLDEN, f"fullsize_{name}.npz")):
            b, f, g = check_batch(name, wc, f"offline chunk {c}")
            compared += b.n_rows
        else:
            b = wl.make_batch(wc, device="cuda")
            f, a = run_batch(b, wc)
            assert (f["flags"] == 0).all() and (a["count"] == 512).all()
            assert (f["rank"] >= 1).all() and (f["rank"] <= w.V).all() and (f["cutoff"] == w.V).all()
            assert (f["maxprob"] > 0).all() and (f["maxprob"] <= 1 + 1e-6).all()
            assert (f["entropy"] >= -1e-5).all() and (f["entropy"] <= np.log(w.V) + 1e-4).all()
            assert (f["logprob"] <= np.log(f["maxprob"]) + 1e-5).all() and (f["margin"] >= 0).all()
        del b
        torch.cuda.empty_cache()
    assert compared == 2 * 32 * 512
    print(f"case offline 512x512: {wl.OFFLINE_CHUNKS} chunks, {compared} rows compared", flush=True)


def test_stream_whole_schedule_every_verdict():
    """256 slots over the 1,024-step schedule (V = 151,936 bf16): every slot's
    count, summaries, score and decision at its finish; every row's features
    on the stored steps; every step's input checksum."""
    w = wl.WORKLOADS["stream_256slots_v151936_bf16"]
    g = load(w.name)
    fin = wl.stream_schedule(w)
    assert np.array_equal(fin, g["fin"])
    n_steps = int(fin.max())
    feature_steps = {int(s): k for k, s in enumerate(g["feature_steps"])}
    st = pr.StreamState(w.n_req, n_steps, q=w.q)
    results = {}
    rows_compared = 0
    print(f"case stream full schedule: {n_steps} steps, {int(g['step_offsets'][-1])} rows", flush=True)
    for step in range(1, n_steps + 1):
        active = np.flatnonzero(fin >= step).astype(np.int32)
        lo, hi = int(g["step_offsets"][step - 1]), int(g["step_offsets"][step])
        assert hi - lo == len(active)
        logits, ids, T = wl.stream_step_inputs(w, step, active, device="cuda", ids=g["ids"][lo:hi])
        ck = wl.combine_checksums(wl.row_checksums(logits))
        assert ck == int(g["checksum_step"][step - 1]), f"step {step}: device-made rows differ from the host's"
        out = st.step(logits, torch.as_tensor(active).cuda(), ids, T, want_features=step in feature_steps)
        if step in feature_steps:
            k = feature_steps[step]
            sel = slice(int(g["feature_offsets"][k]), int(g["feature_offsets"][k + 1]))
            torch.cuda.synchronize()
            compare_rows({key: v.cpu().numpy() for key, v in out.items()}, g, f"step {step}", sel)
            rows_compared += len(active)
        ending = active[fin[active] == step]
        if len(ending):
            res = st.finish(torch.as_tensor(ending).cuda(), w.tau)
            torch.cuda.synchronize()
            for k, s in enumerate(ending):
                results[int(s)] = {key: v[k].cpu().numpy() for key, v in res.items()}
        if step % 128 == 0:
            print(f"  step {step}: {len(active)} active", flush=True)
    st.close()
    assert sorted(results) == list(range(w.n_req))
    a = {key: np.stack([results[s][key] for s in range(w.n_req)]) for key in ("count", "mean", "min", "quant",
                                                                              "score", "ship")}
    compare_requests(a, g, "slot_", w.tau, "stream slots")
    assert np.array_equal(a["count"], fin)
    print(f"case stream: all {w.n_req} slot verdicts compared, {rows_compared} rows on {len(feature_steps)} "
          f"steps compared, {int(a['ship'].sum())} ship", flush=True)
