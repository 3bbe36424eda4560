"""The host side of the seeded logit generator and of the stored expected
values (no GPU): the generator's pieces against independent definitions,
and each stored full-size file against the current generator and oracle."""

import json
import math
import os

import numpy as np
import pytest
import torch
from statistics import NormalDist

import oracle
from paper_2608_28726_amd import workloads as wl
from tests.helpers import ROOT

GOLDEN = os.path.join(ROOT, "tests", "golden")


def _golden_files():
    return sorted(f for f in os.listdir(GOLDEN) if f.startswith("fullsize_") and f.endswith(".npz"))


def test_mix64_array_matches_integer_form():
    rng = np.random.default_rng(1)
    x = rng.integers(0, 2 ** 63, 1000, dtype=np.uint64) * np.uint64(2) + np.uint64(1)
    got = wl.mix64(x)
    for a, b in zip(x.tolist(), got.tolist()):
        assert wl.mix64_int(a) == b


def test_mix64_is_a_bijection_on_a_sample():
    """SplitMix64's output function is invertible (xor-shifts and odd multipliers)."""
    x = np.arange(1 << 16, dtype=np.uint64)
    assert np.unique(wl.mix64(x)).size == x.size


def test_quantile_tables():
    main, tail = wl.normal_tables()
    A, D = main[1:65535, 0], main[1:65535, 1]
    assert (np.diff(main[1:65536, 0]) > 0).all() and (D > 0).all()
    assert main[32768, 0] == 0.0  # Q(1/2)
    assert np.array_equal(A[:100], -main[65535:65435:-1, 0])  # symmetry Q(p) = -Q(1 - p)
    Q = NormalDist().inv_cdf
    assert abs(float(main[1, 0]) - Q(2 ** -16)) < 1e-6 and abs(float(tail[1, 0]) - Q(2 ** -32)) < 1e-6
    assert (np.diff(tail[:, 0]) > 0).all() and (tail[:, 1] > 0).all()
    # the tail table ends where the main table's first knot sits
    assert float(tail[65535, 0] + tail[65535, 1]) == pytest.approx(float(main[1, 0]), abs=1e-6)


def test_normal_deviates_follow_the_normal_law():
    g = wl.normal_from_bits(wl.element_bits(wl.row_key(7, 0), 2_000_000)).astype(np.float64)
    assert abs(g.mean()) < 5 / math.sqrt(g.size)
    assert abs(g.var() - 1.0) < 5 * math.sqrt(2.0 / g.size)
    nd = NormalDist()
    for x in (-3.0, -1.0, 0.0, 0.5, 2.0):  # empirical CDF against Phi
        p = nd.cdf(x)
        assert abs((g <= x).mean() - p) < 5 * math.sqrt(p * (1 - p) / g.size), x
    tail = np.abs(g) > 4.0  # the refined tail cells
    assert abs(tail.mean() - 2 * nd.cdf(-4.0)) < 5 * math.sqrt(2 * nd.cdf(-4.0) / g.size)


def test_bf16_rounding_matches_torch():
    """Round-to-nearest-even to bfloat16, against torch's conversion."""
    rng = np.random.default_rng(3)
    z = np.concatenate([rng.normal(0, 3, 100000), rng.normal(0, 1e-3, 1000), [0.0, -0.0, 1.0]]).astype(np.float32)
    ties = (np.arange(1000, dtype=np.uint32) << np.uint32(16)) | np.uint32(0x3F808000)  # exact halfway values
    z = np.concatenate([z, ties.view(np.float32)])
    want = torch.from_numpy(z).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(wl.bf16_bits(z), want)


def test_host_rows_row_model():
    """Spike on token j with height h, scale s: the row model of every workload."""
    V = 50000
    r = wl.host_row(5, 3, V, "f32", 2.0, 30.0, 123)
    assert r.dtype == np.float32 and r.shape == (V,)
    assert int(np.argmax(r)) == 123
    assert abs(float(np.std(np.delete(r, 123))) - 2.0) < 0.05
    b = wl.host_row(5, 3, V, "bf16", 2.0, 30.0, 123)
    assert np.array_equal(b, wl.bf16_bits(r))
    assert not np.array_equal(r, wl.host_row(5, 4, V, "f32", 2.0, 30.0, 123))  # rows differ
    # the CPU path of fill_logits is the host generator
    t = torch.empty((2, V), dtype=torch.bfloat16)
    wl.fill_logits(t, np.float32([2.0, 1.0]), np.float32([30.0, 0.0]), np.int64([123, -1]), seed=5, row0=3)
    assert np.array_equal(wl.to_host_raw(t)[0], b)


def test_checksums_numpy_and_torch_agree():
    raw = wl.host_rows(9, np.arange(4), 1000, "f32", np.ones(4, np.float32), np.zeros(4, np.float32),
                       np.full(4, -1))
    c = wl.row_checksums(raw)
    w = np.arange(1000) % 65521 + 1
    bits = raw.view(np.uint32).astype(np.int64)
    assert np.array_equal(c, ((bits & 0xFFFF) * w).sum(1) + 7 * ((bits >> 16) * w).sum(1))
    assert wl.combine_checksums(c) == sum(int(v) * (k + 1) for k, v in enumerate(c)) % wl.CHECKSUM_MOD


def test_host_sampler_stays_inside_the_nucleus():
    w = wl.scaled(wl.WORKLOADS["topp_128x256_v262144_f32"], n_req=2, len_hi=3, len_lo=3, V=4096)
    b = wl.make_batch(w, device="cpu")
    o = oracle.token_features_batch(wl.to_host_raw(b.logits), "f32", b.sampled_ids.numpy(), b.temperature.numpy(),
                                    b.top_p.numpy())
    assert (o["flags"] == 0).all() and (o["rank"] <= o["cutoff"]).all()


@pytest.mark.parametrize("fn", _golden_files())
def test_stored_values_match_generator_and_oracle(fn):
    """Each stored file: written by the current oracle sources, its first
    request's (step's) rows regenerate on the host with the stored checksum,
    and the oracle recomputes the stored features of a few of them exactly."""
    from tests.golden import make_fullsize as mk
    d = np.load(os.path.join(GOLDEN, fn), allow_pickle=False)
    meta = json.loads(bytes(d["meta"]))
    assert meta["oracle_hash"] == mk.oracle_hash(), f"{fn} was written by other oracle sources: rerun make_fullsize"
    name = meta["workload"]
    if name.startswith("stream_"):
        w = wl.WORKLOADS[name]
        assert np.array_equal(d["fin"], wl.stream_schedule(w))
        active = np.flatnonzero(d["fin"] >= 1)
        idx, s, h, j = wl.stream_rows(w, 1, active)
        raw = wl.host_rows(wl.stream_seed(w), idx, w.V, w.dtype, s, h, j)
        assert wl.combine_checksums(wl.row_checksums(raw)) == int(d["checksum_step"][0])
        ids, T = d["ids"][:len(active)], np.full(len(active), np.float32(w.T_lo))
        assert np.array_equal(ids, wl.host_sample_ids(raw, T, None, wl.stream_seed(w), idx))
        rows = [0, 1, len(active) - 1]
        P = None
    else:
        w = wl.WORKLOADS[name]
        if "_chunk" in fn:  # a chunk of whole requests of the offline workload
            w = wl.offline_chunk(w, int(fn.split("_chunk")[1].split(".")[0]))
        offsets, s, h, j, T, P = wl.batch_plan(w)
        assert np.array_equal(offsets, d["offsets"]) and np.array_equal(T, d["T"])
        n0 = int(offsets[1])
        raw = wl.host_rows(w.seed, np.arange(n0), w.V, w.dtype, s[:n0], h[:n0], j[:n0])
        assert wl.combine_checksums(wl.row_checksums(raw)) == int(d["checksum_req"][0])
        rows = [0, n0 // 2, n0 - 1]
        assert np.array_equal(d["ids"][:n0], wl.host_sample_ids(raw, T[:n0], None if P is None else P[:n0],
                                                                 w.seed, np.arange(n0)))
        ids = d["ids"]
    for r in rows:
        f = oracle.token_features(raw[r], w.dtype, int(ids[r]), float(T[r]), None if P is None else float(P[r]))
        for k in ("max_logit", "lse", "entropy", "logprob", "maxprob", "margin"):
            assert f[k] == d[k][r] or (math.isnan(f[k]) and math.isnan(d[k][r])), (fn, r, k)
        for k in ("rank", "argmax", "cutoff", "flags"):
            assert f[k] == int(d[k][r]), (fn, r, k)
