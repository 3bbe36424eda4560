"""The paper's verifier head on the GPU (projection + positional encoding,
two encoder layers, mean pool, sigmoid) vs the fp64 oracle."""

import math

import numpy as np
import pytest
import torch

import paper_2608_28726_amd as pr
from oracle import head as ohead
from oracle import sequence as oseq
from paper_2608_28726_amd import workloads as wl
from tests.gpu_common import oracle_features, require_gpu, to_dev
from tests.helpers import assert_floats

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def synthetic_sequence(lengths, seed):
    """Input sequences shaped like the verifier's: l <= 0, m in (0, 1], h <= 0, rho = t / T."""
    rng = np.random.default_rng(seed)
    rows = []
    for n in lengths:
        rows.append(np.stack([-rng.exponential(1.5, n), rng.uniform(0.05, 1.0, n), -rng.uniform(0.0, 3.0, n),
                              (np.arange(n) + 1) / max(n, 1)], axis=1))
    X = np.concatenate(rows).astype(np.float32) if rows else np.zeros((0, 4), np.float32)
    off = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    return X, off


def run_head(X, off, weights, max_len=None):
    Xd = torch.tensor(X, device="cuda").reshape(-1, 4).contiguous()
    s = pr.verifier_head(Xd, torch.tensor(off, device="cuda"), torch.tensor(weights, device="cuda"),
                         max_len=max_len)
    torch.cuda.synchronize()
    return s.cpu().numpy()


@pytest.mark.parametrize("seed", [0, 1])
def test_ragged_lengths(seed):
    """Lengths around every tile and chunk boundary, empty requests included."""
    lengths = [1, 2, 0, 7, 63, 64, 65, 128, 129, 200, 0, 513, 31]
    X, off = synthetic_sequence(lengths, seed)
    weights = wl.head_weights(seed=200 + seed)
    print(f"case head ragged seed={seed} rows={X.shape[0]}", flush=True)
    got = run_head(X, off, weights, max_len=513)
    ref = ohead.head_scores(X.astype(np.float64), off, weights.astype(np.float64))
    assert_floats("head score", got, ref)
    assert np.isnan(got[2]) and np.isnan(got[10])


def test_max_len_and_determinism():
    lengths = [100, 300, 50]
    X, off = synthetic_sequence(lengths, 3)
    weights = wl.head_weights(seed=7)
    a = run_head(X, off, weights, max_len=300)
    b = run_head(X, off, weights, max_len=300)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    c = run_head(X, off, weights, max_len=150)  # request 1 is longer than max_len
    assert np.isnan(c[1]) and c[0] == a[0] and c[2] == a[2]


def test_many_requests():
    """64 requests of U{16..512} tokens, the ragged batch's request shape."""
    rng = np.random.default_rng(11)
    lengths = rng.integers(16, 513, 64).tolist()
    X, off = synthetic_sequence(lengths, 11)
    weights = wl.head_weights(seed=1)
    got = run_head(X, off, weights, max_len=512)
    sample = [0, 5, 17, 33, 63]
    ref = np.array([ohead.head_score(X[off[i]:off[i + 1]].astype(np.float64),
                                     ohead.unpack_weights(weights.astype(np.float64))) for i in sample])
    assert_floats("head score (64 requests)", got[sample], ref)


def test_thousands_of_short_requests():
    """1,500 requests of 0..40 tokens: more requests than the planning
    workgroup has threads, and a deep search for each row's request; every
    score against the oracle."""
    rng = np.random.default_rng(1500)
    lengths = rng.integers(0, 41, 1500).tolist()
    X, off = synthetic_sequence(lengths, 12)
    weights = wl.head_weights(seed=9)
    print(f"case head 1500 requests rows={X.shape[0]}", flush=True)
    got = run_head(X, off, weights, max_len=40)
    ref = ohead.head_scores(X.astype(np.float64), off, weights.astype(np.float64))
    assert_floats("head score (1,500 requests)", got, ref)
    empty = np.asarray(lengths) == 0
    assert np.isnan(got[empty]).all() and np.isfinite(got[~empty]).all()


def test_end_to_end_from_logits():
    """Logits -> verifier input sequence -> head -> ship, both sides from the
    logits: the oracle builds its own X."""
    w = wl.scaled(wl.WORKLOADS["ragged_64req_v151936_bf16"], n_req=4, len_hi=12, V=32000)
    b = wl.make_batch(w, device="cpu")
    logits, ids, T = to_dev(b.logits, b.sampled_ids, b.temperature)
    off = torch.tensor(b.offsets, device="cuda")
    weights = wl.head_weights()
    X = pr.feature_sequence(logits, ids, T, off)
    s = pr.verifier_head(X, off, torch.tensor(weights, device="cuda"), max_len=12)
    ship, _ = pr.route(s, w.tau)
    torch.cuda.synchronize()
    of = oracle_features(logits, ids, T)
    H = oseq.topk_entropy_batch(wl.to_host_raw(logits), "bf16", T.cpu().numpy())
    Xo = oseq.feature_sequence(of, H, b.offsets)
    ref = ohead.head_scores(Xo, b.offsets, weights.astype(np.float64))
    assert_floats("end-to-end head score", s.cpu().numpy(), ref)
    expect = (ref >= w.tau).astype(np.uint8)
    band = np.abs(ref - w.tau) <= 1e-5
    assert np.all((ship.cpu().numpy() == expect) | band)


def test_work_list_edges():
    """The attention's work list: no item at all (every request empty or
    longer than max_len), many empty requests around a few real ones, and
    one request of 1,500 tokens (24 key tiles) among short ones; scores
    against the oracle and bit-identical across calls."""
    weights = wl.head_weights(seed=9)
    X, off = synthetic_sequence([300, 0, 400], 21)
    got = run_head(X, off, weights, max_len=200)  # no request within max_len: an empty list
    assert np.isnan(got).all()
    lengths = [0] * 40 + [5, 0, 70] + [0] * 20
    X, off = synthetic_sequence(lengths, 22)
    got = run_head(X, off, weights, max_len=70)
    ref = ohead.head_scores(X.astype(np.float64), off, weights.astype(np.float64))
    assert_floats("head score (empty requests)", got, ref)
    assert np.isnan(got[[i for i, n in enumerate(lengths) if n == 0]]).all()
    lengths = [1500, 3, 64, 65, 17]
    X, off = synthetic_sequence(lengths, 23)
    print(f"case head work list rows={X.shape[0]}", flush=True)
    got = run_head(X, off, weights, max_len=1500)
    ref = ohead.head_scores(X.astype(np.float64), off, weights.astype(np.float64))
    assert_floats("head score (one long request)", got, ref)
    again = run_head(X, off, weights, max_len=1500)
    assert np.array_equal(got.view(np.uint32), again.view(np.uint32))
