"""Fused sample-and-verify (pr_sample_features): the draws follow the oracle's
distribution softmax(z / T) (chi-square tests at fixed seeds), and every
output of a drawn row equals the oracle's for the drawn token.

The draws are random, so the comparison with the oracle is distributional:
many rows with the same logits (each row draws with its own counter) give
empirical frequencies, tested against the oracle's probabilities. Given the
drawn ids, the features and the verifier input are deterministic and are
compared value by value (R13)."""

import math

import numpy as np
import pytest
import torch
from scipy import stats

import oracle
from oracle import sequence as oseq
import paper_2608_28726_amd as pr
from paper_2608_28726_amd import workloads as wl
from tests.gpu_common import compare_features, dtype_name, oracle_features, require_gpu

pytestmark = pytest.mark.gpu

P_MIN = 1e-5  # p-value below which a frequency test fails (fixed seeds: a pass is reproducible)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _row_tensor(z: np.ndarray, dtype: str, n: int, misalign: bool) -> torch.Tensor:
    """n copies of row z on the GPU; misalign shifts each row by one element
    off the 16-byte boundary (so rows have scalar head elements)."""
    t = torch.from_numpy(z.astype(np.float32)).to(torch.float32 if dtype == "f32" else torch.bfloat16)
    V = z.shape[0]
    if not misalign:
        return t.unsqueeze(0).expand(n, V).contiguous().cuda()
    big = torch.zeros((n, V + 1), dtype=t.dtype)
    big[:, 1:] = t
    return big.cuda()[:, 1:]


def _host_bits(z: np.ndarray, dtype: str) -> np.ndarray:
    """The stored row as the oracle reads it (float32 values or bf16 bits)."""
    t = torch.from_numpy(z.astype(np.float32))
    if dtype == "f32":
        return t.numpy()
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _draw_counts(z, dtype, T, n_rows, reps, misalign=False, seed=1234):
    logits = _row_tensor(z, dtype, n_rows, misalign)
    V = z.shape[0]
    counts = np.zeros(V, dtype=np.int64)
    bad = 0
    for k in range(reps):
        ids, _, _ = pr.sample_features(logits, T, seed=seed, offset=k, features=False)
        torch.cuda.synchronize()
        y = ids.cpu().numpy()
        bad += int(np.count_nonzero((y < 0) | (y >= V)))
        counts += np.bincount(y[(y >= 0) & (y < V)], minlength=V)
    return counts, bad


def _chi_square(counts, p, groups):
    """Pearson's test over the categories `groups` (lists of token ids)."""
    n = counts.sum()
    obs = np.array([counts[g].sum() for g in groups], dtype=np.float64)
    exp = np.array([p[g].sum() for g in groups]) * n
    assert (exp >= 5).all(), exp
    stat = float(((obs - exp) ** 2 / exp).sum())
    return stat, float(stats.chi2.sf(stat, len(groups) - 1))


def _groups_by_mass(p, min_mass):
    """Tokens with at least min_mass each on their own; the rest pooled in
    consecutive index ranges of about min_mass each (so that where in the row
    a token lies is tested too)."""
    heavy = [[int(v)] for v in np.flatnonzero(p >= min_mass)]
    rest = np.flatnonzero((p < min_mass) & (p > 0))
    groups, cur, acc = [], [], 0.0
    for v in rest:
        cur.append(int(v))
        acc += p[v]
        if acc >= min_mass:
            groups.append(cur)
            cur, acc = [], 0.0
    if cur:
        if groups:
            groups[-1].extend(cur)
        else:
            groups.append(cur)
    return heavy + groups


@pytest.mark.parametrize("dtype,n_rows,reps,misalign", [
    ("f32", 4096, 10, False),   # one workgroup of 128 threads per row
    ("bf16", 1000, 40, True),   # 256 threads per row, scalar head elements
    ("f32", 200, 200, True),    # 1,024 threads per row
])
def test_small_row_draws_follow_softmax(dtype, n_rows, reps, misalign):
    rng = np.random.default_rng(11)
    V = 37
    z = rng.normal(0, 1.5, V).astype(np.float32)
    z[[3, 17, 30]] = -np.inf
    T = 0.8
    print(f"case small-row draws {dtype} rows={n_rows} reps={reps} misalign={misalign}", flush=True)
    counts, bad = _draw_counts(z, dtype, T, n_rows, reps, misalign)
    assert bad == 0
    p = oracle.token_probabilities(_host_bits(z, dtype), dtype, T)
    assert counts[p == 0].sum() == 0, "a masked token was drawn"
    stat, pv = _chi_square(counts, p, _groups_by_mass(p, 0.01))
    assert pv > P_MIN, (stat, pv)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_long_row_draws_follow_softmax(dtype):
    """40,000 tokens: a lane scans many buckets, and a ragged tail."""
    rng = np.random.default_rng(12)
    V = 40003
    z = rng.normal(0, 1.0, V).astype(np.float32)
    heavy = rng.choice(V, 24, replace=False)
    z[heavy] = rng.uniform(7.0, 9.5, 24).astype(np.float32)  # about half the mass on 24 tokens
    z[rng.choice(V, 500, replace=False)] = -np.inf
    T = 1.0
    print(f"case long-row draws {dtype}", flush=True)
    counts, bad = _draw_counts(z, dtype, T, 4096, 12)
    assert bad == 0
    p = oracle.token_probabilities(_host_bits(z, dtype), dtype, T)
    assert counts[p == 0].sum() == 0
    groups = _groups_by_mass(p, 0.004)
    stat, pv = _chi_square(counts, p, groups)
    assert pv > P_MIN, (stat, pv, len(groups))


def test_features_and_sequence_for_drawn_tokens():
    w = wl.scaled(wl.WORKLOADS["ragged_64req_v151936_bf16"], n_req=4, len_hi=7, len_lo=2)
    b = wl.make_batch(w, device="cpu")
    logits, T = b.logits.cuda(), b.temperature.cuda()
    offsets = torch.as_tensor(b.offsets).cuda()
    print(f"case features of drawn tokens: {b.n_rows} rows", flush=True)
    ids, feats, X = pr.sample_features(logits, T, seed=7, offset=3, offsets=offsets)
    torch.cuda.synchronize()
    y = ids.cpu().numpy()
    assert ((y >= 0) & (y < w.V)).all()
    g = {k: v.cpu().numpy() for k, v in feats.items()}
    assert (g["rank"] == -1).all()  # "not available" on the fused path
    o = oracle_features(logits, ids, T)
    g["rank"] = o["rank"].copy()
    compare_features(g, o, what="drawn ")
    H = oseq.topk_entropy_batch(wl.to_host_raw(b.logits), dtype_name(logits), b.temperature.numpy())
    Xo = oseq.feature_sequence(o, H, b.offsets)
    Xg = X.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(Xg - Xo) <= 1e-5 + 1e-4 * np.abs(Xo)), (Xg, Xo)
    # the same draw with features only, and with ids only
    ids2, feats2, _ = pr.sample_features(logits, T, seed=7, offset=3)
    ids3, _, _ = pr.sample_features(logits, T, seed=7, offset=3, features=False)
    torch.cuda.synchronize()
    assert torch.equal(ids, ids2) and torch.equal(ids, ids3)
    for k in feats:
        assert torch.equal(feats[k], feats2[k]), k


def test_determinism_and_fresh_offsets():
    w = wl.scaled(wl.WORKLOADS["ragged_64req_v151936_bf16"], n_req=100, len_hi=40, len_lo=30, V=8192)
    b = wl.make_batch(w, device="cuda")
    a1, _, _ = pr.sample_features(b.logits, b.temperature, seed=5, offset=0, features=False)
    a2, _, _ = pr.sample_features(b.logits, b.temperature, seed=5, offset=0, features=False)
    c1, _, _ = pr.sample_features(b.logits, b.temperature, seed=5, offset=1, features=False)
    d1, _, _ = pr.sample_features(b.logits, b.temperature, seed=6, offset=0, features=False)
    torch.cuda.synchronize()
    assert torch.equal(a1, a2)
    # a row whose largest token is not nearly certain draws differently under a new key
    frac_c = (a1 != c1).float().mean().item()
    frac_d = (a1 != d1).float().mean().item()
    assert frac_c > 0.2 and frac_d > 0.2, (frac_c, frac_d)
    # rows keep their draws when the batch around them changes (same tier:
    # more than 2,048 rows, one workgroup of 128 threads per row)
    n = b.n_rows
    assert n > 2200
    sub, _, _ = pr.sample_features(b.logits[100:], b.temperature[100:], seed=5, offset=0, features=False)
    torch.cuda.synchronize()
    # the row index is part of the counter: shifted rows draw afresh, so
    # compare a batch that keeps the indices: the same rows, later ones cut
    cut, _, _ = pr.sample_features(b.logits[: n - 100], b.temperature[: n - 100], seed=5, offset=0,
                                   features=False)
    torch.cuda.synchronize()
    assert torch.equal(cut, a1[: n - 100])
    assert sub.shape[0] == n - 100


def test_undefined_and_degenerate_rows():
    V = 1000
    rows = torch.randn((8, V), dtype=torch.float32)
    rows[0, 5] = float("nan")                 # NaN: undefined
    rows[1, 9] = float("inf")                 # +inf: undefined
    rows[2] = float("-inf")                   # all masked: undefined
    rows[4] = float("-inf")                   # one finite token: always drawn
    rows[4, 321] = 2.0
    rows[5] = float("-inf")                   # three finite tokens
    rows[5, [10, 500, 999]] = torch.tensor([0.0, 1.0, 0.5])
    T = torch.ones(8)
    T[3] = 0.0                                # rejected temperature
    print("case undefined rows", flush=True)
    for off in range(20):
        ids, feats, _ = pr.sample_features(rows.cuda(), T.cuda(), seed=9, offset=off)
        torch.cuda.synchronize()
        y = ids.cpu().numpy()
        fl = feats["flags"].cpu().numpy()
        assert (y[:4] == -1).all(), y
        assert fl[0] & 1 and fl[1] & 1 and fl[2] & 1 and fl[3] & 4
        assert (fl[:4] & 2).all()  # BAD_ID: no token drawn
        assert y[4] == 321 and abs(feats["logprob"][4].item()) < 1e-6
        assert y[5] in (10, 500, 999)
        assert (y[6:] >= 0).all() and (fl[4:] == 0).all()


def test_full_size_draws_are_consistent():
    """The bench batch (64 requests, V = 151,936 bf16): E[log p(y)] = -H per
    row, so the mean of log p(y) + H over the rows is zero within its
    standard error; sampled rows match the oracle for their drawn ids."""
    w = wl.WORKLOADS["ragged_64req_v151936_bf16"]
    b = wl.make_batch(w, device="cuda")
    print(f"case full-size draws: {b.n_rows} rows", flush=True)
    ids, feats, _ = pr.sample_features(b.logits, b.temperature, seed=2024, offset=0)
    torch.cuda.synchronize()
    lp = feats["logprob"].double().cpu().numpy()
    H = feats["entropy"].double().cpu().numpy()
    assert np.isfinite(lp).all() and (ids.cpu().numpy() >= 0).all()
    d = lp + H
    se = math.sqrt(float(np.mean(d * d)) / d.shape[0])
    assert abs(float(d.mean())) < 5 * se, (float(d.mean()), se)
    rows = np.random.default_rng(4).choice(b.n_rows, 12, replace=False)
    sel = torch.as_tensor(rows, device=b.logits.device)
    o = oracle.token_features_batch(wl.to_host_raw(b.logits[sel]), "bf16", ids[sel].cpu().numpy(),
                                    b.temperature[sel].cpu().numpy())
    g = {k: v.cpu().numpy()[rows] for k, v in feats.items()}
    assert (g["rank"] == -1).all()
    g["rank"] = o["rank"].copy()
    compare_features(g, o, what="full-size drawn ")
