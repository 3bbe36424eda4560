"""The paper's verifier input sequence X = (l, m, h, rho) per token (top-K
entropy, position fraction): HIP path vs the fp64 oracle, element by element."""

import numpy as np
import pytest
import torch

import oracle
import paper_2608_28726_amd as pr
from oracle import sequence as oseq
from paper_2608_28726_amd import workloads as wl
from tests.gpu_common import compare_features, dtype_name, gpu_features, oracle_features, require_gpu, to_dev
from tests.helpers import assert_floats

pytestmark = pytest.mark.gpu

# Launch tiers of the sequence kernel (workgroup size by batch size).
TIER_ROWS = {1024: 100, 256: 600, 128: 2048}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def gpu_sequence(logits, ids, T, offsets, P=None, K=20, features=False):
    out = pr.feature_sequence(logits, ids, T, torch.as_tensor(offsets, dtype=torch.int32, device=logits.device),
                              top_p=P, top_k=K, features=features)
    torch.cuda.synchronize()
    if features:
        X, f = out
        return X.cpu().numpy(), {k: v.cpu().numpy() for k, v in f.items()}
    return out.cpu().numpy()


def oracle_sequence(logits, ids, T, offsets, P=None, K=20, rows=None):
    """Oracle X for `rows` (all rows when None): rho from the offsets, the rest per row."""
    rows = np.arange(logits.shape[0]) if rows is None else np.asarray(rows)
    sel = torch.as_tensor(rows, device=logits.device)
    raw = wl.to_host_raw(logits[sel])  # only the rows the oracle computes leave the device
    dt = dtype_name(logits)
    ids_h, T_h = ids[sel].cpu().numpy(), T[sel].cpu().numpy()
    P_h = None if P is None else P[sel].cpu().numpy()
    of = oracle.token_features_batch(raw, dt, ids_h, T_h, P_h)
    H = oseq.topk_entropy_batch(raw, dt, T_h, P_h, K)
    X = np.empty((len(rows), 4))
    X[:, 0] = of["logprob"]
    X[:, 1] = of["maxprob"]
    X[:, 2] = -H
    X[:, 3] = oseq.position_fraction(offsets)[rows]
    return X, of["ambiguous"]


def compare_sequence(Xg, Xo, amb=None, what=""):
    mask = None if amb is None else ~np.asarray(amb)
    for c, name in enumerate(("l", "m", "h", "rho")):
        assert_floats(f"{what}X[:, {c}] ({name})", Xg[:, c], Xo[:, c], mask=mask if c < 3 else None)


def split_offsets(n_rows, n_req, rng, empty=True):
    """Ragged offsets over n_rows rows with n_req requests (some empty)."""
    cuts = np.sort(rng.integers(0, n_rows + 1, n_req - 1))
    off = np.concatenate([[0], cuts, [n_rows]]).astype(np.int32)
    if empty and n_req >= 3:
        off[2] = off[1]  # request 1 is empty
    return off


def test_ragged_bf16_scaled_all_rows():
    """The ragged-batch row model (V = 151,936 bf16, T = 0.7), every row, K = 20."""
    w = wl.scaled(wl.WORKLOADS["ragged_64req_v151936_bf16"], n_req=5, len_hi=20)
    b = wl.make_batch(w, device="cpu")
    logits, ids, T = to_dev(b.logits, b.sampled_ids, b.temperature)
    print(f"case seq ragged_scaled rows={b.n_rows}", flush=True)
    Xg = gpu_sequence(logits, ids, T, b.offsets)
    Xo, _ = oracle_sequence(logits, ids, T, b.offsets)
    compare_sequence(Xg, Xo)


@pytest.mark.parametrize("block", sorted(TIER_ROWS))
@pytest.mark.parametrize("dtype,V", [(torch.bfloat16, 32000), (torch.float32, 8192)])
@pytest.mark.parametrize("K", [1, 5, 20, 32])
def test_tiers_and_k(block, dtype, V, K):
    """Every launch tier, both dtypes, several K: sampled rows against the oracle, rho on all."""
    n = TIER_ROWS[block]
    rng = np.random.default_rng(block * 7 + V + K)
    g = torch.Generator(device="cuda").manual_seed(int(rng.integers(1 << 31)))
    s = torch.tensor(rng.uniform(1, 4, (n, 1)), dtype=torch.float32, device="cuda")
    z = torch.randn(n, V, generator=g, device="cuda") * s
    spike = torch.tensor(rng.integers(0, V, n), device="cuda")
    z[torch.arange(n, device="cuda"), spike] += torch.tensor(rng.uniform(0, 15, n), dtype=torch.float32,
                                                             device="cuda")
    logits = z.to(dtype).contiguous()
    ids = torch.tensor(rng.integers(0, V, n), dtype=torch.int32, device="cuda")
    T = torch.tensor(rng.uniform(0.5, 1.5, n), dtype=torch.float32, device="cuda")
    off = split_offsets(n, max(3, n // 50), rng)
    print(f"case seq tier={block} dtype={dtype} V={V} K={K}", flush=True)
    Xg = gpu_sequence(logits, ids, T, off, K=K)
    rows = np.unique(np.concatenate([[0, n - 1], rng.choice(n, 24, replace=False)]))
    Xo, _ = oracle_sequence(logits, ids, T, off, K=K, rows=rows)
    compare_sequence(Xg[rows], Xo)
    assert_floats("rho all rows", Xg[:, 3], oseq.position_fraction(off))


def _edge_rows(V, rng):
    base = rng.normal(0, 2, V)
    rows = [(np.full(V, 0.5), 0, 1.0), (np.full(V, -1.25), V - 1, 0.7)]
    r = base.copy(); r[: V // 2] = -np.inf
    rows.append((r, V - 1, 0.9))                                       # masked half
    r = np.full(V, -np.inf); r[V - 1] = 1.0
    rows.append((r, 0, 1.0))                                           # one-hot via -inf
    r = np.full(V, -np.inf); r[: min(V, 3)] = [2.0, 1.0, 0.5][: min(V, 3)]
    rows.append((r, 1 % V, 1.0))                                       # fewer than K finite
    r = np.where(rng.random(V) < 0.5, 0.0, -0.0)
    rows.append((r, V // 3, 1.0))                                      # +-0 mix
    r = base.copy(); r[1 % V] = np.nan
    rows.append((r, 0, 1.0))                                           # NaN
    rows.append((np.full(V, -np.inf), 0, 1.0))                         # all -inf
    rows.append((base.copy(), V, 1.0))                                 # bad id
    rows.append((base.copy(), 1, 0.0))                                 # bad temperature
    rows.append((rng.choice([-1.0, 0.0, 0.5, 1.0], size=V), V // 2, 1.0))  # ties everywhere
    rows.append((base * 40.0, int(rng.integers(0, V)), 0.05))          # very peaked
    r = base.copy(); r[rng.choice(V, min(V, 40), replace=False)] = 3.0
    rows.append((r, 0, 1.0))                                           # a 40-way tie at the top
    return rows


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("V", [2, 7, 8, 63, 64, 65, 1000, 32000])
@pytest.mark.parametrize("K", [1, 20, 32])
def test_edge_rows(V, dtype, K):
    rng = np.random.default_rng(V + K)
    rows = _edge_rows(V, rng)
    z = torch.tensor(np.stack([r for r, _, _ in rows]), dtype=torch.float32).to(dtype)
    ids = torch.tensor([y for _, y, _ in rows], dtype=torch.int32)
    T = torch.tensor([t for _, _, t in rows], dtype=torch.float32)
    logits, ids, T = to_dev(z, ids, T)
    off = np.array([0, 4, 4, len(rows)], dtype=np.int32)
    print(f"case seq edge V={V} dtype={dtype} K={K}", flush=True)
    Xg = gpu_sequence(logits, ids, T, off, K=K)
    Xo, _ = oracle_sequence(logits, ids, T, off, K=K)
    compare_sequence(Xg, Xo)


def _crowded_rows(n, V, dtype, block, lanes, per_lane, seed):
    """n rows of N(0, 1) logits; in rows 0..7 the lanes `lanes` of a workgroup
    of `block` threads hold large logits: `per_lane` = "buckets" puts one in
    each of the lane's first 12 steps, "all" makes every logit of the lane
    large. Returns (logits, crafted row indices)."""
    g = torch.Generator(device="cuda").manual_seed(seed)
    z = torch.randn(n, V, generator=g, device="cuda")
    vec = 8 if dtype == torch.bfloat16 else 4
    U = 2 if dtype == torch.bfloat16 else 4
    nvec = V // vec
    crafted = list(range(8))
    for r in crafted:
        for li, lane in enumerate(lanes):
            if per_lane == "buckets":
                for s in range(12):
                    j = lane + s * U * block
                    if j < nvec:
                        z[r, j * vec + (s % vec)] = 8.0 + 0.25 * s + 0.01 * li + 0.5 * r
            else:
                idx = torch.arange(lane, nvec, block, device="cuda")
                el = (idx[:, None] * vec + torch.arange(vec, device="cuda")[None, :]).reshape(-1)
                z[r, el] = 20.0 + torch.randn(el.numel(), generator=g, device="cuda") * (1 + r)
    return z.to(dtype).contiguous(), crafted


@pytest.mark.parametrize("block", sorted(TIER_ROWS))
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("per_lane,lanes", [("buckets", [5]), ("buckets", [3, 64 + 9]), ("all", [5]),
                                            ("all", list(range(40, 56)))])
def test_crowded_lanes(block, dtype, per_lane, lanes):
    """Many of the largest logits in one lane (different buckets, or all of
    its share): the lane's third bucket exceeds the first threshold, its
    entries are withdrawn and its whole share relisted, compacting the list
    when it overflows."""
    n = TIER_ROWS[block]
    V = 262144 if per_lane == "all" else 65536
    logits, crafted = _crowded_rows(n, V, dtype, block, lanes, per_lane, seed=block + len(lanes))
    rng = np.random.default_rng(block)
    ids = torch.tensor(rng.integers(0, V, n), dtype=torch.int32, device="cuda")
    T = torch.tensor(rng.uniform(0.5, 1.5, n), dtype=torch.float32, device="cuda")
    off = np.array([0, n], dtype=np.int32)
    print(f"case seq crowded tier={block} dtype={dtype} {per_lane} lanes={len(lanes)}", flush=True)
    rows = crafted + [n - 1]
    for K in (20, 32):
        Xg = gpu_sequence(logits, ids, T, off, K=K)
        Xo, _ = oracle_sequence(logits, ids, T, off, K=K, rows=rows)
        compare_sequence(Xg[rows], Xo, what=f"K={K} ")


def test_topp_rows():
    """Top-p: the top-K probabilities on the renormalised nucleus; nuclei
    smaller than K (P near 0) sum over the nucleus only."""
    w = wl.scaled(wl.WORKLOADS["topp_128x256_v262144_f32"], n_req=3, len_hi=6)
    b = wl.make_batch(w, device="cpu")
    logits, ids, T, P = to_dev(b.logits, b.sampled_ids, b.temperature, b.top_p)
    P = P.clone()
    P[:3] = torch.tensor([1e-6, 0.02, 1.0], device="cuda")  # k = 1, a few tokens, top-p off
    print(f"case seq topp rows={b.n_rows}", flush=True)
    for K in (1, 20, 32):
        Xg = gpu_sequence(logits, ids, T, b.offsets, P=P, K=K)
        Xo, amb = oracle_sequence(logits, ids, T, b.offsets, P=P, K=K)
        compare_sequence(Xg, Xo, amb, what=f"K={K} ")


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_topp_small_nuclei_bf16_f32(dtype):
    rng = np.random.default_rng(11)
    n, V = 12, 4096
    z = torch.tensor(rng.normal(0, 3, (n, V)), dtype=torch.float32).to(dtype)
    P = torch.tensor(np.linspace(1e-4, 0.9, n), dtype=torch.float32)
    ids = torch.tensor(rng.integers(0, V, n), dtype=torch.int32)
    T = torch.tensor(rng.uniform(0.3, 1.2, n), dtype=torch.float32)
    logits, ids, T, P = to_dev(z, ids, T, P)
    off = np.array([0, 5, n], dtype=np.int32)
    Xg = gpu_sequence(logits, ids, T, off, P=P, K=20)
    Xo, amb = oracle_sequence(logits, ids, T, off, P=P, K=20)
    compare_sequence(Xg, Xo, amb)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_topp_undefined_rows(dtype):
    """The sequence variant on rows with 0 < P < 1 whose distribution is
    undefined (a NaN among the vectors and in the scalar tail, +inf, all
    -inf, a rejected temperature): l, m and h are NaN, rho is not; the
    ordinary rows around them match the oracle."""
    rng = np.random.default_rng(13)
    n, V = 8, 1027
    z = rng.normal(0, 2, (n, V))
    z[0, 100] = np.nan
    z[1, 1026] = np.nan
    z[2, 7] = np.inf
    z[3] = -np.inf
    T = np.full(n, 0.9)
    T[4] = 0.0
    P = np.full(n, 0.85)
    ids = rng.integers(0, V, n)
    logits, ids, T, P = to_dev(torch.tensor(z, dtype=torch.float32).to(dtype), torch.tensor(ids, dtype=torch.int32),
                               torch.tensor(T, dtype=torch.float32), torch.tensor(P, dtype=torch.float32))
    off = np.array([0, 3, 6, n], dtype=np.int32)
    print(f"case seq topp undefined rows {dtype}", flush=True)
    Xg = gpu_sequence(logits, ids, T, off, P=P, K=20)
    assert np.isnan(Xg[:5, :3]).all() and np.isfinite(Xg[:, 3]).all()
    Xo, amb = oracle_sequence(logits, ids, T, off, P=P, K=20)
    compare_sequence(Xg, Xo, amb)


@pytest.mark.parametrize("topp", [False, True])
def test_features_from_the_same_pass(topp):
    """features=True gives the per-token features in the same pass: parity
    with the oracle, X's first two columns are its logprob and maxprob, and
    where pr_token_features takes the same launch shape (one workgroup per
    row: here 600 rows, or any top-p batch) its outputs are bit-identical."""
    if topp:
        w = wl.scaled(wl.WORKLOADS["topp_128x256_v262144_f32"], n_req=3, len_hi=8)
    else:
        w = wl.scaled(wl.WORKLOADS["ragged_64req_v151936_bf16"], n_req=6, len_lo=100, len_hi=100, V=32000)
    b = wl.make_batch(w, device="cpu")
    logits, ids, T, P = to_dev(b.logits, b.sampled_ids, b.temperature, b.top_p)
    Xg, fs = gpu_sequence(logits, ids, T, b.offsets, P=P, features=True)
    compare_features(fs, oracle_features(logits, ids, T, P))
    assert np.array_equal(Xg[:, 0].view(np.uint32), fs["logprob"].view(np.uint32))
    assert np.array_equal(Xg[:, 1].view(np.uint32), fs["maxprob"].view(np.uint32))
    ft = gpu_features(logits, ids, T, P)
    for k in ft:
        assert np.array_equal(fs[k].view(np.uint32), ft[k].view(np.uint32)), k


def test_full_size_ragged_batch():
    """The 64-request V = 151,936 bf16 batch at full size: sampled rows
    against the oracle, rho on every row, two runs bit-identical."""
    w = wl.WORKLOADS["ragged_64req_v151936_bf16"]
    b = wl.make_batch(w, device="cuda")
    n = b.n_rows
    print(f"case seq full rows={n}", flush=True)
    Xg = gpu_sequence(b.logits, b.sampled_ids, b.temperature, b.offsets)
    Xg2 = gpu_sequence(b.logits, b.sampled_ids, b.temperature, b.offsets)
    assert np.array_equal(Xg.view(np.uint32), Xg2.view(np.uint32))
    rng = np.random.default_rng(5)
    rows = np.unique(np.concatenate([[0, n - 1], rng.choice(n, 30, replace=False)]))
    Xo, _ = oracle_sequence(b.logits, b.sampled_ids, b.temperature, b.offsets, rows=rows)
    compare_sequence(Xg[rows], Xo)
    assert_floats("full rho", Xg[:, 3], oseq.position_fraction(b.offsets))
