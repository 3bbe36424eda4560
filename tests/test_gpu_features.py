"""Per-token features: HIP path vs the fp64 oracle, element by element."""

import math

import numpy as np
import pytest
import torch

import paper_2608_28726_amd as pr
from paper_2608_28726_amd import workloads as wl
from tests.gpu_common import compare_features, gpu_features, oracle_features, require_gpu, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _batch_on_gpu(w, lengths=None):
    b = wl.make_batch(w, device="cpu", lengths=lengths)
    logits, ids, T, P = to_dev(b.logits, b.sampled_ids, b.temperature, b.top_p)
    return b, logits, ids, T, P


def test_ragged_bf16_rows_scaled():
    """The ragged-batch row model (V = 151,936 bf16, T = 0.7) on a few requests."""
    w = wl.scaled(wl.WORKLOADS["ragged_64req_v151936_bf16"], n_req=5, len_hi=20)
    b, logits, ids, T, _ = _batch_on_gpu(w)
    print(f"case ragged_scaled rows={b.n_rows}", flush=True)
    compare_features(gpu_features(logits, ids, T), oracle_features(logits, ids, T))


@pytest.mark.parametrize("n_rows,V,dtype", [(1, 151936, torch.bfloat16), (3, 151936, torch.bfloat16),
                                            (7, 262144, torch.float32), (2, 65536 + 24, torch.float32)])
def test_split_rows(n_rows, V, dtype):
    """Few long rows: each row is split over several workgroups and merged."""
    w = wl.scaled(wl.WORKLOADS["ragged_64req_v151936_bf16"], n_req=1, len_hi=n_rows, V=V,
                  dtype="bf16" if dtype == torch.bfloat16 else "f32", seed=1000 + n_rows)
    b, logits, ids, T, _ = _batch_on_gpu(w, lengths=np.array([n_rows]))
    print(f"case split rows={n_rows} V={V}", flush=True)
    assert pr.token_features_workspace(logits) > 0
    compare_features(gpu_features(logits, ids, T), oracle_features(logits, ids, T))


def _special_rows(V, rng):
    """(row values float64, y, T) edge cases for one vocabulary size."""
    rows = []
    base = rng.normal(0, 2, V)
    rows.append((np.full(V, 0.5), 0, 1.0))                    # all equal, y first
    rows.append((np.full(V, -1.25), V - 1, 0.7))              # all equal, y last
    r = base.copy(); r[V // 2] = 30.0
    rows.append((r, V // 2, 1.0))                              # y = argmax
    r = base.copy(); r[: V // 2] = -np.inf
    rows.append((r, V - 1, 0.9))                               # masked half
    r = np.full(V, -np.inf); r[V - 1] = 1.0
    rows.append((r, 0, 1.0))                                   # one-hot via -inf, y masked
    r = np.full(V, -np.inf); r[0] = 1.0; r[V - 1] = -np.inf
    rows.append((r, V - 1, 1.0))                               # y = -inf with -inf ties before it
    r = np.where(rng.random(V) < 0.5, 0.0, -0.0)
    rows.append((r, V // 3, 1.0))                              # +-0 mix
    r = base.copy(); r[1 % V] = np.nan
    rows.append((r, 0, 1.0))                                   # NaN
    r = base.copy(); r[V - 1] = np.inf
    rows.append((r, 0, 1.0))                                   # +inf
    rows.append((np.full(V, -np.inf), 0, 1.0))                 # all -inf
    rows.append((base.copy(), -1, 1.0))                        # bad id
    rows.append((base.copy(), V, 1.0))                         # bad id
    for T in (0.0, -1.0, math.inf, math.nan, 2.0 ** -101):
        rows.append((base.copy(), 1, T))                       # bad temperature
    r = base.copy(); r[0] = np.nan
    rows.append((r, 1, 0.0))                                   # NaN and bad temperature
    rows.append((np.zeros(V), 1, 2.0 ** -100))                 # smallest temperature
    r = rng.choice([-1.0, 0.0, 0.5, 1.0], size=V)
    for y in sorted({0, 1, V // 2, V - 2, V - 1}):
        rows.append((r, y, 1.0))                               # ties everywhere
    r = rng.normal(0, 1e-39, V)
    rows.append((r, 0, 1.0))                                   # subnormals
    r = base.copy(); r[0] = 2.0 ** 102
    rows.append((r, 0, 1.0))                                   # |z| > 2^100 T
    rows.append((base * 40.0, int(rng.integers(0, V)), 0.05))  # very peaked
    return rows


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("V", [2, 7, 8, 63, 64, 65, 1000, 32000])
def test_edge_rows(V, dtype):
    rng = np.random.default_rng(V)
    rows = _special_rows(V, rng)
    z = torch.tensor(np.stack([r for r, _, _ in rows]), dtype=torch.float32).to(dtype)
    ids = torch.tensor([y for _, y, _ in rows], dtype=torch.int32)
    T = torch.tensor([t for _, _, t in rows], dtype=torch.float32)
    logits, ids, T = to_dev(z, ids, T)
    print(f"case edge V={V} dtype={dtype} rows={len(rows)}", flush=True)
    compare_features(gpu_features(logits, ids, T), oracle_features(logits, ids, T))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("V,pad", [(1000, 3), (4093, 5), (151936, 1), (32000, 17)])
def test_strided_unaligned_rows(V, pad, dtype):
    """row_stride > V and rows that start off 16-byte boundaries."""
    rng = np.random.default_rng(V + pad)
    n = 9
    full = torch.tensor(rng.normal(0, 3, (n, V + pad)), dtype=torch.float32).to(dtype)
    ids = torch.tensor(rng.integers(0, V, n), dtype=torch.int32)
    T = torch.tensor(rng.uniform(0.5, 1.5, n), dtype=torch.float32)
    full, ids, T = to_dev(full, ids, T)
    logits = full[:, :V]
    print(f"case strided V={V} pad={pad} dtype={dtype}", flush=True)
    compare_features(gpu_features(logits, ids, T), oracle_features(logits, ids, T))
    off = full[:, 1:V + 1]  # every row starts one element late
    compare_features(gpu_features(off, ids, T), oracle_features(off, ids, T), what="offset ")


def test_deterministic():
    """The no-top-p path has no float atomics: two runs are bit-identical."""
    w = wl.scaled(wl.WORKLOADS["ragged_64req_v151936_bf16"], n_req=3, len_hi=10)
    b, logits, ids, T, _ = _batch_on_gpu(w)
    a1 = gpu_features(logits, ids, T)
    a2 = gpu_features(logits, ids, T)
    for k in a1:
        assert np.array_equal(a1[k].view(np.uint32), a2[k].view(np.uint32)), k
    one = gpu_features(logits[:1].contiguous(), ids[:1].contiguous(), T[:1].contiguous())  # split path
    for k in ("rank", "argmax", "cutoff", "flags"):
        assert one[k][0] == a1[k][0], k


def test_binding_rejects_host_tensors():
    """Every caller-supplied tensor of the binding must live on the logits'
    device: a host tensor is refused with ValueError before anything is
    launched (it would otherwise reach a kernel as a host pointer)."""
    n, V = 4, 256
    logits = torch.randn(n, V, device="cuda")
    ids = torch.zeros(n, dtype=torch.int32, device="cuda")
    T = torch.ones(n, device="cuda")
    good = pr.token_features(logits, ids, T)
    torch.cuda.synchronize()
    for k in ("lse", "rank", "flags"):
        bad = dict(good)
        bad[k] = bad[k].cpu()
        with pytest.raises(ValueError):
            pr.token_features(logits, ids, T, out=bad)
    with pytest.raises(ValueError):
        pr.token_features(logits, ids, T, top_p=0.9, workspace=torch.empty(1 << 20, dtype=torch.uint8))
    with pytest.raises(ValueError):
        pr.sample_features(logits, T.cpu(), seed=1)
    bad = dict(good)
    bad["margin"] = bad["margin"].cpu()
    with pytest.raises(ValueError):
        pr.sample_features(logits, T, seed=1, out=bad)
    offsets = torch.tensor([0, 2, n], dtype=torch.int32, device="cuda")
    with pytest.raises(ValueError):
        pr.request_aggregate(bad, offsets)
    with pytest.raises(ValueError):
        pr.validate_offsets(offsets.cpu(), n)
    st = pr.StreamState(8, 16)
    try:
        with pytest.raises(ValueError):
            st.step(logits, torch.arange(n, dtype=torch.int32), ids, T)
        with pytest.raises(ValueError):
            st.finish(torch.arange(n, dtype=torch.int32), 0.5)
        with pytest.raises(ValueError):
            st.reset(torch.arange(n, dtype=torch.int32))
    finally:
        st.close()
    X = torch.zeros(n, 4, device="cuda")
    w = torch.zeros(pr._abi.PR_HEAD_WEIGHTS, device="cuda")
    with pytest.raises(ValueError):
        pr.verifier_head(X, offsets, w, max_len=4, workspace=torch.empty(1 << 16, dtype=torch.uint8))
    torch.cuda.synchronize()
