"""Top-p (nucleus) features: exact cutoff index, rank and renormalised
features, HIP path vs the fp64 oracle."""

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


def _run(z, ids, T, P, dtype=torch.float32):
    logits, ids, T, P = to_dev(torch.as_tensor(z, dtype=torch.float32).to(dtype), torch.as_tensor(ids, dtype=torch.int32),
                               torch.as_tensor(T, dtype=torch.float32), torch.as_tensor(P, dtype=torch.float32))
    return logits, ids, T, P


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("V", [2, 7, 8, 64, 1000, 32000])
def test_topp_random_rows(V, dtype):
    rng = np.random.default_rng(100 + V)
    n = 24
    z = rng.normal(0, rng.uniform(0.5, 4, (n, 1)), (n, V))
    z[np.arange(n), rng.integers(0, V, n)] += rng.uniform(0, 15, n)
    T = rng.uniform(0.3, 1.2, n)
    P = rng.uniform(0.05, 0.99, n)
    P[:4] = [1.0, 2.0, 1e-7, 0.999]
    ids = rng.integers(0, V, n)
    logits, ids, T, P = _run(z, ids, T, P, dtype)
    print(f"case topp random V={V} {dtype}", flush=True)
    compare_features(gpu_features(logits, ids, T, P), oracle_features(logits, ids, T, P))


def test_topp_special_rows():
    V = 64
    rows, ids, Ts, Ps = [], [], [], []
    def add(z, y, T, P):
        rows.append(np.asarray(z, dtype=np.float64)); ids.append(y); Ts.append(T); Ps.append(P)
    add(np.zeros(V), 3, 1.0, 0.5)            # uniform: k = 32
    add(np.zeros(V), 40, 1.0, 0.5)           # sampled token outside the nucleus
    add(np.zeros(V), 0, 1.0, 0.3)            # k = ceil(0.3 * 64) = 20
    z = np.full(V, -np.inf); z[5] = 1.0
    add(z, 5, 1.0, 0.9)                      # one-hot via -inf
    add(z, 6, 1.0, 0.9)                      # masked sampled token
    add(np.arange(V) * -0.5, 2, 0.7, 0.8)    # geometric
    add(np.zeros(V), 1, 1.0, 0.0)            # P = 0: flagged
    add(np.zeros(V), 1, 1.0, math.nan)       # P = NaN: flagged
    add(np.zeros(V), 1, 1.0, -0.5)           # P < 0: flagged
    add(np.where(np.arange(V) < 10, 2.0, 0.0), 9, 1.0, 0.5)   # tie block at the top
    logits, ids, T, P = _run(np.stack(rows), ids, Ts, Ps)
    compare_features(gpu_features(logits, ids, T, P), oracle_features(logits, ids, T, P))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_topp_undefined_rows_with_a_nucleus(dtype):
    """Rows with 0 < P < 1 whose distribution is undefined: their first pass
    forms no exps, so a NaN must still mark the row (in the vector body and
    in the scalar tail, V = 67); +inf and all -inf rows; a rejected
    temperature (the plain pass); one ordinary row as a control."""
    V = 67
    rng = np.random.default_rng(67)
    base = rng.normal(0, 1, (6, V))
    base[0, 10] = np.nan                     # NaN among the vectors
    base[1, 66] = np.nan                     # NaN in the tail
    base[2, 5] = np.inf                      # +inf
    base[3] = -np.inf                        # every token masked
    T = [1.0, 1.0, 1.0, 1.0, 0.0, 0.8]       # row 4: rejected temperature
    P = [0.9, 0.9, 0.9, 0.9, 0.9, 0.9]
    ids = [3, 4, 5, 6, 7, 8]
    logits, ids, T, P = _run(base, ids, T, P, dtype)
    print(f"case topp undefined rows {dtype}", flush=True)
    g = gpu_features(logits, ids, T, P)
    assert (g["flags"][:4] & pr.FLAG_NONFINITE).all() and g["flags"][4] & pr.FLAG_BAD_TP
    assert g["flags"][5] & (pr.FLAG_NONFINITE | pr.FLAG_BAD_TP) == 0
    compare_features(g, oracle_features(logits, ids, T, P))


@pytest.mark.parametrize("V", [262144, 151936])
def test_topp_massive_ties_radix_path(V):
    """Rows whose boundary bins hold more logits than the LDS sort takes:
    all-equal bf16 rows and rows with a few distinct values."""
    rng = np.random.default_rng(V)
    rows = [np.zeros(V), rng.choice([0.0, 0.5, 1.0], size=V), np.full(V, 3.0)]
    rows[2][: V // 3] = 3.5
    ids = [7, int(rng.integers(0, V)), V - 1]
    logits, ids, T, P = _run(np.stack(rows), ids, [1.0, 0.9, 1.1], [0.37, 0.8, 0.6], torch.bfloat16)
    print(f"case topp ties V={V}", flush=True)
    compare_features(gpu_features(logits, ids, T, P), oracle_features(logits, ids, T, P))


def test_topp_deterministic():
    """Two runs give bit-identical outputs on every path: the two-read
    method (random rows), the three-pass fallback (near-flat row) and its
    radix refinement (tie-heavy rows), whose float atomics only choose bins
    and digits."""
    V = 151936
    rng = np.random.default_rng(5)
    rows = [rng.normal(0, 2, V), rng.normal(0, 0.01, V), np.zeros(V), rng.choice([0.0, 0.5, 1.0], size=V)]
    ids = [int(rng.integers(0, V)) for _ in rows]
    logits, ids, T, P = _run(np.stack(rows), ids, [0.8, 1.2, 1.0, 0.9], [0.9, 0.93, 0.37, 0.8], torch.bfloat16)
    print("case topp deterministic", flush=True)
    a1 = gpu_features(logits, ids, T, P)
    a2 = gpu_features(logits, ids, T, P)
    for k in a1:
        assert np.array_equal(a1[k].view(np.uint32), a2[k].view(np.uint32)), k
    compare_features(a1, oracle_features(logits, ids, T, P))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_topp_histogram_edge_rows(dtype):
    """Rows aimed at each branch of the two-read method: no finite anchor
    (the first vectors all -inf), more logits far above the anchor than the
    list holds, a crossing inside that list (one dominant spike), a nucleus
    spanning the list and the bins, a near-flat row with a wide window, and
    large logits on both sides of the limit on |A0| / T of the binning."""
    V = 65536
    rng = np.random.default_rng(77)
    rows, ids, Ts, Ps = [], [], [], []
    def add(z, y, T, P):
        rows.append(np.asarray(z, dtype=np.float64)); ids.append(int(y)); Ts.append(T); Ps.append(P)
    z = rng.normal(0, 2, V); z[:20000] = -np.inf
    add(z, 30000, 1.0, 0.9)                                  # no finite anchor among the first vectors
    z = rng.normal(0, 1, V); z[40000:41000] = 40.0 + rng.normal(0, 1, 1000)
    add(z, 40500, 1.0, 0.9)                                  # 1,000 logits ~40 nats above the anchor
    z = rng.normal(0, 1, V); z[50000] = 120.0
    add(z, 50000, 1.0, 0.9)                                  # one spike: nucleus = {spike}
    z = rng.normal(0, 1, V); z[60000] = 42.0
    add(z, 123, 4.0, 0.95)                                   # spike 10 nats above the bulk at T = 4
    add(rng.normal(0, 0.01, V), 5, 1.2, 0.93)                # near-flat: wide window
    add(rng.normal(0, 1.5, V) + 3000.0, 77, 1.0, 0.9)        # |A0| / T near 3,000: exact pass, coarse bf
    add(rng.normal(0, 1.5, V) + 30000.0, 78, 1.0, 0.9)       # |A0| / T beyond the binning guard: three passes
    logits, ids, T, P = _run(np.stack(rows), ids, Ts, Ps, dtype)
    print(f"case topp histogram edges {dtype}", flush=True)
    compare_features(gpu_features(logits, ids, T, P), oracle_features(logits, ids, T, P))


def test_topp_workload_scaled():
    """The top-p row model (V = 262,144 float32, T ~ U[0.3,1.2], P ~ U[0.8,0.95]) on a few requests."""
    w = wl.scaled(wl.WORKLOADS["topp_128x256_v262144_f32"], n_req=4, len_hi=6, len_lo=6)
    b = wl.make_batch(w, device="cpu")
    logits, ids, T, P = to_dev(b.logits, b.sampled_ids, b.temperature, b.top_p)
    print(f"case topp workload rows={b.n_rows}", flush=True)
    g = gpu_features(logits, ids, T, P)
    o = oracle_features(logits, ids, T, P)
    compare_features(g, o)
    assert (o["flags"] & pr.FLAG_OUTSIDE_NUCLEUS == 0).all()  # the sampler stays inside the nucleus


def test_topp_bf16_large_vocabulary():
    """The top-p row model on bf16 rows of the MLLM vocabulary (V = 151,936):
    the bf16 instantiation of the two-read method on realistic rows, every
    row against the oracle."""
    w = wl.scaled(wl.WORKLOADS["topp_128x256_v262144_f32"], n_req=6, len_hi=8, V=151936, dtype="bf16")
    b = wl.make_batch(w, device="cpu")
    logits, ids, T, P = to_dev(b.logits, b.sampled_ids, b.temperature, b.top_p)
    assert logits.dtype == torch.bfloat16
    print(f"case topp bf16 V=151936 rows={b.n_rows}", flush=True)
    compare_features(gpu_features(logits, ids, T, P), oracle_features(logits, ids, T, P))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_topp_flat_rows(dtype):
    """Flat and near-flat rows (sigma / T from 0.02 to 2, P from 0.5 to 0.99):
    the rows whose window many buckets reach, which take the float32 pass
    with its certified bound (and the float64 pass where the bound does not
    decide), against the oracle's exact cutoff."""
    V = 131072
    rng = np.random.default_rng(2024)
    n = 32
    sig = np.geomspace(0.02, 2.0, n)
    T = rng.uniform(0.5, 1.5, n)
    z = rng.normal(0, 1, (n, V)) * (sig * T)[:, None] + rng.uniform(-5, 5, (n, 1))
    P = rng.uniform(0.5, 0.99, n)
    ids = rng.integers(0, V, n)
    logits, ids, T, P = _run(z, ids, T, P, dtype)
    print(f"case topp flat rows V={V} {dtype}", flush=True)
    compare_features(gpu_features(logits, ids, T, P), oracle_features(logits, ids, T, P))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_topp_large_windows(dtype):
    """Windows of 513 to 4,096 logits, cut through their sub-buckets: a
    plateau of distinct values, a tie group of 1,500 at the crossing (its
    sub-bucket alone holds more than 512 logits and takes the workgroup
    sort), a window spanning fewer than 256 float steps (one value per
    sub-bucket), and one crossing zero (keys of both signs)."""
    V = 65536
    rng = np.random.default_rng(4096)
    rows, ids, Ps = [], [], []
    def add(z, P):
        pos = np.flatnonzero(z > -10)
        rows.append(z); ids.append(int(pos[len(pos) // 2])); Ps.append(P)
    for n, P in ((600, 0.6), (1500, 0.7), (3000, 0.8), (4000, 0.9)):
        z = np.full(V, -20.0)
        z[rng.choice(V, n, replace=False)] = rng.uniform(0.0, 1e-3, n)
        add(z, P)                                           # plateau of n distinct values
    z = np.full(V, -20.0)
    pos = rng.choice(V, 3000, replace=False)
    z[pos[:1500]] = 0.5
    z[pos[1500:]] = rng.uniform(0.49, 0.51, 1500)
    add(z, 0.5)                                             # 1,500 ties at the crossing
    z = np.full(V, -20.0)
    k = np.repeat(np.arange(200), 10)
    z[rng.choice(V, k.size, replace=False)] = 1.0 + k * 2.0 ** -23
    add(z, 0.6)                                             # 200 values one float step apart, 10 of each
    z = np.full(V, -20.0)
    z[rng.choice(V, 2500, replace=False)] = rng.uniform(-1e-3, 1e-3, 2500)
    add(z, 0.8)                                             # window across zero
    n = len(rows)
    logits, ids, T, P = _run(np.stack(rows), ids, np.ones(n), Ps, dtype)
    print(f"case topp large windows {dtype}", flush=True)
    g = gpu_features(logits, ids, T, P)
    compare_features(g, oracle_features(logits, ids, T, P))
    g2 = gpu_features(logits, ids, T, P)
    for key in g:
        assert np.array_equal(g[key].view(np.uint32), g2[key].view(np.uint32)), key


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_topp_window_size_boundaries(dtype):
    """Windows at the limits of the one-wave cut's sizes (64, 128, 256, 512
    logits per wave, the sub-bucket cut above): a plateau of n values within
    one bin, the rest 20 nats below, the crossing inside the plateau."""
    V = 65536
    rng = np.random.default_rng(640)
    rows, ids, Ps = [], [], []
    for n in (1, 2, 63, 64, 65, 127, 128, 129, 255, 256, 257, 511, 512, 513):
        z = np.full(V, -20.0)
        pos = rng.choice(V, n, replace=False)
        z[pos] = rng.uniform(0.0, 1e-4, n)
        rows.append(z); ids.append(int(pos[0])); Ps.append(0.5)
    n_rows = len(rows)
    logits, ids, T, P = _run(np.stack(rows), ids, np.ones(n_rows), Ps, dtype)
    print(f"case topp window size boundaries {dtype}", flush=True)
    compare_features(gpu_features(logits, ids, T, P), oracle_features(logits, ids, T, P))


def test_topp_large_vocabulary():
    """A vocabulary of 2^20 + 3 (four times the largest workload's): random,
    flat and peaked rows against the oracle's exact cutoff."""
    V = (1 << 20) + 3
    rng = np.random.default_rng(20)
    rows = [rng.normal(0, 2, V), rng.normal(0, 0.01, V), rng.normal(0, 1, V)]
    rows[2][12345] = 40.0
    ids = [int(rng.integers(0, V)), 7, 12345]
    logits, ids, T, P = _run(np.stack(rows), ids, [0.8, 1.2, 1.0], [0.9, 0.93, 0.5])
    print("case topp V = 2^20 + 3", flush=True)
    compare_features(gpu_features(logits, ids, T, P), oracle_features(logits, ids, T, P))


def test_hardware_exp2_bound():
    """The float32 pass of the top-p kernel certifies its masses with a bound
    of 1e-7 on the relative error of the hardware exp2 (the constant
    kExp2RelErr) for arguments in [-100, 100] (its frame keeps t there):
    checked here over every float in [-126, 127]."""
    out = torch.zeros(2, dtype=torch.int64, device="cuda")
    st = wl.tools().prt_exp2_max_rel_err(-126.0, 127.0, out.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    w = out.cpu().numpy()
    err = float(w[:1].view(np.float64)[0])
    x = float(np.array([w[1]], dtype=np.int64).astype(np.uint32).view(np.float32)[0])
    print(f"case exp2 bound: largest relative error {err:.4e} (at x = {x:.9g})", flush=True)
    assert 0.0 < err <= 1.0e-7
    # a sub-range reports a largest error inside it, no larger than the whole range's
    out.zero_()
    assert wl.tools().prt_exp2_max_rel_err(-1.0, 1.0, out.data_ptr(), torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    w = out.cpu().numpy()
    e1 = float(w[:1].view(np.float64)[0])
    x1 = float(np.array([w[1]], dtype=np.int64).astype(np.uint32).view(np.float32)[0])
    assert -1.0 <= x1 <= 1.0 and 0.0 < e1 <= err
