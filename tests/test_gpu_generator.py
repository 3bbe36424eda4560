"""The device logit generator makes the same bits as its host twin, so the
expected values that the oracle computed from host-made rows apply to the
rows the GPU tests make on the device."""

import numpy as np
import pytest
import torch

from paper_2608_28726_amd import workloads as wl
from tests.gpu_common import require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _bits(t: torch.Tensor) -> np.ndarray:
    t = t.cpu()
    return t.view(torch.int16).numpy() if t.dtype == torch.bfloat16 else t.view(torch.int32).numpy()


@pytest.mark.parametrize("n,V,stride,dtype", [
    (64, 151936, 151936, "bf16"),   # about 9.7M elements: the tail cells are hit a few hundred times
    (16, 262144, 262144, "f32"),
    (5, 1001, 1003, "bf16"),        # odd vocabulary and stride: element-wise stores
    (3, 37, 40, "f32"),
    (2, 8, 8, "bf16"),
])
def test_device_rows_equal_host_rows(n, V, stride, dtype):
    rng = np.random.default_rng(n * 7919 + V)
    s = rng.uniform(0.5, 5.0, n).astype(np.float32)
    h = rng.uniform(0.0, 20.0, n).astype(np.float32)
    j = rng.integers(-1, V, n).astype(np.int64)  # -1: no spike
    seed = 0x1234_5678_9ABC_DEF0 + n
    print(f"case generator n={n} V={V} stride={stride} {dtype}", flush=True)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    base = torch.zeros((n, stride), dtype=tdt, device="cuda")
    dev = wl.fill_logits(base[:, :V], s, h, j, seed=seed, row0=11)
    host = wl.host_rows(seed, np.arange(11, 11 + n), V, dtype, s, h, j)
    got = _bits(dev)
    want = host.view(np.int16) if dtype == "bf16" else host.view(np.int32)
    diff = np.argwhere(got != want)
    assert diff.size == 0, f"{len(diff)} elements differ, first {diff[:4].tolist()}"
    assert (_bits(base[:, V:]) == 0).all()  # nothing written past the row
    assert (wl.row_checksums(dev) == wl.row_checksums(host)).all()


def test_device_rows_with_key_indices():
    """Streaming rows are keyed by (step, slot) indices, not by position."""
    w = wl.WORKLOADS["stream_256slots_v151936_bf16"]
    active = np.array([0, 3, 4, 200, 255])
    logits, _, _ = wl.stream_step_inputs(w, 17, active, device="cuda", ids=np.zeros(5, np.int32))
    idx, s, h, j = wl.stream_rows(w, 17, active)
    host = wl.host_rows(wl.stream_seed(w), idx, w.V, w.dtype, s, h, j)
    assert (_bits(logits) == host.view(np.int16)).all()
