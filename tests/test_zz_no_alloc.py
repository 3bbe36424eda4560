"""pr_token_features_noalloc (no workspace, static per-GPU scratch) gives
what pr_token_features gives, call after call on the same scratch."""

import ctypes as C

import numpy as np
import pytest
import torch

import paper_2608_28726_amd as pr
from paper_2608_28726_amd import _abi
from paper_2608_28726_amd import workloads as wl
from tests.gpu_common import require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _noalloc(logits, ids, T, P=None):
    """The entry point called through the C ABI directly."""
    n, V = logits.shape
    out = pr._alloc_features(n, logits.device)
    st = _abi.lib().pr_token_features_noalloc(
        C.c_void_p(logits.data_ptr()), _abi.PR_BF16 if logits.dtype == torch.bfloat16 else _abi.PR_F32, n, V,
        logits.stride(0), C.c_void_p(ids.data_ptr()), C.c_void_p(T.data_ptr()),
        None if P is None else C.c_void_p(P.data_ptr()), C.byref(pr._features_struct(out)),
        C.c_void_p(torch.cuda.current_stream().cuda_stream))
    _abi.check("pr_token_features_noalloc", st)
    return out


def _same(a, b, what):
    torch.cuda.synchronize()
    for k in a:
        x, y = a[k].cpu(), b[k].cpu()
        if x.dtype == torch.float32:
            x, y = x.view(torch.int32), y.view(torch.int32)
        assert torch.equal(x, y), f"{what}: {k} differs"


def _batch(n, V, dtype, seed):
    w = wl.scaled(wl.WORKLOADS["ragged_64req_v151936_bf16"], n_req=1, len_hi=n, len_lo=n, V=V, dtype=dtype,
                  seed=seed)
    b = wl.make_batch(w, device="cuda")
    return b.logits, b.sampled_ids, b.temperature


@pytest.mark.parametrize("shapes", [[(100, 151936, "bf16"), (3, 151936, "bf16")],
                                    [(100, 32000, "f32"), (1, 32000, "f32")]])
def test_noalloc_matches_workspace_entry_point(shapes):
    """Two calls in a row on the same scratch, the second smaller, each
    bit-identical to pr_token_features with a caller workspace."""
    for k, (n, V, dtype) in enumerate(shapes):
        logits, ids, T = _batch(n, V, dtype, 4242 + k)
        assert pr.token_features_workspace(logits) > 0  # the scratch is used at this shape
        print(f"case noalloc n={n} V={V} {dtype}", flush=True)
        _same(_noalloc(logits, ids, T), pr.token_features(logits, ids, T), f"call {k + 1} ({n} rows)")


def test_noalloc_without_scratch_and_with_top_p():
    """Shapes that need no scratch (many rows; top-p) go through unchanged."""
    logits, ids, T = _batch(300, 4096, "f32", 77)
    _same(_noalloc(logits, ids, T), pr.token_features(logits, ids, T), "300 rows")
    P = torch.full((300,), 0.9, dtype=torch.float32, device="cuda")
    _same(_noalloc(logits, ids, T, P), pr.token_features(logits, ids, T, P), "top-p")
    out = pr.token_features_noalloc(logits[:5], ids[:5], T[:5])
    _same(out, pr.token_features(logits[:5], ids[:5], T[:5]), "binding")
    assert np.isfinite(out["lse"].cpu().numpy()).all()
