"""Helpers for the GPU parity tests (imported only by tests marked gpu)."""

from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2608_28726_amd as pr
from paper_2608_28726_amd import workloads as wl
from tests.helpers import assert_floats, assert_ints, ensure_built

FLOATS = ("max_logit", "lse", "entropy", "logprob", "maxprob", "margin")


def require_gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ensure_built()


def dtype_name(logits: torch.Tensor) -> str:
    return "bf16" if logits.dtype == torch.bfloat16 else "f32"


def gpu_features(logits, ids, T, P=None) -> dict:
    f = pr.token_features(logits, ids, T, P)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in f.items()}


def oracle_features(logits, ids, T, P=None, rows=None) -> dict:
    raw = wl.to_host_raw(logits)
    return oracle.token_features_batch(raw, dtype_name(logits), ids.cpu().numpy(), T.cpu().numpy(),
                                       None if P is None else P.cpu().numpy(), rows)


def compare_features(g: dict, o: dict, rows=None, what=""):
    """Element-wise parity of one batch (rows: subset the oracle computed)."""
    if rows is not None:
        g = {k: v[np.asarray(rows)] for k, v in g.items()}
    amb = o["ambiguous"]
    for k in FLOATS:
        assert_floats(f"{what}{k}", g[k], o[k], mask=~amb if k in ("lse", "entropy", "logprob", "maxprob") else None)
    assert_ints(f"{what}rank", g["rank"], o["rank"])
    assert_ints(f"{what}argmax", g["argmax"], o["argmax"])
    assert_ints(f"{what}cutoff", g["cutoff"], o["cutoff"], mask=~amb)
    assert_ints(f"{what}flags", g["flags"].astype(np.int64) & 0xFFFFFFFF, o["flags"], mask=~amb)


def to_dev(*ts):
    return [t.cuda() if t is not None else None for t in ts]
