"""Shared test helpers: library loading and the parity comparison rule."""

from __future__ import annotations

import math
import os

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# Float features agree when |gpu - oracle| <= ATOL + RTOL * |oracle|; infinities
# must match exactly and NaN must meet NaN.
ATOL = 1e-5
RTOL = 1e-4
DECISION_BAND = 1e-5  # ship decisions may differ only when |score - tau| <= this


def ensure_built():
    """Builds the library if no build exists yet (the build is the product's own)."""
    from paper_2608_28726_amd import _abi
    if not os.path.exists(_abi.LIB_PATH):
        from paper_2608_28726_amd import build
        build.build()
    return _abi.lib()


def float_mismatch(gpu, ref, atol=ATOL, rtol=RTOL) -> np.ndarray:
    """Boolean mask of elements that break the tolerance rule."""
    g = np.asarray(gpu, dtype=np.float64)
    o = np.asarray(ref, dtype=np.float64)
    both_nan = np.isnan(g) & np.isnan(o)
    inf_o = np.isinf(o) | np.isinf(g)
    with np.errstate(invalid="ignore"):
        ok = np.abs(g - o) <= atol + rtol * np.abs(o)
    ok = np.where(inf_o, g == o, ok)
    return ~(ok | both_nan)


def tolerance_ratio(gpu, ref, mask=None, atol=ATOL, rtol=RTOL) -> float:
    """Largest |gpu - oracle| / (atol + rtol |oracle|) over the finite pairs
    (1.0 is the edge of the tolerance)."""
    g = np.asarray(gpu, dtype=np.float64)
    o = np.asarray(ref, dtype=np.float64)
    ok = np.isfinite(g) & np.isfinite(o)
    if mask is not None:
        ok &= mask
    if not ok.any():
        return 0.0
    return float(np.max(np.abs(g[ok] - o[ok]) / (atol + rtol * np.abs(o[ok]))))


def assert_floats(name, gpu, ref, mask=None, atol=ATOL, rtol=RTOL):
    bad = float_mismatch(gpu, ref, atol, rtol)
    if mask is not None:
        bad &= mask
    if bad.any():
        i = np.flatnonzero(bad)[:8]
        raise AssertionError(f"{name}: {bad.sum()} mismatches, e.g. rows {i.tolist()}: "
                             f"gpu {np.asarray(gpu)[i].tolist()} oracle {np.asarray(ref)[i].tolist()}")


def assert_ints(name, gpu, ref, mask=None):
    g = np.asarray(gpu, dtype=np.int64)
    o = np.asarray(ref, dtype=np.int64)
    bad = g != o
    if mask is not None:
        bad &= mask
    if bad.any():
        i = np.flatnonzero(bad)[:8]
        raise AssertionError(f"{name}: {bad.sum()} mismatches, e.g. rows {i.tolist()}: "
                             f"gpu {g[i].tolist()} oracle {o[i].tolist()}")


def decisions_agree(ship_gpu, scores_oracle, tau) -> np.ndarray:
    """Mask of requests whose decision matches or whose oracle score is in the band."""
    s = np.asarray(scores_oracle, dtype=np.float64)
    expect = np.where(np.isnan(s), 0, (s >= tau)).astype(np.uint8)
    with np.errstate(invalid="ignore"):
        band = np.abs(s - tau) <= DECISION_BAND
    return (np.asarray(ship_gpu) == expect) | band


def nan_close(a, b):
    a, b = float(a), float(b)
    return (math.isnan(a) and math.isnan(b)) or a == b
