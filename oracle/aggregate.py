"""fp64 oracle: per-request aggregation, summary score and ship rule.

TEST INFRASTRUCTURE ONLY -- see the package docstring. Shares no code with
the HIP library.

Source: Pro-Router, Sec. 3.1. The per-token features of a request's T
generated tokens stack into a sequence X (Sec. 3.1, after Eq. 3); a summary
of that sequence gives one shipping confidence p, and the request ships iff
p >= tau (Sec. 3.1, the paragraph defining the gain, Eq. 1). The ablation
(Sec. 4.2, Table "ablation", row "quantile summary + MLP") shows that a
quantile summary of the sequence is a working verifier input.

Readings where the paper is silent:

R8   The summarised features are the confidence-oriented tuple
     A = (logprob, maxprob, -entropy, margin): the paper negates the entropy
     (h_t = -H_t, Eq. 3) so that larger means more confident, and the
     remaining three already rise with confidence. Each is summarised by its
     count n, mean, minimum and nearest-rank q-quantile: the j-th smallest
     value with j = max(1, ceil(q * n)), the product q * n rounded once in
     float64 (q itself is a float64 parameter, 0.1 by default).
R9   An empty request (n = 0) has NaN summaries; a NaN value anywhere in a
     feature's segment makes that feature's three summaries NaN.
R10  Score s = g(b + sum over nonzero weights w_{f,stat} * A_{f,stat}) with
     g the identity or the logistic sigmoid. Terms with a zero weight are
     skipped (so a -inf summary that is not used cannot poison the score).
     Default: w selects mean(maxprob) only, b = 0, g = identity -- the mean
     of the paper's m_t feature. The paper's own head is a trained
     transformer whose weights are not published: this head is parity
     unpinned against the paper.
R11  Ship iff s >= tau; a NaN score escalates (does not ship).
"""

from __future__ import annotations

import math

import numpy as np

AGG_FEATURES = ("logprob", "maxprob", "neg_entropy", "margin")  # R8, in this order
AGG_STATS = ("mean", "min", "quant")


def _confidence_columns(feats: dict) -> list:
    """The four columns of A (R8) as float64 arrays."""
    return [
        np.asarray(feats["logprob"], dtype=np.float64),
        np.asarray(feats["maxprob"], dtype=np.float64),
        -np.asarray(feats["entropy"], dtype=np.float64),
        np.asarray(feats["margin"], dtype=np.float64),
    ]


def _mean(x: np.ndarray) -> float:
    """Arithmetic mean with the IEEE meaning of infinities."""
    has_pos, has_neg = bool(np.isposinf(x).any()), bool(np.isneginf(x).any())
    if has_pos and has_neg:
        return math.nan
    if has_pos:
        return math.inf
    if has_neg:
        return -math.inf
    return math.fsum(x) / x.shape[0]


def _nearest_rank(x: np.ndarray, q: float) -> float:
    """The j-th smallest element, j = max(1, ceil(q * n)) (R8)."""
    n = x.shape[0]
    j = max(1, math.ceil(float(q) * n))
    j = min(j, n)
    return float(np.sort(x)[j - 1])


def request_aggregate(feats: dict, offsets, q: float = 0.1) -> dict:
    """Per-request summaries (R8, R9).

    ``feats`` holds per-row arrays ``logprob, maxprob, entropy, margin``;
    request i owns rows ``offsets[i] .. offsets[i+1]-1``. Returns ``count``
    (int64[n_req]) and ``mean, min, quant`` (float64[n_req, 4], columns in
    the order of ``AGG_FEATURES``).
    """
    offsets = np.asarray(offsets, dtype=np.int64)
    n_req = offsets.shape[0] - 1
    cols = _confidence_columns(feats)
    count = np.zeros(n_req, dtype=np.int64)
    out = {stat: np.full((n_req, 4), math.nan) for stat in AGG_STATS}
    for i in range(n_req):
        lo, hi = int(offsets[i]), int(offsets[i + 1])
        count[i] = hi - lo
        if hi <= lo:
            continue
        for f, col in enumerate(cols):
            seg = col[lo:hi]
            if np.isnan(seg).any():
                continue
            out["mean"][i, f] = _mean(seg)
            out["min"][i, f] = float(seg.min())
            out["quant"][i, f] = _nearest_rank(seg, q)
    out["count"] = count
    return out


def default_weights() -> np.ndarray:
    """R10 default head: 1.0 on mean(maxprob), zero elsewhere. Shape [3, 4]
    (stat-major: rows mean, min, quant; columns as ``AGG_FEATURES``)."""
    w = np.zeros((3, 4))
    w[0, 1] = 1.0
    return w


def score_from_aggregates(agg: dict, weights=None, bias: float = 0.0, link: str = "identity") -> np.ndarray:
    """Score per request (R10). ``weights`` is [3, 4] stat-major."""
    w = default_weights() if weights is None else np.asarray(weights, dtype=np.float64)
    n_req = agg["count"].shape[0]
    scores = np.empty(n_req)
    for i in range(n_req):
        if agg["count"][i] == 0:
            scores[i] = math.nan
            continue
        s = float(bias)
        for si, stat in enumerate(AGG_STATS):
            for f in range(4):
                if w[si, f] != 0.0:
                    s += w[si, f] * agg[stat][i, f]
        if link == "sigmoid":
            s = 1.0 / (1.0 + math.exp(-s)) if s >= 0 else math.exp(s) / (1.0 + math.exp(s))
        elif link != "identity":
            raise ValueError(f"unknown link {link!r}")
        scores[i] = s
    return scores


def route(scores, tau: float) -> np.ndarray:
    """Ship iff score >= tau; NaN escalates (Sec. 3.1; R11)."""
    s = np.asarray(scores, dtype=np.float64)
    with np.errstate(invalid="ignore"):
        return (s >= float(tau)).astype(np.uint8)
