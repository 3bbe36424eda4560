"""fp64 oracle: the paper's own verifier input sequence.

TEST INFRASTRUCTURE ONLY -- see the package docstring. Shares no code with
the HIP library.

Source: Pro-Router, Sec. 3.1, Eq. 3 and the sentences after it. Each
generated token t of a request contributes the tuple
x_t = (l_t, m_t, h_t, rho_t): the log-probability of the emitted token, the
largest probability, the negated top-K entropy h_t = -H_t with
H_t = -sum over the K most probable tokens of p_t(v) log p_t(v) (K = 20), and
the position fraction rho_t = t / T. Stacked over the request's T tokens they
form the verifier's input X (T rows, 4 columns).

Readings where the paper is silent:

R14  p_t is the decoding distribution after temperature and top-p, the same
     distribution that l_t and m_t are taken on (see features.py, R3 and R4).
     The top-K terms use those probabilities as they are: the K tokens' mass
     is not renormalised to one, as the formula is printed. Where the K-th
     and (K+1)-th largest probabilities tie, every choice gives the same sum.
     Tokens of probability 0 (masked, or outside the nucleus) add nothing, so
     with fewer than K such tokens the sum covers all of them.
R15  t counts a request's generated tokens from 1 and T is their number, so
     rho runs 1/T, 2/T, .., 1. Row r of request i (rows offsets[i] ..
     offsets[i+1]-1) has t = r - offsets[i] + 1.
R16  A row flagged non-finite or with a bad temperature or top-p has NaN in
     l, m and h; rho does not depend on the logits and is always set. A row
     with a bad sampled id has l = NaN and valid m and h.
"""

from __future__ import annotations

import math

import numpy as np

from .features import FLAG_BAD_TP, FLAG_NONFINITE, decode_logits, token_features

PAPER_TOP_K = 20  # Sec. 3.1: K = 20


def topk_entropy(raw_row, dtype: str, T: float, P: float | None = None, K: int = PAPER_TOP_K) -> float:
    """H^{top-K} of one logit row in nats (Sec. 3.1; readings R14, R16).

    The K most probable tokens are the first K of the token order (larger
    logit first), cut to the nucleus when top-p is on. Their probabilities
    p = e_v / S_N come from e_v = exp(u_v - u_argmax) and the nucleus total
    S_N, and log p = (u_v - u_argmax) - log S_N.
    """
    if K < 1:
        raise ValueError("K must be at least 1")
    f = token_features(raw_row, dtype, 0, T, P)
    if f["flags"] & (FLAG_NONFINITE | FLAG_BAD_TP):
        return math.nan
    z = decode_logits(raw_row, dtype)
    V = z.shape[0]
    T = float(np.float32(T))
    idx = np.arange(V)
    order = np.lexsort((idx, -z))
    a = int(order[0])
    u = z / T
    with np.errstate(invalid="ignore", over="ignore"):
        e = np.exp(u - u[a])
    e[np.isneginf(z)] = 0.0
    k = f["cutoff"]
    S_N = math.fsum(e[order[:k]])
    top = order[: min(K, k)]
    live = top[e[top] > 0.0]
    p = e[live] / S_N
    logp = (u[live] - u[a]) - math.log(S_N)
    return float(-math.fsum(p * logp))


def topk_entropy_batch(raw, dtype: str, temps, top_ps=None, K: int = PAPER_TOP_K, rows=None) -> np.ndarray:
    """:func:`topk_entropy` over the rows of ``raw[n_rows, V]`` (float64 array)."""
    raw = np.asarray(raw)
    rows = np.arange(raw.shape[0]) if rows is None else np.asarray(rows)
    return np.array([topk_entropy(raw[r], dtype, float(temps[r]),
                                  None if top_ps is None else float(top_ps[r]), K) for r in rows],
                    dtype=np.float64)


def position_fraction(offsets) -> np.ndarray:
    """rho of every row of a ragged batch (reading R15), float64 [n_rows]."""
    offsets = np.asarray(offsets, dtype=np.int64)
    rho = np.empty(int(offsets[-1] - offsets[0]), dtype=np.float64)
    base = int(offsets[0])
    for i in range(offsets.shape[0] - 1):
        lo, hi = int(offsets[i]), int(offsets[i + 1])
        n = hi - lo
        for t in range(1, n + 1):
            rho[lo - base + t - 1] = t / n
    return rho


def feature_sequence(feats: dict, topk_H, offsets) -> np.ndarray:
    """The stacked inputs X of a ragged batch, float64 [n_rows][4]: columns
    (l, m, h, rho) = (logprob, maxprob, -H^{top-K}, t / T) (Sec. 3.1, Eq. 3)."""
    X = np.empty((len(topk_H), 4), dtype=np.float64)
    X[:, 0] = np.asarray(feats["logprob"], dtype=np.float64)
    X[:, 1] = np.asarray(feats["maxprob"], dtype=np.float64)
    X[:, 2] = -np.asarray(topk_H, dtype=np.float64)
    X[:, 3] = position_fraction(offsets)
    return X
