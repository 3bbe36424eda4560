"""fp64 oracle: per-token confidence features of one vocabulary logit row.

TEST INFRASTRUCTURE ONLY -- see the package docstring. Shares no code with
the HIP library.

Source: Pro-Router, Sec. 3.1. Each decoding step t emits a distribution
p_t over the vocabulary; the verifier reads the log-probability of the
emitted token (l_t = log p_t(y_t)), the maximum probability
(m_t = max_v p_t(v)) and a Shannon entropy of that distribution
(Sec. 3.1, Eq. 3 and the sentence defining H_t). The hot path extends this
to the feature set max logit, logsumexp, softmax entropy, sampled-token
log-probability, top-1/top-2 margin and sampled-token rank, all taken after
temperature and optional top-p (nucleus) truncation.

Readings where the paper is silent:

R1  Logits arrive as IEEE float32 or bfloat16 bit patterns; they are decoded
    exactly to float64. NaN or +inf anywhere, or a row that is all -inf, is
    a non-finite row. -inf alone is a masked token with probability 0.
R2  Token order: v precedes w iff z_v > z_w, or z_v == z_w and v < w, on the
    raw (pre-temperature) values; -0 == +0. argmax is the first token of this
    order, rank(y) is the 1-based position of y in it.
R3  Temperature divides the logits: u = z / T. T must be finite and at least
    2**-100, and |z_argmax| / T must not exceed 2**100; otherwise the row is
    flagged (the bounds keep every scaled logit inside float32's range).
R4  Top-p keeps the shortest prefix of the order whose probability mass
    reaches P: k = min{ j : C_j >= P * S }, C_j the mass of the first j
    tokens, S the total. P >= 1 (or no P) keeps all V tokens; P <= 0 or NaN
    is flagged. Entropy, logsumexp, max probability and the log-probability
    are then taken on the renormalised nucleus; a sampled token outside the
    nucleus has log-probability -inf and is flagged.
R5  Entropy is in nats; 0 * log 0 counts as 0.
R6  margin = (z_argmax - z_second) / T in scaled-logit space over the full
    order (a tie gives 0; top-p does not change it).
R7  A row with a bad sampled id still gets every feature that does not depend
    on the id; log-probability is NaN and rank is -1. The bad-id flag is set
    whenever the id is out of range, also on rows flagged for other reasons.
"""

from __future__ import annotations

import math

import numpy as np

# Row flags. The numeric values are part of the library's interface, so the
# HIP side defines the same bits in its own header.
FLAG_NONFINITE = 1  # NaN or +inf logit, or every logit is -inf      (R1)
FLAG_BAD_ID = 2  # sampled id outside [0, V)                          (R7)
FLAG_BAD_TP = 4  # bad temperature or top-p                           (R3, R4)
FLAG_OUTSIDE_NUCLEUS = 8  # sampled token not inside the top-p nucleus (R4)

_TEMP_RANGE = 2.0 ** 100  # R3: |z_argmax| / T may not exceed this
_MIN_TEMPERATURE = 2.0 ** -100  # R3: smallest accepted temperature

FLOAT_FEATURES = ("max_logit", "lse", "entropy", "logprob", "maxprob", "margin")
INT_FEATURES = ("rank", "argmax", "cutoff")


def decode_logits(raw: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of stored logits (R1).

    ``dtype`` is "f32" (``raw`` holds float32 values) or "bf16" (``raw`` holds
    the uint16 bit patterns; a bfloat16 is the upper half of a float32).
    """
    if dtype == "f32":
        return np.asarray(raw, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        bits = np.asarray(raw, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def _nan_result(V: int, flags: int) -> dict:
    out = {name: math.nan for name in FLOAT_FEATURES}
    out.update({name: -1 for name in INT_FEATURES})
    out["flags"] = flags
    out["ambiguous"] = False
    return out


def token_features(raw_row, dtype: str, y: int, T: float, P: float | None = None) -> dict:
    """Features of one logit row (Sec. 3.1, Eq. 3; readings R1-R7).

    Arguments: ``raw_row`` the stored row (see :func:`decode_logits`), ``y``
    the sampled token id, ``T`` the temperature (a float32 value), ``P`` the
    top-p mass (a float32 value) or None.

    Returns a dict with the float features ``max_logit, lse, entropy,
    logprob, maxprob, margin``, the integers ``rank, argmax, cutoff``, the
    row ``flags`` and ``ambiguous`` (True when the top-p boundary mass lies
    within 1e-12 * S of P * S, so that k is not decided by float64 sums).
    """
    z = decode_logits(raw_row, dtype)
    V = z.shape[0]
    if V < 2:
        raise ValueError("a vocabulary row needs at least two tokens")
    T = float(np.float32(T))
    P = None if P is None else float(np.float32(P))

    bad_id = not (0 <= y < V)
    flags = FLAG_BAD_ID if bad_id else 0  # R7: a bad id is reported in every case
    if np.isnan(z).any() or np.isposinf(z).any() or np.isneginf(z).all():
        flags |= FLAG_NONFINITE
    if not (math.isfinite(T) and T >= _MIN_TEMPERATURE):
        flags |= FLAG_BAD_TP
    if P is not None and (math.isnan(P) or P <= 0.0):
        flags |= FLAG_BAD_TP
    if flags & (FLAG_NONFINITE | FLAG_BAD_TP):
        return _nan_result(V, flags)

    # R2: the order. argmax is the lowest index holding the largest value.
    idx = np.arange(V)
    z_max = z.max()
    a = int(np.flatnonzero(z == z_max)[0])
    if abs(z[a]) > T * _TEMP_RANGE:  # exact: scaling by 2**100 does not round
        return _nan_result(V, flags | FLAG_BAD_TP)
    z_second = np.delete(z, a).max()

    if bad_id:
        rank = -1
    else:
        rank = 1 + int(np.count_nonzero(z > z[y])) + int(np.count_nonzero((z == z[y]) & (idx < y)))

    # R3: temperature, then e_v = exp(u_v - u_a), the unnormalised
    # probabilities relative to the most likely token (e_a = 1).
    u = z / T
    with np.errstate(invalid="ignore", over="ignore"):
        e = np.exp(u - u[a])
    e[np.isneginf(z)] = 0.0
    S = math.fsum(e)

    # R4: top-p nucleus.
    ambiguous = False
    if P is None or P >= 1.0:
        k = V
        nucleus = idx
    else:
        order = np.lexsort((idx, -z))  # the order of R2
        target = P * S
        C = np.cumsum(e[order])
        k = int(np.searchsorted(C, target, side="left")) + 1
        k = min(max(k, 1), V)
        # Re-decide the boundary with correctly rounded prefix sums.
        while k > 1 and math.fsum(e[order[: k - 1]]) >= target:
            k -= 1
        while k < V and math.fsum(e[order[:k]]) < target:
            k += 1
        C_k = math.fsum(e[order[:k]])
        C_km1 = math.fsum(e[order[: k - 1]])
        slack = min(C_k - target, target - C_km1) / S
        ambiguous = bool(slack < 1e-12)
        nucleus = order[:k]

    e_N = e[nucleus]
    S_N = math.fsum(e_N)
    # R5: 0 * log 0 = 0 -- masked tokens (e == 0) contribute nothing.
    live = e_N > 0.0
    d_N = u[nucleus][live] - u[a]
    ent_sum = math.fsum(e_N[live] * d_N)

    lse = u[a] + math.log(S_N)
    entropy = math.log(S_N) - ent_sum / S_N
    maxprob = 1.0 / S_N
    margin = (z[a] - z_second) / T
    if bad_id:
        logprob = math.nan
    elif rank <= k:
        # log p(y) = u_y - lse: finite even where p(y) underflows float64;
        # -inf only for a masked logit (u_y = -inf).
        logprob = u[y] - lse
    else:
        logprob = -math.inf
        flags |= FLAG_OUTSIDE_NUCLEUS

    return {
        "max_logit": float(u[a]),
        "lse": float(lse),
        "entropy": float(entropy),
        "logprob": float(logprob),
        "maxprob": float(maxprob),
        "margin": float(margin),
        "rank": int(rank),
        "argmax": int(a),
        "cutoff": int(k),
        "flags": int(flags),
        "ambiguous": ambiguous,
    }


def token_features_batch(raw, dtype: str, ids, temps, top_ps=None, rows=None) -> dict:
    """:func:`token_features` over the rows of ``raw[n_rows, V]``.

    ``rows`` optionally restricts the work to a subset of row indices (the
    outputs then follow that subset's order). Returns float64 arrays for the
    float features, int64 arrays for the integers and flags, and a bool array
    ``ambiguous``.
    """
    raw = np.asarray(raw)
    rows = np.arange(raw.shape[0]) if rows is None else np.asarray(rows)
    res = [
        token_features(raw[r], dtype, int(ids[r]), float(temps[r]),
                       None if top_ps is None else float(top_ps[r]))
        for r in rows
    ]
    out = {}
    for name in FLOAT_FEATURES:
        out[name] = np.array([d[name] for d in res], dtype=np.float64)
    for name in INT_FEATURES + ("flags",):
        out[name] = np.array([d[name] for d in res], dtype=np.int64)
    out["ambiguous"] = np.array([d["ambiguous"] for d in res], dtype=bool)
    return out
