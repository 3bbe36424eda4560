"""fp64 oracle: the distribution the fused sample-and-verify path draws from.

TEST INFRASTRUCTURE ONLY -- see the package docstring. Shares no code with
the HIP library.

Source: Pro-Router, Sec. 3.1 (the per-token features are read off the
distribution the small model decodes from, softmax of the logits over the
temperature) and Sec. 4.1 (the verifier obtains these distributions as a
side product of decoding). The fused path draws the token y_t from that
distribution in the same pass that computes its features; the oracle gives
the probability of every token, against which the draws are tested, and
the features of a drawn row are those of :func:`oracle.token_features` for
the drawn id.

Reading:

R23  Token v is drawn with probability p_v = e_v / S, e_v = exp((z_v - M)/T),
     S = sum of e_v, over the decoded logits (R1, R3), without top-p.
     Masked tokens (-inf) have p = 0 and are never drawn. A row whose
     distribution is undefined (non-finite logits or a rejected temperature:
     the NONFINITE and BAD_TP rules of R1 and R3) draws no token (id -1).
     The drawn row's features are those of the drawn id, except its rank,
     which the fused pass does not count (it needs z_y before the pass).
"""

from __future__ import annotations

import math

import numpy as np

from .features import FLAG_BAD_TP, FLAG_NONFINITE, decode_logits, token_features


def token_probabilities(raw_row, dtype: str, T: float):
    """p_v of every token of one row (R23), float64; None when the row's
    distribution is undefined."""
    z = decode_logits(raw_row, dtype)
    y0 = int(np.argmax(np.where(np.isnan(z), -np.inf, z)))
    f = token_features(raw_row, dtype, y0, T)  # the row's flags and its maximum
    if f["flags"] & (FLAG_NONFINITE | FLAG_BAD_TP):
        return None
    T = float(np.float32(T))
    u = z / T
    with np.errstate(invalid="ignore", over="ignore"):
        e = np.exp(u - u.max())
    e[np.isneginf(z)] = 0.0
    return e / math.fsum(e)
