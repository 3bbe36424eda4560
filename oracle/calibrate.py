"""fp64 oracle: threshold calibration and the bounded-memory streaming quantile.

TEST INFRASTRUCTURE ONLY -- see the package docstring. Shares no code with
the HIP library.

Threshold calibration. Source: Pro-Router, Sec. 3.1 (the ship rule p >= tau
with tau fixed in advance by calibration on a validation pool) and Sec. 4.1
(the coverage-based rule of selective prediction: a ship fraction q is fixed
and the threshold calibrated on a validation split).

Streaming quantile. Source: R. Jain and I. Chlamtac, "The P-square algorithm
for dynamic calculation of quantiles and histograms without storing
observations", CACM 28(10), 1985: five markers whose heights track the
minimum, the p/2-, p-, (1+p)/2-quantiles and the maximum; each observation
moves the marker positions and a piecewise-parabolic formula adjusts the
heights. It serves the streaming state when no per-token history is kept.

Readings:

R21  tau is the k-th largest score of the pool with k = max(1, ceil(q * n))
     over the n scores that are not NaN (a NaN score always escalates, so it
     is not part of the pool), q * n rounded once in float64; at least a
     fraction q of the pool then ships (more when scores tie at tau). q = 0,
     or a pool with no score, gives tau = +inf: nothing ships.
R22  P-square, as published, with two readings: the desired marker positions
     after n >= 5 observations are taken in closed form,
     n'_i = 1 + (n - 1) * f_i with f = (0, p/2, p, (1+p)/2, 1), instead of
     accumulated increments (the same values without accumulated rounding);
     and with at most 5 observations (the markers are then the sorted
     observations themselves) the estimate is their exact nearest-rank
     p-quantile, as for the exact summary (R8), not the middle marker. A
     NaN observation is not fed to the markers (the feature's summaries are
     NaN anyway, R9). Nor is an infinite one (a margin of +inf from a row
     with one finite logit, a log-prob of -inf): the interpolation is not
     defined on infinite heights (inf - inf), so the estimate becomes NaN
     for the rest of the request and a score that uses it escalates; the
     mean and minimum still include the value.
"""

from __future__ import annotations

import math

import numpy as np


def calibrate_threshold(scores, ship_fraction: float):
    """(tau, n_ship) for a validation pool of scores (reading R21)."""
    s = np.asarray(scores, dtype=np.float64)
    s = s[~np.isnan(s)]
    q = float(ship_fraction)
    if not (0.0 <= q <= 1.0):
        raise ValueError("ship fraction must lie in [0, 1]")
    if q == 0.0 or s.shape[0] == 0:
        return math.inf, 0
    k = max(1, math.ceil(q * s.shape[0]))
    k = min(k, s.shape[0])
    tau = float(np.sort(s)[::-1][k - 1])
    return tau, int(np.count_nonzero(s >= tau))


class P2Quantile:
    """The P-square estimator of the p-quantile (reading R22)."""

    def __init__(self, p: float):
        self.p = float(p)
        self.f = (0.0, self.p / 2.0, self.p, (1.0 + self.p) / 2.0, 1.0)
        self.q = []          # marker heights (the first observations until there are 5)
        self.n = [1, 2, 3, 4, 5]  # marker positions (1-based)
        self.count = 0
        self.poisoned = False  # an infinite observation was seen

    def add(self, x: float) -> None:
        x = float(x)
        if math.isnan(x):
            return
        if math.isinf(x):
            self.poisoned = True
            return
        if self.poisoned:
            return
        self.count += 1
        if self.count <= 5:
            self.q.append(x)
            if self.count == 5:
                self.q.sort()
            return
        q, n = self.q, self.n
        # the cell k with q[k] <= x < q[k+1]; the extreme markers follow the
        # extremes (the maximum is replaced only by a larger value)
        if x < q[0]:
            q[0] = x
            k = 0
        elif x >= q[4]:
            if x > q[4]:
                q[4] = x
            k = 3
        else:
            k = 0
            while not (q[k] <= x < q[k + 1]):
                k += 1
        for i in range(k + 1, 5):
            n[i] += 1
        N = self.count
        for i in (1, 2, 3):
            desired = 1.0 + (N - 1) * self.f[i]
            d = desired - n[i]
            if (d >= 1.0 and n[i + 1] - n[i] > 1) or (d <= -1.0 and n[i - 1] - n[i] < -1):
                s = 1 if d > 0 else -1
                # piecewise-parabolic prediction of the height at n_i + s
                qp = q[i] + s / (n[i + 1] - n[i - 1]) * (
                    (n[i] - n[i - 1] + s) * (q[i + 1] - q[i]) / (n[i + 1] - n[i])
                    + (n[i + 1] - n[i] - s) * (q[i] - q[i - 1]) / (n[i] - n[i - 1]))
                if not (q[i - 1] < qp < q[i + 1]):
                    # linear prediction towards the neighbour in direction s
                    qp = q[i] + s * (q[i + s] - q[i]) / (n[i + s] - n[i])
                q[i] = qp
                n[i] += s

    def estimate(self) -> float:
        if self.count == 0 or self.poisoned:
            return math.nan
        if self.count <= 5:
            v = sorted(self.q)
            j = max(1, math.ceil(self.p * len(v)))
            return v[j - 1]
        return self.q[2]


def p2_quantile(values, p: float) -> float:
    """P-square estimate of the p-quantile of a sequence (NaN: none fed)."""
    est = P2Quantile(p)
    for v in values:
        est.add(v)
    return est.estimate()
