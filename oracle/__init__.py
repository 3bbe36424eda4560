"""Plain fp64 CPU oracle for the token-aware verifier hot path.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import this
package: only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` use it. It shares no code with the HIP library.

The oracle writes out, in float64 and in the order the paper states them,
what the verifier computes (Pro-Router, Sec. 3.1, eq:features and the
ship rule p >= tau):

* :mod:`oracle.features` -- per-token confidence features of one
  vocabulary logit row after temperature and optional top-p.
* :mod:`oracle.aggregate` -- per-request aggregation of those features
  over a ragged batch, the summary score and the ship-or-escalate rule.
* :mod:`oracle.sequence` -- the paper's own verifier input: the top-K
  entropy (K = 20) and the stacked per-token tuples (l, m, h, rho).
* :mod:`oracle.head` -- the paper's verifier head over that input:
  projection with positional encoding, two post-norm encoder layers, mean
  pool and sigmoid (run with seeded synthetic weights).
* :mod:`oracle.sampling` -- the distribution the fused sample-and-verify
  path draws each token from.
* :mod:`oracle.calibrate` -- the threshold tau for a ship fraction on a
  validation pool, and the P-square streaming quantile (bounded memory).

Parity pinning: every function here is pinned by ``tests/test_oracle_pins.py``,
``tests/test_oracle_sequence.py``, ``tests/test_oracle_head.py``,
``tests/test_oracle_calibrate.py`` and ``tests/test_oracle_sampling.py`` against
closed forms, invariants, pure-Python brute force and (for the head) an
independent implementation of the same architecture, except the default
score head (a fixed linear summary chosen because the paper publishes no
trained head weights) and the transformer head's weights, which are *parity
unpinned* against the paper.
"""

from .features import (  # noqa: F401
    FLAG_BAD_ID,
    FLAG_BAD_TP,
    FLAG_NONFINITE,
    FLAG_OUTSIDE_NUCLEUS,
    decode_logits,
    token_features,
    token_features_batch,
)
from .aggregate import (  # noqa: F401
    AGG_FEATURES,
    request_aggregate,
    route,
    score_from_aggregates,
)
from .sequence import (  # noqa: F401
    PAPER_TOP_K,
    feature_sequence,
    position_fraction,
    topk_entropy,
    topk_entropy_batch,
)
from .head import HEAD_WEIGHTS, head_score, head_scores  # noqa: F401,E402
from .calibrate import P2Quantile, calibrate_threshold, p2_quantile  # noqa: F401,E402
from .sampling import token_probabilities  # noqa: F401,E402
