"""Edge-side local resampling of the paper's protocol (Algorithm 1, RESAMPLE(P_hat, Q)).

The cloud step in scalar-q mode (``acespec_verify_tree_scalar_q``) returns, per session,
the number of accepted drafted tokens pi and a top-k sparse target distribution P_hat at
the position where the walk stopped; it does not sample (Section III-B: the cloud "skips
token resampling").  The edge holds its own full draft distribution Q at that position
and draws the corrected token locally:

* after a rejection, from the residual max(0, P_hat - Q) restricted to P_hat's k ids,
  renormalised (from P_hat itself if that residual has no mass);
* after full acceptance, from P_hat (the bonus token).

Draws use the inverse CDF in ascending token-id order with a caller-supplied uniform u in
(0, 1) (the first id whose running mass exceeds u times the total).  This runs on the
edge device's CPU by design, so it is plain numpy.  It is exact only when the k ids cover
the target's whole nucleus; ``residual_law`` exposes the distribution it samples so the
gap to the exact residual can be measured.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np


def residual_law(ids, probs, q, rejected: bool = True) -> Tuple[np.ndarray, np.ndarray]:
    """(ids ascending, normalised weights) of the distribution the edge samples from."""
    ids = np.asarray(ids, dtype=np.int64)
    probs = np.asarray(probs, dtype=np.float64)
    order = np.argsort(ids, kind="stable")
    ids, probs = ids[order], probs[order]
    w = probs
    if rejected:
        r = np.maximum(probs - np.asarray(q, dtype=np.float64)[ids], 0.0)
        if r.sum() > 0.0:
            w = r
    total = w.sum()
    return ids, (w / total if total > 0 else w)


def resample(ids, probs, q, u: float, rejected: bool = True) -> int:
    """The corrected token for one session (inverse CDF at u over residual_law)."""
    sid, w = residual_law(ids, probs, q, rejected)
    c = np.cumsum(w)
    j = int(np.searchsorted(c, u * c[-1], side="right"))
    j = min(j, len(sid) - 1)
    while w[j] == 0.0 and j + 1 < len(sid):   # never return a zero-mass id
        j += 1
    return int(sid[j])
