"""Top-K token selection (paper Section 3.3.3, Eq. topk).

Test infrastructure: used only by tests, the smoke check and the CPU baseline.
"""
from __future__ import annotations

import numpy as np


def select_topk(scores, k: int) -> np.ndarray:
    """Indices of the k largest fp32 scores, returned in ascending index order.

    Eq. topk selects the K highest-scoring tokens.  The paper breaks ties with
    a tiny random perturbation; the deterministic reading used here orders by
    (score descending, index ascending), so among equal scores the lowest
    index wins.  -0.0 and +0.0 are equal; NaN ranks below every number.
    """
    s = np.asarray(scores, dtype=np.float32).astype(np.float64)
    n = s.shape[0]
    if not 0 <= k <= n:
        raise ValueError("k out of range")
    nan = np.isnan(s)
    key = np.where(nan, 0.0, -s) + 0.0          # +0.0 folds -0.0 into +0.0
    idx = np.arange(n)
    order = np.lexsort((idx, key, nan))         # last key is the primary one
    return np.sort(order[:k]).astype(np.int32)
