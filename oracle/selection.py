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


def select_topk_perturbed(scores, delta, k: int) -> np.ndarray:
    """Eq. topk with the paper's tie-break perturbation (Section 3.3): the
    tiny perturbation is added to each score before the selection.  The sums
    are taken in fp32 (one rounding, the arithmetic the scores live in) and
    then selected as in select_topk; ``delta`` is the seeded perturbation."""
    s = np.asarray(scores, dtype=np.float32) + np.asarray(delta, dtype=np.float32)
    return select_topk(s, k)


def select_topk_batched(scores, offsets, k, delta=None) -> np.ndarray:
    """B independent selections over the segments scores[offsets[b]:offsets[b+1]]
    with budgets k[b]; the local index lists concatenated in segment order."""
    out = []
    for b in range(len(k)):
        seg = np.asarray(scores)[offsets[b]:offsets[b + 1]]
        if delta is None:
            out.append(select_topk(seg, int(k[b])))
        else:
            out.append(select_topk_perturbed(seg, np.asarray(delta)[offsets[b]:offsets[b + 1]], int(k[b])))
    return np.concatenate(out).astype(np.int32) if out else np.zeros(0, np.int32)
