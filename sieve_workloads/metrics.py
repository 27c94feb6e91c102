"""Evaluation metrics over search outputs (host-side numpy; not part of the search)."""
from __future__ import annotations

import numpy as np


def pooled_recall(returned_ids, truth_ids) -> tuple[float, int, int]:
    """Pooled filtered top-k recall (Sec. 6.1).

    ``truth_ids`` holds, per query, the threshold-filtered exact top-k ids
    (-1 padded); ``returned_ids`` the ids a search returned (-1 padded).
    R_pool = sum_q |A(q) & G(q)| / sum_q |G(q)|; queries with an empty G(q)
    add nothing to either sum.  Returns (recall, hits, denominator); the
    recall is 1.0 when the denominator is 0.
    """
    returned_ids = np.asarray(returned_ids)
    truth_ids = np.asarray(truth_ids)
    num = den = 0
    for a, g in zip(returned_ids, truth_ids):
        gs = set(int(x) for x in g if x >= 0)
        if not gs:
            continue
        den += len(gs)
        num += len(gs & set(int(x) for x in a if x >= 0))
    return (num / den if den else 1.0), num, den
