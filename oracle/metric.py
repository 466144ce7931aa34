"""fp64 CPU oracle of the Top-k score (section 7.1.2, Eq. (12)): how close the
best measured latency among a cost model's k highest-ranked candidates comes
to the best latency of all candidates, weighted over the subgraphs.

TEST INFRASTRUCTURE ONLY, like the rest of this package: only the tests, the
smoke check and the benchmark's CPU-baseline leg may call it. It shares no
code with the HIP library.

Reading of Eq. (12):
  * a segment is the candidate set of one subgraph s of one model m (the
    pair (m, s)), given by offsets into flat arrays;
  * min_latency of a segment is its lowest measured latency;
  * candidates are ranked by the predicted score, highest first (a higher
    score predicts a faster program); equal scores keep index order and a
    NaN score ranks below every number (the same order as the top-K
    selection of the inference phase);
  * p_latency_i is the measured latency of the i-th ranked candidate, and
    the denominator takes the lowest of the first k (all of them when the
    segment has fewer than k);
  * weight is the subgraph's occurrence count in its model; empty segments
    add nothing to either sum.
Top-k = sum(weight * min_latency) / sum(weight * best of the top k).
"""
from __future__ import annotations

import numpy as np

from oracle import select as osel

f64 = np.float64


def top_k_score(scores, latency, seg_offsets, weight, k):
    """Eq. (12). Returns (score, numerator, denominator)."""
    lat = np.asarray(latency, dtype=f64)
    w = np.asarray(weight, dtype=f64)
    offs = np.asarray(seg_offsets, dtype=np.int64)
    top = osel.topk_segments(scores, offs, k)
    num = den = 0.0
    for g in range(len(offs) - 1):
        lo, hi = int(offs[g]), int(offs[g + 1])
        if hi <= lo:
            continue
        picked = top[g][top[g] >= 0]
        num += w[g] * np.min(lat[lo:hi])
        den += w[g] * np.min(lat[picked])
    return num / den, num, den
