"""fp64 CPU oracle of what consumes the cost model's scores: the top-K
selection of the inference phase (section 3: the cost model picks the best K
candidates of a tuning round to measure) and the RDU sampler's selection of
programs to label (section 4, Alg. 1 with Eq. (1)-(3)).

TEST INFRASTRUCTURE ONLY, like oracle.model: only the tests, the smoke check
and the benchmark's CPU-baseline leg may call it. It shares no code with the
HIP library and takes every input as an argument.

Top-K: per segment (the candidates of one task), the K highest scores,
highest first, equal scores in index order; a NaN score (an invalid program)
ranks below every number.

RDU selection, read from Alg. 1 (one step t; the cost model's update between
steps and the labelling itself are outside):
  * f = the cost model's predictions over the pool, min-max normalised to
    [0, 1] over the whole pool (the paper normalises them before Eq. (1); the
    same normalised values are used in Eq. (2)-(3) and as the weight of d_s);
  * budgets (Calc_Dist and the budget lines): budget[op] = B_t * n_op / N
    with n_op the pool's items of that operator type and N the pool size;
  * repeat until B_t programs are selected (or no candidate is left):
      for every unlabeled candidate x_i, with D_l the labeled set (the
      initial random batch plus everything selected so far, M items):
        d_s = min_{j in D_l} |f_i - f_j|                              Eq. (1)
        mu = (f_i + sum_j f_j) / (M + 1)                              Eq. (2)
        u_s = ((f_i - mu)^2 + sum_j (f_j - mu)^2) / (M + 1)           Eq. (3)
        t_s = f_i * d_s + u_s
      T = argmax t_s (equal scores: the lower index);
      if selected[op_T] < budget[op_T]: label T (selected[op_T] += 1)
      else: T is dropped from the candidates ("continue": it can never fit
      its operator's budget again);
  * the initial batch neither counts toward B_t nor toward the budgets.
"""
from __future__ import annotations

import numpy as np

f64 = np.float64


def topk_segments(scores, seg_offsets, K):
    """Indices [n_seg, K] (global) of each segment's K best scores, best
    first; -1 past the end of a segment shorter than K."""
    s = np.asarray(scores, dtype=f64)
    offs = np.asarray(seg_offsets, dtype=np.int64)
    out = np.full((len(offs) - 1, K), -1, dtype=np.int64)
    for g in range(len(offs) - 1):
        lo, hi = int(offs[g]), int(offs[g + 1])
        # NaN last: sort by (is NaN, -score, index)
        order = sorted(range(lo, hi), key=lambda i: (np.isnan(s[i]), -s[i] if not np.isnan(s[i]) else 0.0, i))
        take = order[:K]
        out[g, :len(take)] = take
    return out


def normalise(scores):
    """Min-max normalisation of the pool's predictions to [0, 1]."""
    f = np.asarray(scores, dtype=f64)
    lo, hi = f.min(), f.max()
    if hi == lo:
        return np.zeros_like(f)
    return (f - lo) / (hi - lo)


def budgets(op, n_ops, n_select):
    """Calc_Dist and the budget lines of Alg. 1: B_t times each operator
    type's share of the pool."""
    op = np.asarray(op)
    counts = np.bincount(op, minlength=n_ops).astype(f64)
    return n_select * counts / len(op)


def rdu_scores(f, labeled, candidates):
    """t_s = f_i d_s + u_s for each candidate (Eq. (1)-(3)), from their
    definitions."""
    fl = f[np.asarray(sorted(labeled), dtype=np.int64)]
    M = len(fl)
    out = np.empty(len(candidates))
    for n, i in enumerate(candidates):
        d = np.min(np.abs(f[i] - fl))
        mu = (f[i] + np.sum(fl)) / (M + 1)
        u = ((f[i] - mu) ** 2 + np.sum((fl - mu) ** 2)) / (M + 1)
        out[n] = f[i] * d + u
    return out


def rdu_select(scores, op, n_ops, initial, n_select):
    """The RDU selection of one step: the indices selected, in order."""
    f = normalise(scores)
    N = len(f)
    budget = budgets(op, n_ops, n_select)
    labeled = set(int(i) for i in initial)
    dropped = set()
    selected = np.zeros(n_ops, dtype=np.int64)
    out = []
    while len(out) < n_select:
        cand = [i for i in range(N) if i not in labeled and i not in dropped]
        if not cand:
            break
        t = rdu_scores(f, labeled, cand)
        T = cand[int(np.argmax(t))]  # first maximum: the lower index
        if selected[op[T]] < budget[op[T]]:
            labeled.add(T)
            selected[op[T]] += 1
            out.append(T)
        else:
            dropped.add(T)
    return out


def rdu_select_pool(scores, op, n_ops, initial, n_select, elems=1 << 22):
    """rdu_select for dataset-sized pools: the same selection loop, with
    Eq. (1)-(3) evaluated for a block of candidates at a time against the
    whole labeled set (the same per-candidate formulas as rdu_scores, as
    numpy array expressions over [candidates, labeled] blocks of about
    `elems` entries instead of a Python loop over candidates). Equal t_s
    keep the lower index, across blocks too."""
    f = normalise(scores)
    op = np.asarray(op)
    N = len(f)
    budget = budgets(op, n_ops, n_select)
    is_cand = np.ones(N, dtype=bool)
    labeled = set(int(i) for i in initial)
    is_cand[np.asarray(sorted(labeled), dtype=np.int64)] = False
    selected = np.zeros(n_ops, dtype=np.int64)
    out = []
    while len(out) < n_select:
        cand = np.nonzero(is_cand)[0]
        if cand.size == 0:
            break
        fl = f[np.asarray(sorted(labeled), dtype=np.int64)]
        M = len(fl)
        step = max(1, elems // max(M, 1))
        best_t, T = -np.inf, -1
        for c0 in range(0, cand.size, step):
            ci = cand[c0:c0 + step]
            fi = f[ci]
            d = np.min(np.abs(fi[:, None] - fl[None, :]), axis=1)             # Eq. (1)
            mu = (fi + np.sum(fl)) / (M + 1)                                    # Eq. (2)
            u = ((fi - mu) ** 2 + np.sum((fl[None, :] - mu[:, None]) ** 2, axis=1)) / (M + 1)  # Eq. (3)
            t = fi * d + u
            k = int(np.argmax(t))
            if t[k] > best_t:
                best_t, T = t[k], int(ci[k])
        if selected[op[T]] < budget[op[T]]:
            labeled.add(T)
            is_cand[T] = False
            selected[op[T]] += 1
            out.append(T)
        else:
            is_cand[T] = False
    return out
