"""fp64 CPU oracle of TCL's ranking objectives: the LambdaRank loss of
section 5.3 (Eq. (6)) and the gated knowledge-distillation loss with the
EWC penalty of section 6 (Eq. (9)-(11)).

TEST INFRASTRUCTURE ONLY, like oracle.model: only the tests, the smoke check
and the benchmark's CPU-baseline leg may call it. It shares no code with the
HIP library and takes every input as an argument.

LambdaRank (Eq. (6)), read with the sign and pair set of the LambdaLoss
formulation it cites (the printed leading minus and the unrestricted sum
over i, j would make the loss symmetric in each pair):
    L = sum over pairs with rel_i > rel_j of
        dNDCG(i, j) * log2(1 + exp(-sigma (s_i - s_j)))
    dNDCG(i, j) = |G_i - G_j| * |1/D_i - 1/D_j|
    G_i = (2^rel_i - 1) / maxDCG,   D_i = log2(1 + r_i)
where s are the model's scores, r_i is the 1-based position of item i when
the items are sorted by score (descending; equal scores keep index order),
rel are the labels min-max normalised to [0, 1] over the batch, and maxDCG
is the DCG of the ideal ordering (items sorted by rel, descending). The
ranks are piecewise constant in s, so dL/ds treats dNDCG as constant (the
LambdaRank gradient). sigma is 1 unless given.

Knowledge distillation (Eq. (9)), one batch j of the KB (student) with
scores P_S, teacher scores P_T and ground-truth labels P_G:
    L_KD = beta * L(P_S; P_G) + (1 - beta) * Phi_j * L(P_S; P_T)
           + lambda/2 * sum_k F_k (theta_k - theta_prev_k)^2
with L(scores; labels) the LambdaRank loss above, Phi_j the teacher-loss
gate of Eq. (10) over the batch losses e_T of Eq. (11), F the diagonal
Fisher information and theta_prev the KB parameters after the previous
platform. The paper uses beta = 0.5 and lambda = 1e4.
"""
from __future__ import annotations

import numpy as np

f64 = np.float64
LN2 = np.log(2.0)


def relevance(labels):
    """Labels -> relevance in [0, 1] by min-max normalisation over the batch
    (all zero when every label is equal)."""
    y = np.asarray(labels, dtype=f64)
    lo, hi = y.min(), y.max()
    if hi == lo:
        return np.zeros_like(y)
    return (y - lo) / (hi - lo)


def ranks_desc(v):
    """1-based position of each item when v is sorted descending, equal values
    keeping index order."""
    v = np.asarray(v, dtype=f64)
    order = sorted(range(len(v)), key=lambda i: (-v[i], i))
    r = np.empty(len(v), dtype=np.int64)
    r[np.asarray(order, dtype=np.int64)] = np.arange(1, len(v) + 1)
    return r


def max_dcg(rel):
    """DCG of the ideal ordering: sum_k (2^rel_(k) - 1) / log2(1 + k) with rel
    sorted descending."""
    srt = np.sort(np.asarray(rel, dtype=f64))[::-1]
    k = np.arange(1, len(srt) + 1, dtype=f64)
    return float(np.sum((np.exp2(srt) - 1.0) / np.log2(1.0 + k)))


def delta_ndcg(scores, labels):
    """The |dNDCG(i, j)| matrix of Eq. (6) at the current ranking."""
    rel = relevance(labels)
    mx = max_dcg(rel)
    if mx <= 0.0:
        return np.zeros((len(rel), len(rel)))
    G = (np.exp2(rel) - 1.0) / mx
    D = np.log2(1.0 + ranks_desc(scores).astype(f64))
    return np.abs(G[:, None] - G[None, :]) * np.abs(1.0 / D[:, None] - 1.0 / D[None, :])


def lambdarank(scores, labels, sigma=1.0):
    """Eq. (6): (loss, dloss/dscores)."""
    s = np.asarray(scores, dtype=f64)
    rel = relevance(labels)
    W = delta_ndcg(s, labels)
    better = rel[:, None] > rel[None, :]          # pair (i, j) with i the more relevant
    x = sigma * (s[:, None] - s[None, :])
    # log2(1 + e^-x), and its derivative -sigmoid(-x) / ln 2
    pair_loss = np.logaddexp(0.0, -x) / LN2
    sig_neg = np.exp(-np.logaddexp(0.0, x))       # 1 / (1 + e^x), without overflow
    loss = float(np.sum(np.where(better, W * pair_loss, 0.0)))
    coef = np.where(better, W * sigma * sig_neg / LN2, 0.0)  # d loss / d s_j of pair (i, j); minus for s_i
    grad = -np.sum(coef, axis=1) + np.sum(coef, axis=0)
    return loss, grad


def teacher_gate(e_T):
    """Eq. (10)-(11): Phi_j = 1 - (e_j - min e) / (max e - min e) for every batch
    j, from the teacher's LambdaRank loss e_j against the ground truth."""
    e = np.asarray(e_T, dtype=f64)
    lo, hi = e.min(), e.max()
    if hi == lo:
        return np.ones_like(e)
    return 1.0 - (e - lo) / (hi - lo)


def ewc(theta, theta_prev, fisher, lam):
    """lambda/2 sum_k F_k (theta_k - theta_prev_k)^2 and its gradient."""
    d = np.asarray(theta, dtype=f64) - np.asarray(theta_prev, dtype=f64)
    F = np.asarray(fisher, dtype=f64)
    return float(0.5 * lam * np.sum(F * d * d)), lam * F * d


def kd_rank_loss(s, t, y, beta=0.5, phi=1.0, sigma=1.0):
    """The two ranking terms of Eq. (9) for one batch:
    (total, L(s; t), L(s; y)) and d total / d s."""
    l_sy, g_sy = lambdarank(s, y, sigma)
    l_st, g_st = lambdarank(s, t, sigma)
    w_t = (1.0 - beta) * phi
    return (beta * l_sy + w_t * l_st, l_st, l_sy), beta * g_sy + w_t * g_st


def distill_step_kd(teacher_blob, tcfg, student_blob, scfg, X, lengths, labels, beta=0.5, phi=1.0,
                    sigma=1.0, lam=0.0, fisher=None, theta_prev=None, m=None, v=None, step=1, lr=1e-3,
                    beta1=0.9, beta2=0.999, eps=1e-8, compute_blob=None, teacher_scores=None):
    """One teacher -> student step on the Eq. (9) objective: the ranking terms
    through the student's backward, the EWC gradient on its master weights,
    then one bias-corrected Adam update. Returns dict(loss=(total, L(s;t),
    L(s;y), ewc), teacher=, student=, grad=, params=, m=, v=)."""
    from . import model as om

    if teacher_scores is None:
        t = om.score(teacher_blob, X, lengths, tcfg)
    else:
        t = np.asarray(teacher_scores, dtype=f64)
    P = om.unpack(student_blob if compute_blob is None else compute_blob, scfg)
    s, caches, top = om.forward(P, X, lengths, scfg, keep=True)
    (tot, l_st, l_sy), ds = kd_rank_loss(s, t, np.asarray(labels, dtype=f64), beta, phi, sigma)
    g = om.pack(om.backward(ds, P, scfg, caches, top), scfg)
    p = np.asarray(student_blob, dtype=f64)
    e_loss = 0.0
    if lam != 0.0:
        e_loss, e_grad = ewc(p, theta_prev, fisher, lam)
        g = g + e_grad
    m = np.zeros_like(p) if m is None else np.asarray(m, dtype=f64)
    v = np.zeros_like(p) if v is None else np.asarray(v, dtype=f64)
    p2, m2, v2 = om.adam_update(p, g, m, v, step, lr, beta1, beta2, eps)
    return dict(loss=(tot + e_loss, l_st, l_sy, e_loss), teacher=t, student=s, grad=g, params=p2, m=m2, v=v2)
