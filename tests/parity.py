"""Tolerances and the ranking check shared by the GPU parity tests.

Score tolerance (per candidate, o = oracle, g = GPU):
  fp32: |g - o| <= 1e-5 + 1e-4 |o|
  bf16: |g - o| <= 2e-2 max(|o|, rms(o))   (relative with a scale floor, so a
        score near zero is judged on the batch's scale, not demanded exact)
Ranking: wherever the oracle's intervals [o - tol, o + tol] of two candidates
do not overlap, the GPU must order them the same way.
"""
import numpy as np

from oracle import model as om

FP32_RTOL, FP32_ATOL = 1e-4, 1e-5
BF16_RTOL = 2e-2


def tolerance(o: np.ndarray, dtype: str) -> np.ndarray:
    o = np.asarray(o, dtype=np.float64)
    if dtype == "f32":
        return FP32_ATOL + FP32_RTOL * np.abs(o)
    scale = np.sqrt(np.mean(o * o))
    return BF16_RTOL * np.maximum(np.abs(o), scale)


def ranking_violations(g: np.ndarray, o: np.ndarray, tol: np.ndarray) -> int:
    """Count pairs (i, j) with o_j - tol_j > o_i + tol_i but g_j <= g_i.

    O(B log B): sort candidates by hi = o + tol; for each j, every i with
    hi_i < lo_j = o_j - tol_j must have g_i < g_j, so it suffices to compare
    g_j with the largest g over that prefix (and count offenders exactly by
    scanning only when the prefix maximum is violated)."""
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    hi, lo = o + tol, o - tol
    order = np.argsort(hi, kind="stable")
    hs, gs = hi[order], g[order]
    pmax = np.maximum.accumulate(gs)
    k = np.searchsorted(hs, lo, side="left")  # number of i with hi_i < lo_j
    bad = 0
    for j in np.nonzero(k > 0)[0]:
        if pmax[k[j] - 1] >= g[j]:
            bad += int(np.sum(gs[:k[j]] >= g[j]))
    return bad


def assert_scores_match(g, o, dtype: str, what: str = ""):
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    assert g.shape == o.shape, (g.shape, o.shape)
    assert np.all(np.isfinite(g)), f"{what}: non-finite GPU scores"
    tol = tolerance(o, dtype)
    err = np.abs(g - o)
    worst = int(np.argmax(err / tol))
    assert np.all(err <= tol), (
        f"{what}: {int(np.sum(err > tol))}/{g.size} scores out of tolerance; worst #{worst}: "
        f"gpu={g[worst]!r} oracle={o[worst]!r} err={err[worst]:.3e} tol={tol[worst]:.3e}")
    v = ranking_violations(g, o, tol)
    assert v == 0, f"{what}: {v} ranking violations"


def oracle_cfg(shape) -> dict:
    return dict(F=shape.F, d_model=shape.d_model, d_inner=shape.d_inner, d_state=shape.d_state,
                d_conv=shape.d_conv, dt_rank=shape.dt_rank, n_layers=shape.n_layers,
                head_hidden=shape.head_hidden, final_norm=shape.final_norm, norm_eps=shape.norm_eps,
                enc_hidden=tuple(shape.enc_hidden), dec_hidden2=shape.dec_hidden2)


def oracle_scores(blob, X, lengths, shape) -> np.ndarray:
    return om.score(blob, X, lengths, oracle_cfg(shape))


def golden_scores(name: str, blob, X, lengths) -> np.ndarray:
    """The fp64 oracle's scores of every program of a named workload, as
    written by tests/golden/make_golden.py; fails if the stored digest does
    not match the inputs being scored."""
    import os

    from tests.golden import make_golden as mg

    path = mg.path(name)
    assert os.path.exists(path), f"missing golden scores {path}: run python -m tests.golden.make_golden {name}"
    with np.load(path, allow_pickle=False) as z:
        scores, sha = z["scores"], str(z["sha256"])
    assert sha == mg.digest(blob, X, lengths), f"{name}: inputs differ from those the golden scores were made from"
    return scores
