"""Pins of the selection oracle (top-K of section 3; the RDU selection of
section 4, Alg. 1 with Eq. (1)-(3)): repeated-argmax brute force, numpy's
population variance and explicit distance matrices, hand-worked pools, and
invariants of the greedy loop."""
import numpy as np
import pytest

from oracle import select as osel


def _brute_topk(s, K):
    """K times: take the largest remaining score (np.nanargmax: the first
    maximum), NaN only once every number is taken (then in index order)."""
    s = np.array(s, dtype=float)
    left = list(range(len(s)))
    out = []
    while left and len(out) < K:
        vals = np.array([s[i] for i in left])
        if np.all(np.isnan(vals)):
            pick = left[0]
        else:
            pick = left[int(np.nanargmax(vals))]
        out.append(pick)
        left.remove(pick)
    return out


def test_topk_against_repeated_argmax():
    rng = np.random.default_rng(0)
    for trial in range(20):
        sizes = rng.integers(0, 40, size=4)
        offs = np.concatenate([[0], np.cumsum(sizes)])
        s = np.round(rng.standard_normal(offs[-1]) * 4) / 4  # many ties
        s[rng.random(offs[-1]) < 0.1] = np.nan
        K = int(rng.integers(1, 12))
        got = osel.topk_segments(s, offs, K)
        for g in range(4):
            ref = [offs[g] + i for i in _brute_topk(s[offs[g]:offs[g + 1]], K)]
            row = got[g]
            assert list(row[:len(ref)]) == ref
            assert np.all(row[len(ref):] == -1)


def test_normalise_and_budgets():
    f = osel.normalise(np.array([3.0, -1.0, 1.0, 7.0]))
    np.testing.assert_allclose(f, [0.5, 0.0, 0.25, 1.0])
    assert not osel.normalise(np.full(5, 2.0)).any()
    b = osel.budgets(np.array([0, 0, 1, 2, 2, 2]), 4, 12)
    np.testing.assert_allclose(b, [4.0, 2.0, 6.0, 0.0])
    assert b.sum() == pytest.approx(12.0)


def test_rdu_scores_against_library_variance_and_distance_matrix():
    rng = np.random.default_rng(1)
    f = rng.random(50)
    labeled = set(rng.choice(50, 9, replace=False).tolist())
    cand = [i for i in range(50) if i not in labeled]
    t = osel.rdu_scores(f, labeled, cand)
    L = np.array(sorted(labeled))
    d = np.abs(np.subtract.outer(f[cand], f[L])).min(axis=1)
    u = np.array([np.var(np.concatenate([[f[i]], f[L]])) for i in cand])  # population variance
    np.testing.assert_allclose(t, f[cand] * d + u, rtol=1e-13)


def test_rdu_hand_worked_pool():
    """f = (0, 1, 0.5, 0.9), initial {0}. Step 1: t = 1.25, 0.3125, 1.0125 ->
    item 1. Step 2 (labeled {0, 1}): t_2 = 0.25 + 1/6, t_3 = 0.09 + 0.2022 ->
    item 2. Then item 3."""
    s = np.array([0.0, 1.0, 0.5, 0.9])
    t1 = osel.rdu_scores(s, {0}, [1, 2, 3])
    np.testing.assert_allclose(t1, [1.25, 0.3125, 1.0125], rtol=1e-14)
    t2 = osel.rdu_scores(s, {0, 1}, [2, 3])
    np.testing.assert_allclose(t2, [0.25 + 1.0 / 6.0, 0.09 + (0.8 / 3) ** 2 / 3 + (1.9 / 3) ** 2 / 3 + (1.1 / 3) ** 2 / 3],
                               rtol=1e-13)
    assert osel.rdu_select(s, np.zeros(4, np.int64), 1, [0], 3) == [1, 2, 3]
    # two operator types, budget 1 each: item 2 (op 0's second pick) is dropped
    assert osel.rdu_select(s, np.array([1, 0, 0, 1]), 2, [0], 2) == [1, 3]
    assert osel.rdu_select(s, np.array([0, 0, 1, 1]), 2, [0], 2) == [1, 2]


def test_rdu_select_invariants():
    rng = np.random.default_rng(2)
    N, n_ops = 300, 5
    s = rng.standard_normal(N)
    op = rng.choice(n_ops, N, p=[0.4, 0.3, 0.15, 0.1, 0.05])
    init = rng.choice(N, 12, replace=False)
    out = osel.rdu_select(s, op, n_ops, init, 40)
    assert len(out) == 40 and len(set(out)) == 40 and not set(out) & set(init.tolist())
    b = osel.budgets(op, n_ops, 40)
    cnt = np.bincount(op[out], minlength=n_ops)
    assert np.all(cnt <= np.ceil(b))
    # a positive affine map of the predictions changes nothing (normalisation)
    assert osel.rdu_select(3.0 * s + 1.0, op, n_ops, init, 40) == out
    # the first pick maximises t_s over every candidate (budgets are not yet binding)
    f = osel.normalise(s)
    cand = [i for i in range(N) if i not in set(init.tolist())]
    t = osel.rdu_scores(f, set(init.tolist()), cand)
    assert out[0] == cand[int(np.argmax(t))]
    # with one operator type the budget never binds: pure greedy argmax
    one = osel.rdu_select(s, np.zeros(N, np.int64), 1, init, 10)
    lab = set(init.tolist())
    for k in one:
        cand = [i for i in range(N) if i not in lab]
        assert k == cand[int(np.argmax(osel.rdu_scores(f, lab, cand)))]
        lab.add(k)


@pytest.mark.parametrize("N,n_ops,n_init,n_select,seed", [(300, 4, 10, 40, 1), (120, 3, 60, 30, 2),
                                                          (500, 1, 1, 20, 3), (400, 6, 5, 60, 4)])
def test_rdu_select_pool_equals_rdu_select(N, n_ops, n_init, n_select, seed):
    """The blocked form for large pools selects exactly what the per-candidate
    loop selects, with small blocks so that the argmax crosses blocks (and
    budgets bind on the skewed pools)."""
    rng = np.random.default_rng(seed)
    s = 0.3 * rng.standard_normal(N)
    p = rng.random(n_ops) + 0.05
    op = rng.choice(n_ops, N, p=p / p.sum())
    init = rng.choice(N, n_init, replace=False)
    ref = osel.rdu_select(s, op, n_ops, init, n_select)
    for elems in (1 << 22, 7 * max(n_init, 1), 1):
        assert osel.rdu_select_pool(s, op, n_ops, init, n_select, elems=elems) == ref


def test_rdu_select_pool_ties_take_the_lower_index():
    """Candidates with identical scores tie in t_s: the lower index wins,
    also when the tie spans two blocks."""
    s = np.array([0.0, 1.0, 0.5, 1.0, 1.0, 0.2])
    op = np.zeros(6, dtype=np.int64)
    for elems in (1 << 22, 1, 2):
        sel = osel.rdu_select_pool(s, op, 1, [0], 3, elems=elems)
        assert sel == osel.rdu_select(s, op, 1, [0], 3)
        assert sel[0] == 1
