"""Parity of the score consumers with the oracle (oracle/select.py), bit-exact
on indices: per-segment top-K (tcl_topk) and the RDU selection of Alg. 1
(tcl_rdu_select).

Top-K compares fp32 scores exactly on both sides, so the indices must be
identical. The RDU selection is an argmax over fp64 t_s; the oracle
computes Eq. (2)-(3) two-pass from their definitions and the kernel from
running sums, so the two t_s differ in the last bits; the selected sequences
must still be identical (seeded continuous scores have no near-ties at that
level) -- and if a step ever differs, the test reports whether the oracle's
own t_s of the two picks tie to 1e-12.
"""
import numpy as np
import pytest
import torch

from oracle import select as osel
from paper_2604_12891_amd import workload as wl

pytestmark = pytest.mark.gpu


def _tb():
    from paper_2604_12891_amd import binding as tb
    return tb


def _dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


@pytest.mark.parametrize("sizes,K", [([0, 1, 5, 64, 65, 300, 4096], 64), ([1000, 3, 2500], 1),
                                     ([70000], 1024), ([257, 1024, 1025], 256), ([5, 7], 10)])
def test_topk_matches_oracle(sizes, K):
    print(f"topk sizes={sizes} K={K}", flush=True)
    rng = np.random.default_rng(sum(sizes) + K)
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    s = (0.3 * rng.standard_normal(offs[-1])).astype(np.float32)
    s[rng.random(offs[-1]) < 0.02] = np.nan          # unscored programs
    s[rng.random(offs[-1]) < 0.05] = 0.125           # ties
    s[rng.random(offs[-1]) < 0.01] = -0.0
    got = _tb().topk(_dev(s, torch.float32), _dev(offs, torch.int32), K)
    torch.cuda.synchronize()
    ref = osel.topk_segments(s, offs, K)
    assert np.array_equal(got.cpu().numpy(), ref)


def test_topk_of_a_scored_round():
    """The top 64 of the headline tuning round's scores as the model would
    produce them (seeded score-like values, one segment per 512 candidates)."""
    w = wl.WORKLOADS["score_B4096_L25_d256_f32"]
    rng = np.random.default_rng(3)
    s = (0.1 * rng.standard_normal(w.B)).astype(np.float32)
    offs = np.arange(0, w.B + 1, 512, dtype=np.int32)
    got = _tb().topk(_dev(s, torch.float32), _dev(offs, torch.int32), 64).cpu().numpy()
    assert np.array_equal(got, osel.topk_segments(s, offs, 64))


def _rdu_case(N, n_ops, n_init, seed):
    rng = np.random.default_rng(seed)
    s = (0.3 * rng.standard_normal(N)).astype(np.float32)
    p = rng.random(n_ops) + 0.2
    op = rng.choice(n_ops, N, p=p / p.sum()).astype(np.int32)
    init = rng.choice(N, n_init, replace=False).astype(np.int32)
    return s, op, init


def _check_rdu(s, op, n_ops, init, n_select):
    sel, cnt = _tb().rdu_select(_dev(s, torch.float32), _dev(op, torch.int32), n_ops, _dev(init, torch.int32),
                                n_select)
    torch.cuda.synchronize()
    got = sel.cpu().numpy().tolist()
    c = int(cnt.cpu().numpy()[0])
    ref = osel.rdu_select(s.astype(np.float64), op, n_ops, init, n_select)
    assert c == len(ref)
    if got[:c] != ref:
        k = next(i for i in range(c) if got[i] != ref[i])
        f = osel.normalise(s.astype(np.float64))
        lab = set(init.tolist()) | set(ref[:k])
        tt = osel.rdu_scores(f, lab, [got[k], ref[k]])
        pytest.fail(f"step {k}: gpu {got[k]} oracle {ref[k]}; oracle t_s {tt[0]!r} vs {tt[1]!r}")
    assert all(g == -1 for g in got[c:])


@pytest.mark.parametrize("N,n_ops,n_init,n_select", [(50, 1, 1, 10), (300, 4, 10, 40), (1000, 8, 32, 64),
                                                     (5000, 16, 64, 32), (64, 3, 60, 10)])
def test_rdu_select_matches_oracle(N, n_ops, n_init, n_select):
    print(f"rdu N={N} ops={n_ops} init={n_init} select={n_select}", flush=True)
    s, op, init = _rdu_case(N, n_ops, n_init, N + n_ops)
    _check_rdu(s, op, n_ops, init, n_select)


def test_rdu_select_budgets_bind_and_pool_runs_out():
    """Skewed operator types so that budgets bind and candidates are dropped;
    then more selections asked than candidates left (the count reports it)."""
    rng = np.random.default_rng(9)
    N = 400
    s = (0.3 * rng.standard_normal(N)).astype(np.float32)
    op = np.where(rng.random(N) < 0.9, 0, 1 + rng.integers(0, 3, N)).astype(np.int32)
    init = rng.choice(N, 8, replace=False).astype(np.int32)
    _check_rdu(s, op, 4, init, 50)
    small_s, small_op = s[:20].copy(), np.zeros(20, np.int32)
    _check_rdu(small_s, small_op, 1, np.array([3, 7], np.int32), 30)


def _check_rdu_pool(s, op, n_ops, init, n_select):
    sel, cnt = _tb().rdu_select(_dev(s, torch.float32), _dev(op, torch.int32), n_ops, _dev(init, torch.int32),
                                n_select)
    torch.cuda.synchronize()
    got = sel.cpu().numpy().tolist()
    c = int(cnt.cpu().numpy()[0])
    ref = osel.rdu_select_pool(s.astype(np.float64), op, n_ops, init, n_select)
    assert c == len(ref) and got[:c] == ref, (got[:c], ref)


def test_rdu_select_grid_stride_pool():
    """A pool of 1.2 M programs: more candidates than one pass of the
    selection grid covers (1024 blocks x 256 threads x 4), so every kernel's
    grid-stride loop runs more than once; 20 operator types, 64 initial
    programs, 6 selections, against the oracle's blocked form."""
    N, n_ops, n_init, n_sel = 1_200_000, 20, 64, 6
    assert N > 1024 * 256 * 4
    print(f"rdu pool N={N} init={n_init} select={n_sel}", flush=True)
    s, op, init = _rdu_case(N, n_ops, n_init, 77)
    _check_rdu_pool(s, op, n_ops, init, n_sel)


def test_rdu_select_large_initial_set():
    """More initial labeled programs (8,500) than the sorted-set path holds
    (8,192): the distances to the initial set come from the direct pass."""
    N, n_ops, n_init, n_sel = 60_000, 8, 8_500, 3
    print(f"rdu N={N} init={n_init} select={n_sel}", flush=True)
    s, op, init = _rdu_case(N, n_ops, n_init, 78)
    _check_rdu_pool(s, op, n_ops, init, n_sel)
