"""Parity of the ranking objectives on the GPU with the fp64 oracle
(oracle/kd.py): tcl_lambdarank (Eq. (6)) on seeded scores and labels, and
tcl_distill_step_kd (Eq. (9): two LambdaRank terms, the teacher gate and the
EWC penalty) end to end.

Tolerances: the kernel computes in fp32 with ranks counted exactly (the same
inputs give the same ranks on both sides, ties broken by index), so the loss
must match to rel 1e-4 and every gradient entry to 1e-4 |g| + 1e-5 max|g|
(sums of up to B terms of one exp and one log each). The distillation step
is held to the bf16 step's bounds (loss rel 2e-2, gradients per tensor
2e-2); its scores come from bf16 models, so the test picks inputs whose
oracle student scores are separated by more than the score tolerance, where
the score ranks (and hence the LambdaRank weights) cannot differ.
"""
import numpy as np
import pytest
import torch

from oracle import kd
from oracle import model as om
from paper_2604_12891_amd import binding as tb
from paper_2604_12891_amd import workload as wl
from tests.parity import oracle_cfg
from tests.test_gpu_distill import LR, _check_params

pytestmark = pytest.mark.gpu


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def _scores_labels(B, seed, ties=False):
    """Score-like values (a model's outputs) and noisy labels of the same items."""
    rng = np.random.default_rng(seed)
    s = (0.3 * rng.standard_normal(B)).astype(np.float32)
    if ties:
        s = (np.round(s * 8) / 8).astype(np.float32)  # many exact ties
    y = (s + 0.2 * rng.standard_normal(B)).astype(np.float32)
    if ties:
        y = (np.round(y * 4) / 4).astype(np.float32)
    return s, y


def _check_rank(B, s, y, sigma, what):
    loss_g, grad_g = tb.lambdarank(_dev(s), _dev(y), sigma)
    torch.cuda.synchronize()
    lo, go = kd.lambdarank(s.astype(np.float64), y.astype(np.float64), sigma)
    lg = float(loss_g.cpu().numpy()[0])
    gg = grad_g.cpu().numpy().astype(np.float64)
    assert abs(lg - lo) <= 1e-4 * abs(lo) + 1e-7, f"{what}: loss {lg} vs {lo}"
    tol = 1e-4 * np.abs(go) + 1e-5 * max(np.abs(go).max(), 1e-30)
    assert np.all(np.abs(gg - go) <= tol), f"{what}: grad max err {np.abs(gg - go).max():.3e}"


@pytest.mark.parametrize("B", [1, 2, 7, 255, 256, 257, 1000, 1024, 3000])
@pytest.mark.parametrize("sigma", [1.0, 2.0])
def test_lambdarank_matches_oracle(B, sigma):
    print(f"lambdarank B={B} sigma={sigma}", flush=True)
    s, y = _scores_labels(B, 100 + B)
    _check_rank(B, s, y, sigma, f"B={B}")


def test_lambdarank_ties_and_degenerate_labels():
    """Exact ties in scores and labels (ranks by index on both sides), equal
    labels (zero loss and gradient), and determinism."""
    s, y = _scores_labels(600, 7, ties=True)
    assert len(np.unique(s)) < 600 and len(np.unique(y)) < 600
    _check_rank(600, s, y, 1.0, "ties")
    loss, g = tb.lambdarank(_dev(s), _dev(np.full(600, 0.25, np.float32)))
    torch.cuda.synchronize()
    assert float(loss.cpu()[0]) == 0.0 and not g.cpu().numpy().any()
    a = tb.lambdarank(_dev(s), _dev(y))[1].cpu().numpy()
    b = tb.lambdarank(_dev(s), _dev(y))[1].cpu().numpy()
    assert np.array_equal(a, b)


def _kd_inputs(B, L, seed):
    tshape = wl.ModelShape(d_model=64, d_inner=128, dt_rank=4, n_layers=2, head_hidden=64)
    sshape = wl.ModelShape(d_model=64, d_inner=128, dt_rank=8, n_layers=2, head_hidden=64)
    rng = np.random.default_rng(seed)
    tblob = wl.round_to_bf16(wl.init_params(tshape, rng, perturb=True))
    sblob = wl.round_to_bf16(wl.init_params(sshape, rng, perturb=True))
    X, lengths = wl.make_inputs(B, L, tshape.F, 1, L, rng)
    t = om.score(tblob, X, lengths, oracle_cfg(tshape))
    s = om.score(sblob, X, lengths, oracle_cfg(sshape))
    labels = (t + 0.05 * rng.standard_normal(B)).astype(np.float32)
    n = sblob.size
    fisher = rng.random(n).astype(np.float32)
    theta_prev = (sblob + 1e-3 * rng.standard_normal(n)).astype(np.float32)
    return tshape, sshape, tblob, sblob, X, lengths, labels, t, s, fisher, theta_prev


def _separated(s, gap):
    return np.diff(np.sort(s)).min() > gap


@pytest.mark.parametrize("ewc_lambda", [0.0, 1e4])
def test_distill_step_kd_matches_oracle(ewc_lambda):
    """One step on Eq. (9) (beta 0.5, phi 0.7, sigma 1) from zero Adam moments:
    the four loss values, every gradient tensor and the updated parameters."""
    B, L = 12, 12
    for seed in range(200, 300):  # the first seed whose student scores are well separated
        inp = _kd_inputs(B, L, seed)
        s = inp[8]
        if _separated(s, 1e-2 * np.abs(s).max()):
            break
    else:
        pytest.fail("no seed with separated student scores")
    tshape, sshape, tblob, sblob, X, lengths, labels, t, s, fisher, theta_prev = inp
    print(f"distill kd seed={seed} ewc={ewc_lambda}", flush=True)
    teacher = tb.CostModel(tb.config_from_shape(tshape, "bf16"), tblob)
    student = tb.CostModel(tb.config_from_shape(sshape, "bf16"), sblob)
    tr = tb.Trainer(teacher, student, lr=LR, max_B=B, max_L=L)
    Xd, Ld, Yd = torch.from_numpy(X).cuda(), torch.from_numpy(lengths).cuda(), torch.from_numpy(labels).cuda()
    Fd, Pd = _dev(fisher), _dev(theta_prev)
    loss = tr.step_kd(Xd, Ld, Yd, beta=0.5, phi=0.7, sigma=1.0, ewc_lambda=ewc_lambda, fisher=Fd, theta_prev=Pd)
    torch.cuda.synchronize()
    lg = loss.cpu().numpy().astype(np.float64)
    gg = tr.grads().astype(np.float64)
    pg = student.get_params().astype(np.float64)
    orc = kd.distill_step_kd(tblob, oracle_cfg(tshape), sblob, oracle_cfg(sshape), X, lengths, labels,
                             beta=0.5, phi=0.7, sigma=1.0, lam=ewc_lambda, fisher=fisher,
                             theta_prev=theta_prev, lr=LR, teacher_scores=t)
    np.testing.assert_allclose(lg[:3], np.array(orc["loss"][:3]), rtol=2e-2, err_msg="loss")
    if ewc_lambda == 0.0:
        assert lg[3] == 0.0
    else:
        assert abs(lg[3] - orc["loss"][3]) <= 1e-4 * orc["loss"][3]
    cfg = oracle_cfg(sshape)
    G, O = om.unpack(gg, cfg), om.unpack(orc["grad"], cfg)
    # a pairwise loss's score gradient sums to zero, so db2 = sum_b dL/ds_b is
    # zero in exact arithmetic and fp32 cancellation noise on the GPU: an
    # absolute floor of 1e-6 of the whole gradient's norm covers it
    floor = 1e-6 * np.linalg.norm(orc["grad"])
    for name in O:
        err, ref = np.linalg.norm(G[name] - O[name]), np.linalg.norm(O[name])
        assert err <= 2e-2 * ref + floor, f"grad {name} rel err {err / max(ref, 1e-30):.3e}"
    _check_params(sblob.astype(np.float64), pg, gg, orc, sshape, "kd")


def test_distill_step_kd_full_batch_runs_and_descends():
    """The distillation workload (B = 1024, L = 25) on the Eq. (9) objective:
    finite losses, the EWC slot equal to its closed form at step 1 (theta =
    theta_prev + delta), and the ranking loss going down over a few steps."""
    w = wl.WORKLOADS["distill_B1024_L25_t256_s128_bf16"]
    (tblob, sblob), X, lengths = wl.make_workload(w.name)
    rng = np.random.default_rng(5)
    labels = (om.score(tblob, X, lengths, oracle_cfg(w.model)) + wl.label_noise(w.B)).astype(np.float32)
    teacher = tb.CostModel(tb.config_from_shape(w.model, "bf16"), tblob)
    student = tb.CostModel(tb.config_from_shape(w.student, "bf16"), sblob)
    Yd = torch.from_numpy(labels).cuda()
    tr = tb.Trainer(teacher, student, lr=LR, max_B=w.B, max_L=w.L)
    n = sblob.size
    fisher = rng.random(n).astype(np.float32)
    delta = (1e-3 * rng.standard_normal(n)).astype(np.float32)
    theta_prev = sblob - delta
    Xd, Ld = torch.from_numpy(X).cuda(), torch.from_numpy(lengths).cuda()
    losses = []
    for _ in range(4):
        loss = tr.step_kd(Xd, Ld, Yd, beta=0.5, phi=0.7, ewc_lambda=1e4, fisher=_dev(fisher),
                          theta_prev=_dev(theta_prev))
        torch.cuda.synchronize()
        losses.append(loss.cpu().numpy().astype(np.float64))
    assert all(np.all(np.isfinite(l)) for l in losses)
    d = (sblob.astype(np.float64) - theta_prev.astype(np.float64))
    ewc1 = 0.5e4 * np.sum(fisher.astype(np.float64) * d * d)
    assert abs(losses[0][3] - ewc1) <= 1e-4 * ewc1
    rank0 = 0.5 * losses[0][2] + 0.5 * 0.7 * losses[0][1]
    rank3 = 0.5 * losses[3][2] + 0.5 * 0.7 * losses[3][1]
    assert rank3 < rank0
