"""A distillation step captured into a HIP graph: every replay is one more
step, equal bit for bit to the same step run uncaptured (the same kernels
on the same inputs in the same order, and Adam's bias correction reads the
step count from the device). Replays are separated by the program's own
uncaptured work and synchronisations, and every replay is compared."""
import numpy as np
import pytest
import torch

from paper_2604_12891_amd import binding as tb
from paper_2604_12891_amd import workload as wl

pytestmark = pytest.mark.gpu
B = 128
STEPS = 4


def _models(w, tblob, sblob):
    teacher = tb.CostModel(tb.config_from_shape(w.model, "bf16"), tblob)
    student = tb.CostModel(tb.config_from_shape(w.student, "bf16"), sblob)
    return teacher, student


def _step(tr, objective, Xd, Ld, Yd, loss, ws, kd):
    if objective == "kd":
        tr.step_kd(Xd, Ld, Yd, loss=loss, workspace=ws, **kd)
    else:
        tr.step(Xd, Ld, Yd, loss=loss, workspace=ws)


@pytest.mark.parametrize("objective", ["mse", "kd"])
def test_distill_graph_replays_equal_uncaptured_steps(objective):
    w = wl.WORKLOADS["distill_B1024_L25_t256_s128_bf16"]
    (tblob, sblob), X, lengths = wl.make_workload(w.name, B=B)
    rng = np.random.default_rng(7)
    labels = rng.standard_normal(B).astype(np.float32)
    Xd, Ld, Yd = (torch.from_numpy(a).cuda() for a in (X, lengths, labels))
    nl = 4 if objective == "kd" else 3
    kd = {}
    if objective == "kd":
        fisher = torch.from_numpy(rng.random(sblob.size).astype(np.float32)).cuda()
        prev = torch.from_numpy((sblob + 1e-3 * rng.standard_normal(sblob.size)).astype(np.float32)).cuda()
        kd = dict(beta=0.5, phi=0.7, sigma=1.0, ewc_lambda=1e4, fisher=fisher, theta_prev=prev)
    print(f"graph replay objective={objective} B={B}", flush=True)

    # uncaptured reference: STEPS steps
    teacher, student = _models(w, tblob, sblob)
    tr = tb.Trainer(teacher, student, lr=1e-3, max_B=B, max_L=w.L)
    ws = tr.workspace(B, w.L)
    loss = torch.empty(nl, device="cuda")
    ref = []
    for _ in range(STEPS):
        _step(tr, objective, Xd, Ld, Yd, loss, ws, kd)
        torch.cuda.synchronize()
        ref.append((loss.cpu().numpy().copy(), student.get_params().copy()))
    tr.close()

    # the same from fresh models: step 1 uncaptured, then one captured step
    # replayed STEPS - 1 times
    teacher2, student2 = _models(w, tblob, sblob)
    tr2 = tb.Trainer(teacher2, student2, lr=1e-3, max_B=B, max_L=w.L)
    ws2 = tr2.workspace(B, w.L)
    loss2 = torch.empty(nl, device="cuda")
    _step(tr2, objective, Xd, Ld, Yd, loss2, ws2, kd)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(loss2.cpu().numpy(), ref[0][0])
    np.testing.assert_array_equal(student2.get_params(), ref[0][1])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _step(tr2, objective, Xd, Ld, Yd, loss2, ws2, kd)
    torch.cuda.synchronize()
    # capturing launched nothing: the parameters are still those of step 1
    np.testing.assert_array_equal(student2.get_params(), ref[0][1])
    for k in range(1, STEPS):
        g.replay()
        torch.cuda.synchronize()
        got_loss, got_params = loss2.cpu().numpy(), student2.get_params()
        print(f"replay {k}: loss {got_loss} (uncaptured {ref[k][0]})", flush=True)
        np.testing.assert_array_equal(got_loss, ref[k][0])
        np.testing.assert_array_equal(got_params, ref[k][1])
        # uncaptured work between replays, on the teacher model too
        t = teacher2.score(Xd, Ld)
        torch.cuda.synchronize()
        assert torch.isfinite(t).all().item()
    tr2.close()


def test_capture_of_an_unseen_shape_is_refused():
    w = wl.WORKLOADS["distill_B1024_L25_t256_s128_bf16"]
    (tblob, sblob), X, lengths = wl.make_workload(w.name, B=16)
    Xd, Ld = torch.from_numpy(X).cuda(), torch.from_numpy(lengths).cuda()
    Yd = torch.zeros(16, device="cuda")
    teacher, student = _models(w, tblob, sblob)
    tr = tb.Trainer(teacher, student, max_B=16, max_L=w.L)
    ws = tr.workspace(16, w.L)
    loss = torch.empty(3, device="cuda")
    before = student.get_params()
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        g.capture_begin()
        try:
            with pytest.raises(tb.TclError, match="cannot be captured"):
                tr.step(Xd, Ld, Yd, loss=loss, workspace=ws, stream=s)
        finally:
            g.capture_end()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(student.get_params(), before)
    # the shape, once run uncaptured, steps normally
    tr.step(Xd, Ld, Yd, loss=loss, workspace=ws)
    torch.cuda.synchronize()
    assert torch.isfinite(loss).all().item()
    tr.close()


@pytest.mark.parametrize("name,B,entry", [("score_B4096_L25_d256_f32", 4096, "score"),
                                          ("score_B4096_L25_d256_f32", 300, "score"),
                                          ("score_B65536_L25_d256_bf16", 2048, "score"),
                                          ("score_B4096_L25_d256_f32", 1000, "noalloc")])
def test_score_graph_replays_equal_uncaptured(name, B, entry):
    """tcl_score (one pass below 2048 programs, two halves on the model's two
    streams from 2048 up) and tcl_score_noalloc captured into a HIP graph:
    every replay, with new features copied into the captured input buffer
    and uncaptured scoring on the same model between replays, equals the
    uncaptured scores of the same inputs bit for bit."""
    w = wl.WORKLOADS[name]
    blob, X, lengths = wl.make_workload(name, B=B)
    model = tb.CostModel(tb.config_from_shape(w.model, w.dtype), blob)
    Xd, Ld = torch.from_numpy(X).cuda(), torch.from_numpy(lengths).cuda()
    out = torch.empty(B, device="cuda")
    ws = model.workspace(B, w.L) if entry == "score" else None
    print(f"score graph {name} B={B} entry={entry}", flush=True)

    def run(o):
        if entry == "score":
            model.score(Xd, Ld, out=o, workspace=ws)
        else:
            model.score_noalloc(Xd, Ld, o)

    run(out)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(out)
    torch.cuda.synchronize()
    rng = np.random.default_rng(3)
    for k in range(3):
        # new inputs in the captured buffers (the same shapes and lengths)
        Xn = X * (1.0 + 0.1 * k) + (0.01 * rng.standard_normal(X.shape)).astype(np.float32) * (X != 0)
        Xd.copy_(torch.from_numpy(Xn.astype(np.float32)))
        ref = torch.empty(B, device="cuda")
        run(ref)  # uncaptured, same model and buffers
        torch.cuda.synchronize()
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        print(f"replay {k}: max |diff| {np.abs(got - ref.cpu().numpy()).max():.3e}", flush=True)
        np.testing.assert_array_equal(got, ref.cpu().numpy())
