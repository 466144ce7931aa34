"""Pins of the whole-model oracle (section 5.2 architecture, the two-MSE
distillation loss, Adam). Each check compares the oracle with something
other than itself: library routines, an independent re-expression built
from torch primitives with autograd, finite differences, closed forms or
invariants the architecture implies."""
import math

import numpy as np
import pytest
import scipy.special
import torch

from oracle import model as om
from paper_2604_12891_amd import workload as wl

TINY_CFG = dict(F=6, d_model=4, d_inner=8, d_state=3, d_conv=4, dt_rank=2, n_layers=2,
                head_hidden=5, final_norm=1, norm_eps=1e-5)


def _cfg(shape: wl.ModelShape) -> dict:
    return dict(F=shape.F, d_model=shape.d_model, d_inner=shape.d_inner, d_state=shape.d_state,
                d_conv=shape.d_conv, dt_rank=shape.dt_rank, n_layers=shape.n_layers,
                head_hidden=shape.head_hidden, final_norm=shape.final_norm, norm_eps=shape.norm_eps,
                enc_hidden=tuple(shape.enc_hidden), dec_hidden2=shape.dec_hidden2)


def _tiny(seed=0, Bn=3, L=7, perturb=True):
    shape = wl.ModelShape(**TINY_CFG)
    rng = np.random.default_rng(seed)
    blob = wl.init_params(shape, rng, perturb=perturb).astype(np.float64)
    X, lengths = wl.make_inputs(Bn, L, shape.F, 1, L, rng)
    return shape, blob, X.astype(np.float64), lengths


# ---------------------------------------------------------------- elementwise

def test_elementwise_against_library():
    x = np.linspace(-40, 40, 2001)
    np.testing.assert_allclose(om.sigmoid(x), scipy.special.expit(x), rtol=1e-15)
    np.testing.assert_allclose(om.softplus(x), np.logaddexp(0.0, x), rtol=1e-15, atol=1e-300)
    np.testing.assert_allclose(om.silu(x), x * scipy.special.expit(x), rtol=1e-15)
    h = 1e-6
    fd = (om.silu(x + h) - om.silu(x - h)) / (2 * h)
    np.testing.assert_allclose(om.silu_grad(x), fd, rtol=1e-6, atol=1e-9)


def test_rmsnorm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(0)
    h = rng.standard_normal((5, 7, 32)) * 3.0
    n, _ = om.rmsnorm(h, np.ones(32), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(n * n, axis=-1)), 1.0, rtol=1e-13)
    n2, _ = om.rmsnorm(h * 7.5, np.ones(32), 0.0)
    np.testing.assert_allclose(n, n2, rtol=1e-13)
    g = rng.standard_normal(32)
    ng, _ = om.rmsnorm(h, g, 1e-5)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(h), (32,), torch.from_numpy(g), eps=1e-5)
    np.testing.assert_allclose(ng, ref.numpy(), rtol=1e-13)


# --------------------------------------------------------------- model-level

def test_layout_matches_workload_generator():
    for shape in (wl.TINY, wl.D256, wl.STUDENT, wl.ModelShape(**TINY_CFG), wl.PAPER_CPU, wl.PAPER_GPU):
        cfg = _cfg(shape)
        assert [(n, tuple(s)) for n, s in om.layout(cfg)] == [(n, tuple(s)) for n, s in wl.param_layout(shape)]


def test_pool_equals_mean_at_full_length():
    shape, blob, X, _ = _tiny(Bn=4, L=6)
    cfg = _cfg(shape)
    P = om.unpack(blob, cfg)
    lengths = np.full(4, 6)
    s, _, top = om.forward(P, X, lengths, cfg, keep=True)
    np.testing.assert_allclose(top["pooled"], np.mean(top["hf"], axis=1), rtol=1e-14)


def test_padding_invariance():
    """Values in rows t >= length never change a score (causal model, masked pool)."""
    shape, blob, X, lengths = _tiny(Bn=5, L=9)
    cfg = _cfg(shape)
    s0 = om.score(blob, X, lengths, cfg)
    X2 = X.copy()
    pad = np.arange(9)[None, :] >= lengths[:, None]
    X2[pad] = np.random.default_rng(1).standard_normal((pad.sum(), shape.F)) * 10
    np.testing.assert_array_equal(om.score(blob, X2, lengths, cfg), s0)


def test_permutation_and_batch_independence():
    shape, blob, X, lengths = _tiny(Bn=6, L=8)
    cfg = _cfg(shape)
    s = om.score(blob, X, lengths, cfg)
    perm = np.random.default_rng(2).permutation(6)
    np.testing.assert_allclose(om.score(blob, X[perm], lengths[perm], cfg), s[perm], rtol=1e-13)
    for b in range(6):
        one = om.score(blob, X[b:b + 1], lengths[b:b + 1], cfg)
        np.testing.assert_allclose(one, s[b:b + 1], rtol=1e-13)
    # a program is scored the same whatever the padded length of its batch
    Xw = np.concatenate([X, np.zeros((6, 5, shape.F))], axis=1)
    np.testing.assert_allclose(om.score(blob, Xw, lengths, cfg), s, rtol=1e-13)


def test_token_causality_of_hidden_states():
    """Changing token t0's features leaves every hidden state before t0 unchanged."""
    shape, blob, X, lengths = _tiny(Bn=2, L=8)
    cfg = _cfg(shape)
    cfg_nohead = dict(cfg)
    P = om.unpack(blob, cfg)
    lengths = np.full(2, 8)
    _, _, top0 = om.forward(P, X, lengths, cfg_nohead, keep=True)
    X2 = X.copy()
    X2[:, 5] += 1.0
    _, _, top1 = om.forward(P, X2, lengths, cfg_nohead, keep=True)
    assert np.array_equal(top0["h_last"][:, :5], top1["h_last"][:, :5])
    assert not np.allclose(top0["h_last"][:, 5], top1["h_last"][:, 5])


# ------------------------------------------------- independent torch re-expression

def _torch_block(h, Pt, l, cfg):
    """One Mamba block with its residual, in torch primitives, the SSM in its
    explicit (quadratic) convolution form instead of the recurrence."""
    F = torch.nn.functional
    E, N, R, K = cfg["d_inner"], cfg["d_state"], cfg["dt_rank"], cfg["d_conv"]
    L = h.shape[1]
    causal = torch.tril(torch.ones(L, L, dtype=torch.float64))
    p = f"blk{l}."
    n = F.rms_norm(h, (cfg["d_model"],), Pt[p + "g"], eps=cfg["norm_eps"])
    xz = F.linear(n, Pt[p + "W_in"])
    xs, z = xz[..., :E], xz[..., E:]
    xc = F.conv1d(xs.transpose(1, 2), Pt[p + "conv_w"][:, None, :], Pt[p + "conv_b"],
                  padding=K - 1, groups=E)[..., :L].transpose(1, 2)
    u = F.silu(xc)
    xdbl = F.linear(u, Pt[p + "W_x"])
    dtr, Bm, Cm = xdbl[..., :R], xdbl[..., R:R + N], xdbl[..., R + N:]
    dt = F.softplus(F.linear(dtr, Pt[p + "W_dt"], Pt[p + "b_dt"]))
    A = -torch.exp(Pt[p + "A_log"])
    cum = torch.cumsum(dt[..., None] * A, dim=1)                  # [B,L,E,N]
    seg = cum[:, :, None] - cum[:, None, :]                        # [B,t,k,E,N]
    mask = causal[None, :, :, None, None]
    decay = torch.exp(torch.where(mask > 0, seg, torch.full_like(seg, -1e30))) * mask
    y = torch.einsum("btn,btken,bkn,bke->bte", Cm, decay, Bm, dt * u)
    y = y + Pt[p + "D"] * u
    return h + F.linear(y * F.silu(z), Pt[p + "W_out"])


def _torch_pool(h, Pt, lengths, cfg):
    F = torch.nn.functional
    L = h.shape[1]
    hf = F.rms_norm(h, (cfg["d_model"],), Pt["g_f"], eps=cfg["norm_eps"])
    valid = (torch.arange(L)[None, :] < torch.as_tensor(lengths)[:, None]).double()
    return (hf * valid[..., None]).sum(1) / torch.as_tensor(lengths, dtype=torch.float64)[:, None]


def _torch_model_scores(Pt, X, lengths, cfg):
    """The same model written with torch primitives, and the SSM in its
    explicit (quadratic) convolution form instead of the recurrence."""
    F = torch.nn.functional
    # encoder: Linear layers with a ReLU between consecutive ones
    enc = [F.linear(X, Pt["W0"], Pt["b0"])]
    for i in range(1, len(cfg.get("enc_hidden", ())) + 1):
        enc.append(F.linear(F.relu(enc[-1]), Pt[f"W0_{i}"], Pt[f"b0_{i}"]))
    h = enc[-1]
    for l in range(cfg["n_layers"]):
        h = _torch_block(h, Pt, l, cfg)
    pooled = _torch_pool(h, Pt, lengths, cfg)
    r1 = F.relu(F.linear(pooled, Pt["W1"], Pt["b1"]))
    if cfg.get("dec_hidden2", 0):
        return F.linear(F.relu(F.linear(r1, Pt["W2"], Pt["b2"])), Pt["W3"], Pt["b3"])[:, 0]
    return F.linear(r1, Pt["W2"], Pt["b2"])[:, 0]


def test_forward_and_gradients_match_torch_reexpression():
    shape, blob, X, lengths = _tiny(seed=3, Bn=4, L=7)
    cfg = _cfg(shape)
    P = om.unpack(blob, cfg)
    s, caches, top = om.forward(P, X, lengths, cfg, keep=True)
    Pt = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in P.items()}
    st = _torch_model_scores(Pt, torch.from_numpy(X), lengths, cfg)
    np.testing.assert_allclose(s, st.detach().numpy(), rtol=1e-11, atol=1e-13)
    ds = np.random.default_rng(4).standard_normal(4)
    G = om.backward(ds, P, cfg, caches, top)
    (st * torch.from_numpy(ds)).sum().backward()
    for k in P:
        np.testing.assert_allclose(G[k], Pt[k].grad.numpy(), rtol=1e-9, atol=1e-12, err_msg=k)


def test_gradients_against_finite_differences():
    shape, blob, X, lengths = _tiny(seed=5, Bn=2, L=5)
    cfg = _cfg(shape)
    P = om.unpack(blob, cfg)
    t = np.array([0.3, -0.2])
    y = np.array([0.1, 0.5])

    def loss_of(b):
        s = om.score(b, X, lengths, cfg)
        return om.distill_loss(s, t, y)[0][0]

    s, caches, top = om.forward(P, X, lengths, cfg, keep=True)
    _, ds = om.distill_loss(s, t, y)
    g = om.pack(om.backward(ds, P, cfg, caches, top), cfg)
    h = 1e-6
    fd = np.empty_like(blob)
    for i in range(blob.size):
        bp, bm = blob.copy(), blob.copy()
        bp[i] += h
        bm[i] -= h
        fd[i] = (loss_of(bp) - loss_of(bm)) / (2 * h)
    np.testing.assert_allclose(g, fd, rtol=1e-5, atol=1e-9)


def test_mse_loss_gradient_closed_form():
    rng = np.random.default_rng(6)
    s, t, y = rng.standard_normal(7), rng.standard_normal(7), rng.standard_normal(7)
    (tot, mt, ml), ds = om.distill_loss(s, t, y)
    assert math.isclose(mt, float(np.sum((s - t) ** 2)) / 7, rel_tol=1e-14)
    assert math.isclose(tot, mt + ml, rel_tol=1e-15)
    np.testing.assert_allclose(ds, (2.0 / 7) * (2 * s - t - y), rtol=1e-14)


def test_adam_first_step_closed_form_and_torch():
    rng = np.random.default_rng(7)
    p = rng.standard_normal(50)
    g = rng.standard_normal(50) * np.logspace(-6, 1, 50)
    p1, m1, v1 = om.adam_update(p, g, np.zeros(50), np.zeros(50), 1, 1e-3)
    # at step 1 the bias-corrected moments are g and g^2
    np.testing.assert_allclose(p1, p - 1e-3 * g / (np.abs(g) + 1e-8), rtol=1e-13)
    # a few more steps against torch.optim.Adam
    pt = torch.tensor(p, requires_grad=True)
    opt = torch.optim.Adam([pt], lr=1e-3, betas=(0.9, 0.999), eps=1e-8)
    pp, m, v = p.copy(), np.zeros(50), np.zeros(50)
    for step in range(1, 5):
        gs = g * (1 + 0.1 * step)
        pt.grad = torch.tensor(gs)
        opt.step()
        pp, m, v = om.adam_update(pp, gs, m, v, step, 1e-3)
    np.testing.assert_allclose(pp, pt.detach().numpy(), rtol=1e-12, atol=1e-15)


def test_distill_step_moves_loss_down():
    shape, blob, X, lengths = _tiny(seed=8, Bn=6, L=6)
    cfg = _cfg(shape)
    tshape, tblob, _, _ = _tiny(seed=9, Bn=6, L=6)
    labels = np.zeros(6)
    r = om.distill_step(tblob, cfg, blob, cfg, X, lengths, labels, lr=1e-2)
    r2 = om.distill_step(tblob, cfg, r["params"], cfg, X, lengths, labels, m=r["m"], v=r["v"], step=2, lr=1e-2)
    assert r2["loss"][0] < r["loss"][0]
