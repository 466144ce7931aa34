"""Pins of the progressive KB + AC forward (section 6, Fig. 6, Eq. (7)).

The oracle is checked against an independent torch re-expression of both
columns (torch Linear/ReLU/RMSNorm, the SSM in its explicit convolution
form, the KB's layer inputs captured as it runs), against the plain model
when every alpha is zero, and against structural facts of Eq. (7): an AC
layer reads the KB's input to the same layer (so the KB's output layer
feeds nothing), the score is affine in the last layer's alpha, and the KB
reaches the AC through every lateral."""
import numpy as np
import pytest
import torch

from oracle import model as om
from oracle import progressive as op
from paper_2604_12891_amd import workload as wl
from tests.test_oracle_model import _cfg, _torch_block, _torch_pool

F = torch.nn.functional

BASE = wl.ModelShape(F=6, d_model=4, d_inner=8, d_state=3, d_conv=4, dt_rank=2, n_layers=2, head_hidden=5)
VARIANT = wl.ModelShape(F=5, d_model=4, d_inner=4, d_state=2, d_conv=4, dt_rank=2, n_layers=1,
                        head_hidden=6, enc_hidden=(3, 7), dec_hidden2=3)


def _draw(shape, a, seed, Bn=4, L=7):
    rng = np.random.default_rng(seed)
    kb = wl.init_params(shape, rng, perturb=True).astype(np.float64)
    ac = wl.init_params(shape, rng, perturb=True).astype(np.float64)
    lat = wl.init_lateral(shape, a, rng).astype(np.float64)
    X, lengths = wl.make_inputs(Bn, L, shape.F, 1, L, rng)
    return kb, ac, lat, X.astype(np.float64), lengths


def _torch_column(Pt, X, lengths, cfg, Q=None, kb_in=None):
    """Both columns in torch; returns (scores, inputs of every layer)."""
    ins, i = [], 0

    def lat(pre):
        if Q is None or i == 0:
            return pre
        p = f"lat{i - 1}."
        return pre + Q[p + "alpha"] * F.linear(F.relu(F.linear(kb_in[i], Q[p + "V"], Q[p + "c"])), Q[p + "U"])

    h = X
    n_enc = len(cfg.get("enc_hidden", ())) + 1
    for e in range(n_enc):
        ins.append(h)
        sfx = f"_{e}" if e else ""
        pre = lat(F.linear(h, Pt[f"W0{sfx}"], Pt[f"b0{sfx}"]))
        h = F.relu(pre) if e < n_enc - 1 else pre
        i += 1
    for l in range(cfg["n_layers"]):
        ins.append(h)
        h = lat(_torch_block(h, Pt, l, cfg))
        i += 1
    v = _torch_pool(h, Pt, lengths, cfg)
    dec = [("W1", "b1"), ("W2", "b2")] + ([("W3", "b3")] if cfg.get("dec_hidden2", 0) else [])
    for k, (wn, bn) in enumerate(dec):
        ins.append(v)
        pre = lat(F.linear(v, Pt[wn], Pt[bn]))
        v = F.relu(pre) if k < len(dec) - 1 else pre
        i += 1
    return v[:, 0], ins


def _t(d):
    return {k: torch.tensor(v, dtype=torch.float64) for k, v in d.items()}


def test_lateral_layout_matches_generator():
    for shape in (BASE, VARIANT, wl.PAPER_CPU, wl.D256):
        for a in (4, 8):
            assert [(n, tuple(s)) for n, s in op.lateral_layout(_cfg(shape), a)] == \
                   [(n, tuple(s)) for n, s in wl.lateral_layout(shape, a)]


@pytest.mark.parametrize("shape,a", [(BASE, 3), (BASE, 8), (VARIANT, 5)])
def test_progressive_matches_torch_reexpression(shape, a):
    kb, ac, lat, X, lengths = _draw(shape, a, 1)
    cfg = _cfg(shape)
    s = op.progressive_scores(kb, ac, lat, a, X, lengths, cfg)
    Xt = torch.from_numpy(X)
    _, kb_in = _torch_column(_t(om.unpack(kb, cfg)), Xt, lengths, cfg)
    st, _ = _torch_column(_t(om.unpack(ac, cfg)), Xt, lengths, cfg, _t(op.unpack_lateral(lat, cfg, a)), kb_in)
    np.testing.assert_allclose(s, st.numpy(), rtol=1e-11, atol=1e-13)
    # and the KB column alone is the plain model
    np.testing.assert_allclose(op.kb_forward(kb, X, lengths, cfg)[0], om.score(kb, X, lengths, cfg), rtol=1e-13)


def test_zero_alpha_gives_the_plain_model():
    for shape in (BASE, VARIANT):
        kb, ac, lat, X, lengths = _draw(shape, 4, 2)
        cfg = _cfg(shape)
        Q = op.unpack_lateral(lat, cfg, 4)
        for k in Q:
            if k.endswith("alpha"):
                Q[k][:] = 0.0
        flat = np.concatenate([Q[n].reshape(-1) for n, _ in op.lateral_layout(cfg, 4)])
        np.testing.assert_allclose(op.progressive_scores(kb, ac, flat, 4, X, lengths, cfg),
                                   om.score(ac, X, lengths, cfg), rtol=1e-13)


def test_lateral_reads_the_kb_input_of_the_same_layer():
    """No AC layer reads the KB's output layer: changing the KB's last
    decoder layer leaves the AC's scores alone, while changing the KB's first
    encoder layer or its second-to-last decoder layer changes them."""
    for shape in (BASE, VARIANT):
        kb, ac, lat, X, lengths = _draw(shape, 4, 3)
        cfg = _cfg(shape)
        s0 = op.progressive_scores(kb, ac, lat, 4, X, lengths, cfg)
        P = om.unpack(kb, cfg)
        last = "W3" if shape.dec_hidden2 else "W2"
        prev = "W2" if shape.dec_hidden2 else "W1"
        for name, moves in [(last, False), ("W0", True), (prev, True)]:
            Q = {k: v.copy() for k, v in P.items()}
            Q[name] = Q[name] * 1.7 + 0.1
            s1 = op.progressive_scores(om.pack(Q, cfg), ac, lat, 4, X, lengths, cfg)
            if moves:
                assert not np.allclose(s1, s0, rtol=1e-9), name
            else:
                np.testing.assert_array_equal(s1, s0)


def test_score_is_affine_in_the_last_alpha():
    """The score layer has no outer activation: s(t alpha_last) is affine in t."""
    kb, ac, lat, X, lengths = _draw(VARIANT, 4, 4)
    cfg = _cfg(VARIANT)
    Q = op.unpack_lateral(lat, cfg, 4)
    j = len(op.layer_widths(cfg)) - 2
    names = [n for n, _ in op.lateral_layout(cfg, 4)]

    def at(t):
        R = {k: v.copy() for k, v in Q.items()}
        R[f"lat{j}.alpha"] = Q[f"lat{j}.alpha"] * t
        return op.progressive_scores(kb, ac, np.concatenate([R[n].reshape(-1) for n in names]), 4, X, lengths, cfg)

    s0, s1, s3 = at(0.0), at(1.0), at(3.0)
    np.testing.assert_allclose(s3 - s0, 3.0 * (s1 - s0), rtol=1e-11, atol=1e-14)
    assert not np.allclose(s1, s0)


def test_first_layer_has_no_lateral_and_each_lateral_matters():
    """There is one adapter per layer after the first; zeroing any single
    adapter's alpha changes the scores (decoder widths of 8, so that no
    ReLU layer is dead on every program of the batch)."""
    shape = wl.ModelShape(F=5, d_model=4, d_inner=4, d_state=2, d_conv=4, dt_rank=2, n_layers=1,
                          head_hidden=8, enc_hidden=(3, 7), dec_hidden2=8)
    kb, ac, lat, X, lengths = _draw(shape, 4, 5, Bn=8)
    cfg = _cfg(shape)
    assert len(op.lateral_layout(cfg, 4)) == 4 * (len(op.layer_widths(cfg)) - 1)
    s0 = op.progressive_scores(kb, ac, lat, 4, X, lengths, cfg)
    Q = op.unpack_lateral(lat, cfg, 4)
    names = [n for n, _ in op.lateral_layout(cfg, 4)]
    for j in range(len(op.layer_widths(cfg)) - 1):
        R = {k: v.copy() for k, v in Q.items()}
        R[f"lat{j}.alpha"][:] = 0.0
        s1 = op.progressive_scores(kb, ac, np.concatenate([R[n].reshape(-1) for n in names]), 4, X, lengths, cfg)
        assert not np.allclose(s1, s0, rtol=1e-12), j
