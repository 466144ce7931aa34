"""Pins of the oracle's form of the paper's own model (section 5.2: a
three-layer encoder 64/128/128 and decoder 64/32/1 around one Mamba block
with Table 2's best hyper-parameters [1, 8, 1, 4]) and of the Top-k score
(Eq. (12)).

The model size is pinned to the paper's 0.35 MB (Table 3); the forward pass
to the independent torch re-expression (library Linear/ReLU/RMSNorm, the
SSM in its explicit convolution form); the layer stacks to reductions that
must give back the one-Linear encoder and two-layer decoder. The Top-k score
is pinned to a hand-worked pair of subgraphs, a rank-counting brute force
and the metric's limits."""
import numpy as np
import pytest
import torch

from oracle import metric as omet
from oracle import model as om
from paper_2604_12891_amd import workload as wl
from tests.test_oracle_model import _cfg, _torch_model_scores


def _draw(shape, seed, Bn, L):
    rng = np.random.default_rng(seed)
    blob = wl.init_params(shape, rng, perturb=True).astype(np.float64)
    X, lengths = wl.make_inputs(Bn, L, shape.F, 1, L, rng)
    return blob, X.astype(np.float64), lengths


def test_paper_model_size_is_035_mb():
    """Table 3 gives the model 0.35 MB: 92,097 fp32 values for the 26 x 22
    CPU features (91,969 for 41 x 20) are 0.351 MiB."""
    for shape, n in ((wl.PAPER_CPU, 92097), (wl.PAPER_GPU, 91969)):
        count = sum(int(np.prod(s)) for _, s in om.layout(_cfg(shape)))
        assert count == n
        assert round(count * 4 / 2**20, 2) == 0.35


TINY_VARIANT = wl.ModelShape(F=5, d_model=4, d_inner=4, d_state=2, d_conv=4, dt_rank=2, n_layers=1,
                             head_hidden=6, enc_hidden=(3, 7), dec_hidden2=3)


@pytest.mark.parametrize("shape,Bn,L", [(TINY_VARIANT, 4, 7), (wl.PAPER_CPU, 3, 6), (wl.PAPER_GPU, 2, 9)])
def test_variant_forward_matches_torch_reexpression(shape, Bn, L):
    blob, X, lengths = _draw(shape, 11, Bn, L)
    cfg = _cfg(shape)
    P = om.unpack(blob, cfg)
    s = om.forward(P, X, lengths, cfg)
    Pt = {k: torch.tensor(v, dtype=torch.float64) for k, v in P.items()}
    st = _torch_model_scores(Pt, torch.from_numpy(X), lengths, cfg)
    np.testing.assert_allclose(s, st.numpy(), rtol=1e-11, atol=1e-13)


def test_relu_sits_between_layers_not_after_the_last():
    """With the block switched off (W_out = 0) and eps ~ 0, RMSNorm is odd, so
    negating the last encoder layer (no ReLU after it) equals negating W1.
    Negating a hidden layer instead is not the same as negating the layer
    after it, because a ReLU sits between them."""
    shape = TINY_VARIANT
    blob, X, lengths = _draw(shape, 5, 4, 7)
    cfg = dict(_cfg(shape), norm_eps=1e-300)
    P0 = om.unpack(blob, _cfg(shape))
    P0["blk0.W_out"][:] = 0.0

    def flip(P, *names):
        Q = {k: v.copy() for k, v in P.items()}
        for n in names:
            Q[n] *= -1.0
        return Q

    np.testing.assert_allclose(om.forward(flip(P0, "W0_2", "b0_2"), X, lengths, cfg),
                               om.forward(flip(P0, "W1"), X, lengths, cfg), rtol=1e-12, atol=1e-12)
    assert not np.allclose(om.forward(flip(P0, "W0_1", "b0_1"), X, lengths, cfg),
                           om.forward(flip(P0, "W0_2"), X, lengths, cfg))


def test_stacks_reduce_to_the_one_layer_forms():
    """Encoder F -> d -> d with an identity second layer and non-negative
    first-layer pre-activations is the one-Linear encoder; decoder
    d -> h -> h -> 1 with an identity middle layer is the two-layer one."""
    d, h = 4, 6
    var = wl.ModelShape(F=5, d_model=d, d_inner=8, d_state=3, d_conv=3, dt_rank=2, n_layers=2,
                        head_hidden=h, enc_hidden=(d,), dec_hidden2=h)
    base = wl.ModelShape(F=5, d_model=d, d_inner=8, d_state=3, d_conv=3, dt_rank=2, n_layers=2,
                         head_hidden=h)
    blob, X, lengths = _draw(var, 8, 5, 6)
    cv, cb = _cfg(var), _cfg(base)
    P = om.unpack(blob, cv)
    P["W0"] = np.abs(P["W0"])
    P["b0"] = np.abs(P["b0"])  # features are >= 0, so W0 x + b0 >= 0
    P["W0_1"] = np.eye(d)
    P["b0_1"] = np.zeros(d)
    P["W2"] = np.eye(h)
    P["b2"] = np.zeros(h)
    Pb = {k: v for k, v in P.items() if k in dict(om.layout(cb))}
    Pb["W2"], Pb["b2"] = P["W3"], P["b3"]
    np.testing.assert_allclose(om.forward(P, X, lengths, cv), om.forward(Pb, X, lengths, cb), rtol=1e-13)


# ---------------------------------------------------------------- Eq. (12)

def test_topk_score_hand_worked():
    """Subgraph A (weight 2): latencies 3, 1, 2 with scores 0.9, 0.1, 0.5,
    ranked 0, 2, 1. Subgraph B (weight 1): latencies 4, 5 with scores 0.2,
    0.3, ranked 1, 0. Top-1 = (2*1 + 4) / (2*3 + 5), Top-2 = 6 / (2*2 + 4),
    Top-3 = 1."""
    lat = [3.0, 1.0, 2.0, 4.0, 5.0]
    sc = np.array([0.9, 0.1, 0.5, 0.2, 0.3], np.float32)
    offs, w = [0, 3, 5], [2.0, 1.0]
    assert omet.top_k_score(sc, lat, offs, w, 1)[0] == pytest.approx(6.0 / 11.0, rel=1e-15)
    assert omet.top_k_score(sc, lat, offs, w, 2)[0] == pytest.approx(0.75, rel=1e-15)
    assert omet.top_k_score(sc, lat, offs, w, 3)[0] == 1.0


def _brute_top_k(scores, lat, offs, w, k):
    """Rank of i = how many candidates of its subgraph come before it (a
    larger score, or an equal one at a lower index; NaN after numbers)."""
    num = den = 0.0
    for g in range(len(offs) - 1):
        idx = list(range(offs[g], offs[g + 1]))
        if not idx:
            continue

        def before(j, i):
            sj, si = scores[j], scores[i]
            if np.isnan(si) and not np.isnan(sj):
                return True
            if np.isnan(sj) and not np.isnan(si):
                return False
            if np.isnan(si) and np.isnan(sj):
                return j < i
            return sj > si or (sj == si and j < i)

        rank = {i: sum(before(j, i) for j in idx if j != i) for i in idx}
        num += w[g] * min(lat[i] for i in idx)
        den += w[g] * min(lat[i] for i in idx if rank[i] < k)
    return num / den


def test_topk_score_against_rank_counting():
    rng = np.random.default_rng(21)
    for trial in range(15):
        sizes = rng.integers(0, 25, size=6)
        offs = np.concatenate([[0], np.cumsum(sizes)])
        n = int(offs[-1])
        sc = (np.round(rng.standard_normal(n) * 3) / 3).astype(np.float32)  # ties
        sc[rng.random(n) < 0.1] = np.nan
        lat = rng.lognormal(0.0, 1.0, n)
        w = rng.integers(1, 5, size=6).astype(float)
        for k in (1, 3, 10):
            got = omet.top_k_score(sc, lat, offs, w, k)[0]
            assert got == pytest.approx(_brute_top_k(sc, lat, offs, w, k), rel=1e-14)


def test_topk_score_limits():
    rng = np.random.default_rng(22)
    offs = np.array([0, 40, 41, 100, 100, 160])
    n = int(offs[-1])
    lat = rng.lognormal(0.0, 0.5, n)
    w = np.array([1.0, 3.0, 2.0, 5.0, 1.0])
    perfect = (-lat).astype(np.float32)   # predicts the latency order (fp32 keeps it here)
    assert len(np.unique(perfect)) == n
    for k in (1, 5, 60):
        assert omet.top_k_score(perfect, lat, offs, w, k)[0] == 1.0
    sc = rng.standard_normal(n).astype(np.float32)
    vals = [omet.top_k_score(sc, lat, offs, w, k)[0] for k in range(1, 62)]
    assert all(0.0 < v <= 1.0 for v in vals)
    assert all(b >= a for a, b in zip(vals, vals[1:]))     # more candidates can only help
    assert vals[-1] == 1.0                                 # k >= every subgraph's size
    worst = lat.astype(np.float32)                         # predicts the reverse order
    mins = [lat[a:b].min() for a, b in zip(offs[:-1], offs[1:]) if b > a]
    maxs = [lat[a:b].max() for a, b in zip(offs[:-1], offs[1:]) if b > a]
    ws = [w[g] for g in range(5) if offs[g + 1] > offs[g]]
    assert omet.top_k_score(worst, lat, offs, w, 1)[0] == pytest.approx(np.dot(ws, mins) / np.dot(ws, maxs),
                                                                         rel=1e-14)
