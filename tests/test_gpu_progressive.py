"""Parity of the progressive KB + AC forward (tcl_progressive_score, Eq. (7))
with the fp64 oracle (oracle/progressive.py) on the same seeded inputs.

The AC's scores are held to the fp32 score tolerance and ranking check of
the other scoring tests: every layer is the same fp32 arithmetic as
tcl_score plus two fp32 GEMMs per adapter."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import progressive as op
from paper_2604_12891_amd import binding as tb
from paper_2604_12891_amd import workload as wl
from tests.parity import assert_scores_match, oracle_cfg
from tests.test_gpu_score import _sample

pytestmark = pytest.mark.gpu

NAME = "progressive_B4096_L41_F20_a8_f32"


def _prog(shape, kb, ac, lat, a, f32_matmul="split"):
    cfg = tb.config_from_shape(shape, "f32", f32_matmul)
    K, A = tb.CostModel(cfg, kb), tb.CostModel(cfg, ac)
    return tb.Progressive(K, A, a, lat)


def _run(p, X, lengths):
    out = p.score(torch.from_numpy(X).cuda(), torch.from_numpy(lengths).cuda())
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _oracle(shape, kb, ac, lat, a, X, lengths):
    return op.progressive_scores(kb, ac, lat, a, X, lengths, oracle_cfg(shape))


@pytest.mark.parametrize("f32_matmul", ["split", "native"])
def test_paper_model_progressive_small_batch(f32_matmul):
    w = wl.WORKLOADS[NAME]
    print(f"tcl_progressive_score {NAME} B=300 {f32_matmul}", flush=True)
    (kb, ac, lat), X, lengths = wl.make_workload(NAME, B=300, perturb=True)
    g = _run(_prog(w.model, kb, ac, lat, w.adapter, f32_matmul), X, lengths)
    assert_scores_match(g, _oracle(w.model, kb, ac, lat, w.adapter, X, lengths), "f32", NAME)


def test_paper_model_progressive_full_size_sampled():
    w = wl.WORKLOADS[NAME]
    print(f"tcl_progressive_score {NAME} full batch", flush=True)
    (kb, ac, lat), X, lengths = wl.make_workload(NAME)
    g = _run(_prog(w.model, kb, ac, lat, w.adapter), X, lengths)
    assert np.all(np.isfinite(g))
    idx = _sample(lengths, 64)
    assert_scores_match(g[idx], _oracle(w.model, kb, ac, lat, w.adapter, X[idx], lengths[idx]), "f32", NAME)


@pytest.mark.parametrize("a", [4, 8, 16, 64])
def test_base_architecture_progressive(a):
    """The one-Linear encoder, two blocks with d_state 16, the two-layer
    decoder; adapter widths 4, 8 and 16 (the fused per-row adapter kernel)
    and 64 (= d, two GEMMs)."""
    shape = wl.TINY
    rng = np.random.default_rng(60 + a)
    kb = wl.init_params(shape, rng, perturb=True)
    ac = wl.init_params(shape, rng, perturb=True)
    lat = wl.init_lateral(shape, a, rng)
    X, lengths = wl.make_inputs(130, 25, shape.F, 1, 25, rng)
    print(f"tcl_progressive_score tiny a={a}", flush=True)
    g = _run(_prog(shape, kb, ac, lat, a), X, lengths)
    assert_scores_match(g, _oracle(shape, kb, ac, lat, a, X, lengths), "f32", f"tiny a={a}")


def test_zero_alpha_equals_plain_scoring_and_invalid_lengths():
    """alpha = 0 gives tcl_score of the AC; an invalid length gives NaN on
    both entry points."""
    shape = wl.PAPER_CPU
    rng = np.random.default_rng(70)
    kb = wl.init_params(shape, rng, perturb=True)
    ac = wl.init_params(shape, rng, perturb=True)
    lat = wl.init_lateral(shape, 8, rng)
    names = [n for n, _ in wl.lateral_layout(shape, 8)]
    parts, off = [], 0
    for n, s in wl.lateral_layout(shape, 8):
        k = int(np.prod(s))
        v = lat[off:off + k].copy()
        if n.endswith("alpha"):
            v[:] = 0.0
        parts.append(v)
        off += k
    lat0 = np.concatenate(parts)
    assert len(names) and off == lat.size
    X, lengths = wl.make_inputs(40, 26, shape.F, 1, 26, rng)
    lengths[[3, 17]] = [0, 27]
    print("tcl_progressive_score alpha=0", flush=True)
    p = _prog(shape, kb, ac, lat0, 8)
    g = _run(p, X, lengths)
    s = p.ac.score(torch.from_numpy(X).cuda(), torch.from_numpy(lengths).cuda())
    torch.cuda.synchronize()
    s = s.cpu().numpy()
    assert np.isnan(g[3]) and np.isnan(g[17]) and np.isnan(s[3]) and np.isnan(s[17])
    ok = np.ones(40, bool)
    ok[[3, 17]] = False
    np.testing.assert_allclose(g[ok], s[ok], rtol=1e-5, atol=1e-6)


def test_one_program():
    w = wl.WORKLOADS[NAME]
    (kb, ac, lat), X, lengths = wl.make_workload(NAME, B=5, perturb=True)
    print("tcl_progressive_score B=1", flush=True)
    g = _run(_prog(w.model, kb, ac, lat, w.adapter), X[:1], lengths[:1])
    assert_scores_match(g, _oracle(w.model, kb, ac, lat, w.adapter, X[:1], lengths[:1]), "f32", "B=1")


def test_create_rejects_bad_arguments():
    L = tb.lib()
    shape = wl.TINY
    rng = np.random.default_rng(1)
    blob = wl.init_params(shape, rng)
    f32 = tb.CostModel(tb.config_from_shape(shape), blob)
    f32b = tb.CostModel(tb.config_from_shape(shape), blob)
    bf = tb.CostModel(tb.config_from_shape(shape, "bf16"), wl.round_to_bf16(blob))
    bf2 = tb.CostModel(tb.config_from_shape(shape, "bf16"), wl.round_to_bf16(blob))
    other_shape = wl.ModelShape(d_model=64, d_inner=128, dt_rank=8, n_layers=2, head_hidden=64)
    other = tb.CostModel(tb.config_from_shape(other_shape), wl.init_params(other_shape, rng))
    lat = wl.init_lateral(shape, 8, rng)
    h = ctypes.c_void_p()

    def create(k, a, adapter=8, params=lat, n=None):
        return L.tcl_lateral_create(k.handle, a.handle, adapter, params.ctypes.data,
                                    params.size if n is None else n, ctypes.byref(h))

    assert create(f32, f32) == -1                  # the same model twice
    assert create(f32, other) == -1               # architectures differ
    assert create(bf, bf2) == -2                  # fp32 models only
    assert create(f32, f32b, adapter=6) == -2
    assert create(f32, f32b, n=lat.size - 1) == -1
    assert create(f32, f32b) == 0
    assert L.tcl_lateral_destroy(h) == 0
