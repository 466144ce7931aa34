"""The seeded generator: reproducible, and its weights follow the init recipe."""
import math

import numpy as np
import pytest
import scipy.stats

from paper_2604_12891_amd import workload as wl


def test_reproducible():
    p1, X1, l1 = wl.make_workload("score_B64_L25_d64_f32")
    p2, X2, l2 = wl.make_workload("score_B64_L25_d64_f32")
    assert np.array_equal(p1, p2) and np.array_equal(X1, X2) and np.array_equal(l1, l2)


def test_inputs_recipe():
    _, X, lengths = wl.make_workload("score_B64_L25_d64_f32", B=512)
    assert X.dtype == np.float32 and lengths.dtype == np.int32
    assert lengths.min() >= 5 and lengths.max() <= 25
    pad = np.arange(25)[None, :] >= lengths[:, None]
    assert np.all(X[pad] == 0) and np.all(X[~pad] > 0)
    # features are log1p of a lognormal(0,1): exp(x)-1 is lognormal
    z = np.log(np.expm1(X[~pad].ravel()[:20000].astype(np.float64)))
    assert scipy.stats.kstest(z, "norm").pvalue > 1e-4


def test_init_recipe():
    shape = wl.D256
    P = wl.unpack(wl.init_params(shape, np.random.default_rng(0)), shape)
    assert np.abs(P["W0"]).max() <= 1 / math.sqrt(164)
    assert np.abs(P["blk0.W_in"]).max() <= 1 / math.sqrt(256)
    assert np.abs(P["blk0.W_out"]).max() <= 1 / math.sqrt(512)
    assert np.abs(P["blk0.W_dt"]).max() <= 1 / math.sqrt(16)
    np.testing.assert_array_equal(P["blk1.A_log"], np.tile(np.log(np.arange(1, 17)), (512, 1)).astype(np.float32))
    assert np.all(P["blk2.D"] == 1) and np.all(P["g_f"] == 1)
    dt0 = np.logaddexp(0.0, P["blk3.b_dt"].astype(np.float64))
    assert dt0.min() >= 1e-3 * (1 - 1e-5) and dt0.max() <= 1e-1 * (1 + 1e-5)
    u = (np.log(dt0) - math.log(1e-3)) / (math.log(1e-1) - math.log(1e-3))
    assert scipy.stats.kstest(u, "uniform").pvalue > 1e-3


def test_bf16_rounding():
    a = np.array([1.0, 1.00390625, 1.005859375, -3.14159, 1e-30, 65504.0], dtype=np.float32)
    r = wl.round_to_bf16(a)
    assert np.all((r.view(np.uint32) & 0xFFFF) == 0)
    t = np.asarray(__import__("torch").tensor(a).bfloat16().float())
    np.testing.assert_array_equal(r, t)


def test_distill_workload_pair():
    (t, s), X, lengths = wl.make_workload("distill_B1024_L25_t256_s128_bf16", B=8)
    assert t.size == wl.param_count(wl.D256) and s.size == wl.param_count(wl.STUDENT)
    assert np.all((s.view(np.uint32) & 0xFFFF) == 0)


@pytest.mark.parametrize("name", ["score_B4096_L25_d256_f32", "score_B65536_L25_d256_bf16",
                                  "score_B8192_L256_d256_f32"])
def test_golden_scores_are_the_oracles(name):
    """The stored full-batch scores were written from today's generator
    (digest) and are the oracle's: a seeded sample of programs, including
    the first and the last, rescored by the oracle here agrees to rounding."""
    from oracle import model as om
    from tests.parity import golden_scores, oracle_cfg

    w = wl.WORKLOADS[name]
    blob, X, lengths = wl.make_workload(name)
    g = golden_scores(name, blob, X, lengths)
    assert g.shape == (w.B,) and np.all(np.isfinite(g))
    idx = np.unique(np.concatenate([[0, w.B - 1], np.random.default_rng(7).choice(w.B, 6, replace=False)]))
    o = om.score(blob, X[idx], lengths[idx], oracle_cfg(w.model))
    np.testing.assert_allclose(g[idx], o, rtol=1e-12, atol=1e-14)
