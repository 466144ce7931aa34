"""The C ABI without a GPU: the library loads, exports every entry point that
include/tcl.h declares, and rejects bad arguments before touching a device."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import model as om
from paper_2604_12891_amd import binding as tb
from paper_2604_12891_amd import workload as wl

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "tcl.h")


def declared_symbols():
    text = open(HEADER).read()
    return re.findall(r"TCL_API\s+[\w\s\*]+?\b(tcl_\w+)\s*\(", text)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(tb.lib_path()):
        pytest.fail("libtcl.so is not built (run __graft_entry__.build())")
    return tb.lib()


def test_exports_every_declared_symbol(lib):
    names = declared_symbols()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
    # and the binding declares a signature for each of them
    assert set(names) <= set(tb._SIGS)


@pytest.mark.parametrize("shape", [wl.TINY, wl.D256, wl.STUDENT, wl.PAPER_CPU, wl.PAPER_GPU])
def test_param_count_matches_oracle_layout(lib, shape):
    cfg = tb.config_from_shape(shape)
    n = lib.tcl_param_count(ctypes.byref(cfg))
    ocfg = dict(F=shape.F, d_model=shape.d_model, d_inner=shape.d_inner, d_state=shape.d_state,
                d_conv=shape.d_conv, dt_rank=shape.dt_rank, n_layers=shape.n_layers,
                head_hidden=shape.head_hidden, enc_hidden=shape.enc_hidden, dec_hidden2=shape.dec_hidden2)
    assert n == sum(int(np.prod(s)) for _, s in om.layout(ocfg)) == wl.param_count(shape)


def _create(lib, cfg, blob, n=None):
    h = ctypes.c_void_p()
    st = lib.tcl_cost_model_create(ctypes.byref(cfg) if cfg is not None else None,
                                   blob.ctypes.data if blob is not None else None,
                                   (0 if blob is None else blob.size) if n is None else n, ctypes.byref(h))
    return st, h


def test_create_rejects_bad_arguments(lib):
    cfg = tb.config_from_shape(wl.TINY)
    blob = np.zeros(wl.param_count(wl.TINY), np.float32)
    st, h = _create(lib, None, blob)
    assert st == -1 and h.value is None
    st, _ = _create(lib, cfg, None)
    assert st == -1
    st, _ = _create(lib, cfg, blob, n=blob.size - 1)
    assert st == -1 and b"needs" in lib.tcl_last_error()
    for field, value in [("d_state", 4), ("d_model", 96), ("dt_rank", 6), ("head_hidden", 300), ("F", 2000),
                         ("d_conv", 5), ("dec_hidden2", 300)]:
        bad = tb.config_from_shape(wl.TINY)
        setattr(bad, field, value)
        st, _ = _create(lib, bad, np.zeros(lib.tcl_param_count(ctypes.byref(bad)), np.float32))
        assert st == -2, field
    # the multi-layer encoder: fp32 only, widths multiples of 4, no e2 without e1
    for shape, dtype, enc, want in [(wl.TINY, "bf16", (64, 128), -2), (wl.TINY, "f32", (62, 0), -2),
                                    (wl.TINY, "f32", (0, 64), -1)]:
        bad = tb.config_from_shape(shape, dtype)
        bad.enc_hidden[0], bad.enc_hidden[1] = enc
        st, _ = _create(lib, bad, np.zeros(lib.tcl_param_count(ctypes.byref(bad)), np.float32))
        assert st == want, (dtype, enc)
    bad = tb.config_from_shape(wl.PAPER_CPU)
    bad.dt_rank = 12  # d_state 8 takes dt_rank 4, 8 or 16
    st, _ = _create(lib, bad, np.zeros(lib.tcl_param_count(ctypes.byref(bad)), np.float32))
    assert st == -2
    bad = tb.config_from_shape(wl.TINY)
    bad.norm_eps = 0.0
    st, _ = _create(lib, bad, blob)
    assert st == -1
    bad = tb.config_from_shape(wl.TINY)
    bad.f32_matmul = 3
    st, _ = _create(lib, bad, blob)
    assert st == -1 and b"f32_matmul" in lib.tcl_last_error()


def test_calls_on_null_handles(lib):
    assert lib.tcl_cost_model_destroy(None) == 0
    assert lib.tcl_score(None, 1, 1, None, None, None, None, 0, None) == -1
    assert lib.tcl_score_workspace_bytes(None, 4, 4) == 0
    assert lib.tcl_get_params(None, None, 0) == -1
    assert lib.tcl_test_gemm_f32(0, 4, 4, None, None, None, None, -1, 0, None) == -1
    assert lib.tcl_test_scan_f32(1, 16, 8, 4, 0, *([None] * 4), 16, *([None] * 6)) in (-1, -2)
    assert lib.tcl_teacher_gate(0, None, None, None) == -1
    assert lib.tcl_teacher_gate(4, None, None, None) == -1
    assert lib.tcl_test_distill_step_kd_ranked(None, 1, 1, *([None] * 8), 0, None) == -1


def test_split_gemm_entry_rejects_bad_arguments(lib):
    """Argument checks of tcl_test_gemm_split run on the host."""
    fake = 1 << 20
    args = dict(M=8, N=8, K=8, A=fake, offs=None, B=0, L=0, W=fake, bias=None, C=fake, variant=-1,
                epilogue=0, Wsplit=fake, stream=None)

    def call(**kw):
        a = dict(args, **kw)
        return lib.tcl_test_gemm_split(*a.values())

    assert call(K=6) == -1            # K % 4
    assert call(variant=8) == -1
    assert call(epilogue=4) == -1
    assert call(epilogue=3) == -1     # the gather needs offsets and B, L
    assert call(epilogue=3, offs=fake, B=2, L=3) == -1  # ... and the bias
    assert call(epilogue=1, bias=fake) == -1
    assert call(Wsplit=None) == -1
    assert call(A=fake + 4) == -1     # alignment
    assert call(K=320, variant=1) == -2
    assert call(K=320, variant=2) == -2
    assert call(N=300, variant=3) == -2
    assert call(K=600, variant=3) == -2


def test_bf16_gemm_entry_rejects_bad_arguments(lib):
    """Argument checks run on the host, before any device work."""
    fake = 1 << 20  # never dereferenced: every call below fails its checks first
    args = dict(kind=0, tile=-1, M=8, N=8, K=8, A=fake, offs=None, B=0, L=0, W=fake, bias=None, gain=None,
                C=fake, stream=None)

    def call(**kw):
        a = dict(args, **kw)
        return lib.tcl_test_gemm_bf16(*a.values())

    assert call(kind=7) == -1
    assert call(kind=-1) == -1
    assert call(tile=9) == -1
    assert call(N=6) == -1            # N % 4
    assert call(K=12) == -1           # bf16 A needs K % 8
    assert call(kind=5, K=6) == -1    # fp32 A needs K % 4
    assert call(A=None) == -1
    assert call(kind=2) == -1         # the RMSNorm variant needs the gain
    assert call(kind=4) == -1         # the gather needs offsets and B, L
    assert call(kind=4, offs=fake, B=2, L=3) == -1  # ... and the bias
    assert call(C=fake + 4) == -1     # alignment


def test_offsets_entry_rejects_bad_arguments(lib):
    """Argument checks run on the host, before any device work."""
    fake = 1 << 20  # never dereferenced
    assert lib.tcl_test_offsets(0, 25, fake, fake, None, None) == -1
    assert lib.tcl_test_offsets(4, 0, fake, fake, None, None) == -1
    assert lib.tcl_test_offsets(4, 25, None, fake, None, None) == -1
    assert lib.tcl_test_offsets(4, 25, fake, None, fake, None) == -1


@pytest.mark.parametrize("shape", [wl.TINY, wl.PAPER_CPU])
def test_lateral_param_count_matches_oracle_layout(lib, shape):
    from oracle import progressive as op
    cfg = tb.config_from_shape(shape)
    ocfg = dict(F=shape.F, d_model=shape.d_model, d_inner=shape.d_inner, d_state=shape.d_state,
                d_conv=shape.d_conv, dt_rank=shape.dt_rank, n_layers=shape.n_layers,
                head_hidden=shape.head_hidden, enc_hidden=shape.enc_hidden, dec_hidden2=shape.dec_hidden2)
    for a in (4, 8, 32):
        n = lib.tcl_lateral_param_count(ctypes.byref(cfg), a)
        assert n == sum(int(np.prod(s)) for _, s in op.lateral_layout(ocfg, a))
        assert n == sum(int(np.prod(s)) for _, s in wl.lateral_layout(shape, a))
    assert lib.tcl_lateral_param_count(ctypes.byref(cfg), 0) == 0


def test_progressive_calls_on_null_handles(lib):
    h = ctypes.c_void_p()
    assert lib.tcl_lateral_create(None, None, 8, None, 0, ctypes.byref(h)) == -1 and h.value is None
    assert lib.tcl_lateral_destroy(None) == 0
    assert lib.tcl_progressive_workspace_bytes(None, 4, 4) == 0
    assert lib.tcl_progressive_score(None, 1, 1, None, None, None, None, 0, None) == -1
