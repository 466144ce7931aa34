"""tcl_score_noalloc (the scoring entry point that allocates nothing, for
callers under graph capture or in serving loops) against tcl_score: the same
scores bit for bit on two calls in a row, the second with a smaller batch,
through the C ABI; batches beyond the library's scratch buffer are refused
before anything is enqueued."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2604_12891_amd import binding as tb
from paper_2604_12891_amd import workload as wl

pytestmark = pytest.mark.gpu


def _noalloc(lib, m, X, lengths, stream=None):
    B, L, _ = X.shape
    out = torch.full((B,), float("nan"), device="cuda")
    st = lib.tcl_score_noalloc(m.handle, B, L, X.data_ptr(), lengths.data_ptr(), out.data_ptr(),
                               None if stream is None else ctypes.c_void_p(stream.cuda_stream))
    return st, out


def _reference(m, X, lengths):
    ws = torch.empty(m.workspace_bytes(X.shape[0], X.shape[1]), dtype=torch.uint8, device="cuda")
    return m.score(X, lengths, workspace=ws)


@pytest.mark.parametrize("name,dtype,B1,B2,L2", [
    ("score_B4096_L25_d256_f32", "f32", 1300, 37, 19),
    ("score_B65536_L25_d256_bf16", "bf16", 1400, 260, 25),
    ("paper_B4096_L41_F20_f32", "f32", 2000, 5, 41),
])
def test_noalloc_matches_tcl_score(name, dtype, B1, B2, L2):
    lib = tb.lib()
    w = wl.WORKLOADS[name]
    blob, X, lengths = wl.make_workload(name, B=B1)
    m = tb.CostModel(tb.config_from_shape(w.model, dtype), blob)
    assert lib.tcl_score_noalloc_max_bytes() == 256 << 20
    assert m.workspace_bytes(B1, w.L) <= lib.tcl_score_noalloc_max_bytes()
    Xd, Ld = torch.from_numpy(X).cuda(), torch.from_numpy(lengths).cuda()
    print(f"noalloc {name} B={B1}", flush=True)
    st, g1 = _noalloc(lib, m, Xd, Ld)
    assert st == 0, lib.tcl_last_error()
    # a second call in a row, smaller (fewer programs, shorter padding), on
    # another stream: the buffer still holds the first call's contents
    X2 = np.ascontiguousarray(X[B1 - B2:, :L2])
    l2 = np.minimum(lengths[B1 - B2:], L2).astype(np.int32)
    X2[np.arange(L2)[None, :] >= l2[:, None]] = 0
    X2d, l2d = torch.from_numpy(X2).cuda(), torch.from_numpy(l2).cuda()
    s = torch.cuda.Stream()
    torch.cuda.current_stream().synchronize()
    with torch.cuda.stream(s):
        st2, g2 = _noalloc(lib, m, X2d, l2d, stream=s)
    assert st2 == 0, lib.tcl_last_error()
    s.synchronize()
    r1 = _reference(m, Xd, Ld)
    r2 = _reference(m, X2d, l2d)
    torch.cuda.synchronize()
    assert torch.equal(g1, r1), float((g1 - r1).abs().max())
    assert torch.equal(g2, r2), float((g2 - r2).abs().max())
    assert torch.isfinite(g1).all() and torch.isfinite(g2).all()


def test_noalloc_refuses_what_does_not_fit():
    lib = tb.lib()
    w = wl.WORKLOADS["score_B4096_L25_d256_f32"]
    blob, X, lengths = wl.make_workload(w.name, B=8)
    m = tb.CostModel(tb.config_from_shape(w.model), blob)
    B = 4096
    assert m.workspace_bytes(B // 2, w.L) > lib.tcl_score_noalloc_max_bytes()
    out = torch.full((B,), 7.0, device="cuda")
    Xd = torch.zeros(B, w.L, w.model.F, device="cuda")
    Ld = torch.full((B,), 25, dtype=torch.int32, device="cuda")
    assert lib.tcl_score_noalloc(m.handle, B, w.L, Xd.data_ptr(), Ld.data_ptr(), out.data_ptr(), None) == -2
    assert b"scratch" in lib.tcl_last_error()
    m.timing(True)
    assert lib.tcl_score_noalloc(m.handle, 8, w.L, Xd.data_ptr(), Ld.data_ptr(), out.data_ptr(), None) == -1
    m.timing(False)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())  # nothing was enqueued
