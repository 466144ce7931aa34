"""End-to-end parity of tcl_score against the fp64 oracle on the same seeded
inputs: scores within the fp32 tolerance, and no ranking inversion wherever
the oracle's tolerance intervals of two candidates are disjoint.

Full-size workloads are scored whole on the GPU, in the launch configuration
the benchmark times, and every program is compared with the oracle's
full-batch scores, written by tests/golden/make_golden.py (which calls only
the oracle and the seeded generator); the ranking check runs over the whole
batch.
"""
import numpy as np
import pytest
import torch

from paper_2604_12891_amd import binding as tb
from paper_2604_12891_amd import workload as wl
from tests.parity import assert_scores_match, golden_scores, oracle_scores

pytestmark = pytest.mark.gpu


def _model(shape, blob, dtype="f32", f32_matmul="split"):
    return tb.CostModel(tb.config_from_shape(shape, dtype, f32_matmul), blob)


def _score(model, X, lengths):
    out = model.score(torch.from_numpy(X).cuda(), torch.from_numpy(lengths).cuda())
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _sample(lengths, n, seed=0):
    """n seeded random program indices plus the shortest, the longest, the
    first and the last program (the pinned four are always kept)."""
    rng = np.random.default_rng(seed)
    idx = set(rng.choice(len(lengths), size=n, replace=False).tolist())
    idx |= {int(np.argmin(lengths)), int(np.argmax(lengths)), 0, len(lengths) - 1}
    return np.array(sorted(idx))


@pytest.mark.parametrize("f32_matmul", ["split", "split_bf16", "native"])
@pytest.mark.parametrize("perturb", [False, True])
def test_tiny_full_batch(perturb, f32_matmul):
    w = wl.WORKLOADS["score_B64_L25_d64_f32"]
    print(f"tcl_score {w.name} perturb={perturb} {f32_matmul}", flush=True)
    blob, X, lengths = wl.make_workload(w.name, perturb=perturb)
    g = _score(_model(w.model, blob, f32_matmul=f32_matmul), X, lengths)
    assert_scores_match(g, oracle_scores(blob, X, lengths, w.model), "f32", w.name)


@pytest.mark.parametrize("f32_matmul", ["split", "split_bf16", "native"])
def test_headline_full_batch(f32_matmul):
    """The headline round (B = 4096, L = 25), scored whole in the launch
    configuration the benchmark times: every program against the oracle's
    stored full-batch scores, and the ranking check over the whole batch."""
    w = wl.WORKLOADS["score_B4096_L25_d256_f32"]
    print(f"tcl_score {w.name} full batch {f32_matmul}", flush=True)
    blob, X, lengths = wl.make_workload(w.name)
    o = golden_scores(w.name, blob, X, lengths)
    g = _score(_model(w.model, blob, f32_matmul=f32_matmul), X, lengths)
    assert_scores_match(g, o, "f32", w.name)


@pytest.mark.parametrize("f32_matmul", ["split", "split_bf16", "native"])
def test_headline_shape_perturbed_weights(f32_matmul):
    w = wl.WORKLOADS["score_B4096_L25_d256_f32"]
    blob, X, lengths = wl.make_workload(w.name, B=160, perturb=True)
    print(f"tcl_score {w.name} B=160 perturbed {f32_matmul}", flush=True)
    g = _score(_model(w.model, blob, f32_matmul=f32_matmul), X, lengths)
    assert_scores_match(g, oracle_scores(blob, X, lengths, w.model), "f32", w.name + " perturbed")


@pytest.mark.parametrize("f32_matmul", ["split", "native"])
def test_long_sequences_full_batch(f32_matmul):
    """B = 8192 programs of 64..256 tokens: every program against the
    oracle's stored scores, ranking over the whole batch."""
    w = wl.WORKLOADS["score_B8192_L256_d256_f32"]
    print(f"tcl_score {w.name} full batch {f32_matmul}", flush=True)
    blob, X, lengths = wl.make_workload(w.name)
    o = golden_scores(w.name, blob, X, lengths)
    g = _score(_model(w.model, blob, f32_matmul=f32_matmul), X, lengths)
    assert_scores_match(g, o, "f32", w.name)


def test_long_sequences_chunked_scan_full_shape():
    """The long-sequence workload's own programs through the chunked
    two-level scan: a batch of 96 of them (sampled with the first and last,
    the shortest and the longest) is too small to fill the GPU with one
    thread per (program, channel), so tcl_score scans each program in
    concurrent chunks; scores against the oracle's stored ones."""
    w = wl.WORKLOADS["score_B8192_L256_d256_f32"]
    blob, X, lengths = wl.make_workload(w.name)
    o = golden_scores(w.name, blob, X, lengths)
    idx = _sample(lengths, 92, seed=3)
    assert {0, w.B - 1} <= set(idx.tolist())
    print(f"tcl_score {w.name} {len(idx)} sampled programs (chunked scan)", flush=True)
    g = _score(_model(w.model, blob), X[idx], lengths[idx])
    assert_scores_match(g, o[idx], "f32", w.name + " chunked")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_long_sequences_small_batch(dtype):
    """A batch too small to fill the GPU with one thread per (program,
    channel): tcl_score runs the chunked two-level scan here."""
    w = wl.WORKLOADS["score_B8192_L256_d256_f32"]
    blob, X, lengths = wl.make_workload(w.name, B=6, perturb=True)
    lengths[0], lengths[1] = 256, 64
    X[np.arange(256)[None, :] >= lengths[:, None]] = 0
    if dtype == "bf16":
        blob = wl.round_to_bf16(blob)
    print(f"tcl_score B=6 L=256 {dtype} (chunked scan)", flush=True)
    g = _score(_model(w.model, blob, dtype), X, lengths)
    assert_scores_match(g, oracle_scores(blob, X, lengths, w.model), dtype, "small batch, long sequences")


@pytest.mark.parametrize("perturb", [False, True])
def test_tiny_bf16(perturb):
    """The bf16 path (bf16 weights and activations, fp32 accumulation and scan
    state) on the small model; weights are bf16-representable on both sides."""
    shape = wl.TINY
    blob = wl.round_to_bf16(wl.init_params(shape, np.random.default_rng(21), perturb=perturb))
    X, lengths = wl.make_inputs(64, 25, shape.F, 5, 25, np.random.default_rng(22))
    print(f"tcl_score tiny bf16 perturb={perturb}", flush=True)
    g = _score(_model(shape, blob, "bf16"), X, lengths)
    assert_scores_match(g, oracle_scores(blob, X, lengths, shape), "bf16", "tiny bf16")


def test_bf16_pool_full_batch():
    """B = 65536 programs, bf16: every program against the oracle's stored
    scores (bf16 tolerance), ranking over the whole batch."""
    w = wl.WORKLOADS["score_B65536_L25_d256_bf16"]
    print(f"tcl_score {w.name} full batch", flush=True)
    blob, X, lengths = wl.make_workload(w.name)
    o = golden_scores(w.name, blob, X, lengths)
    g = _score(_model(w.model, blob, "bf16"), X, lengths)
    assert_scores_match(g, o, "bf16", w.name)


def test_bf16_perturbed_weights():
    w = wl.WORKLOADS["score_B65536_L25_d256_bf16"]
    blob, X, lengths = wl.make_workload(w.name, B=128, perturb=True)
    print(f"tcl_score {w.name} B=128 perturbed", flush=True)
    g = _score(_model(w.model, blob, "bf16"), X, lengths)
    assert_scores_match(g, oracle_scores(blob, X, lengths, w.model), "bf16", w.name + " perturbed")


@pytest.mark.parametrize("case", ["B1", "L1", "all_full", "odd_B", "len_1_and_L"])
def test_edge_shapes(case):
    shape = wl.TINY
    rng = np.random.default_rng(11)
    blob = wl.init_params(shape, rng, perturb=True)
    B, L = {"B1": (1, 25), "L1": (37, 1), "all_full": (20, 25), "odd_B": (37, 13), "len_1_and_L": (33, 30)}[case]
    X, lengths = wl.make_inputs(B, L, shape.F, 1, L, rng)
    if case == "all_full":
        lengths[:] = L
        X, _ = wl.make_inputs(B, L, shape.F, L, L, rng)
    if case == "len_1_and_L":
        lengths[::2] = 1
        lengths[1::2] = L
        X[np.arange(L)[None, :] >= lengths[:, None]] = 0
    print(f"tcl_score edge {case} B={B} L={L}", flush=True)
    g = _score(_model(shape, blob), X, lengths)
    assert_scores_match(g, oracle_scores(blob, X, lengths, shape), "f32", case)


@pytest.mark.parametrize("L", [4096, 4097])
def test_long_padding_around_the_ordering_limit(L):
    """The offsets kernel lists programs longest first (a counting sort over
    L + 1 length buckets) for L up to 4096, and the sequential scan hands
    them out in that order; above it the scan takes them in index order.
    Enough programs for the sequential scan (>= 1024 wavefronts of 64
    channels), padded to L; the oracle scores the same programs padded only
    to their longest (a program's score reads its own tokens alone)."""
    shape = wl.ModelShape(F=8, d_model=64, d_inner=512, dt_rank=4, n_layers=2, head_hidden=64)
    rng = np.random.default_rng(L)
    blob = wl.init_params(shape, rng, perturb=True)
    B = 130
    X, lengths = wl.make_inputs(B, L, shape.F, 1, 20, rng)
    for b, n in ((5, 300), (129, 299)):
        lengths[b] = n
        X[b, :n] = np.log1p(rng.lognormal(0.0, 1.0, size=(n, shape.F))).astype(np.float32)
    print(f"tcl_score B={B} L={L} (longest program 300 tokens)", flush=True)
    g = _score(_model(shape, blob), X, lengths)
    Lmax = int(lengths.max())
    assert_scores_match(g, oracle_scores(blob, np.ascontiguousarray(X[:, :Lmax]), lengths, shape), "f32",
                        f"L={L}")


def test_padding_never_read_and_invalid_lengths():
    """Rows past each length hold NaN and must not be read; programs with a
    length outside [1, L] score NaN without disturbing the others."""
    shape = wl.TINY
    rng = np.random.default_rng(12)
    blob = wl.init_params(shape, rng, perturb=True)
    B, L = 24, 25
    X, lengths = wl.make_inputs(B, L, shape.F, 1, L, rng)
    Xn = X.copy()
    Xn[np.arange(L)[None, :] >= lengths[:, None]] = np.nan
    bad = lengths.copy()
    bad[3], bad[10], bad[17] = 0, L + 1, -5
    print("tcl_score NaN padding + invalid lengths", flush=True)
    m = _model(shape, blob)
    g = _score(m, Xn, bad)
    ok = np.ones(B, bool)
    ok[[3, 10, 17]] = False
    assert np.all(np.isnan(g[~ok]))
    assert_scores_match(g[ok], oracle_scores(blob, X[ok], lengths[ok], shape), "f32", "nan padding")


def test_deterministic_and_batch_independent():
    w = wl.WORKLOADS["score_B4096_L25_d256_f32"]
    blob, X, lengths = wl.make_workload(w.name, B=300)
    print("tcl_score determinism B=300", flush=True)
    m = _model(w.model, blob)
    g1 = _score(m, X, lengths)
    g2 = _score(m, X, lengths)
    assert np.array_equal(g1, g2)
    sub = np.arange(40, 57)
    g3 = _score(m, X[sub], lengths[sub])
    np.testing.assert_allclose(g3, g1[sub], rtol=1e-5, atol=1e-6)


def test_set_get_params_roundtrip():
    shape = wl.TINY
    rng = np.random.default_rng(13)
    b1 = wl.init_params(shape, rng, perturb=True)
    b2 = wl.init_params(shape, rng, perturb=True)
    X, lengths = wl.make_inputs(16, 25, shape.F, 5, 25, rng)
    m = _model(shape, b1)
    assert np.array_equal(m.get_params(), b1)
    m.set_params(b2)
    assert np.array_equal(m.get_params(), b2)
    g = _score(m, X, lengths)
    assert_scores_match(g, oracle_scores(b2, X, lengths, shape), "f32", "set_params")


def test_workspace_too_small_is_rejected():
    shape = wl.TINY
    m = _model(shape, wl.init_params(shape, np.random.default_rng(0)))
    X = torch.zeros(4, 25, shape.F, device="cuda")
    lens = torch.full((4,), 5, dtype=torch.int32, device="cuda")
    ws = torch.empty(m.workspace_bytes(4, 25) - 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(tb.TclError) as e:
        m.score(X, lens, workspace=ws)
    assert e.value.status == -3


def test_two_concurrent_halves_match_separate_calls():
    """A batch of >= 2048 programs runs as two halves on the model's two
    streams; its scores are the same bits as scoring the programs in
    smaller single-stream batches (every kernel treats rows and programs
    independently and in a fixed order), and the workspace query covers
    both halves."""
    w = wl.WORKLOADS["score_B4096_L25_d256_f32"]
    blob, X, lengths = wl.make_workload(w.name)
    m = _model(w.model, blob)
    B, L = X.shape[:2]
    assert m.workspace_bytes(B, L) >= 2 * m.workspace_bytes(1000, L)
    print("tcl_score two halves vs batches of 1000", flush=True)
    g = _score(m, X, lengths)
    parts = [_score(m, X[i:i + 1000], lengths[i:i + 1000]) for i in range(0, B, 1000)]
    np.testing.assert_array_equal(g, np.concatenate(parts))
    # one pass over the whole batch: the same bits
    m.set_score_streams(1)
    np.testing.assert_array_equal(_score(m, X, lengths), g)
    m.set_score_streams(2)
    for bad in (0, 3, -1):
        with pytest.raises(tb.TclError):
            m.set_score_streams(bad)
    # and on a non-default stream, twice in a row
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        out = torch.empty(B, device="cuda")
        for _ in range(2):
            m.score(torch.from_numpy(X).cuda(), torch.from_numpy(lengths).cuda(), out=out, stream=s)
    s.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy(), g)


@pytest.mark.parametrize("B", [2048, 2049, 2051])
def test_two_halves_edges(B):
    """The split at B = 2048 (halves of 1024), odd B (the second half one
    program longer), invalid and empty programs on both sides of the split
    point: scores match the one-pass run bit for bit, invalid ones are NaN,
    and a workspace one byte short is refused."""
    w = wl.WORKLOADS["score_B4096_L25_d256_f32"]
    blob, X, lengths = wl.make_workload(w.name, B=B, perturb=True)
    h = B // 2
    lengths = lengths.copy()
    lengths[[h - 1, h, h + 1, 0, B - 1]] = [0, 26, 1, -3, 25]
    X = X.copy()
    X[h + 1, 1:] = 0.0
    m = _model(w.model, blob)
    print(f"tcl_score two halves B={B}", flush=True)
    g2 = _score(m, X, lengths)
    m.set_score_streams(1)
    g1 = _score(m, X, lengths)
    m.set_score_streams(2)
    np.testing.assert_array_equal(g2, g1)
    bad = np.zeros(B, bool)
    bad[[h - 1, h, 0]] = True
    assert np.all(np.isnan(g2[bad])) and np.all(np.isfinite(g2[~bad]))
    idx = np.array([1, h + 1, h + 2, B - 1])
    assert_scores_match(g2[idx], oracle_scores(blob, X[idx], lengths[idx], w.model), "f32", "split edges")
    L = X.shape[1]
    need = m.workspace_bytes(B, L)
    ws = torch.empty(need - 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(tb.TclError):
        m.score(torch.from_numpy(X).cuda(), torch.from_numpy(lengths).cuda(), workspace=ws)
