"""Seeded synthetic workloads for the TCL Mamba cost model.

This module is the one piece shared by the HIP path's callers (tests,
bench) and by the fp64 oracle's callers: it draws inputs and initial
weights from seeded generators and does none of the model's arithmetic.
It imports nothing else from this package.

Inputs stand in for the paper's tensor-program feature sequences
(section 5.1): the paper's datasets (Tenset plus its own i7 / 3080 Ti
traces) are not available, so each candidate program is a zero-padded
sequence of per-statement feature vectors with F = 164 entries (Ansor's
per-statement feature count quoted in section 5.1), each entry
log1p(lognormal(0, 1)), and a per-program length drawn uniformly.

Weight initialisation recipe:
  * Linear weights and biases ~ U(-1/sqrt(fan_in), +1/sqrt(fan_in));
    in_proj, x_proj and out_proj carry no bias;
  * depthwise conv weight and bias ~ U(-1/sqrt(d_conv), +1/sqrt(d_conv));
  * A_log[e, n] = log(n + 1) for every channel e, D = 1;
  * dt bias b_dt = dt0 + log(-expm1(-dt0)) with dt0 log-uniform in
    [1e-3, 1e-1], so that softplus(b_dt) = dt0;
  * RMSNorm gains = 1.
`perturb=True` additionally jitters the gains, D, A_log and the dt bias so
that an indexing mistake in any of them changes the result (the plain
recipe makes them constant along a dimension).

Canonical parameter order (one flat fp32 blob, every matrix row-major in
[out, in] layout):
  W0[d,F], b0[d],
  per block: g[d], W_in[2E,d], conv_w[E,K], conv_b[E], W_x[R+2N,E],
             W_dt[E,R], b_dt[E], A_log[E,N], D[E], W_out[d,E],
  g_f[d], W1[h,d], b1[h], W2[1,h], b2[1]
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Tuple

import numpy as np

ROOT_SEED = 12891


@dataclasses.dataclass(frozen=True)
class ModelShape:
    F: int = 164
    d_model: int = 256
    d_inner: int = 512
    d_state: int = 16
    d_conv: int = 4
    dt_rank: int = 16
    n_layers: int = 4
    head_hidden: int = 256
    final_norm: int = 1
    norm_eps: float = 1e-5
    enc_hidden: Tuple[int, ...] = ()  # hidden widths of a multi-layer encoder
    dec_hidden2: int = 0  # second hidden width of a three-layer decoder (0: two layers)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    B: int
    L: int
    len_lo: int
    len_hi: int
    dtype: str  # "f32" or "bf16"
    seed_index: int
    student: ModelShape | None = None  # distillation only
    adapter: int = 0  # progressive KB + AC forward: the lateral adapters' width


TINY = ModelShape(d_model=64, d_inner=128, dt_rank=4, n_layers=2, head_hidden=64)
D256 = ModelShape()
STUDENT = ModelShape(d_model=128, d_inner=256, dt_rank=8, n_layers=2, head_hidden=128)
# The paper's own model (section 5.2 and Table 2's best hyper-parameters): an
# encoder of three Linear layers F -> 64 -> 128 -> 128, one Mamba block with
# d_model 128, expand 1, d_state 8, d_conv 4, a decoder 128 -> 64 -> 32 -> 1;
# dt_rank = ceil(d_model / 16). Features per statement: 22 for the CPU
# traces, 20 for the GPU ones (section 5.1).
PAPER_CPU = ModelShape(F=22, d_model=128, d_inner=128, d_state=8, d_conv=4, dt_rank=8, n_layers=1,
                       head_hidden=64, enc_hidden=(64, 128), dec_hidden2=32)
PAPER_GPU = dataclasses.replace(PAPER_CPU, F=20)

WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in [
        Workload("score_B64_L25_d64_f32", TINY, 64, 25, 5, 25, "f32", 0),
        Workload("score_B4096_L25_d256_f32", D256, 4096, 25, 5, 25, "f32", 1),
        Workload("score_B65536_L25_d256_bf16", D256, 65536, 25, 5, 25, "bf16", 2),
        Workload("score_B8192_L256_d256_f32", D256, 8192, 256, 64, 256, "f32", 3),
        Workload("distill_B1024_L25_t256_s128_bf16", D256, 1024, 25, 5, 25, "bf16", 4, STUDENT),
        # the paper's model on its own input shapes: 26 x 22 (CPU) and 41 x 20 (GPU)
        Workload("paper_B4096_L26_F22_f32", PAPER_CPU, 4096, 26, 5, 26, "f32", 5),
        Workload("paper_B4096_L41_F20_f32", PAPER_GPU, 4096, 41, 8, 41, "f32", 6),
        # the CKD framework's continual-learning forward: frozen KB and active
        # column, both the paper's model, joined by lateral adapters of width 8
        Workload("progressive_B4096_L41_F20_a8_f32", PAPER_GPU, 4096, 41, 8, 41, "f32", 7, adapter=8),
    ]
}
WORKLOAD_ORDER = list(WORKLOADS)


def _rng(*path: int) -> np.random.Generator:
    ss = np.random.SeedSequence(ROOT_SEED)
    for p in path:
        ss = ss.spawn(p + 1)[p]
    return np.random.Generator(np.random.PCG64(ss))


def param_layout(m: ModelShape) -> List[Tuple[str, Tuple[int, ...]]]:
    """Names and shapes of the parameters, in canonical blob order."""
    d, E, N, K, R, F, h = m.d_model, m.d_inner, m.d_state, m.d_conv, m.dt_rank, m.F, m.head_hidden
    dims = [F, *m.enc_hidden, d]
    out: List[Tuple[str, Tuple[int, ...]]] = []
    for i in range(len(dims) - 1):
        sfx = f"_{i}" if i else ""
        out += [(f"W0{sfx}", (dims[i + 1], dims[i])), (f"b0{sfx}", (dims[i + 1],))]
    for l in range(m.n_layers):
        out += [
            (f"blk{l}.g", (d,)),
            (f"blk{l}.W_in", (2 * E, d)),
            (f"blk{l}.conv_w", (E, K)),
            (f"blk{l}.conv_b", (E,)),
            (f"blk{l}.W_x", (R + 2 * N, E)),
            (f"blk{l}.W_dt", (E, R)),
            (f"blk{l}.b_dt", (E,)),
            (f"blk{l}.A_log", (E, N)),
            (f"blk{l}.D", (E,)),
            (f"blk{l}.W_out", (d, E)),
        ]
    out += [("g_f", (d,)), ("W1", (h, d)), ("b1", (h,))]
    if m.dec_hidden2:
        out += [("W2", (m.dec_hidden2, h)), ("b2", (m.dec_hidden2,)), ("W3", (1, m.dec_hidden2)), ("b3", (1,))]
    else:
        out += [("W2", (1, h)), ("b2", (1,))]
    return out


def layer_widths(m: ModelShape) -> List[Tuple[int, int]]:
    """(n_in, n_out) of every layer in forward order: the encoder's Linear
    layers, the Mamba blocks, the decoder's Linear layers."""
    dims = [m.F, *m.enc_hidden, m.d_model]
    out = [(dims[i], dims[i + 1]) for i in range(len(dims) - 1)]
    out += [(m.d_model, m.d_model)] * m.n_layers
    dec = [m.d_model, m.head_hidden] + ([m.dec_hidden2] if m.dec_hidden2 else []) + [1]
    out += [(dec[i], dec[i + 1]) for i in range(len(dec) - 1)]
    return out


def lateral_layout(m: ModelShape, a: int) -> List[Tuple[str, Tuple[int, ...]]]:
    """Lateral adapters (KB -> AC, one per layer after the first, forward
    order): V[a, n_in], c[a], U[n_out, a], alpha[n_out]."""
    out: List[Tuple[str, Tuple[int, ...]]] = []
    for j, (n_in, n_out) in enumerate(layer_widths(m)[1:]):
        out += [(f"lat{j}.V", (a, n_in)), (f"lat{j}.c", (a,)), (f"lat{j}.U", (n_out, a)),
                (f"lat{j}.alpha", (n_out,))]
    return out


def init_lateral(m: ModelShape, a: int, rng: np.random.Generator) -> np.ndarray:
    """Flat fp32 lateral blob: V, c ~ U(+-1/sqrt(n_in)), U ~ U(+-1/sqrt(a)),
    alpha ~ U(0.5, 1.5) (so that every adapter visibly contributes)."""
    parts = []
    for (n_in, _), j in zip(layer_widths(m)[1:], range(len(layer_widths(m)) - 1)):
        bv, bu = 1.0 / math.sqrt(n_in), 1.0 / math.sqrt(a)
        parts += [rng.uniform(-bv, bv, size=(a, n_in)), rng.uniform(-bv, bv, size=a)]
        n_out = layer_widths(m)[j + 1][1]
        parts += [rng.uniform(-bu, bu, size=(n_out, a)), rng.uniform(0.5, 1.5, size=n_out)]
    return np.concatenate([np.asarray(p, dtype=np.float32).reshape(-1) for p in parts])


def param_count(m: ModelShape) -> int:
    return sum(int(np.prod(s)) for _, s in param_layout(m))


def init_params(m: ModelShape, rng: np.random.Generator, perturb: bool = False) -> np.ndarray:
    """Flat fp32 parameter blob in canonical order."""
    parts = []
    fan_in = 0
    for name, shape in param_layout(m):
        base = name.split(".")[-1]
        if base in ("W_in", "W_x", "W_dt", "W_out", "W1", "W2", "W3") or base.startswith("W0"):
            bound = 1.0 / math.sqrt(shape[1])
            a = rng.uniform(-bound, bound, size=shape)
        elif base in ("b1", "b2", "b3") or base.startswith("b0"):
            bound = 1.0 / math.sqrt(fan_in)  # fan-in of the weight just before
            a = rng.uniform(-bound, bound, size=shape)
        elif base in ("conv_w", "conv_b"):
            bound = 1.0 / math.sqrt(m.d_conv)
            a = rng.uniform(-bound, bound, size=shape)
        elif base in ("g", "g_f"):
            a = np.ones(shape)
            if perturb:
                a = a + 0.2 * rng.standard_normal(shape)
        elif base == "A_log":
            a = np.tile(np.log(np.arange(1, m.d_state + 1, dtype=np.float64)), (shape[0], 1))
            if perturb:
                a = a + 0.3 * rng.standard_normal(shape)
        elif base == "D":
            a = np.ones(shape)
            if perturb:
                a = a + 0.5 * rng.standard_normal(shape)
        elif base == "b_dt":
            lo, hi = math.log(1e-3), math.log(1e-1)
            dt0 = np.exp(rng.uniform(lo, hi, size=shape))
            a = dt0 + np.log(-np.expm1(-dt0))  # inverse of softplus at dt0
        else:  # pragma: no cover - layout and init must list the same names
            raise KeyError(name)
        if base.startswith("W") and len(shape) == 2:
            fan_in = shape[1]
        parts.append(np.asarray(a, dtype=np.float32).reshape(-1))
    return np.concatenate(parts)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns fp32."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    nan = np.isnan(a)
    out = r.astype(np.uint32).view(np.float32).copy()
    out[nan] = np.nan
    return out


def unpack(blob: np.ndarray, m: ModelShape) -> Dict[str, np.ndarray]:
    out, off = {}, 0
    for name, shape in param_layout(m):
        n = int(np.prod(shape))
        out[name] = blob[off : off + n].reshape(shape)
        off += n
    assert off == blob.size
    return out


def make_inputs(B: int, L: int, F: int, len_lo: int, len_hi: int, rng: np.random.Generator):
    """Features [B,L,F] fp32 (zero past each length) and lengths [B] int32."""
    lengths = rng.integers(len_lo, len_hi + 1, size=B).astype(np.int32)
    X = np.log1p(rng.lognormal(0.0, 1.0, size=(B, L, F))).astype(np.float32)
    X[np.arange(L)[None, :] >= lengths[:, None]] = 0.0
    return X, lengths


def make_workload(name: str, B: int | None = None, perturb: bool = False):
    """Seeded (params, X, lengths) for a named workload.

    `B` overrides the batch size (a smaller batch is its own draw from the
    same seed path). For the distillation workload `params` is the pair
    (teacher_blob, student_blob); both are bf16-representable. For the
    progressive workload it is (kb_blob, ac_blob, lateral_blob).
    """
    w = WORKLOADS[name]
    Bn = w.B if B is None else B
    prng = _rng(w.seed_index, 0)
    if w.adapter:
        params = (init_params(w.model, prng, perturb), init_params(w.model, _rng(w.seed_index, 1), perturb),
                  init_lateral(w.model, w.adapter, _rng(w.seed_index, 4)))
    elif w.student is None:
        params = init_params(w.model, prng, perturb)
        if w.dtype == "bf16":
            params = round_to_bf16(params)
    else:
        t = round_to_bf16(init_params(w.model, prng, perturb))
        s = round_to_bf16(init_params(w.student, _rng(w.seed_index, 1), perturb))
        params = (t, s)
    X, lengths = make_inputs(Bn, w.L, w.model.F, w.len_lo, w.len_hi, _rng(w.seed_index, 2))
    return params, X, lengths


def label_noise(B: int, seed_index: int = 4, sigma: float = 0.05) -> np.ndarray:
    """N(0, sigma^2) noise added to teacher scores to form synthetic labels."""
    return (sigma * _rng(seed_index, 3).standard_normal(B)).astype(np.float32)


def random_tensor(shape, seed_path=(9, 9), scale=1.0, dist="normal") -> np.ndarray:
    r = _rng(*seed_path)
    if dist == "normal":
        a = scale * r.standard_normal(shape)
    else:
        a = scale * r.uniform(-1.0, 1.0, size=shape)
    return a.astype(np.float32)
