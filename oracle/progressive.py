"""fp64 CPU oracle of the progressive KB + AC forward of the CKD framework
(section 6, Fig. 6, Eq. (7)): during continual learning the frozen knowledge
base (KB) runs on the programs, and every layer of the active column (AC)
takes, beside its own input, the KB's input to the same layer through a
lateral adapter.

TEST INFRASTRUCTURE ONLY, like oracle.model: only the tests, the smoke check
and the benchmark's CPU-baseline leg may call it. It shares no code with the
HIP library and takes every input as an argument.

Reading of Eq. (7), h_i = s(W_i h_{i-1} + alpha_i * U_i s(V_i h^KB_{i-1} + c_i) + b_i):
  * the layers i are, in order, the encoder's Linear layers, the Mamba
    blocks and the decoder's Linear layers (section 6 names encoder, Mamba
    block and decoder as the layers); KB and AC share the architecture;
  * the first layer has no lateral input: both columns read the same
    features;
  * s inside the adapter is ReLU; the outer s is the layer's own activation
    (ReLU between Linear layers, none after the encoder's last layer, none
    on the score);
  * for a Mamba block the AC's own term is the block itself with its
    residual, h_{i-1} + Block(RMSNorm(h_{i-1})); the adapter's output is added
    to it (the block has no output bias, so b_i is absent there);
  * the lateral input of the decoder's first layer is the KB's decoder
    input: its pooled, normalised vector; the other decoder layers take the
    KB's hidden decoder activations;
  * adapters: V_i [a, n_{i-1}], c_i [a], U_i [n_i, a], alpha_i [n_i], with
    one adapter width a for every lateral (the paper gives none).
Lateral parameters of a model: for each lateral layer in forward order,
  lat{j}.V, lat{j}.c, lat{j}.U, lat{j}.alpha.
"""
from __future__ import annotations

from typing import Dict, List, Tuple

import numpy as np

from oracle import model as om

f64 = np.float64


def layer_widths(cfg: dict) -> List[Tuple[str, int, int]]:
    """(kind, n_in, n_out) of every layer in forward order; kind is "enc",
    "block" or "dec"."""
    dims = om.encoder_dims(cfg)
    out = [("enc", dims[i], dims[i + 1]) for i in range(len(dims) - 1)]
    d = cfg["d_model"]
    out += [("block", d, d)] * cfg["n_layers"]
    h, h2 = cfg["head_hidden"], cfg.get("dec_hidden2", 0)
    dec = [d, h] + ([h2] if h2 else []) + [1]
    out += [("dec", dec[i], dec[i + 1]) for i in range(len(dec) - 1)]
    return out


def lateral_layout(cfg: dict, a: int) -> List[Tuple[str, Tuple[int, ...]]]:
    """Lateral adapters of every layer but the first, in forward order."""
    names = []
    for j, (_, n_in, n_out) in enumerate(layer_widths(cfg)[1:]):
        p = f"lat{j}."
        names += [(p + "V", (a, n_in)), (p + "c", (a,)), (p + "U", (n_out, a)), (p + "alpha", (n_out,))]
    return names


def unpack_lateral(blob, cfg: dict, a: int) -> Dict[str, np.ndarray]:
    blob = np.asarray(blob, dtype=f64)
    out, off = {}, 0
    for name, shape in lateral_layout(cfg, a):
        n = int(np.prod(shape))
        out[name] = blob[off:off + n].reshape(shape).copy()
        off += n
    if off != blob.size:
        raise ValueError(f"blob has {blob.size} values, layout needs {off}")
    return out


def _relu(x):
    return np.maximum(x, 0.0)


def _adapter(Q, j, h_kb):
    """alpha_j * U_j ReLU(V_j h_kb + c_j)."""
    p = f"lat{j}."
    return Q[p + "alpha"] * (_relu(h_kb @ Q[p + "V"].T + Q[p + "c"]) @ Q[p + "U"].T)


def _column(P, X, lengths, cfg, Q=None, kb_inputs=None):
    """One column's forward. Returns the score and the input of every layer
    (the h_{i-1} that the AC's adapters read). With Q and kb_inputs, the
    column is the AC: layer i > 0 adds adapter i-1 applied to kb_inputs[i]."""
    X = np.asarray(X, dtype=f64)
    lengths = np.asarray(lengths)
    Bn, L, _ = X.shape
    layers = layer_widths(cfg)
    n_enc = len(om.encoder_dims(cfg)) - 1
    inputs = []
    i = 0

    def lateral(pre):
        if Q is None or i == 0:
            return pre
        return pre + _adapter(Q, i - 1, kb_inputs[i])

    h = X
    for e in range(n_enc):
        inputs.append(h)
        sfx = f"_{e}" if e else ""
        pre = lateral(h @ P[f"W0{sfx}"].T + P[f"b0{sfx}"])
        h = _relu(pre) if e < n_enc - 1 else pre
        i += 1
    for l in range(cfg["n_layers"]):
        inputs.append(h)
        h = lateral(om._block_forward(h, P, l, cfg, keep=False)[0])
        i += 1
    if cfg.get("final_norm", 1):
        hf, _ = om.rmsnorm(h, P["g_f"], cfg["norm_eps"])
    else:
        hf = h
    mask = (np.arange(L)[None, :] < lengths[:, None]).astype(f64)
    v = np.sum(hf * mask[:, :, None], axis=1) / lengths[:, None].astype(f64)
    names = [("W1", "b1"), ("W2", "b2")] + ([("W3", "b3")] if cfg.get("dec_hidden2", 0) else [])
    for k, (wn, bn) in enumerate(names):
        inputs.append(v)
        pre = lateral(v @ P[wn].T + P[bn])
        v = _relu(pre) if k < len(names) - 1 else pre
        i += 1
    assert i == len(layers)
    return v[:, 0], inputs


def kb_forward(kb_blob, X, lengths, cfg):
    """The KB's scores and the input of each of its layers."""
    return _column(om.unpack(kb_blob, cfg), X, lengths, cfg)


def progressive_scores(kb_blob, ac_blob, lat_blob, a, X, lengths, cfg):
    """The AC's scores (the CL phase's prediction p_t, Eq. (8)) with every
    layer after the first reading the KB through Eq. (7)."""
    _, kb_in = kb_forward(kb_blob, X, lengths, cfg)
    s, _ = _column(om.unpack(ac_blob, cfg), X, lengths, cfg, unpack_lateral(lat_blob, cfg, a), kb_in)
    return s
