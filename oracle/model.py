"""fp64 CPU oracle of TCL's Mamba cost model: forward scoring, backward, Adam.

TEST INFRASTRUCTURE ONLY. This is the plain, slow, obviously correct
definition that the HIP library is checked against. Only the test suite,
the smoke check and the CPU-baseline leg of the benchmark may import or
call it; the product path never does. It shares no code with the HIP
path: it has its own parameter layout, its own arithmetic, and takes all
inputs (weights, features, lengths, labels) as arguments.

Everything is numpy float64. Matrix products use numpy's matmul (a
library primitive); everything else is written out step by step in the
order the model defines it, with no fusion or reordering.

What the model computes (section 5.2 of the paper, Fig. 5, Eq. (4)-(5)):
  encoder: one Linear F -> d_model, or (the paper's form, section 5.2: three
    Linear layers of widths 64, 128, 128) Linear F -> e_1, ReLU, ...,
    Linear e_k -> d_model, with cfg["enc_hidden"] = (e_1, ..., e_k)
  -> n_layers x [ h <- h + MambaBlock(RMSNorm(h)) ]
  -> final RMSNorm ("normalized again", section 5.2)
  -> masked mean-pool over the valid tokens of each program
  -> decoder Linear(d, h) -> ReLU -> Linear(h, 1) = score, or (the paper's
    three layers of widths 64, 32, 1) Linear(d, h) -> ReLU -> Linear(h, h2)
    -> ReLU -> Linear(h2, 1) with cfg["dec_hidden2"] = h2.
The paper names no activation inside its encoder and decoder; a ReLU sits
between consecutive Linear layers and none after the last one (a stack of
Linear layers without one would collapse to a single Linear).

Mamba block (the selective SSM that section 5.2 builds on):
  [x | z] = in_proj(n)                       (no bias)
  u       = SiLU(causal depthwise conv1d(x) + conv_b)
  [dt_r | B | C] = x_proj(u)                 (no bias)
  dt      = softplus(dt_proj(dt_r) + b_dt)
  A       = -exp(A_log)                      (diagonal, one row per channel)
  Eq. (4) discretised with zero-order hold on A and Euler on B:
      s_t = exp(dt_t * A) * s_{t-1} + dt_t * u_t * B_t,   s_{-1} = 0
  Eq. (5) read as y = C s (the printed C z' is taken as a typo):
      y_t = C_t . s_t + D * u_t
  out     = out_proj(y * SiLU(z))            (no bias)

Readings of points the paper leaves open (all listed in the design notes):
the conv is a cross-correlation with d_conv-1 zeros on the left of each
program (its last tap multiplies the current token); the x_proj output
splits as [dt_r (R), B (N), C (N)]; RMSNorm uses eps=1e-5 and a gain; the
state starts at zero for every program; padded tokens (t >= length) are
computed but excluded from the pool, so they cannot change any score.

Distillation step (the teacher -> student knowledge distillation of
section 6, with the loss simplified to two mean squared errors):
  L = mean_b (s_b - t_b)^2 + mean_b (s_b - y_b)^2
where t = frozen teacher scores and y = labels; gradients of every student
parameter by hand-derived reverse-mode differentiation (checked against
finite differences in the tests), then one bias-corrected Adam update.
"""
from __future__ import annotations

from typing import Dict, List, Tuple

import numpy as np

f64 = np.float64


# --------------------------------------------------------------------------
# parameter layout
# --------------------------------------------------------------------------

def encoder_dims(cfg: dict) -> List[int]:
    """Widths along the encoder: F, the hidden widths, d_model."""
    return [cfg["F"], *cfg.get("enc_hidden", ()), cfg["d_model"]]


def layout(cfg: dict) -> List[Tuple[str, Tuple[int, ...]]]:
    """Canonical flat-blob order: the encoder's Linear layers W0, b0 (then
    W0_1, b0_1, ... for a multi-layer encoder), per block [g, W_in, conv_w,
    conv_b, W_x, W_dt, b_dt, A_log, D, W_out], then g_f, W1, b1, W2, b2 (and
    W3, b3 for a three-layer decoder). Matrices are [out, in] row-major."""
    d, E, N = cfg["d_model"], cfg["d_inner"], cfg["d_state"]
    K, R, h = cfg["d_conv"], cfg["dt_rank"], cfg["head_hidden"]
    h2 = cfg.get("dec_hidden2", 0)
    dims = encoder_dims(cfg)
    names = []
    for i in range(len(dims) - 1):
        sfx = f"_{i}" if i else ""
        names += [(f"W0{sfx}", (dims[i + 1], dims[i])), (f"b0{sfx}", (dims[i + 1],))]
    for l in range(cfg["n_layers"]):
        p = f"blk{l}."
        names += [
            (p + "g", (d,)), (p + "W_in", (2 * E, d)), (p + "conv_w", (E, K)),
            (p + "conv_b", (E,)), (p + "W_x", (R + 2 * N, E)), (p + "W_dt", (E, R)),
            (p + "b_dt", (E,)), (p + "A_log", (E, N)), (p + "D", (E,)),
            (p + "W_out", (d, E)),
        ]
    names += [("g_f", (d,)), ("W1", (h, d)), ("b1", (h,))]
    if h2:
        names += [("W2", (h2, h)), ("b2", (h2,)), ("W3", (1, h2)), ("b3", (1,))]
    else:
        names += [("W2", (1, h)), ("b2", (1,))]
    return names


def unpack(blob, cfg: dict) -> Dict[str, np.ndarray]:
    blob = np.asarray(blob, dtype=f64)
    out, off = {}, 0
    for name, shape in layout(cfg):
        n = int(np.prod(shape))
        out[name] = blob[off:off + n].reshape(shape).copy()
        off += n
    if off != blob.size:
        raise ValueError(f"blob has {blob.size} values, layout needs {off}")
    return out


def pack(P: Dict[str, np.ndarray], cfg: dict) -> np.ndarray:
    return np.concatenate([np.asarray(P[n], dtype=f64).reshape(-1) for n, _ in layout(cfg)])


# --------------------------------------------------------------------------
# elementwise pieces
# --------------------------------------------------------------------------

def sigmoid(x):
    x = np.asarray(x, dtype=f64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def silu(x):
    return x * sigmoid(x)


def silu_grad(x):
    s = sigmoid(x)
    return s * (1.0 + x * (1.0 - s))


def softplus(x):
    """log(1 + e^x), written so it neither overflows nor loses digits."""
    x = np.asarray(x, dtype=f64)
    return np.maximum(x, 0.0) + np.log1p(np.exp(-np.abs(x)))


def rmsnorm(h, g, eps):
    """n = h * (mean(h^2) + eps)^(-1/2) * g over the last axis."""
    r = 1.0 / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps)
    return h * r * g, r


def rmsnorm_backward(dn, h, r, g):
    """Gradients of n = h*r*g: returns (dh, dg)."""
    d = h.shape[-1]
    dg = np.sum(dn * h * r, axis=tuple(range(h.ndim - 1)))
    gd = dn * g
    dh = r * gd - (r ** 3) / d * h * np.sum(gd * h, axis=-1, keepdims=True)
    return dh, dg


# --------------------------------------------------------------------------
# conv and scan
# --------------------------------------------------------------------------

def causal_conv1d(x, w, b):
    """xc[b,t,e] = b[e] + sum_k w[e,k] * x[b, t-(K-1)+k, e], x = 0 at t < 0."""
    Bn, L, E = x.shape
    K = w.shape[1]
    out = np.broadcast_to(b, (Bn, L, E)).astype(f64).copy()
    for k in range(K):
        shift = K - 1 - k  # how far back tap k looks
        if shift >= L:
            continue
        out[:, shift:, :] += w[:, k] * x[:, :L - shift, :]
    return out


def causal_conv1d_backward(dxc, x, w):
    Bn, L, E = x.shape
    K = w.shape[1]
    dx = np.zeros_like(x)
    dw = np.zeros_like(w)
    for k in range(K):
        shift = K - 1 - k
        if shift >= L:
            continue
        dx[:, :L - shift, :] += w[:, k] * dxc[:, shift:, :]
        dw[:, k] = np.sum(dxc[:, shift:, :] * x[:, :L - shift, :], axis=(0, 1))
    db = np.sum(dxc, axis=(0, 1))
    return dx, dw, db


def selective_scan(u, dt, A, Bm, Cm, D, return_states=False):
    """Sequential recurrence of Eq. (4)-(5) after discretisation.

    u, dt: [B,L,E]; A: [E,N]; Bm, Cm: [B,L,N]; D: [E].
    s_t = exp(dt_t A) * s_{t-1} + (dt_t u_t) B_t ; y_t = sum_n C_t s_t + D u_t.
    """
    Bn, L, E = u.shape
    N = A.shape[1]
    s = np.zeros((Bn, E, N), dtype=f64)
    y = np.empty((Bn, L, E), dtype=f64)
    states = np.empty((Bn, L, E, N), dtype=f64) if return_states else None
    for t in range(L):
        a = np.exp(dt[:, t, :, None] * A[None, :, :])
        s = a * s + (dt[:, t, :] * u[:, t, :])[:, :, None] * Bm[:, t, None, :]
        y[:, t, :] = np.einsum("ben,bn->be", s, Cm[:, t, :]) + D * u[:, t, :]
        if return_states:
            states[:, t] = s
    return (y, states) if return_states else y


def selective_scan_backward(dy, u, dt, A, Bm, Cm, D, states):
    """Reverse-mode gradients of selective_scan.

    With a_t = exp(dt_t A), the adjoint of the state obeys
      g_t = C_t * dy_t + a_{t+1} * g_{t+1}   (g_L = 0),
    and each input's gradient collects the terms where it enters s_t or y_t.
    Returns du, ddt, dA, dB, dC, dD.
    """
    Bn, L, E = u.shape
    N = A.shape[1]
    du = dy * D
    dD = np.sum(dy * u, axis=(0, 1))
    ddt = np.zeros_like(dt)
    dA = np.zeros_like(A)
    dB = np.zeros_like(Bm)
    dC = np.einsum("bte,bten->btn", dy, states)
    g = np.zeros((Bn, E, N), dtype=f64)
    a_next = np.zeros((Bn, E, N), dtype=f64)
    for t in range(L - 1, -1, -1):
        g = dy[:, t, :, None] * Cm[:, t, None, :] + a_next * g
        a_t = np.exp(dt[:, t, :, None] * A[None])
        s_prev = states[:, t - 1] if t > 0 else np.zeros((Bn, E, N), dtype=f64)
        # s_t = a_t * s_prev + dt u B
        du[:, t, :] += dt[:, t, :] * np.einsum("ben,bn->be", g, Bm[:, t, :])
        dB[:, t, :] = np.einsum("ben,be->bn", g, dt[:, t, :] * u[:, t, :])
        da = g * s_prev  # d/d a_t
        ddt[:, t, :] = (np.einsum("ben,bn->be", g, Bm[:, t, :]) * u[:, t, :]
                        + np.sum(da * a_t * A[None], axis=-1))
        dA += np.sum(da * a_t * dt[:, t, :, None], axis=0)
        a_next = a_t
    return du, ddt, dA, dB, dC, dD


# --------------------------------------------------------------------------
# model
# --------------------------------------------------------------------------

def _block_forward(h, P, l, cfg, keep):
    p = f"blk{l}."
    E, N, R = cfg["d_inner"], cfg["d_state"], cfg["dt_rank"]
    n, r = rmsnorm(h, P[p + "g"], cfg["norm_eps"])
    xz = n @ P[p + "W_in"].T
    xs, z = xz[..., :E], xz[..., E:]
    xc = causal_conv1d(xs, P[p + "conv_w"], P[p + "conv_b"])
    u = silu(xc)
    xdbl = u @ P[p + "W_x"].T
    dtr, Bm, Cm = xdbl[..., :R], xdbl[..., R:R + N], xdbl[..., R + N:]
    v = dtr @ P[p + "W_dt"].T + P[p + "b_dt"]
    dt = softplus(v)
    A = -np.exp(P[p + "A_log"])
    if keep:
        y, states = selective_scan(u, dt, A, Bm, Cm, P[p + "D"], return_states=True)
    else:
        y, states = selective_scan(u, dt, A, Bm, Cm, P[p + "D"]), None
    yg = y * silu(z)
    out = h + yg @ P[p + "W_out"].T
    cache = None
    if keep:
        cache = dict(h=h, n=n, r=r, xs=xs, z=z, xc=xc, u=u, dtr=dtr, Bm=Bm, Cm=Cm,
                     v=v, dt=dt, A=A, y=y, states=states, yg=yg)
    return out, cache


def _block_backward(dout, P, l, cfg, c, G):
    p = f"blk{l}."
    E = cfg["d_inner"]
    dh = dout.copy()                                   # residual path
    G[p + "W_out"] = np.einsum("btd,bte->de", dout, c["yg"])
    dyg = dout @ P[p + "W_out"]
    sz = silu(c["z"])
    dy = dyg * sz
    dz = dyg * c["y"] * silu_grad(c["z"])
    du, ddt, dA, dB, dC, dD = selective_scan_backward(
        dy, c["u"], c["dt"], c["A"], c["Bm"], c["Cm"], P[p + "D"], c["states"])
    G[p + "D"] = dD
    G[p + "A_log"] = dA * c["A"]                       # A = -exp(A_log)
    dv = ddt * sigmoid(c["v"])                         # softplus' = sigmoid
    G[p + "W_dt"] = np.einsum("bte,btr->er", dv, c["dtr"])
    G[p + "b_dt"] = np.sum(dv, axis=(0, 1))
    ddtr = dv @ P[p + "W_dt"]
    dxdbl = np.concatenate([ddtr, dB, dC], axis=-1)
    G[p + "W_x"] = np.einsum("btj,bte->je", dxdbl, c["u"])
    du = du + dxdbl @ P[p + "W_x"]
    dxc = du * silu_grad(c["xc"])
    dxs, dcw, dcb = causal_conv1d_backward(dxc, c["xs"], P[p + "conv_w"])
    G[p + "conv_w"] = dcw
    G[p + "conv_b"] = dcb
    dxz = np.concatenate([dxs, dz], axis=-1)
    n = c["n"]
    G[p + "W_in"] = np.einsum("btj,btd->jd", dxz, n)
    dn = dxz @ P[p + "W_in"]
    dh_n, dg = rmsnorm_backward(dn, c["h"], c["r"], P[p + "g"])
    G[p + "g"] = dg
    return dh + dh_n


def forward(P, X, lengths, cfg, keep=False):
    """Scores [B] (and, with keep=True, every intermediate for backward)."""
    X = np.asarray(X, dtype=f64)
    lengths = np.asarray(lengths)
    Bn, L, _ = X.shape
    h = X @ P["W0"].T + P["b0"]
    for i in range(1, len(encoder_dims(cfg)) - 1):
        h = np.maximum(h, 0.0) @ P[f"W0_{i}"].T + P[f"b0_{i}"]
    caches = []
    for l in range(cfg["n_layers"]):
        h, c = _block_forward(h, P, l, cfg, keep)
        caches.append(c)
    if cfg.get("final_norm", 1):
        hf, rf = rmsnorm(h, P["g_f"], cfg["norm_eps"])
    else:
        hf, rf = h, None
    mask = (np.arange(L)[None, :] < lengths[:, None]).astype(f64)
    pooled = np.sum(hf * mask[:, :, None], axis=1) / lengths[:, None].astype(f64)
    a1 = pooled @ P["W1"].T + P["b1"]
    r1 = np.maximum(a1, 0.0)
    if cfg.get("dec_hidden2", 0):
        r2 = np.maximum(r1 @ P["W2"].T + P["b2"], 0.0)
        s = (r2 @ P["W3"].T)[:, 0] + P["b3"][0]
    else:
        s = (r1 @ P["W2"].T)[:, 0] + P["b2"][0]
    if not keep:
        return s
    if cfg.get("enc_hidden") or cfg.get("dec_hidden2", 0):
        raise NotImplementedError("gradients cover the one-Linear encoder and two-layer decoder")
    top = dict(X=X, h_last=h, hf=hf, rf=rf, mask=mask, lengths=lengths,
               pooled=pooled, a1=a1, r1=r1)
    return s, caches, top


def score(blob, X, lengths, cfg):
    """Candidate scores [B] for a flat parameter blob (higher ranks first)."""
    return forward(unpack(blob, cfg), X, lengths, cfg)


def backward(ds, P, cfg, caches, top):
    """Gradients of sum_b ds_b * s_b with respect to every parameter."""
    G: Dict[str, np.ndarray] = {}
    G["W2"] = (ds @ top["r1"])[None, :]
    G["b2"] = np.array([np.sum(ds)])
    dr1 = ds[:, None] * P["W2"][0][None, :]
    da1 = dr1 * (top["a1"] > 0)
    G["W1"] = da1.T @ top["pooled"]
    G["b1"] = np.sum(da1, axis=0)
    dpooled = da1 @ P["W1"]
    lengths = top["lengths"].astype(f64)
    dhf = (dpooled / lengths[:, None])[:, None, :] * top["mask"][:, :, None]
    if cfg.get("final_norm", 1):
        dh, G["g_f"] = rmsnorm_backward(dhf, top["h_last"], top["rf"], P["g_f"])
    else:
        dh, G["g_f"] = dhf, np.zeros_like(P["g_f"])
    for l in range(cfg["n_layers"] - 1, -1, -1):
        dh = _block_backward(dh, P, l, cfg, caches[l], G)
    G["W0"] = np.einsum("btd,btf->df", dh, top["X"])
    G["b0"] = np.sum(dh, axis=(0, 1))
    return G


# --------------------------------------------------------------------------
# distillation step
# --------------------------------------------------------------------------

def distill_loss(s, t, y):
    """(total, mse_teacher, mse_label) and dL/ds for L = mse(s,t) + mse(s,y)."""
    Bn = s.shape[0]
    mt = np.mean((s - t) ** 2)
    ml = np.mean((s - y) ** 2)
    ds = (2.0 / Bn) * (s - t) + (2.0 / Bn) * (s - y)
    return (mt + ml, mt, ml), ds


def adam_update(p, g, m, v, step, lr, beta1=0.9, beta2=0.999, eps=1e-8):
    """One bias-corrected Adam step (no weight decay); step counts from 1."""
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** step)
    vhat = v / (1.0 - beta2 ** step)
    return p - lr * mhat / (np.sqrt(vhat) + eps), m, v


def distill_step(teacher_blob, tcfg, student_blob, scfg, X, lengths, labels,
                 m=None, v=None, step=1, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                 compute_blob=None, teacher_scores=None):
    """One teacher->student step.

    `student_blob` holds the master weights that Adam updates; the forward and
    backward use `compute_blob` when given (the bf16-rounded copy of the
    master), else the master itself. `teacher_scores`, when given, are the
    teacher's scores of this batch (saves recomputing them).
    Returns dict(loss=(total, mt, ml), teacher=t, student=s, grad=flat,
    params=new master, m=, v=).
    """
    if teacher_scores is None:
        t = score(teacher_blob, X, lengths, tcfg)
    else:
        t = np.asarray(teacher_scores, dtype=f64)
    P = unpack(student_blob if compute_blob is None else compute_blob, scfg)
    s, caches, top = forward(P, X, lengths, scfg, keep=True)
    loss, ds = distill_loss(s, t, np.asarray(labels, dtype=f64))
    G = backward(ds, P, scfg, caches, top)
    g = pack(G, scfg)
    p = np.asarray(student_blob, dtype=f64)
    m = np.zeros_like(p) if m is None else np.asarray(m, dtype=f64)
    v = np.zeros_like(p) if v is None else np.asarray(v, dtype=f64)
    p2, m2, v2 = adam_update(p, g, m, v, step, lr, beta1, beta2, eps)
    return dict(loss=loss, teacher=t, student=s, grad=g, params=p2, m=m2, v=v2)
