"""Kernel-level parity on the GPU: each kernel through its own C-ABI entry
point against the oracle's matching piece on the same seeded inputs.

Tolerances are derived from the fp32 arithmetic each kernel performs:
  GEMM:  |c - c*| <= (K + 2) 2^-24 sum_k |a_k w_k|  (worst-case bound of an
         fp32 dot product of length K; inputs are exact in fp64)
  conv:  rtol 1e-5 on a scale of |b| + sum |w x| (4 FMAs, expf, one divide)
  scan:  rtol 1e-4 on the output scale (16-term state sums over <= L steps,
         exp2 of v_exp_f32, log1pf/expf in softplus)
"""
import numpy as np
import pytest
import torch

from oracle import model as om
from paper_2604_12891_amd import binding as tb
from paper_2604_12891_amd import workload as wl

pytestmark = pytest.mark.gpu
U = 2.0 ** -24


def _dev(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


def _offs(lengths):
    return np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)


def _pack(padded, lengths):
    return np.concatenate([padded[b, :lengths[b]] for b in range(len(lengths))], axis=0)


def _unpack(packed, lengths, L):
    B = len(lengths)
    out = np.zeros((B, L) + packed.shape[1:], dtype=packed.dtype)
    o = _offs(lengths)
    for b in range(B):
        out[b, :lengths[b]] = packed[o[b]:o[b + 1]]
    return out


@pytest.mark.parametrize("M,N,K", [(1, 64, 4), (31, 48, 512), (129, 256, 164), (1000, 1024, 256),
                                   (257, 256, 512), (77, 100, 36)])
@pytest.mark.parametrize("bias", [False, True])
@pytest.mark.parametrize("tile", [-1, 2, 3, 4, 5, 6, 7])
def test_gemm_f32(M, N, K, bias, tile):
    print(f"gemm M={M} N={N} K={K} bias={bias} tile={tile}", flush=True)
    rng = np.random.default_rng(M * 7 + N + K)
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = rng.standard_normal((N, K)).astype(np.float32)
    bv = rng.standard_normal(N).astype(np.float32) if bias else None
    C = tb.gemm_f32(_dev(A), _dev(W), _dev(bv) if bias else None, tile=tile)
    torch.cuda.synchronize()
    ref = A.astype(np.float64) @ W.astype(np.float64).T
    bound = (K + 2) * U * (np.abs(A).astype(np.float64) @ np.abs(W).astype(np.float64).T)
    if bias:
        ref += bv
        bound += U * np.abs(ref)
    err = np.abs(C.cpu().numpy() - ref)
    assert np.all(err <= bound + 1e-30), float(np.max(err / (bound + 1e-30)))


@pytest.mark.parametrize("M,N,K", [(77, 100, 36), (1000, 1024, 256), (257, 256, 512)])
@pytest.mark.parametrize("tile", [-1, 0, 3, 5, 7])
@pytest.mark.parametrize("epilogue", [1, 2])
def test_gemm_f32_epilogues(M, N, K, tile, epilogue):
    """The residual (C += A W^T, in place) and RMSNorm row-scale epilogues."""
    print(f"gemm epilogue={epilogue} M={M} N={N} K={K} tile={tile}", flush=True)
    rng = np.random.default_rng(M + 3 * N + 7 * K + epilogue)
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = rng.standard_normal((N, K)).astype(np.float32)
    C0 = rng.standard_normal((M, N)).astype(np.float32)
    C = _dev(C0)
    tb.gemm_f32(_dev(A), _dev(W), out=C, tile=tile, epilogue=epilogue)
    torch.cuda.synchronize()
    A64, W64 = A.astype(np.float64), W.astype(np.float64)
    prod = A64 @ W64.T
    bound = (K + 2) * U * (np.abs(A64) @ np.abs(W64).T)
    if epilogue == 1:
        ref = C0 + prod
        bound = bound + U * np.abs(ref)
    else:
        rstd = 1.0 / np.sqrt(np.mean(A64 * A64, axis=1, keepdims=True) + 1e-5)
        ref = rstd * prod
        bound = rstd * bound + (K + 8) * U * np.abs(ref)  # the row statistic's own rounding
    err = np.abs(C.cpu().numpy() - ref)
    assert np.all(err <= bound + 1e-30), float(np.max(err / (bound + 1e-30)))


@pytest.mark.parametrize("M,N,K", [(1, 64, 64), (300, 100, 128), (1000, 256, 164), (777, 1024, 256),
                                   (129, 36, 256), (40000, 96, 192)])
@pytest.mark.parametrize("mode", ["plain", "bias", "norm"])
def test_gemm_f32_row_panels(M, N, K, mode):
    """Row-panel tile (A held in registers): plain, + bias, RMSNorm row scale;
    ragged M and N, every supported K."""
    print(f"gemm panel mode={mode} M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M + 5 * N + 11 * K + len(mode))
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = rng.standard_normal((N, K)).astype(np.float32)
    bv = rng.standard_normal(N).astype(np.float32) if mode == "bias" else None
    C = tb.gemm_f32(_dev(A), _dev(W), _dev(bv) if bv is not None else None, tile=8,
                    epilogue=2 if mode == "norm" else 0)
    torch.cuda.synchronize()
    A64, W64 = A.astype(np.float64), W.astype(np.float64)
    ref = A64 @ W64.T
    bound = (K + 2) * U * (np.abs(A64) @ np.abs(W64).T)
    if mode == "bias":
        ref += bv
        bound += U * np.abs(ref)
    elif mode == "norm":
        rstd = 1.0 / np.sqrt(np.mean(A64 * A64, axis=1, keepdims=True) + 1e-5)
        ref = rstd * ref
        bound = rstd * bound + (K + 8) * U * np.abs(ref)
    err = np.abs(C.cpu().numpy() - ref)
    assert np.all(err <= bound + 1e-30), float(np.max(err / (bound + 1e-30)))


@pytest.mark.parametrize("M,N,K", [(1, 64, 512), (300, 100, 384), (777, 256, 512), (1000, 48, 256),
                                   (40000, 96, 500)])
@pytest.mark.parametrize("mode", ["plain", "bias", "resid"])
def test_gemm_f32_row_panels16(M, N, K, mode):
    """16-row panels (16x16 MFMA blocks, K up to 512): plain, + bias, and the
    residual epilogue C += A W^T in place; ragged M, N and K."""
    print(f"gemm panel16 mode={mode} M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M + 7 * N + 13 * K + len(mode))
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = rng.standard_normal((N, K)).astype(np.float32)
    bv = rng.standard_normal(N).astype(np.float32) if mode == "bias" else None
    C0 = rng.standard_normal((M, N)).astype(np.float32)
    C = _dev(C0)
    tb.gemm_f32(_dev(A), _dev(W), _dev(bv) if bv is not None else None, out=C, tile=9,
                epilogue=1 if mode == "resid" else 0)
    torch.cuda.synchronize()
    A64, W64 = A.astype(np.float64), W.astype(np.float64)
    ref = A64 @ W64.T
    bound = (K + 2) * U * (np.abs(A64) @ np.abs(W64).T)
    if mode == "bias":
        ref += bv
    elif mode == "resid":
        ref += C0
    if mode != "plain":
        bound += U * np.abs(ref)
    err = np.abs(C.cpu().numpy() - ref)
    assert np.all(err <= bound + 1e-30), float(np.max(err / (bound + 1e-30)))


def test_gemm_f32_row_panels_refuse_unsupported():
    """No residual epilogue and only K in {64, 128, 164, 192, 256} on 32-row
    panels; no RMSNorm on 16-row panels."""
    rng = np.random.default_rng(9)
    A = _dev(rng.standard_normal((64, 256)).astype(np.float32))
    W = _dev(rng.standard_normal((64, 256)).astype(np.float32))
    with pytest.raises(tb.TclError):
        tb.gemm_f32(A, W, out=torch.zeros(64, 64, device="cuda"), tile=8, epilogue=1)
    A2 = _dev(rng.standard_normal((64, 100)).astype(np.float32))
    W2 = _dev(rng.standard_normal((64, 100)).astype(np.float32))
    with pytest.raises(tb.TclError):
        tb.gemm_f32(A2, W2, tile=8)
    with pytest.raises(tb.TclError):
        tb.gemm_f32(A, W, tile=9, epilogue=2)


@pytest.mark.parametrize("M,N,K", [(1, 64, 8), (31, 48, 512), (129, 256, 168), (1000, 1024, 256),
                                   (257, 256, 512), (77, 100, 40)])
@pytest.mark.parametrize("bias", [False, True])
def test_gemm_bf16(M, N, K, bias):
    """bf16 x bf16 products are exact in fp32; only the fp32 accumulation rounds."""
    print(f"gemm_bf16 M={M} N={N} K={K} bias={bias}", flush=True)
    rng = np.random.default_rng(M * 5 + N + K)
    A = wl.round_to_bf16(rng.standard_normal((M, K)).astype(np.float32))
    W = wl.round_to_bf16(rng.standard_normal((N, K)).astype(np.float32))
    bv = rng.standard_normal(N).astype(np.float32) if bias else None
    C = tb.gemm_bf16(_dev(A, torch.bfloat16), _dev(W, torch.bfloat16), _dev(bv) if bias else None)
    torch.cuda.synchronize()
    ref = A.astype(np.float64) @ W.astype(np.float64).T
    bound = (K + 2) * U * (np.abs(A).astype(np.float64) @ np.abs(W).astype(np.float64).T)
    if bias:
        ref += bv
        bound += U * np.abs(ref)
    err = np.abs(C.cpu().numpy() - ref)
    assert np.all(err <= bound + 1e-30), float(np.max(err / (bound + 1e-30)))


@pytest.mark.parametrize("B,L", [(1, 25), (37, 25), (4096, 25), (32768, 25), (40001, 4096), (5000, 4097),
                                 (1000, 1)])
def test_offsets_and_longest_first_order(B, L):
    """Index work, bit-exact: the packed offsets are the prefix sums of the
    valid lengths (a length outside [1, L] packs nothing); for L <= 4096 the
    order is a permutation of the programs by non-increasing valid length
    (equal lengths may come in any order), above that it is not written.
    Also with the lengths at a 4-byte offset (the kernel's scalar path)."""
    print(f"offsets B={B} L={L}", flush=True)
    rng = np.random.default_rng(B + L)
    lengths = rng.integers(1, L + 1, size=B + 1).astype(np.int32)
    if B >= 8:
        bad = rng.choice(B, size=3, replace=False)
        lengths[bad] = (0, -3, L + 1)
    for shift in (0, 1):
        ln = lengths[shift:shift + B]
        Ld = torch.from_numpy(lengths).cuda()[shift:shift + B]
        ordd = torch.full((B,), -7, dtype=torch.int32, device="cuda")
        offs = tb.offsets(Ld, L, ord=ordd)
        torch.cuda.synchronize()
        valid = np.where((ln >= 1) & (ln <= L), ln, 0).astype(np.int64)
        assert np.array_equal(offs.cpu().numpy(), np.concatenate([[0], np.cumsum(valid)])), (B, L, shift)
        o = ordd.cpu().numpy()
        if L <= 4096:
            assert np.array_equal(np.sort(o), np.arange(B)), "not a permutation"
            v = valid[o]
            assert np.all(v[:-1] >= v[1:]), "not longest first"
        else:
            assert np.all(o == -7), "the order was written above the limit"


def _bf16_w(N, K, rng):
    """W [N, round_up(K, 8)] bf16-exact, zero-padded in K as the kernels expect."""
    Kw = (K + 7) // 8 * 8
    W = np.zeros((N, Kw), np.float32)
    W[:, :K] = wl.round_to_bf16(rng.standard_normal((N, K)).astype(np.float32))
    return W


_BF16_KINDS = ["f32", "bf16", "norm", "resid", "gather", "f32a", "f32a_resid"]


@pytest.mark.parametrize("tile", [-1, 0, 1, 2, 3, 4, 5, 6, 7, 8])
@pytest.mark.parametrize("kind", _BF16_KINDS)
def test_gemm_bf16_variants(kind, tile):
    """Every bf16 GEMM variant the model runs, on every tile, with ragged M, N
    and K. Where the kernel rounds an fp32 operand to bf16 (A, or A * gain),
    the same rounding is applied on the host first (the products of bf16
    values are then exact), so the bound is that of fp32 accumulation, plus
    the bf16 unit roundoff 2^-8 where the output is bf16."""
    print(f"gemm_bf16 kind={kind} tile={tile}", flush=True)
    rng = np.random.default_rng(_BF16_KINDS.index(kind) * 10 + tile + 1)
    f32a = kind in ("norm", "gather", "f32a", "f32a_resid")
    if kind.startswith("f32a") and tile in (7, 8):
        # the fp32-A kinds (the distillation backward) run on tiles only: an
        # explicit row-panel tile is refused
        A = _dev(rng.standard_normal((64, 164)).astype(np.float32))
        W = _dev(_bf16_w(196, 164, rng), torch.bfloat16)
        out = torch.zeros(64, 196, device="cuda")
        k = tb.GEMM_BF16_F32A if kind == "f32a" else tb.GEMM_BF16_F32A_RESID
        with pytest.raises(tb.TclError):
            tb.gemm_bf16(A, W, out=out, kind=k, tile=tile)
        return
    # bf16 rows of C must be 16-byte aligned for the row-panel tile
    M, N, K = 1000, (200 if kind in ("bf16", "norm") else 196), (164 if f32a else 168)
    W = _bf16_w(N, K, rng)
    Wk = W[:, :K].astype(np.float64)
    bv = rng.standard_normal(N).astype(np.float32)
    gain = (1.0 + 0.5 * rng.standard_normal(K)).astype(np.float32)
    Wd = _dev(W, torch.bfloat16)
    if kind == "gather":
        lengths = rng.integers(0, 26, size=45).astype(np.int32)
        lengths[3] = 0
        lengths[7] = 25
        Bp, L = len(lengths), 25
        Ap = rng.standard_normal((Bp, L, K)).astype(np.float32)
        out = torch.full((Bp * L, N), float("nan"), device="cuda")
        tb.gemm_bf16(_dev(Ap), Wd, bias=_dev(bv), out=out, kind=tb.GEMM_BF16_GATHER, tile=tile,
                     offs=_dev(_offs(lengths), torch.int32))
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        Mv = int(lengths.sum())
        assert np.all(np.isnan(got[Mv:])), "rows past the packed tokens were written"
        got = got[:Mv]
        Ah = wl.round_to_bf16(_pack(Ap, lengths)).astype(np.float64)
        ref = Ah @ Wk.T + bv
        bound = (K + 2) * U * (np.abs(Ah) @ np.abs(Wk).T) + U * np.abs(ref)
    elif kind in ("f32a", "f32a_resid"):
        A = (2.0 * rng.standard_normal((M, K))).astype(np.float32)
        Ah = wl.round_to_bf16(A).astype(np.float64)  # the kernel rounds A to bf16 (RNE) as it stages it
        prod = Ah @ Wk.T
        mag = (K + 2) * U * (np.abs(Ah) @ np.abs(Wk).T)
        if kind == "f32a":
            got = tb.gemm_bf16(_dev(A), Wd, kind=tb.GEMM_BF16_F32A, tile=tile)
            ref, bound = prod, mag + U * np.abs(prod)
        else:
            C0 = rng.standard_normal((M, N)).astype(np.float32)
            got = _dev(C0)
            tb.gemm_bf16(_dev(A), Wd, out=got, kind=tb.GEMM_BF16_F32A_RESID, tile=tile)
            ref, bound = C0 + prod, mag + U * np.abs(C0 + prod)
        torch.cuda.synchronize()
        got = got.cpu().numpy()
    elif kind == "norm":
        A = (3.0 * rng.standard_normal((M, K))).astype(np.float32)
        out = tb.gemm_bf16(_dev(A), Wd, gain=_dev(gain), kind=tb.GEMM_BF16_NORM, tile=tile)
        torch.cuda.synchronize()
        got = out.float().cpu().numpy()
        Ah = wl.round_to_bf16(A * gain[None, :]).astype(np.float64)  # fp32 product, then RNE
        rstd = 1.0 / np.sqrt(np.mean(A.astype(np.float64) ** 2, axis=1) + 1e-5)
        ref = rstd[:, None] * (Ah @ Wk.T)
        bound = ((K + 4) * U * rstd[:, None] * (np.abs(Ah) @ np.abs(Wk).T)
                 + (2.0 ** -8 + 8 * U) * np.abs(ref))
    else:
        A = wl.round_to_bf16(rng.standard_normal((M, K)).astype(np.float32))
        Ad = _dev(A, torch.bfloat16)
        A64 = A.astype(np.float64)
        prod = A64 @ Wk.T
        mag = (K + 2) * U * (np.abs(A64) @ np.abs(Wk).T)
        if kind == "f32":
            got = tb.gemm_bf16(Ad, Wd, bias=_dev(bv), kind=tb.GEMM_BF16_F32, tile=tile)
            ref, bound = prod + bv, mag + U * np.abs(prod + bv)
        elif kind == "bf16":
            got = tb.gemm_bf16(Ad, Wd, kind=tb.GEMM_BF16_BF16, tile=tile)
            ref, bound = prod, mag + 2.0 ** -8 * np.abs(prod) * (1 + 1e-3)
        else:
            C0 = rng.standard_normal((M, N)).astype(np.float32)
            got = _dev(C0)
            tb.gemm_bf16(Ad, Wd, out=got, kind=tb.GEMM_BF16_RESID, tile=tile)
            ref, bound = C0 + prod, mag + U * np.abs(C0 + prod)
        torch.cuda.synchronize()
        got = got.float().cpu().numpy()
    err = np.abs(got.astype(np.float64) - ref)
    assert np.all(err <= bound + 1e-30), (kind, tile, float(np.max(err / (bound + 1e-30))))


def test_gemm_bf16_panel_rejects_unaligned_rows():
    """The row-panel tile stores 16-byte row segments: bf16 rows of 196
    columns (392 bytes) are refused when it is asked for explicitly, and the
    model's tile choice falls back to the tiled kernel for them."""
    rng = np.random.default_rng(3)
    M = 140000  # enough rows for the model's policy to want row panels
    A = _dev(wl.round_to_bf16(rng.standard_normal((M, 64)).astype(np.float32)), torch.bfloat16)
    W = _dev(_bf16_w(196, 64, rng), torch.bfloat16)
    with pytest.raises(tb.TclError):
        tb.gemm_bf16(A, W, kind=tb.GEMM_BF16_BF16, tile=7)
    out = tb.gemm_bf16(A, W, kind=tb.GEMM_BF16_BF16, tile=-1)
    torch.cuda.synchronize()
    ref = A.float().cpu().numpy().astype(np.float64) @ W.float().cpu().numpy().astype(np.float64).T
    np.testing.assert_allclose(out.float().cpu().numpy(), ref, rtol=2.0 ** -7, atol=1e-3)


@pytest.mark.parametrize("K", [1, 3, 4])
def test_conv_silu_f32(K):
    rng = np.random.default_rng(K)
    lengths = np.array([1, 2, 3, 4, 25, 0, 17, 5, 9], dtype=np.int32)
    B, L, E, ldx = len(lengths), 25, 192, 448
    print(f"conv K={K} B={B} E={E}", flush=True)
    x = rng.standard_normal((B, L, E))
    w = rng.uniform(-0.5, 0.5, (E, K))
    b = rng.uniform(-0.5, 0.5, E)
    xp = np.zeros((int(lengths.sum()), ldx), np.float32)
    xp[:, :E] = _pack(x, lengths)
    out = torch.full((int(lengths.sum()), E), float("nan"), device="cuda")
    tb.conv_silu_f32(_dev(_offs(lengths), torch.int32), _dev(xp), _dev(w.astype(np.float32)),
                     _dev(b.astype(np.float32)), E, out, ldx=ldx)
    torch.cuda.synchronize()
    xr = _unpack(xp[:, :E].astype(np.float64), lengths, L)
    wf, bf = w.astype(np.float32).astype(np.float64), b.astype(np.float32).astype(np.float64)
    expect = _pack(om.silu(om.causal_conv1d(xr, wf, bf)), lengths)
    scale = np.abs(bf) + _pack(om.causal_conv1d(np.abs(xr), np.abs(wf), 0 * bf), lengths)
    np.testing.assert_array_less(np.abs(out.cpu().numpy() - expect), 1e-5 * scale + 1e-7)


@pytest.mark.parametrize("E,N", [(512, 48), (128, 20), (64, 64), (320, 33)])
def test_xproj_conv_f32(E, N):
    """The fused conv + SiLU + x_proj kernel: u is the same bits as the
    stand-alone conv kernel's, both within the conv bound of the oracle's
    conv, and xdbl = u W^T within the split GEMM's fp32 bound. Programs of
    length 1..4 around wavefront and panel edges, an empty program, a
    ragged last panel, and a row count bound above the packed rows."""
    rng = np.random.default_rng(E + N)
    L = 40
    lengths = np.concatenate([[1, 2, 3, 4, 0, 40, 31, 33, 1, 1, 1, 29, 3], rng.integers(1, L + 1, 60)])
    lengths = lengths.astype(np.int32)
    B = len(lengths)
    M = int(lengths.sum())
    rows = M + 77
    ldx = 2 * E
    print(f"xproj_conv E={E} N={N} B={B} M={M}", flush=True)
    x = rng.standard_normal((B, L, E))
    w = rng.uniform(-0.5, 0.5, (E, 4)).astype(np.float32)
    b = rng.uniform(-0.5, 0.5, E).astype(np.float32)
    W = (rng.uniform(-1, 1, (N, E)) / np.sqrt(E)).astype(np.float32)
    xp = rng.standard_normal((rows, ldx)).astype(np.float32)  # rows past M and the z half: noise
    xp[:M, :E] = _pack(x, lengths)
    offs = _dev(_offs(lengths), torch.int32)
    u, xdbl = tb.xproj_conv_f32(offs, _dev(xp), _dev(w), _dev(b), _dev(W), rows, E, ldx=ldx)
    ref_u = torch.full((M, E), float("nan"), device="cuda")
    tb.conv_silu_f32(offs, _dev(xp), _dev(w), _dev(b), E, ref_u, ldx=ldx)
    torch.cuda.synchronize()
    u, xdbl, ref_u = u.cpu().numpy(), xdbl.cpu().numpy(), ref_u.cpu().numpy()
    assert np.all(np.isnan(u[M:])) and np.all(np.isnan(xdbl[M:]))
    np.testing.assert_array_equal(u[:M].view(np.uint32), ref_u.view(np.uint32))
    xr = _unpack(xp[:M, :E].astype(np.float64), lengths, L)
    wf, bf = w.astype(np.float64), b.astype(np.float64)
    expect = _pack(om.silu(om.causal_conv1d(xr, wf, bf)), lengths)
    scale = np.abs(bf) + _pack(om.causal_conv1d(np.abs(xr), np.abs(wf), 0 * bf), lengths)
    np.testing.assert_array_less(np.abs(u[:M] - expect), 1e-5 * scale + 1e-7)
    ref, bound = _split_ref(u[:M], W, "plain")
    err = np.abs(xdbl[:M] - ref)
    assert np.all(err <= bound + 1e-30), float(np.max(err / (bound + 1e-30)))


@pytest.mark.parametrize("E,N", [(512, 48), (128, 20), (256, 64)])
def test_xproj_conv_bf16(E, N):
    """The bf16 fused kernel: u (bf16) within the conv bound of the oracle's
    conv plus one bf16 rounding, and xdbl = u W^T from the kernel's own bf16
    u within the fp32 accumulation bound (bf16 products are exact); program
    edges around wavefront and panel boundaries, an empty program, a ragged
    last panel."""
    rng = np.random.default_rng(E + 3 * N)
    L = 40
    lengths = np.concatenate([[1, 2, 3, 4, 0, 40, 31, 33, 1, 1, 1, 29, 3], rng.integers(1, L + 1, 60)])
    lengths = lengths.astype(np.int32)
    B = len(lengths)
    M = int(lengths.sum())
    rows = M + 77
    ldx = 2 * E
    print(f"xproj_conv_bf16 E={E} N={N} B={B} M={M}", flush=True)
    xp = torch.from_numpy(rng.standard_normal((rows, ldx)).astype(np.float32)).to(torch.bfloat16)
    w = rng.uniform(-0.5, 0.5, (E, 4)).astype(np.float32)
    b = rng.uniform(-0.5, 0.5, E).astype(np.float32)
    W = torch.from_numpy((rng.uniform(-1, 1, (N, E)) / np.sqrt(E)).astype(np.float32)).to(torch.bfloat16)
    offs = _dev(_offs(lengths), torch.int32)
    u, xdbl = tb.xproj_conv_bf16(offs, xp.cuda(), _dev(w), _dev(b), W.cuda(), rows, E, ldx=ldx)
    torch.cuda.synchronize()
    u = u.float().cpu().numpy().astype(np.float64)
    xdbl = xdbl.cpu().numpy()
    assert np.all(np.isnan(xdbl[M:])) and np.all(u[M:] == 0)
    xf = xp.float().numpy().astype(np.float64)[:M, :E]
    xr = _unpack(xf, lengths, L)
    wf, bf = w.astype(np.float64), b.astype(np.float64)
    expect = _pack(om.silu(om.causal_conv1d(xr, wf, bf)), lengths)
    scale = np.abs(bf) + _pack(om.causal_conv1d(np.abs(xr), np.abs(wf), 0 * bf), lengths)
    np.testing.assert_array_less(np.abs(u[:M] - expect), 1e-5 * scale + 2.0 ** -8 * np.abs(expect) + 1e-7)
    W64 = W.float().numpy().astype(np.float64)
    ref = u[:M] @ W64.T
    bound = (E + 2) * U * (np.abs(u[:M]) @ np.abs(W64).T)
    err = np.abs(xdbl[:M] - ref)
    assert np.all(err <= bound + 1e-30), float(np.max(err / (bound + 1e-30)))


def test_xproj_conv_rejects_unsupported():
    offs = _dev(_offs(np.array([3, 2], np.int32)), torch.int32)
    for E, N in [(96, 48), (576, 48), (128, 65)]:
        with pytest.raises(tb.TclError):
            tb.xproj_conv_f32(offs, torch.zeros(5, 2 * E, device="cuda"), torch.zeros(E, 4, device="cuda"),
                              torch.zeros(E, device="cuda"), torch.zeros(N, E, device="cuda"), 5, E)


@pytest.mark.parametrize("R", [4, 16])
@pytest.mark.parametrize("L", [1, 25, 70, 256])
@pytest.mark.parametrize("chunks", [0, 1, 2, 3, 5, 8])
def test_scan_f32(R, L, chunks):
    """chunks = 0: sequential scan; > 0: the chunked two-level scan."""
    N, E = 16, 320
    rng = np.random.default_rng(R * 100 + L)
    lengths = rng.integers(1, L + 1, size=11).astype(np.int32)
    lengths[0] = L
    lengths[1] = 1
    B = len(lengths)
    print(f"scan R={R} L={L} B={B} E={E} chunks={chunks}", flush=True)
    rows = int(lengths.sum())
    u = rng.standard_normal((rows, E)).astype(np.float32)
    z = rng.standard_normal((rows, E)).astype(np.float32)
    xdbl = (0.5 * rng.standard_normal((rows, R + 2 * N))).astype(np.float32)
    W_dt = rng.uniform(-0.5, 0.5, (E, R)).astype(np.float32)
    b_dt = np.log(np.expm1(np.exp(rng.uniform(np.log(1e-3), np.log(1e-1), E)))).astype(np.float32)
    A_log = (np.log(np.arange(1, N + 1))[None, :] + 0.3 * rng.standard_normal((E, N))).astype(np.float32)
    D = rng.standard_normal(E).astype(np.float32)
    out = torch.full((rows, E), float("nan"), device="cuda")
    tb.scan_f32(_dev(_offs(lengths), torch.int32), _dev(u), _dev(xdbl), _dev(z), _dev(W_dt), _dev(b_dt),
                _dev(A_log), _dev(D), out, chunks=chunks)
    torch.cuda.synchronize()
    f = lambda a: a.astype(np.float64)
    up, zp, xd = (_unpack(f(a), lengths, L) for a in (u, z, xdbl))
    dt = om.softplus(xd[..., :R] @ f(W_dt).T + f(b_dt))
    y = om.selective_scan(up, dt, -np.exp(f(A_log)), xd[..., R:R + N], xd[..., R + N:], f(D))
    expect = _pack(y * om.silu(zp), lengths)
    got = out.cpu().numpy()
    scale = np.sqrt(np.mean(expect ** 2))
    err = np.abs(got - expect)
    assert np.all(err <= 1e-4 * (np.abs(expect) + scale)), float(np.max(err / (np.abs(expect) + scale)))


def test_scan_chunked_at_long_sequence_shape():
    """The long-sequence workload's scan shape (B = 8192 programs of 64..256
    tokens, E = 512, N = 16, R = 16) through the chunked two-level scan
    forced to 8 chunks per program (tcl_score picks the sequential scan at
    this batch size): every element against the sequential scan (the same
    recurrence, its chunks stitched through per-chunk affine summaries, so
    equal to rounding: 1e-4 of |y| plus the output's rms), and a sample of
    programs, the first and last among them, against the oracle."""
    N, E, R, L, B = 16, 512, 16, 256, 8192
    rng = np.random.default_rng(8192)
    lengths = rng.integers(64, L + 1, size=B).astype(np.int32)
    rows = int(lengths.sum())
    u = rng.standard_normal((rows, E), dtype=np.float32)
    z = rng.standard_normal((rows, E), dtype=np.float32)
    xdbl = 0.5 * rng.standard_normal((rows, R + 2 * N), dtype=np.float32)
    W_dt = rng.uniform(-0.25, 0.25, (E, R)).astype(np.float32)
    b_dt = np.log(np.expm1(np.exp(rng.uniform(np.log(1e-3), np.log(1e-1), E)))).astype(np.float32)
    A_log = (np.log(np.arange(1, N + 1))[None, :] + 0.3 * rng.standard_normal((E, N))).astype(np.float32)
    D = rng.standard_normal(E).astype(np.float32)
    print(f"scan B={B} rows={rows} E={E}: chunked (8) vs sequential", flush=True)
    offs = _offs(lengths)
    d = [_dev(a) for a in (u, xdbl, z, W_dt, b_dt, A_log, D)]
    od = _dev(offs, torch.int32)
    seq = torch.full((rows, E), float("nan"), device="cuda")
    chk = torch.full((rows, E), float("nan"), device="cuda")
    tb.scan_f32(od, *d, seq, chunks=0)
    tb.scan_f32(od, *d, chk, chunks=8)
    torch.cuda.synchronize()
    scale = float(torch.sqrt(torch.mean(seq.double() ** 2)))
    bad = (chk - seq).abs() > 1e-4 * (seq.abs() + scale)
    assert not torch.isnan(chk).any() and int(bad.sum()) == 0, int(bad.sum())
    idx = np.unique(np.concatenate([[0, B - 1], rng.choice(B, 4, replace=False)]))
    f = lambda a: a.astype(np.float64)
    got = chk.cpu().numpy()
    for b in idx:
        r0, r1 = int(offs[b]), int(offs[b + 1])
        dt = om.softplus(f(xdbl[r0:r1, :R]) @ f(W_dt).T + f(b_dt))
        y = om.selective_scan(f(u[r0:r1])[None], dt[None], -np.exp(f(A_log)), f(xdbl[r0:r1, R:R + N])[None],
                              f(xdbl[r0:r1, R + N:])[None], f(D))[0]
        expect = y * om.silu(f(z[r0:r1]))
        err = np.abs(got[r0:r1] - expect)
        assert np.all(err <= 1e-4 * (np.abs(expect) + scale)), (int(b), float(np.max(err)))


@pytest.mark.parametrize("chunks", [0, 4])
def test_scan_in_place_matches_out_of_place(chunks):
    """The model runs the scan with out aliasing u; results must not change."""
    N, E, R = 16, 128, 4
    rng = np.random.default_rng(3)
    lengths = np.array([25, 3, 14], np.int32)
    rows = int(lengths.sum())
    args = [rng.standard_normal((rows, E)).astype(np.float32),
            (0.5 * rng.standard_normal((rows, R + 2 * N))).astype(np.float32),
            rng.standard_normal((rows, E)).astype(np.float32),
            rng.uniform(-0.5, 0.5, (E, R)).astype(np.float32),
            np.full(E, -3.0, np.float32),
            np.tile(np.log(np.arange(1, N + 1)), (E, 1)).astype(np.float32),
            np.ones(E, np.float32)]
    d = [_dev(a) for a in args]
    offs = _dev(_offs(lengths), torch.int32)
    out = torch.empty_like(d[0])
    tb.scan_f32(offs, *d, out, chunks=chunks)
    u_copy = d[0].clone()
    tb.scan_f32(offs, u_copy, *d[1:], u_copy, chunks=chunks)
    torch.cuda.synchronize()
    assert torch.equal(out, u_copy)


# ---------------------------------------------------------------- split path (fp32 on bf16 MFMA)
# Both operands split exactly into three bf16 parts; the three dropped part
# products are at most 2^-23 |a w| = 2U |a w| per product, so the bound is the
# fp32 dot-product bound with two more units: (K + 4) U sum |a_k w_k|.

def _split_ref(A, W, mode, bv=None, C0=None):
    A64, W64 = A.astype(np.float64), W.astype(np.float64)
    K = A.shape[1]
    ref = A64 @ W64.T
    bound = (K + 4) * U * (np.abs(A64) @ np.abs(W64).T)
    if mode == "bias":
        ref = ref + bv
        bound = bound + U * np.abs(ref)
    elif mode == "resid":
        ref = ref + C0
        bound = bound + U * np.abs(ref)
    elif mode == "norm":
        rstd = 1.0 / np.sqrt(np.mean(A64 * A64, axis=1, keepdims=True) + 1e-5)
        ref = rstd * ref
        bound = rstd * bound + (K + 8) * U * np.abs(ref)
    return ref, bound


@pytest.mark.parametrize("M,N,K", [(1, 64, 4), (129, 256, 164), (1000, 1024, 256), (77, 100, 36),
                                   (300, 48, 64), (40000, 96, 192)])
@pytest.mark.parametrize("mode", ["plain", "bias", "norm"])
@pytest.mark.parametrize("variant", [1, 4])
def test_gemm_split32(M, N, K, mode, variant):
    """32-row split panels (K <= 256), one wavefront per panel row group
    (variant 1) or the K halves on two (variant 4): plain, + bias, RMSNorm
    row scale; ragged M, N and K (K % 8 == 4 exercises a half-filled last k
    unit; K <= 128 leaves the upper half empty)."""
    print(f"gemm split32 variant={variant} mode={mode} M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M + 3 * N + 17 * K + len(mode))
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = rng.standard_normal((N, K)).astype(np.float32)
    bv = rng.standard_normal(N).astype(np.float32) if mode == "bias" else None
    C = tb.gemm_split(_dev(A), _dev(W), _dev(bv) if bv is not None else None, variant=variant,
                      epilogue=2 if mode == "norm" else 0)
    torch.cuda.synchronize()
    ref, bound = _split_ref(A, W, mode, bv)
    err = np.abs(C.cpu().numpy() - ref)
    assert np.all(err <= bound + 1e-30), float(np.max(err / (bound + 1e-30)))


@pytest.mark.parametrize("M,N,K", [(1, 64, 512), (31, 48, 500), (257, 256, 512), (77, 100, 64),
                                   (200, 256, 128), (65, 40, 256), (40000, 96, 512)])
@pytest.mark.parametrize("mode", ["plain", "bias", "resid"])
def test_gemm_split16(M, N, K, mode):
    """16-row split panels (K up to 512): plain, + bias, and the residual
    epilogue C += A W^T in place; ragged M, N and K."""
    print(f"gemm split16 mode={mode} M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M + 7 * N + 19 * K + len(mode))
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = rng.standard_normal((N, K)).astype(np.float32)
    bv = rng.standard_normal(N).astype(np.float32) if mode == "bias" else None
    C0 = rng.standard_normal((M, N)).astype(np.float32)
    C = _dev(C0)
    tb.gemm_split(_dev(A), _dev(W), _dev(bv) if bv is not None else None, out=C, variant=2,
                  epilogue=1 if mode == "resid" else 0)
    torch.cuda.synchronize()
    ref, bound = _split_ref(A, W, mode, bv, C0)
    err = np.abs(C.cpu().numpy() - ref)
    assert np.all(err <= bound + 1e-30), float(np.max(err / (bound + 1e-30)))


@pytest.mark.parametrize("variant", [1, 4])
def test_gemm_split_gather(variant):
    """The input Linear on the split path: rows gathered from padded [B, L, F]
    features by token offsets, + bias; the padding (NaN here) is never read."""
    rng = np.random.default_rng(41)
    B, L, K, N = 37, 25, 164, 256
    lengths = rng.integers(1, L + 1, B).astype(np.int32)
    X = rng.standard_normal((B, L, K)).astype(np.float32)
    for b in range(B):
        X[b, lengths[b]:] = np.nan
    W = rng.standard_normal((N, K)).astype(np.float32)
    bv = rng.standard_normal(N).astype(np.float32)
    offs = _offs(lengths)
    C = tb.gemm_split(_dev(X), _dev(W), _dev(bv), variant=variant, epilogue=3, offs=_dev(offs, torch.int32))
    torch.cuda.synchronize()
    Ap = _pack(X, lengths)
    ref, bound = _split_ref(Ap, W, "bias", bv)
    got = C.cpu().numpy()[:offs[-1]]
    err = np.abs(got - ref)
    assert np.all(np.isfinite(got))
    assert np.all(err <= bound + 1e-30), float(np.max(err / (bound + 1e-30)))


# ---------------------------------------------------------------- two-part fp16 split (TCL_F32_MATMUL_SPLIT)
# Each operand (after an exact power-of-two scale) is h + 2^-11 l + r with
# |r| <= 2^-22 |x|; three of the four part products are kept. Per product the
# two r and the dropped 2^-22 l_a l_w add at most 3 * 2^-22 = 12 U of |a w|,
# so the element bound is the fp32 dot-product bound with 16 more units.

def _f16_ref(A, W, mode, bv=None):
    A64, W64 = A.astype(np.float64), W.astype(np.float64)
    K = A.shape[1]
    ref = A64 @ W64.T
    bound = (K + 16) * U * (np.abs(A64) @ np.abs(W64).T)
    if mode == "bias":
        ref = ref + bv
        bound = bound + U * np.abs(ref)
    elif mode == "norm":
        rstd = 1.0 / np.sqrt(np.mean(A64 * A64, axis=1, keepdims=True) + 1e-5)
        ref = rstd * ref
        bound = rstd * bound + (K + 8) * U * np.abs(ref)
    return ref, bound


@pytest.mark.parametrize("M,N,K", [(1, 64, 64), (129, 256, 164), (1000, 1024, 256), (77, 100, 60),
                                   (300, 48, 128), (40000, 96, 192), (33, 1024, 252)])
@pytest.mark.parametrize("mode", ["plain", "bias", "norm"])
def test_gemm_f16split(M, N, K, mode):
    """The two-part fp16 panels (variant 5): plain, + bias, RMSNorm row scale;
    ragged M, N and K; rows spanning 10^-30 .. 10^30 in magnitude (10^-15 ..
    10^15 with the RMSNorm, whose fp32 sum of squares bounds the range as in
    every fp32 kernel; the per-row power-of-two scale keeps every row inside
    fp16's range) and one all-zero row."""
    print(f"gemm f16split mode={mode} M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M + 3 * N + 17 * K + len(mode) + 5)
    A = rng.standard_normal((M, K))
    span = 15 if mode == "norm" else 30
    A *= 10.0 ** rng.integers(-span, span + 1, size=(M, 1))
    A[M // 2] = 0.0
    A = A.astype(np.float32)
    W = rng.standard_normal((N, K)).astype(np.float32)
    bv = rng.standard_normal(N).astype(np.float32) if mode == "bias" else None
    C = tb.gemm_split(_dev(A), _dev(W), _dev(bv) if bv is not None else None, variant=5,
                      epilogue=2 if mode == "norm" else 0)
    torch.cuda.synchronize()
    ref, bound = _f16_ref(A, W, mode, bv)
    got = C.cpu().numpy()
    err = np.abs(got - ref)
    assert np.all(np.isfinite(got))
    assert np.all(err <= bound + 1e-300), float(np.max(err / (bound + 1e-300)))


def test_gemm_f16split_gather():
    """The input Linear on the fp16 split path: rows gathered from padded
    [B, L, F] features by token offsets, + bias; NaN padding never read."""
    rng = np.random.default_rng(43)
    B, L, K, N = 37, 25, 164, 256
    lengths = rng.integers(1, L + 1, B).astype(np.int32)
    X = np.log1p(rng.lognormal(0.0, 1.0, (B, L, K))).astype(np.float32)
    for b in range(B):
        X[b, lengths[b]:] = np.nan
    W = rng.uniform(-1, 1, (N, K)).astype(np.float32) / np.float32(np.sqrt(K))
    bv = rng.standard_normal(N).astype(np.float32)
    offs = _offs(lengths)
    C = tb.gemm_split(_dev(X), _dev(W), _dev(bv), variant=5, epilogue=3, offs=_dev(offs, torch.int32))
    torch.cuda.synchronize()
    ref, bound = _f16_ref(_pack(X, lengths), W, "bias", bv)
    got = C.cpu().numpy()[:offs[-1]]
    assert np.all(np.isfinite(got))
    err = np.abs(got - ref)
    assert np.all(err <= bound + 1e-30), float(np.max(err / (bound + 1e-30)))


def test_gemm_f16split_error_against_native_fp32():
    """On the model's in_proj and out_proj shapes (unit-scale rows, weights
    U(+-1/sqrt K)) the two-part fp16 paths' rms error against fp64 is within
    4x of the fp32 matrix cores' (each operand carries 22 of fp32's 24 bits,
    so a product is off by up to 12 units of fp32 rounding against the fp32
    kernel's one); both within the element bounds above."""
    rng = np.random.default_rng(8)
    M, N, K = 4096, 1024, 256
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.uniform(-1, 1, (N, K)) / np.sqrt(K)).astype(np.float32)
    ref = A.astype(np.float64) @ W.astype(np.float64).T
    h = tb.gemm_split(_dev(A), _dev(W), variant=5).cpu().numpy()
    n = tb.gemm_f32(_dev(A), _dev(W), tile=8).cpu().numpy()
    e_h = float(np.sqrt(np.mean((h - ref) ** 2)))
    e_n = float(np.sqrt(np.mean((n - ref) ** 2)))
    print(f"M={M} N={N} K={K}: rms error fp16 split {e_h:.3e}, native fp32 {e_n:.3e}", flush=True)
    assert e_h <= 4.0 * e_n
    # out_proj's shape on the all-N kernel
    M, N, K = 4096, 256, 512
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.uniform(-1, 1, (N, K)) / np.sqrt(K)).astype(np.float32)
    ref = A.astype(np.float64) @ W.astype(np.float64).T
    h = tb.gemm_split(_dev(A), _dev(W), variant=6).cpu().numpy()
    n = tb.gemm_f32(_dev(A), _dev(W), tile=9).cpu().numpy()
    e_h = float(np.sqrt(np.mean((h - ref) ** 2)))
    e_n = float(np.sqrt(np.mean((n - ref) ** 2)))
    print(f"M={M} N={N} K={K}: rms error fp16 split {e_h:.3e}, native fp32 {e_n:.3e}", flush=True)
    assert e_h <= 4.0 * e_n


@pytest.mark.parametrize("M,N,K", [(1, 64, 512), (31, 48, 500), (257, 256, 512), (77, 100, 64),
                                   (200, 256, 128), (65, 40, 256), (40000, 96, 512), (129, 256, 384),
                                   (40000, 256, 512)])
@pytest.mark.parametrize("mode", ["plain", "bias", "resid"])
def test_gemm_f16acc(M, N, K, mode):
    """The two-part fp16 panels with all N in registers (variant 6: out_proj's
    kernel): plain, + bias, and the residual epilogue C += A W^T in place;
    ragged M, N and K; each row's 128-wide K chunks scaled by independent
    powers of ten between 10^-20 and 10^20, so the running row scale drops
    (and the accumulators are rescaled) at every kind of chunk boundary."""
    print(f"gemm f16acc mode={mode} M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M + 5 * N + 23 * K + len(mode))
    A = rng.standard_normal((M, K))
    nch = (K + 127) // 128
    A *= np.repeat(10.0 ** rng.integers(-20, 21, size=(M, nch)), 128, axis=1)[:, :K]
    A[M // 2] = 0.0
    A = A.astype(np.float32)
    W = rng.standard_normal((N, K)).astype(np.float32)
    bv = rng.standard_normal(N).astype(np.float32) if mode == "bias" else None
    C0 = rng.standard_normal((M, N)).astype(np.float32)
    C = _dev(C0)
    tb.gemm_split(_dev(A), _dev(W), _dev(bv) if bv is not None else None, out=C, variant=6,
                  epilogue=1 if mode == "resid" else 0)
    torch.cuda.synchronize()
    ref, bound = _f16_ref(A, W, "bias" if mode == "bias" else "plain", bv)
    if mode == "resid":
        ref = ref + C0
        bound = bound + U * np.abs(ref)
    got = C.cpu().numpy()
    assert np.all(np.isfinite(got))
    err = np.abs(got - ref)
    assert np.all(err <= bound + 1e-300), float(np.max(err / (bound + 1e-300)))


def test_gemm_split_error_matches_native_fp32():
    """The split path is as accurate as the fp32 matrix cores: on the model's
    projection shapes its rms error against fp64 stays within 1.5x of the
    fp32 MFMA kernel's (and both within the fp32 bound above)."""
    rng = np.random.default_rng(7)
    for (M, N, K, variant, tile) in [(4096, 1024, 256, 1, 8), (4096, 1024, 256, 4, 8), (4096, 256, 512, 3, 9),
                                     (4096, 256, 512, 2, 9)]:
        A = rng.standard_normal((M, K)).astype(np.float32)
        W = (rng.uniform(-1, 1, (N, K)) / np.sqrt(K)).astype(np.float32)
        ref = A.astype(np.float64) @ W.astype(np.float64).T
        s = tb.gemm_split(_dev(A), _dev(W), variant=variant).cpu().numpy()
        n = tb.gemm_f32(_dev(A), _dev(W), tile=tile).cpu().numpy()
        e_split = float(np.sqrt(np.mean((s - ref) ** 2)))
        e_nat = float(np.sqrt(np.mean((n - ref) ** 2)))
        print(f"M={M} N={N} K={K}: rms error split {e_split:.3e}, native fp32 {e_nat:.3e}", flush=True)
        assert e_split <= 1.5 * e_nat


def test_gemm_split_refuses_unsupported():
    rng = np.random.default_rng(3)
    A = _dev(rng.standard_normal((64, 320)).astype(np.float32))
    W = _dev(rng.standard_normal((64, 320)).astype(np.float32))
    with pytest.raises(tb.TclError):        # 32-row panels stop at K = 256
        tb.gemm_split(A, W, variant=1)
    with pytest.raises(tb.TclError):        # ... also with K in two halves
        tb.gemm_split(A, W, variant=4)
    with pytest.raises(tb.TclError):        # K = 320 rounds up to 384: no 16-row kernel
        tb.gemm_split(A, W, variant=2)
    A2 = _dev(rng.standard_normal((64, 256)).astype(np.float32))
    W2 = _dev(rng.standard_normal((64, 256)).astype(np.float32))
    with pytest.raises(tb.TclError):        # no residual epilogue on streaming 32-row panels
        tb.gemm_split(A2, W2, out=torch.zeros(64, 64, device="cuda"), variant=1, epilogue=1)
    with pytest.raises(tb.TclError):
        tb.gemm_split(A2, W2, out=torch.zeros(64, 64, device="cuda"), variant=4, epilogue=1)
    with pytest.raises(tb.TclError):        # no RMSNorm on 16-row panels
        tb.gemm_split(A2, W2, variant=2, epilogue=2)
    with pytest.raises(tb.TclError):        # no RMSNorm with all of N in registers
        tb.gemm_split(A2, W2, variant=3, epilogue=2)
    W3 = _dev(rng.standard_normal((300, 256)).astype(np.float32))
    with pytest.raises(tb.TclError):        # ... which holds N <= 256
        tb.gemm_split(A2, W3, variant=3)


@pytest.mark.parametrize("M,N,K", [(1, 64, 512), (31, 48, 500), (257, 256, 512), (77, 100, 64),
                                   (200, 256, 128), (65, 40, 256), (129, 200, 164), (40000, 256, 512),
                                   (300, 96, 384)])
@pytest.mark.parametrize("mode", ["plain", "bias", "resid"])
def test_gemm_split32acc(M, N, K, mode):
    """32-row split panels with all N columns accumulated in registers (N <=
    256, K <= 512 in chunks of 256): plain, + bias, residual in place."""
    print(f"gemm split32acc mode={mode} M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M + 11 * N + 23 * K + len(mode))
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = rng.standard_normal((N, K)).astype(np.float32)
    bv = rng.standard_normal(N).astype(np.float32) if mode == "bias" else None
    C0 = rng.standard_normal((M, N)).astype(np.float32)
    C = _dev(C0)
    tb.gemm_split(_dev(A), _dev(W), _dev(bv) if bv is not None else None, out=C, variant=3,
                  epilogue=1 if mode == "resid" else 0)
    torch.cuda.synchronize()
    ref, bound = _split_ref(A, W, mode, bv, C0)
    err = np.abs(C.cpu().numpy() - ref)
    assert np.all(err <= bound + 1e-30), float(np.max(err / (bound + 1e-30)))
