"""Pins of the oracle's selective scan and causal conv to what the mathematics
fixes (section 5.2, Eq. (4)-(5), discretised: a_t = exp(dt_t A), B_bar = dt_t B).
None of these re-types the oracle's recurrence: each compares it with a
different formula, a library routine, or an identity."""
import numpy as np
import pytest
import scipy.signal

from oracle import model as om


def _scan_inputs(rng, Bn=2, L=6, E=3, N=4, dt_scale=0.5):
    u = rng.standard_normal((Bn, L, E))
    dt = dt_scale * rng.uniform(0.05, 1.0, size=(Bn, L, E))
    A = -rng.uniform(0.2, 3.0, size=(E, N))
    Bm = rng.standard_normal((Bn, L, N))
    Cm = rng.standard_normal((Bn, L, N))
    D = rng.standard_normal(E)
    return u, dt, A, Bm, Cm, D


def _explicit_form(u, dt, A, Bm, Cm, D):
    """y_t = sum_{k<=t} C_t . (prod_{j=k+1..t} exp(dt_j A)) . dt_k B_k u_k + D u_t,
    by brute force over every (b, t, e, k, n)."""
    Bn, L, E = u.shape
    N = A.shape[1]
    y = np.zeros((Bn, L, E))
    for b in range(Bn):
        for t in range(L):
            for e in range(E):
                acc = 0.0
                for k in range(t + 1):
                    for n in range(N):
                        decay = 1.0
                        for j in range(k + 1, t + 1):
                            decay *= np.exp(dt[b, j, e] * A[e, n])
                        acc += Cm[b, t, n] * decay * dt[b, k, e] * Bm[b, k, n] * u[b, k, e]
                y[b, t, e] = acc + D[e] * u[b, t, e]
    return y


def test_scan_equals_explicit_convolution_form():
    rng = np.random.default_rng(1)
    args = _scan_inputs(rng)
    np.testing.assert_allclose(om.selective_scan(*args), _explicit_form(*args), rtol=1e-12, atol=1e-12)


def test_scan_causality():
    rng = np.random.default_rng(2)
    u, dt, A, Bm, Cm, D = _scan_inputs(rng, L=9)
    y0 = om.selective_scan(u, dt, A, Bm, Cm, D)
    for t0 in (0, 4, 8):
        u2, dt2, B2, C2 = u.copy(), dt.copy(), Bm.copy(), Cm.copy()
        u2[:, t0] += 1.0
        dt2[:, t0] *= 1.7
        B2[:, t0] -= 0.5
        C2[:, t0] += 0.25
        y1 = om.selective_scan(u2, dt2, A, B2, C2, D)
        assert np.array_equal(y0[:, :t0], y1[:, :t0])
        assert not np.allclose(y0[:, t0], y1[:, t0])


def test_scan_length_one():
    rng = np.random.default_rng(3)
    u, dt, A, Bm, Cm, D = _scan_inputs(rng, L=1)
    expect = np.einsum("bn,bn->b", Cm[:, 0], Bm[:, 0])[:, None] * dt[:, 0] * u[:, 0] + D * u[:, 0]
    np.testing.assert_allclose(om.selective_scan(u, dt, A, Bm, Cm, D)[:, 0], expect, rtol=1e-13)


def test_scan_zero_input():
    rng = np.random.default_rng(4)
    u, dt, A, Bm, Cm, D = _scan_inputs(rng)
    y = om.selective_scan(np.zeros_like(u), dt, A, Bm, Cm, D)
    assert np.array_equal(y, np.zeros_like(y))


def test_scan_lti_matches_lfilter():
    """With dt, B, C constant in t every state is a first-order IIR filter."""
    rng = np.random.default_rng(5)
    Bn, L, E, N = 2, 40, 3, 5
    u = rng.standard_normal((Bn, L, E))
    dtv = rng.uniform(0.01, 0.5, size=E)
    A = -rng.uniform(0.1, 4.0, size=(E, N))
    Bv, Cv, D = rng.standard_normal(N), rng.standard_normal(N), rng.standard_normal(E)
    dt = np.broadcast_to(dtv, (Bn, L, E)).copy()
    Bm = np.broadcast_to(Bv, (Bn, L, N)).copy()
    Cm = np.broadcast_to(Cv, (Bn, L, N)).copy()
    y = om.selective_scan(u, dt, A, Bm, Cm, D)
    expect = np.zeros_like(u)
    for b in range(Bn):
        for e in range(E):
            for n in range(N):
                s = scipy.signal.lfilter([dtv[e] * Bv[n]], [1.0, -np.exp(dtv[e] * A[e, n])], u[b, :, e])
                expect[b, :, e] += Cv[n] * s
            expect[b, :, e] += D[e] * u[b, :, e]
    np.testing.assert_allclose(y, expect, rtol=1e-10, atol=1e-12)


def test_scan_limits():
    rng = np.random.default_rng(6)
    u, dt, A, Bm, Cm, D = _scan_inputs(rng)
    # dt -> 0: the state never fills, y -> D u
    y = om.selective_scan(u, 1e-12 * np.ones_like(dt), A, Bm, Cm, D)
    np.testing.assert_allclose(y, D * u, rtol=1e-9, atol=1e-9)
    # dt |A| >> 1: the state forgets everything before t
    big = 200.0 * np.ones_like(dt)
    A2 = -np.ones_like(A)
    y = om.selective_scan(u, big, A2, Bm, Cm, D)
    expect = np.einsum("btn,btn->bt", Cm, Bm)[:, :, None] * big * u + D * u
    np.testing.assert_allclose(y, expect, rtol=1e-9)


def test_scan_backward_against_finite_differences():
    rng = np.random.default_rng(7)
    u, dt, A, Bm, Cm, D = _scan_inputs(rng, Bn=2, L=5, E=3, N=3)
    w = rng.standard_normal(u.shape)  # objective sum(w * y)
    _, states = om.selective_scan(u, dt, A, Bm, Cm, D, return_states=True)
    grads = om.selective_scan_backward(w, u, dt, A, Bm, Cm, D, states)
    args = [u, dt, A, Bm, Cm, D]
    h = 1e-6
    for i, g in enumerate(grads):
        x = args[i]
        fd = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            ap, am = list(args), list(args)
            ap[i], am[i] = xp, xm
            fd[idx] = (np.sum(w * om.selective_scan(*ap)) - np.sum(w * om.selective_scan(*am))) / (2 * h)
        np.testing.assert_allclose(g, fd, rtol=1e-6, atol=1e-8)


def test_conv_matches_numpy_convolve():
    rng = np.random.default_rng(8)
    Bn, L, E, K = 3, 11, 4, 4
    x = rng.standard_normal((Bn, L, E))
    w = rng.standard_normal((E, K))
    b = rng.standard_normal(E)
    y = om.causal_conv1d(x, w, b)
    for bb in range(Bn):
        for e in range(E):
            # the last tap multiplies the current token: a causal convolution
            # with the kernel reversed
            expect = np.convolve(x[bb, :, e], w[e, ::-1])[:L] + b[e]
            np.testing.assert_allclose(y[bb, :, e], expect, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("L", [1, 2, 3])
def test_conv_shorter_than_kernel(L):
    rng = np.random.default_rng(9)
    x = rng.standard_normal((2, L, 3))
    w = rng.standard_normal((3, 4))
    b = rng.standard_normal(3)
    y = om.causal_conv1d(x, w, b)
    for e in range(3):
        expect = np.convolve(x[0, :, e], w[e, ::-1])[:L] + b[e]
        np.testing.assert_allclose(y[0, :, e], expect, rtol=1e-13)


def test_conv_backward_against_finite_differences():
    rng = np.random.default_rng(10)
    x = rng.standard_normal((2, 6, 3))
    w = rng.standard_normal((3, 4))
    b = rng.standard_normal(3)
    gout = rng.standard_normal(x.shape)
    dx, dw, db = om.causal_conv1d_backward(gout, x, w)
    h = 1e-6
    for arr, g, which in ((x, dx, 0), (w, dw, 1), (b, db, 2)):
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            a1, a2 = arr.copy(), arr.copy()
            a1[idx] += h
            a2[idx] -= h
            args1, args2 = [x, w, b], [x, w, b]
            args1[which], args2[which] = a1, a2
            fd[idx] = (np.sum(gout * om.causal_conv1d(*args1)) - np.sum(gout * om.causal_conv1d(*args2))) / (2 * h)
        np.testing.assert_allclose(g, fd, rtol=1e-7, atol=1e-9)
