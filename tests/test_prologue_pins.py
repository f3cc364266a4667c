"""Pins of the fp64 prologue oracle (short causal conv + SiLU + L2 norm) against
facts fixed independently of it: numpy's convolution, the SiLU definition via
scipy's logistic function, unit norms, causality, sequence isolation, and
central finite differences of its hand-written backward."""
import numpy as np
import pytest
from scipy.special import expit

from oracle.prologue import K_CONV, prologue_bwd, prologue_fwd


def rel(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


def draw(seed, B=2, T=23, H=2, D=5, K=K_CONV):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((B, T, H, D)), 0.5 * rng.standard_normal((H, D, K))


def test_conv_matches_numpy_convolve():
    # u_t = sum_j w[j] x_{t-(K-1)+j}: numpy's full convolution with the taps
    # reversed, truncated to the first T outputs (zero history)
    x, w = draw(1)
    y = prologue_fwd(x, w, False)
    for b in range(2):
        for h in range(2):
            for c in range(5):
                u = np.convolve(x[b, :, h, c], w[h, c, ::-1])[:x.shape[1]]
                assert rel(y[b, :, h, c], u * expit(u)) < 1e-14


def test_impulse_response_orientation():
    x = np.zeros((1, 10, 1, 1))
    x[0, 3, 0, 0] = 1.0
    w = np.array([[[0.1, 0.2, 0.3, 0.4]]])
    y = prologue_fwd(x, w, False)
    u = np.zeros(10)
    u[3:7] = [0.4, 0.3, 0.2, 0.1]  # the newest tap (j = K-1) acts first
    assert rel(y[0, :, 0, 0], u * expit(u)) < 1e-15


def test_normalised_rows_have_unit_norm():
    x, w = draw(2, D=16)
    y = prologue_fwd(3.0 * x, w, True)
    n = np.linalg.norm(y, axis=-1)
    assert np.all(n <= 1.0) and np.all(n > 0.999)


def test_causal_and_sequences_isolated():
    x, w = draw(3, B=1, T=30)
    cu = np.array([0, 7, 7, 19, 30])
    y = prologue_fwd(x, w, True, cu_seqlens=cu)
    x2 = x.copy()
    x2[0, 12] += 5.0                      # inside the third sequence [7, 19)
    y2 = prologue_fwd(x2, w, True, cu_seqlens=cu)
    changed = np.any(y2 != y, axis=(2, 3))[0]
    assert not changed[:12].any() and not changed[19:].any() and changed[12]
    # packed sequences equal separate calls
    for a, e in ((0, 7), (7, 19), (19, 30)):
        ys = prologue_fwd(x[:, a:e], w, True)
        assert np.array_equal(ys, y[:, a:e])


@pytest.mark.parametrize("normalize", [False, True])
def test_backward_matches_finite_differences(normalize):
    x, w = draw(4, B=1, T=9, H=1, D=4)
    cu = None
    rng = np.random.default_rng(5)
    dy = rng.standard_normal(x.shape)
    dx, dw = prologue_bwd(x, w, normalize, dy, cu_seqlens=cu)

    def loss(xx, ww):
        return float(np.sum(dy * prologue_fwd(xx, ww, normalize, cu_seqlens=cu)))

    h = 1e-6
    for idx in np.ndindex(*x.shape):
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        fd = (loss(xp, w) - loss(xm, w)) / (2 * h)
        assert abs(fd - dx[idx]) < 1e-7 * max(1.0, abs(fd)), idx
    for idx in np.ndindex(*w.shape):
        wp, wm = w.copy(), w.copy()
        wp[idx] += h
        wm[idx] -= h
        fd = (loss(x, wp) - loss(x, wm)) / (2 * h)
        assert abs(fd - dw[idx]) < 1e-7 * max(1.0, abs(fd)), idx


def test_backward_packed_matches_per_sequence():
    x, w = draw(6, B=1, T=25, H=2, D=3)
    cu = np.array([0, 2, 2, 14, 25])
    dy = np.random.default_rng(7).standard_normal(x.shape)
    dx, dw = prologue_bwd(x, w, True, dy, cu_seqlens=cu)
    dw_sum = np.zeros_like(w)
    for a, e in ((0, 2), (2, 14), (14, 25)):
        dxs, dws = prologue_bwd(x[:, a:e], w, True, dy[:, a:e])
        assert rel(dxs, dx[:, a:e]) < 1e-14
        dw_sum += dws
    assert rel(dw_sum, dw) < 1e-13


def test_gate_matches_definition_and_finite_differences():
    from oracle.prologue import gate_bwd, gate_fwd

    rng = np.random.default_rng(9)
    o, z, dy = (rng.standard_normal((2, 5, 3, 4)) for _ in range(3))
    assert rel(gate_fwd(o, z), o * expit(z)) < 1e-15
    assert np.all(gate_fwd(o, np.full_like(z, 0.0)) == 0.5 * o)   # sigmoid(0) = 1/2
    do, dz = gate_bwd(o, z, dy)
    h = 1e-6
    fo = (np.sum(dy * gate_fwd(o + h, z)) - np.sum(dy * gate_fwd(o - h, z))) / (2 * h)
    fz = (np.sum(dy * gate_fwd(o, z + h)) - np.sum(dy * gate_fwd(o, z - h))) / (2 * h)
    # a uniform shift probes the sum of each gradient
    assert abs(fo - np.sum(do)) < 1e-7 * max(1.0, abs(fo))
    assert abs(fz - np.sum(dz)) < 1e-7 * max(1.0, abs(fz))
    for idx in [(0, 0, 0, 0), (1, 4, 2, 3), (0, 2, 1, 1)]:
        e = np.zeros_like(z)
        e[idx] = h
        fd = (np.sum(dy * gate_fwd(o, z + e)) - np.sum(dy * gate_fwd(o, z - e))) / (2 * h)
        assert abs(fd - dz[idx]) < 1e-8
        fd = (np.sum(dy * gate_fwd(o + e, z)) - np.sum(dy * gate_fwd(o - e, z))) / (2 * h)
        assert abs(fd - do[idx]) < 1e-8
