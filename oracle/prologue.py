"""fp64 reference of the Comba layer's input prologue (Section 3.4, Neural Architecture).

TEST INFRASTRUCTURE ONLY: imported by tests/ and bench.py's cpu_baseline leg,
never by the product path.

The layer turns the projected q, k, v pre-activations into the operator's inputs
with a short causal convolution per channel (token shift), the SiLU feature map,
and, for q and k, an L2 normalisation over each head's channels:

    u_t[c] = sum_{j < K} w[c, j] x_{t - (K-1) + j}[c]      (x = 0 before the sequence start)
    s_t    = SiLU(u_t) = u_t * sigmoid(u_t)
    y_t    = s_t / sqrt(|s_t|^2 + eps)    (q and k)        or  y_t = s_t  (v)

Readings where the paper is silent: kernel size K = 4, depthwise (one filter per
channel, no bias), zero padding at each sequence start, eps = 1e-6 inside the
square root.  The backward is written out by hand:

    dy -> ds = (dy - y <y, dy>) / sqrt(|s|^2 + eps)        (normalised), ds = dy (v)
    du = ds * sigmoid(u) * (1 + u (1 - sigmoid(u)))
    dx_t[c] = sum_j w[c, j] du_{t + (K-1) - j}[c]           (inside the sequence)
    dw[c, j] = sum_t du_t[c] x_{t - (K-1) + j}[c]

Layouts: x, y, dy, dx [B, T, H, D] (or B = 1, packed, with cu_seqlens); w, dw
[H, D, K].  Plain loops over tokens, vectorised over channels.
"""
from __future__ import annotations

import numpy as np

K_CONV = 4
EPS = 1e-6


def _segments(B, T, cu_seqlens):
    """(row, token start, token end) of every sequence."""
    if cu_seqlens is None:
        return [(b, 0, T) for b in range(B)]
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    return [(0, int(cu[s]), int(cu[s + 1])) for s in range(len(cu) - 1)]


def _conv(x, w, b, a, e):
    """Causal depthwise conv over tokens a..e-1 of row b: [e-a, H, D]."""
    K = w.shape[-1]
    seg = x[b, a:e]
    u = np.zeros_like(seg)
    for t in range(e - a):
        for j in range(K):
            src = t - (K - 1) + j
            if src >= 0:
                u[t] += w[..., j] * seg[src]
    return u


def _sigmoid(u):
    return 1.0 / (1.0 + np.exp(-u))


def prologue_fwd(x, w, normalize, *, cu_seqlens=None, eps=EPS):
    """y = [L2-normalised] SiLU(causal depthwise conv(x)), fp64."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    B, T = x.shape[:2]
    y = np.zeros_like(x)
    for b, a, e in _segments(B, T, cu_seqlens):
        u = _conv(x, w, b, a, e)
        s = u * _sigmoid(u)
        if normalize:
            s = s / np.sqrt(np.sum(s * s, axis=-1, keepdims=True) + eps)
        y[b, a:e] = s
    return y


def prologue_bwd(x, w, normalize, dy, *, cu_seqlens=None, eps=EPS):
    """(dx, dw) of L = <dy, y>, fp64."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    dy = np.asarray(dy, np.float64)
    B, T = x.shape[:2]
    K = w.shape[-1]
    dx = np.zeros_like(x)
    dw = np.zeros_like(w)
    for b, a, e in _segments(B, T, cu_seqlens):
        u = _conv(x, w, b, a, e)
        sg = _sigmoid(u)
        s = u * sg
        g = dy[b, a:e]
        if normalize:
            n = np.sqrt(np.sum(s * s, axis=-1, keepdims=True) + eps)
            yv = s / n
            ds = (g - yv * np.sum(yv * g, axis=-1, keepdims=True)) / n
        else:
            ds = g
        du = ds * sg * (1.0 + u * (1.0 - sg))
        seg = x[b, a:e]
        L = e - a
        for t in range(L):
            for j in range(K):
                src = t - (K - 1) + j          # x_src feeds u_t through tap j
                if src >= 0:
                    dx[b, a + src] += w[..., j] * du[t]
                    dw[..., j] += du[t] * seg[src]
    return dx, dw


def gate_fwd(o, z):
    """Output gate of the layer (Section 3.4: sigmoid gating): y = o * sigmoid(z), fp64."""
    o = np.asarray(o, np.float64)
    z = np.asarray(z, np.float64)
    return o * _sigmoid(z)


def gate_bwd(o, z, dy):
    """(do, dz) of L = <dy, y>: do = dy sigmoid(z), dz = dy o sigmoid(z) (1 - sigmoid(z))."""
    o = np.asarray(o, np.float64)
    z = np.asarray(z, np.float64)
    dy = np.asarray(dy, np.float64)
    sg = _sigmoid(z)
    return dy * sg, dy * o * sg * (1.0 - sg)
