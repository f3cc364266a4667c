"""Chunk-wise reformulation of the Comba recurrence in NumPy fp64 -- TEST INFRASTRUCTURE ONLY.

Follows Section 3.3 of the paper step by step, in the paper's own orientation
(state S in R^{dv x dk}); only tests may use it.  Per chunk of C tokens with
start state S (rows r = 1..C of the chunk matrices, in-chunk cumulative
log-gates G_r = sum_{j<=r} g_j, so alpha^{1:r} = exp(G_r)):

* Eq. prepare-WY_M: M = (I + strictlower(Diag(bt) (A^{(i-1)/j} o K K^T)))^{-1},
  where A^{(i-1)/j} has entries alpha^{1:i-1} / alpha^{1:j}; the inverse is
  taken by row-wise forward substitution, as the paper prescribes.
* W = M Diag(bt o alpha^{0..C-1}) K,   U = M Diag(beta) V.
* Matrix form (end of Section 3.3):
      S_next = alpha^{1:C} S + (U - W S^T)^T Diag(alpha^{i->C}) K
      O      = Diag(alpha^{1:r}) Qt S^T + Tril(Qt K^T o A^{i/j}) (U - W S^T)
  with Qt = Q - d K; alpha^{i->C} = alpha^{1:C} / alpha^{1:i} and Tril includes
  the diagonal.

Readings taken where the paper's index notation is loose (see the design notes):
gate ratios are always formed as exp(G_a - G_b) of cumulative log-gates, the
product alpha^{1:0} is 1, the triangular part inside M is strict while the
output's Tril includes the diagonal, and a sequence's last chunk may be shorter
than C.
"""
from __future__ import annotations

import numpy as np


def forward_substitution_inverse(L: np.ndarray) -> np.ndarray:
    """(I + L)^{-1} for strictly lower-triangular L, row by row (Gaussian elimination)."""
    n = L.shape[0]
    M = np.zeros_like(L)
    for i in range(n):
        row = np.zeros(n)
        row[i] = 1.0
        for j in range(i):
            row -= L[i, j] * M[j]
        M[i] = row
    return M


def _chunk(Q, K, V, g, b, bt, d, S):
    """One chunk: returns (O, S_next, intermediates)."""
    n = Q.shape[0]
    G = np.cumsum(g)                          # log alpha^{1:r}
    Gm1 = np.concatenate([[0.0], G[:-1]])     # log alpha^{1:r-1}
    ii, jj = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    strict = ii > jj
    incl = ii >= jj
    A_prev = np.exp(np.where(strict, Gm1[:, None] - G[None, :], -np.inf))   # A^{(i-1)/j}
    A_cur = np.exp(np.where(incl, G[:, None] - G[None, :], -np.inf))       # A^{i/j}
    L = np.where(strict, bt[:, None] * (A_prev * (K @ K.T)), 0.0)
    M = forward_substitution_inverse(L)
    W = M @ (np.diag(bt * np.exp(Gm1)) @ K)
    U = M @ (np.diag(b) @ V)
    Qt = Q - d * K
    pseudo_v = U - W @ S.T                    # (U - W S^T), C x dv
    O = np.diag(np.exp(G)) @ Qt @ S.T + np.where(incl, (Qt @ K.T) * A_cur, 0.0) @ pseudo_v
    decay_to_end = np.exp(G[-1] - G)          # alpha^{i->C}
    S_next = np.exp(G[-1]) * S + pseudo_v.T @ np.diag(decay_to_end) @ K
    inter = {"M": M, "W": W, "U": U, "S": S.copy(), "G": G, "pseudo_v": pseudo_v}
    return O, S_next, inter


def chunk_fwd(q, k, v, g, beta, d, h0=None, *, chunk=64, cu_seqlens=None, beta_tilde=None,
              return_intermediates=False):
    """Chunk-form forward.  Shapes as ``oracle.step_fwd``; h0/ht use the [dk, dv] layout.

    Returns (o [B,T,H,dv], ht [N,H,dk,dv]) and, if requested, a dict mapping
    (sequence, head, chunk) to that chunk's M, W, U, start state S (dv x dk),
    cumulative gates G and pseudo-values U - W S^T.
    """
    q = np.asarray(q, dtype=np.float64)
    B, T, H, dk = q.shape
    dv = np.shape(v)[-1]
    Ttot = B * T
    qq = q.reshape(Ttot, H, dk)
    kk = np.asarray(k, np.float64).reshape(Ttot, H, dk)
    vv = np.asarray(v, np.float64).reshape(Ttot, H, dv)
    gg = np.asarray(g, np.float64).reshape(Ttot, H)
    bb = np.asarray(beta, np.float64).reshape(Ttot, H)
    bt = bb if beta_tilde is None else np.asarray(beta_tilde, np.float64).reshape(Ttot, H)
    dd = np.asarray(d, np.float64).reshape(H)
    if cu_seqlens is None:
        cu = np.arange(B + 1, dtype=np.int64) * T
    else:
        cu = np.asarray(cu_seqlens, dtype=np.int64)
    N = len(cu) - 1
    o = np.zeros((Ttot, H, dv))
    ht = np.zeros((N, H, dk, dv))
    inters = {}
    for s in range(N):
        for h in range(H):
            S = np.zeros((dv, dk)) if h0 is None else np.asarray(h0, np.float64)[s, h].T.copy()
            for c, a in enumerate(range(int(cu[s]), int(cu[s + 1]), chunk)):
                e = min(a + chunk, int(cu[s + 1]))
                O, S, inter = _chunk(qq[a:e, h], kk[a:e, h], vv[a:e, h], gg[a:e, h],
                                     bb[a:e, h], bt[a:e, h], dd[h], S)
                o[a:e, h] = O
                if return_intermediates:
                    inters[(s, h, c)] = inter
            ht[s, h] = S.T
    o = o.reshape(B, T, H, dv)
    if return_intermediates:
        return o, ht, inters
    return o, ht
