"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

None of these compare the oracle with itself: each checks a closed form, a
reduction to a textbook model, an invariant, a second independent formulation
(the chunk form of Section 3.3 vs the step form of Eq. comba-S), or finite
differences.  A plausible slip in the oracle (dropped term, wrong sign or
index, transposed state, off-by-one gate product) fails at least one of them.
"""
import numpy as np
import pytest

import oracle
from comba_inputs import random_case
from oracle.chunk import chunk_fwd, forward_substitution_inverse


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.max(np.abs(b))
    return np.max(np.abs(a - b)) / (den if den > 0 else 1.0)


# ---------------------------------------------------------------------------
# Chunk-wise reformulation (Section 3.3) == step recurrence (Eq. comba-S)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("C", [1, 2, 4, 16, 64])
@pytest.mark.parametrize("T", [1, 63, 64, 65, 200])
def test_chunk_form_equals_step_form(C, T):
    w = random_case(B=2, T=T, H=2, dk=8, dv=6, seed=100 + T + C, beta_tilde=True)
    bt = w.extra["beta_tilde"]
    o, ht = oracle.step_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0, beta_tilde=bt)
    oc, hc = chunk_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0, chunk=C, beta_tilde=bt)
    assert rel(oc, o) < 1e-12
    assert rel(hc, ht) < 1e-12


def test_chunk_form_equals_step_form_varlen_full_width():
    w = random_case(T=0, H=2, dk=64, dv=64, seed=7, seqlens=[1, 64, 130, 77])
    o, ht = oracle.step_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0, cu_seqlens=w.cu_seqlens)
    oc, hc = chunk_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0, cu_seqlens=w.cu_seqlens)
    assert rel(oc, o) < 1e-12
    assert rel(hc, ht) < 1e-12


def test_chunk_form_strong_decay_no_overflow():
    # log-gates far below fp32 exp range inside one chunk: ratios are formed as
    # exp(G_a - G_b) of cumulative gates, so nothing overflows
    w = random_case(B=1, T=130, H=1, dk=8, dv=8, seed=3, gate_scale=20.0)
    o, ht = oracle.step_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0)
    with np.errstate(over="raise", invalid="raise"):
        oc, hc = chunk_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0)
    assert np.all(np.isfinite(oc))
    assert rel(oc, o) < 1e-12


# ---------------------------------------------------------------------------
# Reductions to textbook models
# ---------------------------------------------------------------------------
def _la_case(T=40, dk=6, dv=5, seed=0):
    w = random_case(B=1, T=T, H=1, dk=dk, dv=dv, seed=seed, h0=False)
    g = np.zeros_like(w.g)
    beta = np.ones_like(w.beta)
    bt = np.zeros_like(w.beta)
    return w, g, beta, bt


def test_reduces_to_causal_linear_attention():
    # bt = 0, beta = 1, alpha = 1, d = 0: o_t = sum_{i<=t} v_i (k_i . q_t)
    # (plain linear attention, Table 1 LA row and Eq. seq-parallel of Section 2.1)
    w, g, beta, bt = _la_case()
    d = np.zeros(1)
    o, _ = oracle.step_fwd(w.q, w.k, w.v, g, beta, d, None, beta_tilde=bt)
    q, k, v = (x[0, :, 0].astype(np.float64) for x in (w.q, w.k, w.v))
    T = q.shape[0]
    ref = np.zeros((T, v.shape[1]))
    for t in range(T):
        for i in range(t + 1):
            ref[t] += v[i] * np.dot(k[i], q[t])
    assert rel(o[0, :, 0], ref) < 1e-13
    oc, _ = chunk_fwd(w.q, w.k, w.v, g, beta, d, None, chunk=16, beta_tilde=bt)
    assert rel(oc[0, :, 0], ref) < 1e-13


def test_reduces_to_scalar_gated_linear_attention():
    # bt = 0, beta = 1, any alpha: o_t = sum_{i<=t} (prod_{j=i+1..t} alpha_j) v_i k_i^T q~_t
    # (Mamba2-style scalar gate row of Table 1), with the output correction q~ = q - d k
    w = random_case(B=1, T=50, H=1, dk=6, dv=5, seed=1, h0=False)
    beta = np.ones_like(w.beta)
    bt = np.zeros_like(w.beta)
    o, _ = oracle.step_fwd(w.q, w.k, w.v, w.g, beta, w.d, None, beta_tilde=bt)
    q, k, v = (x[0, :, 0].astype(np.float64) for x in (w.q, w.k, w.v))
    alpha = np.exp(w.g[0, :, 0].astype(np.float64))
    qt = q - float(w.d[0]) * k
    T = q.shape[0]
    ref = np.zeros((T, v.shape[1]))
    for t in range(T):
        for i in range(t + 1):
            ref[t] += np.prod(alpha[i + 1:t + 1]) * v[i] * np.dot(k[i], qt[t])
    assert rel(o[0, :, 0], ref) < 1e-12


def test_reduces_to_gated_delta_rule_explicit_matrices():
    # Eq. comba-S written with explicit dv x dk matrices and explicit transition
    # matrices (alpha_t I - bt_t k k^T), in the paper's S orientation
    w = random_case(B=1, T=30, H=1, dk=5, dv=4, seed=2, beta_tilde=True)
    bt = w.extra["beta_tilde"]
    o, ht = oracle.step_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0, beta_tilde=bt)
    q, k, v = (x[0, :, 0].astype(np.float64) for x in (w.q, w.k, w.v))
    S = w.h0[0, 0].astype(np.float64).T
    ref = []
    for t in range(q.shape[0]):
        A = np.exp(float(w.g[0, t, 0])) * np.eye(5) - float(bt[0, t, 0]) * np.outer(k[t], k[t])
        S = S @ A + float(w.beta[0, t, 0]) * np.outer(v[t], k[t])
        ref.append(S @ (q[t] - float(w.d[0]) * k[t]))
    assert rel(o[0, :, 0], np.array(ref)) < 1e-13
    assert rel(ht[0, 0], S.T) < 1e-13


def test_delta_rule_memorization():
    # alpha = beta = bt = 1 and |k| = 1: the transition is a Householder
    # projection, so S_t k_t = v_t (Section 2.2, delta rule); with q = (1+d) k
    # the corrected query is k itself and o_t = v_t exactly.
    w = random_case(B=1, T=40, H=2, dk=8, dv=8, seed=4)
    k = w.k.astype(np.float64)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)   # unit norm in fp64
    g = np.zeros_like(w.g)
    one = np.ones_like(w.beta)
    q = (1.0 + w.d[None, None, :, None].astype(np.float64)) * k
    o, _ = oracle.step_fwd(q, k, w.v, g, one, w.d, w.h0)
    assert rel(o, w.v) < 1e-12
    oc, _ = chunk_fwd(q, k, w.v, g, one, w.d, w.h0, chunk=16)
    assert rel(oc, w.v) < 1e-12


def test_output_correction_cancels_query():
    # q = d k: the corrected query q - d k is exactly zero, so o == 0
    w = random_case(B=1, T=33, H=2, dk=6, dv=4, seed=5)
    q = w.d[None, None, :, None].astype(np.float64) * w.k.astype(np.float64)
    o, ht = oracle.step_fwd(q, w.k, w.v, w.g, w.beta, w.d, w.h0)
    assert np.max(np.abs(o)) == 0.0
    assert np.max(np.abs(ht)) > 0


def test_frozen_state_when_nothing_is_written():
    # beta = bt = 0: only the scalar gate acts, S_t = alpha^{1:t} S_0,
    # o_t = alpha^{1:t} h0^T (q_t - d k_t)
    w = random_case(B=1, T=20, H=1, dk=6, dv=5, seed=6)
    zero = np.zeros_like(w.beta)
    o, ht = oracle.step_fwd(w.q, w.k, w.v, w.g, zero, w.d, w.h0)
    gam = np.exp(np.cumsum(w.g[0, :, 0].astype(np.float64)))
    qt = w.q[0, :, 0].astype(np.float64) - float(w.d[0]) * w.k[0, :, 0].astype(np.float64)
    ref = gam[:, None] * (qt @ w.h0[0, 0].astype(np.float64))
    assert rel(o[0, :, 0], ref) < 1e-13
    assert rel(ht[0, 0], gam[-1] * w.h0[0, 0]) < 1e-13


def test_transition_identity_unit_keys():
    # with |k_t| = 1: S_t k_t - beta_t v_t = (alpha_t - bt_t) S_{t-1} k_t
    # (apply one step at a time through h0 -> ht)
    w = random_case(B=1, T=12, H=1, dk=7, dv=3, seed=8, beta_tilde=True)
    bt = w.extra["beta_tilde"]
    kk = w.k.astype(np.float64)
    kk /= np.linalg.norm(kk, axis=-1, keepdims=True)   # unit norm in fp64
    H = w.h0.astype(np.float64)
    for t in range(12):
        sl = slice(t, t + 1)
        _, H2 = oracle.step_fwd(w.q[:, sl], kk[:, sl], w.v[:, sl], w.g[:, sl],
                                w.beta[:, sl], w.d, H, beta_tilde=bt[:, sl])
        k = kk[0, t, 0]
        lhs = H2[0, 0].T @ k - float(w.beta[0, t, 0]) * w.v[0, t, 0].astype(np.float64)
        rhs = (np.exp(float(w.g[0, t, 0])) - float(bt[0, t, 0])) * (H[0, 0].T @ k)
        assert rel(lhs, rhs) < 1e-12
        H = H2


# ---------------------------------------------------------------------------
# WY representation (Eqs. wy1, wy2) and UT transform (Eq. prepare-WY_M)
# ---------------------------------------------------------------------------
def test_wy_representation_matches_explicit_products():
    # D^r = prod_{i<=r} (alpha_i - bt_i k_i k_i^T) = alpha^{1:r} I - sum_i alpha^{i:r} w_i k_i^T
    # H^r (zero start) = sum_i alpha^{i:r} u_i k_i^T, using W, U from the UT transform
    w = random_case(B=1, T=16, H=1, dk=6, dv=4, seed=9, beta_tilde=True, h0=False)
    bt = w.extra["beta_tilde"][0, :, 0].astype(np.float64)
    _, _, inter = chunk_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, None, chunk=16,
                            beta_tilde=w.extra["beta_tilde"], return_intermediates=True)
    W, U, G = inter[(0, 0, 0)]["W"], inter[(0, 0, 0)]["U"], inter[(0, 0, 0)]["G"]
    k = w.k[0, :, 0].astype(np.float64)
    v = w.v[0, :, 0].astype(np.float64)
    g = w.g[0, :, 0].astype(np.float64)
    b = w.beta[0, :, 0].astype(np.float64)
    D = np.eye(6)
    Hm = np.zeros((4, 6))
    for r in range(16):
        A = np.exp(g[r]) * np.eye(6) - bt[r] * np.outer(k[r], k[r])
        D = D @ A
        Hm = Hm @ A + b[r] * np.outer(v[r], k[r])
        ratio = np.exp(G[r] - G[:r + 1])            # alpha^{i:r}, i = 1..r
        D_wy = np.exp(G[r]) * np.eye(6) - (W[:r + 1] * ratio[:, None]).T @ k[:r + 1]
        H_wy = (U[:r + 1] * ratio[:, None]).T @ k[:r + 1]
        assert rel(D_wy, D) < 1e-12
        assert rel(H_wy, Hm) < 1e-12


def test_forward_substitution_inverse_is_inverse():
    rng = np.random.default_rng(0)
    L = np.tril(rng.standard_normal((20, 20)), -1)
    M = forward_substitution_inverse(L)
    assert rel(M @ (np.eye(20) + L), np.eye(20)) < 1e-12
    assert np.allclose(np.triu(M, 1), 0.0) and np.allclose(np.diag(M), 1.0)


# ---------------------------------------------------------------------------
# Structural invariants
# ---------------------------------------------------------------------------
def test_segment_invariance_bit_exact():
    # constant-memory recurrence: running [0, T) == running [0, c) then [c, T) from ht
    w = random_case(B=1, T=150, H=2, dk=8, dv=8, seed=10)
    o, ht = oracle.step_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0)
    for cut in (1, 64, 97):
        a, b = slice(0, cut), slice(cut, 150)
        o1, h1 = oracle.step_fwd(w.q[:, a], w.k[:, a], w.v[:, a], w.g[:, a], w.beta[:, a], w.d, w.h0)
        o2, h2 = oracle.step_fwd(w.q[:, b], w.k[:, b], w.v[:, b], w.g[:, b], w.beta[:, b], w.d, h1)
        assert np.array_equal(np.concatenate([o1, o2], axis=1), o)
        assert np.array_equal(h2, ht)


def test_varlen_equals_per_sequence_bit_exact():
    lens = [5, 64, 70, 1]
    w = random_case(T=0, H=2, dk=8, dv=4, seed=11, seqlens=lens)
    o, ht = oracle.step_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0, cu_seqlens=w.cu_seqlens)
    cu = w.cu_seqlens
    for s in range(len(lens)):
        sl = slice(int(cu[s]), int(cu[s + 1]))
        os_, hs = oracle.step_fwd(w.q[:, sl], w.k[:, sl], w.v[:, sl], w.g[:, sl], w.beta[:, sl],
                                  w.d, w.h0[s:s + 1])
        assert np.array_equal(os_, o[:, sl])
        assert np.array_equal(hs[0], ht[s])


def test_joint_linearity_in_values_and_initial_state():
    w = random_case(B=2, T=40, H=2, dk=6, dv=5, seed=12)
    o, ht = oracle.step_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0)
    c = 2.5
    o2, ht2 = oracle.step_fwd(w.q, w.k, c * w.v.astype(np.float64), w.g, w.beta, w.d,
                              c * w.h0.astype(np.float64))
    assert rel(o2, c * o) < 1e-14
    assert rel(ht2, c * ht) < 1e-14


# ---------------------------------------------------------------------------
# Backward: finite differences and Euler identities
# ---------------------------------------------------------------------------
def _loss(w, dO, dht, **kw):
    o, ht = oracle.step_fwd(w["q"], w["k"], w["v"], w["g"], w["beta"], w["d"], w["h0"], **kw)
    return float(np.sum(o * dO) + np.sum(ht * dht))


@pytest.mark.parametrize("seqlens", [None, [3, 9, 1]])
def test_backward_matches_finite_differences(seqlens):
    if seqlens is None:
        case = random_case(B=2, T=11, H=2, dk=5, dv=4, seed=13, dht=True, beta_tilde=True)
    else:
        case = random_case(T=0, H=2, dk=4, dv=3, seed=14, dht=True, beta_tilde=True,
                           seqlens=seqlens)
    kw = {"cu_seqlens": case.cu_seqlens}
    base = {n: getattr(case, n).astype(np.float64) for n in ("q", "k", "v", "g", "beta", "d", "h0")}
    base["bt"] = case.extra["beta_tilde"].astype(np.float64)
    dO = case.dO.astype(np.float64)
    dht = case.dht.astype(np.float64)
    grads = oracle.step_bwd(base["q"], base["k"], base["v"], base["g"], base["beta"], base["d"],
                            base["h0"], dO, dht, beta_tilde=base["bt"], **kw)
    gname = {"q": "dq", "k": "dk", "v": "dv", "g": "dg", "beta": "dbeta", "d": "dd",
             "h0": "dh0", "bt": "dbeta_tilde"}
    rng = np.random.default_rng(99)
    eps = 1e-6
    for name, gkey in gname.items():
        for _ in range(3):
            direction = rng.standard_normal(base[name].shape)
            p = dict(base)
            m = dict(base)
            p[name] = base[name] + eps * direction
            m[name] = base[name] - eps * direction

            def L(x):
                xx = {kk: vv for kk, vv in x.items() if kk != "bt"}
                return _loss(xx, dO, dht, beta_tilde=x["bt"], **kw)

            fd = (L(p) - L(m)) / (2 * eps)
            an = float(np.sum(grads[gkey] * direction))
            assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (name, fd, an)


def test_backward_tied_beta_is_sum_of_both_roles():
    # with bt == beta (the operator's reading) dbeta is the total derivative
    w = random_case(B=1, T=9, H=1, dk=4, dv=3, seed=15, dht=True)
    g_sep = oracle.step_bwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0, w.dO, w.dht,
                            beta_tilde=w.beta)
    g_tied = oracle.step_bwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0, w.dO, w.dht)
    assert rel(g_tied["dbeta"], g_sep["dbeta"] + g_sep["dbeta_tilde"]) < 1e-14
    eps = 1e-6
    dirn = np.random.default_rng(1).standard_normal(w.beta.shape)
    lp = _loss({"q": w.q, "k": w.k, "v": w.v, "g": w.g, "beta": w.beta + eps * dirn, "d": w.d,
                "h0": w.h0}, w.dO, w.dht)
    lm = _loss({"q": w.q, "k": w.k, "v": w.v, "g": w.g, "beta": w.beta - eps * dirn, "d": w.d,
                "h0": w.h0}, w.dO, w.dht)
    assert abs((lp - lm) / (2 * eps) - np.sum(g_tied["dbeta"] * dirn)) < 1e-7


def test_euler_identity_values_and_state():
    # o and ht are jointly linear (degree-1 homogeneous) in (v, h0), so
    # <dv, v> + <dh0, h0> = <dO, o> + <dht, ht>
    w = random_case(B=2, T=70, H=2, dk=8, dv=6, seed=16, dht=True)
    o, ht = oracle.step_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0)
    gr = oracle.step_bwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0, w.dO, w.dht)
    lhs = np.sum(gr["dv"] * w.v) + np.sum(gr["dh0"] * w.h0)
    rhs = np.sum(w.dO * o) + np.sum(w.dht * ht)
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(rhs))


def test_euler_identity_query_and_feedback_scalar():
    # o is jointly linear in (q, d) while ht does not depend on them:
    # <dq, q> + sum_h dd_h d_h = <dO, o>
    w = random_case(B=2, T=70, H=2, dk=8, dv=6, seed=17, dht=True)
    o, _ = oracle.step_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0)
    gr = oracle.step_bwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0, w.dO, w.dht)
    lhs = np.sum(gr["dq"] * w.q) + np.sum(gr["dd"] * w.d)
    rhs = np.sum(w.dO * o)
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(rhs))


def test_backward_segment_chaining():
    # gradients through a split run chained by dht -> dh0 equal the one-pass gradients
    w = random_case(B=1, T=90, H=1, dk=6, dv=5, seed=18, dht=True)
    full = oracle.step_bwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0, w.dO, w.dht)
    cut = 40
    a, b = slice(0, cut), slice(cut, 90)
    _, h1 = oracle.step_fwd(w.q[:, a], w.k[:, a], w.v[:, a], w.g[:, a], w.beta[:, a], w.d, w.h0)
    g2 = oracle.step_bwd(w.q[:, b], w.k[:, b], w.v[:, b], w.g[:, b], w.beta[:, b], w.d, h1,
                         w.dO[:, b], w.dht)
    g1 = oracle.step_bwd(w.q[:, a], w.k[:, a], w.v[:, a], w.g[:, a], w.beta[:, a], w.d, w.h0,
                         w.dO[:, a], g2["dh0"])
    for key in ("dq", "dk", "dv", "dg", "dbeta"):
        assert rel(np.concatenate([g1[key], g2[key]], axis=1), full[key]) < 1e-12
    assert rel(g1["dd"] + g2["dd"], full["dd"]) < 1e-12
    assert rel(g1["dh0"], full["dh0"]) < 1e-12


def test_iplr_reflections_preserve_the_state_norm():
    # Comba-iplr's transition alpha (I - 2 c k k^T) in SPLR form has beta~ =
    # 2 alpha c.  With alpha = 1, c = 1, beta = 0 and |k| = 1 every transition
    # is a Householder reflection (orthogonal, its own inverse): the state's
    # Frobenius norm never changes, and a key repeated twice gives the state back.
    w = random_case(B=1, T=24, H=2, dk=8, dv=5, seed=41, h0=True)
    k = w.k.astype(np.float64)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    g = np.zeros_like(w.g)
    zero = np.zeros_like(w.beta)
    two = np.full_like(w.beta, 2.0)
    _, ht = oracle.step_fwd(w.q, k, w.v, g, zero, w.d, w.h0, beta_tilde=two)
    h0 = w.h0.astype(np.float64)
    for h in range(2):
        assert abs(np.linalg.norm(ht[0, h]) / np.linalg.norm(h0[0, h]) - 1.0) < 1e-13
    assert rel(ht, h0) > 0.1  # the reflections did act on the state
    kk = k.copy()
    kk[:, 1::2] = kk[:, 0::2]  # every key twice in a row
    _, ht2 = oracle.step_fwd(w.q, kk, w.v, g, zero, w.d, w.h0, beta_tilde=two)
    assert rel(ht2, w.h0) < 1e-13
    # and the chunk form agrees across chunk boundaries
    _, htc = chunk_fwd(w.q, kk, w.v, g, zero, w.d, w.h0, chunk=8, beta_tilde=two)
    assert rel(htc, w.h0) < 1e-12
