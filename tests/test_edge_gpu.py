"""GPU edge cases of the chunk-wise operator beyond the unit-norm regime.

* Keys and queries off the unit sphere.  Eq. comba-S defines the recurrence for
  any k; the layer normalises q and k upstream (Section 3.4), so the operator
  itself must stay exact when it does not.  The feedback strength is chosen so
  that every transition alpha I - beta~ k k^T stays contractive
  (beta~ |k|^2 <= 1 + alpha), which keeps the states bounded as in the paper.
  One case drives the UT-transform inverse M = (I + L)^{-1} (Eq. prepare-WY_M)
  to its largest entries within that limit: nearly parallel keys with
  beta~ |k|^2 close to 1 + alpha give rows of slowly decaying alternating
  entries near 2, so M R cancels heavily.
* Non-finite inputs.  A NaN in v and an Inf in dO inside one sequence and head
  of a packed batch must make that sequence's outputs and gradients
  non-finite, while every other sequence and head stays bitwise equal to a
  clean run (the chunk states and the inverse are stored with per-block scales,
  which must not swallow a NaN).
"""
import copy

import numpy as np
import pytest

from comba_inputs import bf16_round, random_case
from gpu_helpers import check_bwd, check_fwd, gpu_bwd, gpu_fwd

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _log(msg):
    print(msg, flush=True)


def _scale_qk(w, norm):
    # q, k are unit rows rounded to bf16; a power-of-two norm keeps them exact
    w.q = (w.q * np.float32(norm)).astype(np.float32)
    w.k = (w.k * np.float32(norm)).astype(np.float32)


def _contractive_beta_tilde(w, frac, seed):
    # beta~_t = frac_t (1 + alpha_t) / |k_t|^2 with frac_t = sigmoid(N(0,1)) * frac,
    # rounded to the input dtype (rounded down where rounding would cross the limit)
    rng = np.random.default_rng(seed)
    alpha = np.exp(w.g.astype(np.float64))
    kk = np.sum(w.k.astype(np.float64) ** 2, axis=-1)
    c = frac / (1.0 + np.exp(-rng.standard_normal(w.g.shape)))
    limit = (1.0 + alpha) / np.maximum(kk, 1e-30)
    bt = bf16_round((c * limit).astype(np.float32)) if w.in_dtype == "bf16" else \
        (c * limit).astype(np.float32)
    over = bt.astype(np.float64) * kk > 1.0 + alpha
    bt[over] = np.nextafter(bt[over], np.float32(0)) if w.in_dtype == "f32" else \
        bf16_round(bt[over] * np.float32(0.99))
    assert np.all(bt.astype(np.float64) * kk <= 1.0 + alpha)
    return bt


def _unit_case(d, norm, tied):
    seed = {"128": 101, "256": 202}[str(d)] + (0 if norm < 1 else 10) + (0 if tied else 1)
    T = 200 if d == 128 else 150
    w = random_case(seed=seed, B=2 if d == 128 else 1, T=T, H=2, dk=d, dv=d, in_dtype="bf16",
                    dht=True)
    _scale_qk(w, norm)
    if tied:
        # beta~ = beta: scale beta itself into the contractive range
        kk = np.sum(w.k.astype(np.float64) ** 2, axis=-1)
        lim = (1.0 + np.exp(w.g.astype(np.float64))) / kk
        w.beta = bf16_round(np.minimum(w.beta, 0.98 * lim).astype(np.float32))
        assert np.all(w.beta.astype(np.float64) * kk <= 1.0 + np.exp(w.g.astype(np.float64)))
    else:
        w.extra["beta_tilde"] = _contractive_beta_tilde(w, 1.0, seed + 1000)
    return w


UNNORM = [(d, norm, tied) for d in (128, 256) for norm in (0.25, 2.0) for tied in (True, False)]


@pytest.mark.parametrize("d,norm,tied", UNNORM,
                         ids=["d%d_norm%g_%s" % (d, n, "tied" if t else "sep")
                              for d, n, t in UNNORM])
def test_unnormalised_keys(d, norm, tied):
    w = _unit_case(d, norm, tied)
    ef = check_fwd(w)
    eb = check_bwd(w)
    _log("unnormalised |q|=|k|=%g d=%d %s: fwd %s bwd %s" % (norm, d, "tied" if tied else "sep",
                                                            ef, eb))


def _max_inverse_entry(w):
    # host fp64 max |M| over the chunks of the case (the quantity the case is
    # built to stress; not compared with anything)
    worst = 0.0
    bt = w.extra.get("beta_tilde", w.beta)
    for b in range(w.B):
        for h in range(w.H):
            for c0 in range(0, w.T, 64):
                k = w.k[b, c0:c0 + 64, h].astype(np.float64)
                n = k.shape[0]
                G = np.cumsum(w.g[b, c0:c0 + n, h].astype(np.float64))
                Gm = np.concatenate([[0.0], G[:-1]])
                L = np.tril(bt[b, c0:c0 + n, h, None] * np.exp(Gm[:, None] - G[None, :]) *
                            (k @ k.T), -1)
                worst = max(worst, float(np.max(np.abs(np.linalg.inv(np.eye(n) + L)))))
    return worst


@pytest.mark.parametrize("d", [128, 256])
def test_inverse_with_large_entries(d):
    # nearly parallel keys of norm 2, weak decay, beta~ |k|^2 ~ 0.99 (1 + alpha):
    # the transitions flip the shared key direction each token (eigenvalue
    # ~ -0.98) and M's rows hold ~64 alternating entries of size ~2
    rng = np.random.default_rng(303 + d)
    w = random_case(seed=303 + d, B=1, T=192, H=2, dk=d, dv=d, in_dtype="bf16", dht=True)
    u = rng.standard_normal((1, 1, 2, d))
    u /= np.linalg.norm(u, axis=-1, keepdims=True)
    k = u + 0.05 * rng.standard_normal(w.k.shape) / np.sqrt(d)
    k = 2.0 * k / np.linalg.norm(k, axis=-1, keepdims=True)
    w.k = bf16_round(k.astype(np.float32))
    w.g = (w.g * np.float32(0.02)).astype(np.float32)
    alpha = np.exp(w.g.astype(np.float64))
    kk = np.sum(w.k.astype(np.float64) ** 2, axis=-1)
    bt = bf16_round((0.99 * (1.0 + alpha) / kk).astype(np.float32))
    over = bt.astype(np.float64) * kk > 1.0 + alpha
    bt[over] = bf16_round(bt[over] * np.float32(0.995))
    assert np.all(bt.astype(np.float64) * kk <= 1.0 + alpha)
    w.extra["beta_tilde"] = bt
    mmax = _max_inverse_entry(w)
    assert mmax > 1.8, mmax  # the case does reach the large-entry regime
    ef = check_fwd(w)
    eb = check_bwd(w)
    _log("large inverse entries d=%d (max |M| = %.3f): fwd %s bwd %s" % (d, mmax, ef, eb))


# ------------------------------------------------------------ non-finite inputs
def _nonfinite_case(d, in_dtype="bf16"):
    # three sequences of 3000 tokens, two heads: 144 chunk slots x 2 heads = 288
    # chunk-heads, more than one per CU, so the persistent gradient kernel
    # carries a workgroup from a poisoned chunk-head on to a clean one
    return random_case(seed=505 + d, T=0, H=2, dk=d, dv=d, in_dtype=in_dtype, dht=True,
                       seqlens=[3000, 3000, 3000])


NONFINITE = [(128, "stateless", "v"), (128, "saved", "v"), (256, "stateless", "v"),
             (256, "saved", "v"), (128, "saved", "k"), (128, "saved", "q"),
             (64, "saved", "v_f32")]


@pytest.mark.parametrize("d,pair,where", NONFINITE,
                         ids=["d%d_%s_%s" % c for c in NONFINITE])
def test_nonfinite_values_stay_in_their_sequence(d, pair, where):
    # a NaN in one token of v (or k, or q) of sequence 0, head 0, and an Inf in
    # dO further along the same sequence; "v_f32" is the fp32-input path
    import torch
    import paper_2506_02475_amd as comba
    from gpu_helpers import to_device

    clean = _nonfinite_case(d, "f32" if where.endswith("f32") else "bf16")
    bad = copy.deepcopy(clean)
    seq, h = 0, 0
    a0 = int(clean.cu_seqlens[seq])
    t_nan, t_inf = a0 + 330, a0 + 2400       # chunk 5 and chunk 37 of sequence 0
    getattr(bad, where.split("_")[0])[0, t_nan, h, 7] = np.nan
    bad.dO[0, t_inf, h, 3] = np.inf

    def run(w):
        a = to_device(w)
        args = (a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"], a["h0"])
        kw = dict(cu_seqlens=a["cu_seqlens"], cu_seqlens_host=w.cu_seqlens)
        if pair == "saved":
            o, ht, ws = comba.comba_chunk_fwd_save(*args, **kw)
            gr = comba.comba_chunk_bwd_saved(*args, a["dO"], a["dht"], workspace=ws, **kw)
        else:
            o, ht = comba.comba_chunk_fwd(*args, **kw)
            gr = comba.comba_chunk_bwd(*args, a["dO"], a["dht"], **kw)
        torch.cuda.synchronize()
        out = {"o": o, "ht": ht}
        out.update(gr)
        return {k_: v_.cpu().numpy() for k_, v_ in out.items()}

    rc = run(clean)
    rb = run(bad)
    for name, x in rc.items():
        assert np.all(np.isfinite(x)), ("clean run", name)
    cu = clean.cu_seqlens
    a, b = int(cu[seq]), int(cu[seq + 1])
    poisoned = np.zeros(clean.T, bool)
    poisoned[a:b] = True
    for name in ("o", "dq", "dk", "dv", "dg", "dbeta"):
        x, y = rb[name][0], rc[name][0]        # [T, H, ...]
        # every other sequence, and the other head everywhere, bitwise equal
        assert np.array_equal(x[~poisoned], y[~poisoned]), name
        assert np.array_equal(x[:, 1 - h], y[:, 1 - h]), name
        # the poisoned sequence and head carries non-finite values
        assert not np.all(np.isfinite(x[a:b, h])), name
    for name in ("ht", "dh0"):
        x, y = rb[name], rc[name]              # [N, H, dk, dv]
        for s_ in range(len(cu) - 1):
            for hh in range(clean.H):
                if (s_, hh) == (seq, h) and not (name == "ht" and where == "q"):
                    assert not np.all(np.isfinite(x[s_, hh])), name
                else:
                    # (the states never depend on q: a NaN in q leaves ht exact)
                    assert np.array_equal(x[s_, hh], y[s_, hh]), (name, s_, hh)
    # dd sums over every sequence of a head
    assert not np.isfinite(rb["dd"][h]) and rb["dd"][1 - h] == rc["dd"][1 - h]
    # outputs before the poisoned chunk are untouched (causality)
    c_nan = a + (t_nan - a) // 64 * 64
    assert np.array_equal(rb["o"][0, a:c_nan, h], rc["o"][0, a:c_nan, h])
    _log("non-finite d=%d %s %s: o untouched before token %d; %d of %d tokens hold a non-finite value" % (
        d, pair, where, c_nan - a, int(np.sum((~np.isfinite(rb["o"][0, a:b, h])).any(-1))), b - a))
