"""Shared helpers for the GPU parity tests: move a seeded workload to the
device, call the HIP path through the C ABI, and compare with the fp64 oracle."""
import numpy as np

import oracle


def maxrel(x, ref):
    """Norm-wise max relative error ||x - ref||_inf / ||ref||_inf (ref = oracle)."""
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.max(np.abs(ref)) if ref.size else 0.0
    num = np.max(np.abs(x - ref)) if ref.size else 0.0
    if den == 0.0:
        return num
    return num / den


def maxrel_by_slice(x, ref, offsets):
    """Largest norm-wise relative error over the (sequence, head) slices of a
    per-token tensor [B, T, H, ...] (ref = oracle); ``offsets`` are the
    sequences' token offsets into the flattened B*T axis.  Every slice is
    measured against its own largest reference value, so the small entries of
    one sequence or head are not hidden behind another's."""
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    H = ref.shape[2]
    xf = x.reshape((-1, H) + ref.shape[3:])
    rf = ref.reshape((-1, H) + ref.shape[3:])
    worst = 0.0
    for s in range(len(offsets) - 1):
        a, b = int(offsets[s]), int(offsets[s + 1])
        if b <= a:
            continue
        for h in range(H):
            worst = max(worst, maxrel(xf[a:b, h], rf[a:b, h]))
    return worst


def elementwise_floor(x, ref, floor=1e-2):
    """Largest elementwise relative error |x - y| / max(|y|, floor * ||y||_inf),
    for information: near zero a purely elementwise ratio is ill-posed."""
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    den = np.maximum(np.abs(ref), floor * np.max(np.abs(ref)))
    den = np.where(den > 0, den, 1.0)
    return float(np.max(np.abs(x - ref) / den))


def tol_for(w):
    # tolerances stated for the operator: 1e-5 (fp32 inputs), 2e-3 (bf16 inputs,
    # fp32 accumulation), on the norm-wise max relative error
    return 1e-5 if w.in_dtype == "f32" else 2e-3


def to_device(w, device="cuda"):
    import torch

    dt = torch.float32 if w.in_dtype == "f32" else torch.bfloat16

    def t(x, dtype=None):
        if x is None:
            return None
        return torch.from_numpy(np.ascontiguousarray(x)).to(device=device, dtype=dtype or torch.float32)

    out = dict(q=t(w.q, dt), k=t(w.k, dt), v=t(w.v, dt), g=t(w.g), beta=t(w.beta, dt), d=t(w.d),
               h0=t(w.h0), dO=t(w.dO, dt), dht=t(w.dht),
               beta_tilde=t(w.extra.get("beta_tilde"), dt))
    out["cu_seqlens"] = None if w.cu_seqlens is None else \
        torch.from_numpy(w.cu_seqlens.astype(np.int32)).to(device)
    return out


def gpu_fwd(w, **kw):
    import torch
    import paper_2506_02475_amd as comba

    a = to_device(w)
    o, ht = comba.comba_chunk_fwd(a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"], a["h0"],
                                  beta_tilde=a["beta_tilde"], cu_seqlens=a["cu_seqlens"], **kw)
    torch.cuda.synchronize()
    return o.cpu().numpy(), (None if ht is None else ht.cpu().numpy())


def gpu_bwd(w, **kw):
    import torch
    import paper_2506_02475_amd as comba

    a = to_device(w)
    gr = comba.comba_chunk_bwd(a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"], a["h0"],
                               a["dO"], a["dht"], beta_tilde=a["beta_tilde"],
                               cu_seqlens=a["cu_seqlens"], **kw)
    torch.cuda.synchronize()
    return {k: (None if v is None else v.cpu().numpy()) for k, v in gr.items()}


def _offsets(w):
    return w.seq_offsets


def check_fwd(w, heads=None, tol=None):
    """GPU forward vs oracle; returns the error dict (asserts within tolerance).

    Norm-wise max relative error per output tensor (the stated metric) and per
    (sequence, head) slice ("o@seq,head"), both held to ``tol``; the floored
    elementwise error ("o~ew") is reported only."""
    tol = tol_for(w) if tol is None else tol
    o, ht = gpu_fwd(w)
    ro, rht = oracle.workload_fwd(w, heads=heads)
    sel = slice(None) if heads is None else list(heads)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(ht)), w.spec.name
    hts = ht[:, sel]
    errs = {"o": maxrel(o[:, :, sel], ro), "ht": maxrel(hts, rht),
            "o@seq,head": maxrel_by_slice(o[:, :, sel], ro, _offsets(w)),
            "ht@seq,head": max((maxrel(hts[a, b], rht[a, b]) for a in range(rht.shape[0])
                                for b in range(rht.shape[1])), default=0.0)}
    for name, e in errs.items():
        assert e <= tol, (w.spec.name, name, e, tol)
    errs["o~ew"] = elementwise_floor(o[:, :, sel], ro)
    return errs


def check_bwd(w, heads=None, tol=None):
    """GPU backward vs oracle, metrics as in check_fwd; dd per head as well."""
    tol = tol_for(w) if tol is None else tol
    gr = gpu_bwd(w)
    ref = oracle.workload_bwd(w, heads=heads)
    sel = slice(None) if heads is None else list(heads)
    errs = {}
    names = ("dq", "dk", "dv", "dg", "dbeta") + (("dbeta_tilde",) if "dbeta_tilde" in ref else ())
    assert ("dbeta_tilde" in gr) == ("dbeta_tilde" in ref)
    for name in names:
        errs[name] = maxrel(gr[name][:, :, sel], ref[name])
        errs[name + "@seq,head"] = maxrel_by_slice(gr[name][:, :, sel], ref[name], _offsets(w))
    errs["dd"] = maxrel(gr["dd"][sel], ref["dd"])
    # dd_h = -sum_t <k_t, dq~_t> over every token of head h: per head, its
    # error is held against the magnitude of the terms it sums (a per-head
    # relative error is ill-conditioned when the terms cancel; reported only)
    ddiff = np.abs(gr["dd"][sel] - ref["dd"])
    terms = np.einsum("bthd,bthd->h", np.abs(w.k[:, :, sel].astype(np.float64)),
                      np.abs(ref["dq"]))
    errs["dd@head/terms"] = float(np.max(ddiff / np.maximum(terms, 1e-30)))
    rdd = np.abs(ref["dd"])
    info_dd = float(np.max(ddiff / np.maximum(rdd, max(1e-7 * np.max(rdd), 1e-30))))
    errs["dh0"] = maxrel(gr["dh0"][:, sel], ref["dh0"])
    for name, e in errs.items():
        assert np.isfinite(e) and e <= tol, (w.spec.name, name, e, tol)
    for name in names:
        errs[name + "~ew"] = elementwise_floor(gr[name][:, :, sel], ref[name])
    errs["dd@head~rel"] = info_dd
    return errs


def bar_errors(errs):
    """The entries of an error dict that are held to the tolerance (the
    informational floored-elementwise and per-head-relative figures, whose
    keys contain '~', are dropped)."""
    return {k: v for k, v in errs.items() if "~" not in k}
