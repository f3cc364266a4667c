"""fp64 CPU oracle for the Comba chunk-wise operator -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, the smoke check and the benchmark's CPU-baseline leg may use
this package.  The product path (the HIP library and its binding) never
imports, links or calls it, and it imports nothing from the product package.

Two independent formulations of the same result:

* ``step_fwd`` / ``step_bwd`` -- the token-by-token recurrence of Eq. comba-S
  (Section 3) and its reverse-mode derivative, in C (``comba_step.c``), fp64,
  threaded over independent (sequence, head) pairs.
* ``chunk.chunk_fwd`` -- the chunk-wise reformulation of Section 3.3 (WY/UT
  transform with one triangular inverse, Eqs. wy1, wy2, prepare-WY_M and the
  inter/intra-chunk matrix form), in NumPy fp64.  It must agree with the step
  form for every chunk size.

Parity status: the forward step form, the backward step form and the chunk form
are all pinned by the tests in ``tests/test_oracle_*.py`` (closed-form
reductions, invariants, finite differences); no function here is unpinned.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "comba_step.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (fp64, -O2, pthreads)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-pthread", "-o", tmp, _SRC,
                               "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build()
            lib = ctypes.CDLL(_LIB)
            P = ctypes.c_void_p
            I = ctypes.c_int
            lib.oracle_fwd.argtypes = [I, P, I, I, I] + [P] * 10 + [I]
            lib.oracle_fwd.restype = I
            lib.oracle_bwd.argtypes = [I, P, I, I, I] + [P] * 18 + [I]
            lib.oracle_bwd.restype = I
            _lib = lib
    return _lib


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except Exception:  # pragma: no cover
        return os.cpu_count() or 1


def _f64(x, shape=None):
    if x is None:
        return None
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    if shape is not None:
        a = a.reshape(shape)
    return a


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _offsets(B, T, cu_seqlens):
    if cu_seqlens is None:
        return np.ascontiguousarray(np.arange(B + 1, dtype=np.int64) * T)
    return np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int64))


def step_fwd(q, k, v, g, beta, d, h0=None, *, cu_seqlens=None, beta_tilde=None,
             nthreads=None):
    """Forward of the step recurrence.

    q, k [B,T,H,dk]; v [B,T,H,dv]; g, beta [B,T,H]; d [H]; h0 [N,H,dk,dv] or None.
    ``beta_tilde`` defaults to ``beta`` (the operator's b == 1 reading).
    Returns (o [B,T,H,dv], ht [N,H,dk,dv]) in fp64.
    """
    q = _f64(q)
    B, T, H, dk = q.shape
    dv = np.shape(v)[-1]
    Ttot = B * T
    cu = _offsets(B, T, cu_seqlens)
    N = len(cu) - 1
    qq = q.reshape(Ttot, H, dk)
    kk = _f64(k, (Ttot, H, dk))
    vv = _f64(v, (Ttot, H, dv))
    gg = _f64(g, (Ttot, H))
    bb = _f64(beta, (Ttot, H))
    bt = bb if beta_tilde is None else _f64(beta_tilde, (Ttot, H))
    dd = _f64(d, (H,))
    hh = _f64(h0, (N, H, dk, dv))
    o = np.zeros((Ttot, H, dv))
    ht = np.zeros((N, H, dk, dv))
    rc = _load().oracle_fwd(N, _ptr(cu), H, dk, dv, _ptr(qq), _ptr(kk), _ptr(vv), _ptr(gg),
                            _ptr(bb), _ptr(bt), _ptr(dd), _ptr(hh), _ptr(o), _ptr(ht),
                            nthreads or default_threads())
    if rc != 0:
        raise RuntimeError("oracle_fwd failed (%d)" % rc)
    return o.reshape(B, T, H, dv), ht


def step_bwd(q, k, v, g, beta, d, h0, dO, dht=None, *, cu_seqlens=None, beta_tilde=None,
             nthreads=None):
    """Reverse-mode gradients of L = <dO, o> + <dht, ht> for the step recurrence.

    Returns a dict with dq, dk [B,T,H,dk]; dv [B,T,H,dv]; dg, dbeta [B,T,H];
    dd [H]; dh0 [N,H,dk,dv].  When ``beta_tilde`` is None (bt == beta) the
    returned ``dbeta`` is the total derivative through both roles of beta;
    otherwise ``dbeta`` and ``dbeta_tilde`` are returned separately.
    """
    q = _f64(q)
    B, T, H, dk = q.shape
    dv = np.shape(v)[-1]
    Ttot = B * T
    cu = _offsets(B, T, cu_seqlens)
    N = len(cu) - 1
    qq = q.reshape(Ttot, H, dk)
    kk = _f64(k, (Ttot, H, dk))
    vv = _f64(v, (Ttot, H, dv))
    gg = _f64(g, (Ttot, H))
    bb = _f64(beta, (Ttot, H))
    bt = bb if beta_tilde is None else _f64(beta_tilde, (Ttot, H))
    dd = _f64(d, (H,))
    hh = _f64(h0, (N, H, dk, dv))
    dOo = _f64(dO, (Ttot, H, dv))
    dhtt = _f64(dht, (N, H, dk, dv))
    out = {
        "dq": np.zeros((Ttot, H, dk)), "dk": np.zeros((Ttot, H, dk)),
        "dv": np.zeros((Ttot, H, dv)), "dg": np.zeros((Ttot, H)),
        "dbeta": np.zeros((Ttot, H)), "dbeta_tilde": np.zeros((Ttot, H)),
        "dd_part": np.zeros((N, H)), "dh0": np.zeros((N, H, dk, dv)),
    }
    rc = _load().oracle_bwd(N, _ptr(cu), H, dk, dv, _ptr(qq), _ptr(kk), _ptr(vv), _ptr(gg),
                            _ptr(bb), _ptr(bt), _ptr(dd), _ptr(hh), _ptr(dOo), _ptr(dhtt),
                            _ptr(out["dq"]), _ptr(out["dk"]), _ptr(out["dv"]), _ptr(out["dg"]),
                            _ptr(out["dbeta"]), _ptr(out["dbeta_tilde"]), _ptr(out["dd_part"]),
                            _ptr(out["dh0"]), nthreads or default_threads())
    if rc != 0:
        raise RuntimeError("oracle_bwd failed (%d)" % rc)
    res = {
        "dq": out["dq"].reshape(B, T, H, dk), "dk": out["dk"].reshape(B, T, H, dk),
        "dv": out["dv"].reshape(B, T, H, dv), "dg": out["dg"].reshape(B, T, H),
        "dd": np.sum(out["dd_part"], axis=0), "dh0": out["dh0"],
    }
    if beta_tilde is None:
        res["dbeta"] = (out["dbeta"] + out["dbeta_tilde"]).reshape(B, T, H)
    else:
        res["dbeta"] = out["dbeta"].reshape(B, T, H)
        res["dbeta_tilde"] = out["dbeta_tilde"].reshape(B, T, H)
    return res


def _workload_beta_tilde(w, sel):
    bt = w.extra.get("beta_tilde")
    return None if bt is None else bt[:, :, sel]


def workload_fwd(w, *, heads=None, nthreads=None):
    """Oracle forward on a comba_inputs.Workload (optionally a subset of heads);
    a separate feedback strength in ``w.extra['beta_tilde']`` is used when present."""
    sel = slice(None) if heads is None else list(heads)
    h0 = None if w.h0 is None else w.h0[:, sel]
    return step_fwd(w.q[:, :, sel], w.k[:, :, sel], w.v[:, :, sel], w.g[:, :, sel],
                    w.beta[:, :, sel], w.d[sel], h0, cu_seqlens=w.cu_seqlens,
                    beta_tilde=_workload_beta_tilde(w, sel), nthreads=nthreads)


def workload_bwd(w, *, heads=None, nthreads=None):
    """Oracle backward on a comba_inputs.Workload (optionally a subset of heads)."""
    sel = slice(None) if heads is None else list(heads)
    h0 = None if w.h0 is None else w.h0[:, sel]
    dht = None if w.dht is None else w.dht[:, sel]
    return step_bwd(w.q[:, :, sel], w.k[:, :, sel], w.v[:, :, sel], w.g[:, :, sel],
                    w.beta[:, :, sel], w.d[sel], h0, w.dO[:, :, sel], dht,
                    cu_seqlens=w.cu_seqlens, beta_tilde=_workload_beta_tilde(w, sel),
                    nthreads=nthreads)
