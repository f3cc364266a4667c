"""Seeded synthetic inputs for the Comba chunk-wise operator.

This module is input plumbing only: it draws random tensors with the shapes and
value distributions of the Comba layer's operator inputs and rounds them to the
storage precision.  It performs none of the recurrence's arithmetic, so both the
fp64 oracle and the HIP path can consume exactly the same values.

Distributions follow the gate parameterisation of the paper (Section 3.2,
Table 5): log alpha = -softplus(x) so that alpha is in (0, 1), beta = sigmoid(x),
q and k L2-normalised per token and head (Section 3.4), v standard normal.  The
output-feedback scalar d is one value per head (Eq. comba-S).

Layouts (all C-contiguous):
    q, k       [B, T, H, dk]
    v, dO      [B, T, H, dv]
    g, beta    [B, T, H]          g = log alpha (always fp32)
    d          [H]                (always fp32)
    h0, dht    [N, H, dk, dv]     (always fp32; state stored as S^T, see Eq. comba-S)
    cu_seqlens [N + 1] int32      (varlen only; then B == 1 and T is the packed total)

Arrays are returned as float32 numpy arrays whose values are exactly
representable in the storage dtype (bf16 inputs are pre-rounded, round to
nearest even), so widening them to fp64 (oracle) or narrowing them to bf16
(GPU) is exact.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

__all__ = [
    "WorkloadSpec",
    "Workload",
    "WORKLOADS",
    "attach_beta_tilde",
    "prologue_case",
    "bf16_round",
    "generate",
    "random_case",
]


_SLAB = 1 << 20  # elements per in-place processing slab (bounds temporaries)


def bf16_round_(x: np.ndarray) -> np.ndarray:
    """Round a float32 array to the nearest bfloat16 in place (ties to even)."""
    assert x.dtype == np.float32 and x.flags.c_contiguous
    u = x.reshape(-1).view(np.uint32)
    for a in range(0, u.size, _SLAB):
        blk = u[a:a + _SLAB]
        lsb = (blk >> np.uint32(16)) & np.uint32(1)
        blk += np.uint32(0x7FFF)
        blk += lsb
        blk &= np.uint32(0xFFFF0000)
    return x


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    return bf16_round_(np.array(x, dtype=np.float32, order="C", copy=True))


def _normal(rng, shape) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    rng.standard_normal(dtype=np.float32, out=out)
    return out


def _softplus(x: np.ndarray) -> np.ndarray:
    # numerically safe log(1 + e^x) in float32
    return np.logaddexp(np.float32(0.0), x).astype(np.float32)


def _sigmoid(x: np.ndarray) -> np.ndarray:
    return (1.0 / (1.0 + np.exp(-x.astype(np.float64)))).astype(np.float32)


def _l2norm_(x: np.ndarray) -> np.ndarray:
    """Normalise a float32 array to unit L2 norm along the last axis, in place."""
    flat = x.reshape(-1, x.shape[-1])
    rows = max(1, _SLAB // x.shape[-1])
    for a in range(0, flat.shape[0], rows):
        blk = flat[a:a + rows]
        n = np.sqrt(np.einsum("ij,ij->i", blk, blk))
        blk /= np.maximum(n, np.float32(1e-12))[:, None]
    return x


def _l2norm(x: np.ndarray) -> np.ndarray:
    return _l2norm_(np.array(x, dtype=np.float32, order="C", copy=True))


@dataclass(frozen=True)
class WorkloadSpec:
    """One named synthetic workload (shapes, dtypes, distributions, seed)."""

    name: str
    H: int
    dk: int
    dv: int
    B: int = 1
    T: int = 0                     # per-sequence length (fixed-length batches)
    nseq_varlen: int = 0           # > 0: packed variable-length batch of this many sequences
    len_range: tuple = (0, 0)      # inclusive [lo, hi] for varlen lengths
    chunk: int = 64
    in_dtype: str = "bf16"         # "f32" or "bf16" for q, k, v, beta, dO
    work: str = "fwd"              # "fwd" or "fwdbwd"
    d_mode: str = "uniform"        # "const:<x>" or "uniform"
    h0_mode: str = "zero"          # "zero" or "normal:<std>"
    seed: int = 0
    description: str = ""


# The five parity/benchmark workloads.  Shapes are those of the paper's 340M and
# 1.3B model layers (Section 4.1: 340M and 1.3B models; head dim 128).
WORKLOADS = [
    WorkloadSpec("tiny_f32_fwd", B=1, H=1, T=256, dk=64, dv=64, in_dtype="f32", work="fwd",
                 d_mode="const:0.5", h0_mode="zero", seed=0,
                 description="tiny fp32 forward, B1 H1 T256 d64"),
    WorkloadSpec("l340m_fwd", B=8, H=8, T=2048, dk=128, dv=128, in_dtype="bf16", work="fwd",
                 d_mode="uniform", h0_mode="normal:0.02", seed=1,
                 description="340M-shape layer forward, B8 H8 T2048 d128 bf16"),
    WorkloadSpec("l340m_fwdbwd", B=8, H=8, T=2048, dk=128, dv=128, in_dtype="bf16",
                 work="fwdbwd", d_mode="uniform", h0_mode="normal:0.02", seed=2,
                 description="340M-shape layer forward+backward, B8 H8 T2048 d128 bf16"),
    WorkloadSpec("l1p3b_fwdbwd", B=4, H=16, T=4096, dk=128, dv=128, in_dtype="bf16",
                 work="fwdbwd", d_mode="uniform", h0_mode="zero", seed=3,
                 description="1.3B-shape layer forward+backward, B4 H16 T4096 d128 bf16"),
    WorkloadSpec("varlen_512k_fwd", nseq_varlen=16, len_range=(1024, 65536), H=16, dk=128,
                 dv=128, in_dtype="bf16", work="fwd", d_mode="uniform",
                 h0_mode="normal:0.02", seed=4,
                 description="packed varlen forward, 16 seqs of U[1024,65536] tokens, H16 d128"),
]


@dataclass
class Workload:
    spec: WorkloadSpec
    B: int
    T: int
    H: int
    dk: int
    dv: int
    chunk: int
    in_dtype: str
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    g: np.ndarray
    beta: np.ndarray
    d: np.ndarray
    h0: Optional[np.ndarray]
    dO: Optional[np.ndarray] = None
    dht: Optional[np.ndarray] = None
    cu_seqlens: Optional[np.ndarray] = None
    extra: dict = field(default_factory=dict)

    @property
    def nseq(self) -> int:
        return self.B if self.cu_seqlens is None else len(self.cu_seqlens) - 1

    @property
    def seq_offsets(self) -> np.ndarray:
        """Token offsets [N+1] into the flattened [B*T] token axis."""
        if self.cu_seqlens is not None:
            return self.cu_seqlens.astype(np.int64)
        return np.arange(self.B + 1, dtype=np.int64) * self.T

    @property
    def tokens(self) -> int:
        return self.B * self.T


def _draw_d(rng, mode: str, H: int) -> np.ndarray:
    if mode.startswith("const:"):
        return np.full(H, float(mode.split(":")[1]), dtype=np.float32)
    if mode == "uniform":
        return rng.uniform(0.0, 1.0, size=H).astype(np.float32)
    raise ValueError(mode)


def _draw_h0(rng, mode: str, shape) -> Optional[np.ndarray]:
    if mode == "zero":
        return None
    if mode.startswith("normal:"):
        std = float(mode.split(":")[1])
        return (rng.standard_normal(shape, dtype=np.float32) * np.float32(std)).astype(np.float32)
    raise ValueError(mode)


def _fill_head(child_seed, h, arrays, in_dtype):
    """Draw one head's slices, in order q, k, v, gate noise, beta noise, dO."""
    rng = np.random.default_rng(child_seed)
    q, k, v, g, beta, dO = arrays
    B, T = q.shape[:2]
    for dst, norm in ((q, True), (k, True), (v, False)):
        x = _normal(rng, (B, T, dst.shape[-1]))
        if norm:
            _l2norm_(x)
        if in_dtype == "bf16":
            bf16_round_(x)
        dst[:, :, h, :] = x
    g[:, :, h] = -_softplus(_normal(rng, (B, T)))
    b = _sigmoid(_normal(rng, (B, T)))
    beta[:, :, h] = bf16_round_(b) if in_dtype == "bf16" else b
    if dO is not None:
        x = _normal(rng, (B, T, dO.shape[-1]))
        if in_dtype == "bf16":
            bf16_round_(x)
        dO[:, :, h, :] = x


def attach_beta_tilde(w: Workload, form: str = "b_beta", seed: int = 0) -> Workload:
    """Give ``w`` a separate state-feedback strength in ``w.extra['beta_tilde']``.

    Forms (Section 3.2 and the SPLR/IPLR comparison of Section 3):
      "b_beta"       beta~ = b_h * beta with one b_h = sigmoid(N(0,1)) per head
                     (the paper's default parameterisation, b in (0, 1));
      "independent"  beta~ = sigmoid(N(0,1)) per token, independent of beta;
      "iplr"         beta~ = 2 alpha c with c = sigmoid(N(0,1)) per token: the
                     IPLR transition alpha (I - 2 c k k^T) written in SPLR form
                     (beta~ up to 2, transition eigenvalues down to -alpha).
    The draws come from a PCG64 stream seeded with ``seed``; the result is
    rounded to the storage dtype like beta.
    """
    rng = np.random.default_rng(seed)
    shp = w.beta.shape
    if form == "b_beta":
        b = _sigmoid(rng.standard_normal(w.H, dtype=np.float32))
        bt = w.beta * b[None, None, :]
    elif form == "independent":
        bt = _sigmoid(rng.standard_normal(shp, dtype=np.float32))
    elif form == "iplr":
        c = _sigmoid(rng.standard_normal(shp, dtype=np.float32))
        bt = np.float32(2.0) * np.exp(w.g) * c
    else:
        raise ValueError(form)
    bt = np.ascontiguousarray(bt, dtype=np.float32)
    w.extra["beta_tilde"] = bf16_round(bt) if w.in_dtype == "bf16" else bt
    return w


def prologue_case(*, B=1, T=64, H=1, dk=64, dv=64, seed=0, in_dtype="bf16", seqlens=None,
                  tap_scale=0.5) -> dict:
    """Seeded inputs of the layer prologue: pre-activations xq, xk [B,T,H,dk] and xv
    [B,T,H,dv] ~ N(0,1) (bf16-representable for bf16 inputs), taps wq, wk, wv
    [H,d,4] ~ tap_scale * N(0,1) (fp32), output gradients gq, gk, gv ~ N(0,1)
    (fp32), and cu_seqlens for packed sequences (then B = 1, T = sum)."""
    rng = np.random.default_rng(seed)
    cu = None
    if seqlens is not None:
        cu = np.zeros(len(seqlens) + 1, dtype=np.int32)
        cu[1:] = np.cumsum(seqlens)
        B, T = 1, int(cu[-1])
    out = {"cu_seqlens": cu, "B": B, "T": T, "H": H, "dk": dk, "dv": dv, "in_dtype": in_dtype}
    for n, dd in (("xq", dk), ("xk", dk), ("xv", dv)):
        x = rng.standard_normal((B, T, H, dd), dtype=np.float32)
        out[n] = bf16_round(x) if in_dtype == "bf16" else x
    for n, dd in (("wq", dk), ("wk", dk), ("wv", dv)):
        out[n] = (np.float32(tap_scale) * rng.standard_normal((H, dd, 4), dtype=np.float32))
    for n, dd in (("gq", dk), ("gk", dk), ("gv", dv)):
        out[n] = rng.standard_normal((B, T, H, dd), dtype=np.float32)
    return out


def generate(spec, *, with_grad: Optional[bool] = None, threads: Optional[int] = None) -> Workload:
    """Draw the seeded inputs of one workload.

    ``spec`` is a WorkloadSpec or an index into WORKLOADS.  A root PCG64 stream
    seeded with spec.seed draws, in order, the varlen lengths (if any), d and
    h0; each head h then draws its own q, k, v, gate noise, beta noise and dO
    from child stream h of SeedSequence(spec.seed) (heads are filled in
    parallel threads; the values do not depend on the thread count).
    """
    import os
    from concurrent.futures import ThreadPoolExecutor

    if isinstance(spec, int):
        spec = WORKLOADS[spec]
    ss = np.random.SeedSequence(spec.seed)
    root_seed, head_seeds = ss.spawn(1)[0], None
    rng = np.random.default_rng(root_seed)
    cu = None
    if spec.nseq_varlen > 0:
        lo, hi = spec.len_range
        lens = rng.integers(lo, hi, size=spec.nseq_varlen, endpoint=True)
        cu = np.zeros(spec.nseq_varlen + 1, dtype=np.int32)
        cu[1:] = np.cumsum(lens)
        B, T = 1, int(cu[-1])
    else:
        B, T = spec.B, spec.T
    H, dk, dv = spec.H, spec.dk, spec.dv
    d = _draw_d(rng, spec.d_mode, H)
    N = B if cu is None else len(cu) - 1
    h0 = _draw_h0(rng, spec.h0_mode, (N, H, dk, dv))
    if with_grad is None:
        with_grad = spec.work == "fwdbwd"
    q = np.empty((B, T, H, dk), np.float32)
    k = np.empty((B, T, H, dk), np.float32)
    v = np.empty((B, T, H, dv), np.float32)
    g = np.empty((B, T, H), np.float32)
    beta = np.empty((B, T, H), np.float32)
    dO = np.empty((B, T, H, dv), np.float32) if with_grad else None
    head_seeds = np.random.SeedSequence(spec.seed).spawn(1 + H)[1:]
    arrays = (q, k, v, g, beta, dO)
    if threads is None:
        try:
            threads = len(os.sched_getaffinity(0))
        except Exception:  # pragma: no cover
            threads = os.cpu_count() or 1
    with ThreadPoolExecutor(max_workers=max(1, min(threads, H, 16))) as ex:
        list(ex.map(lambda h: _fill_head(head_seeds[h], h, arrays, spec.in_dtype), range(H)))
    return Workload(spec=spec, B=B, T=T, H=H, dk=dk, dv=dv, chunk=spec.chunk,
                    in_dtype=spec.in_dtype, q=q, k=k, v=v, g=g, beta=beta, d=d, h0=h0,
                    dO=dO, dht=None, cu_seqlens=cu)


def random_case(*, B=1, T=64, H=1, dk=16, dv=16, seed=0, in_dtype="f32", seqlens=None,
                h0=True, grad=True, dht=False, gate_scale=1.0, d_range=(0.0, 1.0),
                normalize=True, beta_tilde=False) -> Workload:
    """A small general-purpose case for tests (same distributions, free shapes).

    ``seqlens`` (list of ints) builds a packed variable-length batch (B must be 1).
    ``gate_scale`` scales the softplus argument noise's magnitude so tests can
    reach strong and weak decay.  ``beta_tilde`` adds an independent feedback
    strength in ``extra['beta_tilde']`` (stored like beta: bf16-representable
    for bf16 inputs).
    """
    rng = np.random.default_rng(seed)
    cu = None
    if seqlens is not None:
        assert B == 1
        cu = np.zeros(len(seqlens) + 1, dtype=np.int32)
        cu[1:] = np.cumsum(seqlens)
        T = int(cu[-1])
    q = rng.standard_normal((B, T, H, dk), dtype=np.float32)
    k = rng.standard_normal((B, T, H, dk), dtype=np.float32)
    if normalize:
        q, k = _l2norm(q), _l2norm(k)
    v = rng.standard_normal((B, T, H, dv), dtype=np.float32)
    g = (-_softplus(np.float32(gate_scale) * rng.standard_normal((B, T, H), dtype=np.float32)))
    beta = _sigmoid(rng.standard_normal((B, T, H), dtype=np.float32))
    d = rng.uniform(d_range[0], d_range[1], size=H).astype(np.float32)
    N = B if cu is None else len(cu) - 1
    h0a = (rng.standard_normal((N, H, dk, dv), dtype=np.float32) * np.float32(0.1)) if h0 else None
    dO = rng.standard_normal((B, T, H, dv), dtype=np.float32) if grad else None
    dhta = rng.standard_normal((N, H, dk, dv), dtype=np.float32) if dht else None
    extra = {}
    if beta_tilde:
        extra["beta_tilde"] = _sigmoid(rng.standard_normal((B, T, H), dtype=np.float32))
    if in_dtype == "bf16":
        q, k, v, beta = bf16_round(q), bf16_round(k), bf16_round(v), bf16_round(beta)
        if dO is not None:
            dO = bf16_round(dO)
        if beta_tilde:
            extra["beta_tilde"] = bf16_round(extra["beta_tilde"])
    spec = WorkloadSpec("random", H=H, dk=dk, dv=dv, B=B, T=T, in_dtype=in_dtype,
                        work="fwdbwd" if grad else "fwd", seed=seed)
    return Workload(spec=spec, B=B, T=T, H=H, dk=dk, dv=dv, chunk=64, in_dtype=in_dtype,
                    q=q, k=k, v=v, g=g.astype(np.float32), beta=beta, d=d, h0=h0a, dO=dO,
                    dht=dhta, cu_seqlens=cu, extra=extra)
