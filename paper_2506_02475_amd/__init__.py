"""MI355X (gfx950) chunk-wise Comba operator: Python binding of libcomba.so.

The binding only marshals arguments: it checks dtypes/shapes/devices of torch
tensors, allocates outputs and the workspace with torch (device memory and the
current stream are the only things torch provides), and calls the C ABI of
``include/comba.h``.  Every step of the computation runs in the HIP kernels.
There is no fallback: if the library is missing or no GPU is present, the
calls raise.

    o, ht = comba_chunk_fwd(q, k, v, g, beta, d, h0)
    grads = comba_chunk_bwd(q, k, v, g, beta, d, h0, dO, dht)

Shapes (see include/comba.h): q, k [B,T,H,dk]; v, dO [B,T,H,dv]; g, beta [B,T,H];
d [H]; h0, dht [N,H,dk,dv].  q, k, v, beta, dO share one dtype (bfloat16 or
float32); g, d and states are float32; all outputs are float32.  Pass
``cu_seqlens`` (int32 [N+1] on the device) for a packed variable-length batch
with B == 1.  ``beta_tilde=`` ([B,T,H], the dtype of q) gives the state
feedback strength its own value (Section 3.2; omitted: tied to beta); the
backward then also returns ``dbeta_tilde`` and ``dbeta`` covers the write
strength only.
"""
from __future__ import annotations

import ctypes
import os
import re
import threading

__all__ = ["comba_chunk_fwd", "comba_chunk_bwd", "comba_chunk_fwd_save", "comba_chunk_bwd_saved",
           "comba_chunk_fwd_noalloc", "noalloc_scratch_bytes",
           "comba_recurrent_fwd", "comba_prologue_fwd", "comba_prologue_bwd",
           "comba_gate_fwd", "comba_gate_bwd",
           "load_library", "library_path",
           "profile_enable", "profile_read",
           "fwd_workspace_bytes", "bwd_workspace_bytes", "exported_symbols", "CombaError",
           "CombaShape", "COMBA_F32", "COMBA_BF16", "CHUNK"]

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "libcomba.so")
_HEADER = os.path.join(os.path.dirname(_PKG), "include", "comba.h")
_lock = threading.Lock()
_lib = None

COMBA_F32 = 0
COMBA_BF16 = 1
CHUNK = 64


class CombaError(RuntimeError):
    pass


class CombaShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("T", ctypes.c_int32), ("H", ctypes.c_int32),
                ("dk", ctypes.c_int32), ("dv", ctypes.c_int32), ("chunk", ctypes.c_int32),
                ("num_seqs", ctypes.c_int32), ("cu_seqlens", ctypes.c_void_p),
                ("cu_seqlens_host", ctypes.c_void_p), ("in_dtype", ctypes.c_int)]


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load libcomba.so (built by ``paper_2506_02475_amd.build``); raises if absent."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH):
                raise ImportError("libcomba.so is not built; run "
                                  "`python -m paper_2506_02475_amd.build` (hipcc, gfx950)")
            lib = ctypes.CDLL(_LIB_PATH)
            P, Z, I = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
            SP = ctypes.POINTER(CombaShape)
            lib.comba_fwd_workspace_bytes.argtypes = [SP]
            lib.comba_fwd_workspace_bytes.restype = Z
            lib.comba_bwd_workspace_bytes.argtypes = [SP]
            lib.comba_bwd_workspace_bytes.restype = Z
            lib.comba_chunk_fwd.argtypes = [SP] + [P] * 10 + [P, Z, P]
            lib.comba_chunk_fwd.restype = I
            lib.comba_chunk_bwd.argtypes = [SP] + [P] * 18 + [P, Z, P]
            lib.comba_chunk_bwd.restype = I
            lib.comba_chunk_fwd_save.argtypes = [SP] + [P] * 10 + [P, Z, P]
            lib.comba_chunk_fwd_save.restype = I
            lib.comba_chunk_bwd_saved.argtypes = [SP] + [P] * 18 + [P, Z, P]
            lib.comba_chunk_bwd_saved.restype = I
            lib.comba_chunk_fwd_noalloc.argtypes = [SP] + [P] * 10 + [P]
            lib.comba_chunk_fwd_noalloc.restype = I
            lib.comba_noalloc_scratch_bytes.argtypes = []
            lib.comba_noalloc_scratch_bytes.restype = Z
            lib.comba_recurrent_fwd.argtypes = [SP] + [P] * 10 + [P]
            lib.comba_recurrent_fwd.restype = I
            lib.comba_prologue_fwd.argtypes = [SP] + [P] * 9 + [P]
            lib.comba_prologue_fwd.restype = I
            lib.comba_prologue_bwd.argtypes = [SP] + [P] * 15 + [P, Z, P]
            lib.comba_prologue_bwd.restype = I
            lib.comba_prologue_workspace_bytes.argtypes = [SP]
            lib.comba_prologue_workspace_bytes.restype = Z
            lib.comba_gate_fwd.argtypes = [SP, P, P, P, P]
            lib.comba_gate_fwd.restype = I
            lib.comba_gate_bwd.argtypes = [SP, P, P, P, P, P, P]
            lib.comba_gate_bwd.restype = I
            lib.comba_profile_enable.argtypes = [I]
            lib.comba_profile_enable.restype = I
            lib.comba_profile_read.argtypes = [P, P, I]
            lib.comba_profile_read.restype = I
            lib.comba_profile_select.argtypes = [ctypes.c_char_p]
            lib.comba_profile_select.restype = I
            lib.comba_status_string.argtypes = [I]
            lib.comba_status_string.restype = ctypes.c_char_p
            _lib = lib
    return _lib


def profile_enable(on: bool = True) -> None:
    """Turn per-stage HIP-event timing of the entry points on or off (this thread)."""
    _check(load_library().comba_profile_enable(1 if on else 0))


def profile_select(stage=None) -> None:
    """Record only the named stage's start and end in later timing sessions of
    this thread (None: every stage)."""
    _check(load_library().comba_profile_select(None if stage is None else stage.encode()))


def profile_read(capacity: int = 4096):
    """(stage name, ms) of every stage recorded since profile_enable(True)."""
    cap = capacity
    ms = (ctypes.c_float * cap)()
    names = (ctypes.c_char_p * cap)()
    n = load_library().comba_profile_read(ms, names, cap)
    if n < 0:
        raise CombaError("comba: profile_read failed")
    return [(names[i].decode(), float(ms[i])) for i in range(n)]


def exported_symbols():
    """Function names declared in include/comba.h (the C ABI)."""
    with open(_HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(comba_[a-z_]+)\s*\(", text)))


def _check(status: int):
    if status != 0:
        msg = load_library().comba_status_string(status).decode()
        raise CombaError("comba: %s (status %d)" % (msg, status))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _make_shape(B, T, H, dk, dv, N, cu_ptr, dtype_code, chunk=CHUNK, cu_host=None):
    """The C shape struct.  ``cu_host`` is a host int32 array of the offsets (a
    numpy array or a CPU tensor, kept alive by the caller for the call); the
    library then rejects a malformed offset table before any launch."""
    hp = None
    if cu_host is not None:
        hp = ctypes.c_void_p(cu_host.ctypes.data if hasattr(cu_host, "ctypes")
                             else cu_host.data_ptr())
    shp = CombaShape(B, T, H, dk, dv, chunk, N, cu_ptr, hp, dtype_code)
    shp._keep = cu_host  # the host offsets live as long as the struct
    return shp


def _host_offsets(cu_seqlens_host, n):
    """A contiguous host int32 copy of the offsets (or None), checked for length."""
    if cu_seqlens_host is None:
        return None
    import numpy as np

    if hasattr(cu_seqlens_host, "detach"):  # torch tensor
        if cu_seqlens_host.is_cuda:
            raise CombaError("comba: cu_seqlens_host must be in host memory")
        cu_seqlens_host = cu_seqlens_host.detach().numpy()
    a = np.ascontiguousarray(np.asarray(cu_seqlens_host), dtype=np.int32)
    if a.ndim != 1 or a.size != n:
        raise CombaError("comba: cu_seqlens_host must hold the N + 1 offsets of cu_seqlens")
    return a


def fwd_workspace_bytes(B, T, H, dk, dv, *, num_seqs=None, varlen=False, bf16=True) -> int:
    N = B if num_seqs is None else num_seqs
    shp = _make_shape(B, T, H, dk, dv, N, ctypes.c_void_p(1) if varlen else None,
                      COMBA_BF16 if bf16 else COMBA_F32)
    return int(load_library().comba_fwd_workspace_bytes(ctypes.byref(shp)))


def bwd_workspace_bytes(B, T, H, dk, dv, *, num_seqs=None, varlen=False, bf16=True) -> int:
    N = B if num_seqs is None else num_seqs
    shp = _make_shape(B, T, H, dk, dv, N, ctypes.c_void_p(1) if varlen else None,
                      COMBA_BF16 if bf16 else COMBA_F32)
    return int(load_library().comba_bwd_workspace_bytes(ctypes.byref(shp)))


def _prepare(q, k, v, g, beta, d, h0, cu_seqlens, extra=(), cu_seqlens_host=None):
    import torch

    if not q.is_cuda:
        raise CombaError("comba: tensors must be on a GPU device")
    if q.dtype == torch.bfloat16:
        code = COMBA_BF16
    elif q.dtype == torch.float32:
        code = COMBA_F32
    else:
        raise CombaError("comba: q must be bfloat16 or float32")
    for name, t in (("k", k), ("v", v), ("beta", beta)) + tuple(extra):
        if t.dtype != q.dtype:
            raise CombaError("comba: %s must have the dtype of q" % name)
    for name, t in (("g", g), ("d", d)):
        if t.dtype != torch.float32:
            raise CombaError("comba: %s must be float32" % name)
    tensors = [q, k, v, g, beta, d] + [t for _, t in extra]
    if h0 is not None:
        tensors.append(h0)
    for t in tensors:
        if not t.is_contiguous() or t.device != q.device:
            raise CombaError("comba: all tensors must be contiguous and on one device")
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    if k.shape != q.shape or v.shape[:3] != (B, T, H) or g.shape != (B, T, H) \
            or beta.shape != (B, T, H) or d.shape != (H,):
        raise CombaError("comba: inconsistent shapes")
    if cu_seqlens is not None:
        if cu_seqlens.dtype != torch.int32 or not cu_seqlens.is_contiguous() \
                or cu_seqlens.device != q.device or B != 1:
            raise CombaError("comba: cu_seqlens must be contiguous int32 on the device, B == 1")
        N = cu_seqlens.numel() - 1
    else:
        if cu_seqlens_host is not None:
            raise CombaError("comba: cu_seqlens_host needs cu_seqlens")
        N = B
    if h0 is not None and (h0.dtype != torch.float32 or tuple(h0.shape) != (N, H, dk, dv)):
        raise CombaError("comba: h0 must be float32 [N,H,dk,dv]")
    shp = _make_shape(B, T, H, dk, dv, N, _ptr(cu_seqlens), code,
                      cu_host=_host_offsets(cu_seqlens_host, N + 1))
    return shp, (B, T, H, dk, dv, N)


def _beta_tilde(beta_tilde, beta):
    if beta_tilde is None:
        return ()
    if tuple(beta_tilde.shape) != tuple(beta.shape):
        raise CombaError("comba: beta_tilde must have the shape of beta [B,T,H]")
    return (("beta_tilde", beta_tilde),)


def _fwd(save, q, k, v, g, beta, d, h0, cu_seqlens, output_final_state, workspace, stream,
         beta_tilde, cu_seqlens_host=None):
    import torch

    lib = load_library()
    shp, (B, T, H, dk, dv, N) = _prepare(q, k, v, g, beta, d, h0, cu_seqlens,
                                         extra=_beta_tilde(beta_tilde, beta),
                                         cu_seqlens_host=cu_seqlens_host)
    o = torch.empty((B, T, H, dv), dtype=torch.float32, device=q.device)
    ht = torch.empty((N, H, dk, dv), dtype=torch.float32, device=q.device) \
        if output_final_state else None
    size_fn = lib.comba_bwd_workspace_bytes if save else lib.comba_fwd_workspace_bytes
    nbytes = size_fn(ctypes.byref(shp))
    if nbytes == 0:
        _check(2)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    st = torch.cuda.current_stream(q.device).cuda_stream if stream is None else stream
    fn = lib.comba_chunk_fwd_save if save else lib.comba_chunk_fwd
    _check(fn(ctypes.byref(shp), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
              _ptr(beta_tilde), _ptr(d), _ptr(h0), _ptr(o), _ptr(ht), _ptr(workspace),
              ctypes.c_size_t(workspace.numel()), ctypes.c_void_p(st)))
    return o, ht, workspace


def comba_chunk_fwd(q, k, v, g, beta, d, h0=None, *, beta_tilde=None, cu_seqlens=None,
                    cu_seqlens_host=None, output_final_state=True, workspace=None, stream=None):
    """Chunk-wise forward.  Returns (o [B,T,H,dv] fp32, ht [N,H,dk,dv] fp32 or None).

    ``cu_seqlens_host`` (optional, every entry point): a host copy of the
    offsets (numpy array or CPU tensor); the library then rejects a malformed
    table with a shape error before any launch."""
    o, ht, _ = _fwd(False, q, k, v, g, beta, d, h0, cu_seqlens, output_final_state, workspace,
                    stream, beta_tilde, cu_seqlens_host)
    return o, ht


def comba_chunk_fwd_save(q, k, v, g, beta, d, h0=None, *, beta_tilde=None, cu_seqlens=None,
                         cu_seqlens_host=None, output_final_state=True, workspace=None,
                         stream=None):
    """Forward that also keeps the backward's state in a backward-sized workspace.

    Returns (o, ht, workspace); pass the same inputs and `workspace` to
    comba_chunk_bwd_saved."""
    return _fwd(True, q, k, v, g, beta, d, h0, cu_seqlens, output_final_state, workspace,
                stream, beta_tilde, cu_seqlens_host)


def noalloc_scratch_bytes() -> int:
    """Size of the static device scratch behind comba_chunk_fwd_noalloc."""
    return int(load_library().comba_noalloc_scratch_bytes())


def comba_chunk_fwd_noalloc(q, k, v, g, beta, d, h0=None, *, beta_tilde=None, cu_seqlens=None,
                            cu_seqlens_host=None, o=None, ht=None, output_final_state=True,
                            stream=None):
    """Chunk-wise forward whose library call allocates nothing (its workspace is
    the library's static device scratch).  ``o`` [B,T,H,dv] and ``ht``
    [N,H,dk,dv] (float32, contiguous) may be passed in so that the call
    allocates nothing on the Python side either.  Returns (o, ht)."""
    import torch

    lib = load_library()
    shp, (B, T, H, dk, dv, N) = _prepare(q, k, v, g, beta, d, h0, cu_seqlens,
                                         extra=_beta_tilde(beta_tilde, beta),
                                         cu_seqlens_host=cu_seqlens_host)
    for name, t, shape in (("o", o, (B, T, H, dv)), ("ht", ht, (N, H, dk, dv))):
        if t is not None and (t.dtype != torch.float32 or tuple(t.shape) != shape
                              or not t.is_contiguous() or t.device != q.device):
            raise CombaError("comba: %s must be contiguous float32 %s on the device"
                             % (name, list(shape)))
    if o is None:
        o = torch.empty((B, T, H, dv), dtype=torch.float32, device=q.device)
    if ht is None and output_final_state:
        ht = torch.empty((N, H, dk, dv), dtype=torch.float32, device=q.device)
    st = torch.cuda.current_stream(q.device).cuda_stream if stream is None else stream
    _check(lib.comba_chunk_fwd_noalloc(ctypes.byref(shp), _ptr(q), _ptr(k), _ptr(v), _ptr(g),
                                       _ptr(beta), _ptr(beta_tilde), _ptr(d), _ptr(h0), _ptr(o),
                                       _ptr(ht), ctypes.c_void_p(st)))
    return o, ht


def comba_recurrent_fwd(q, k, v, g, beta, d, h0=None, *, beta_tilde=None, cu_seqlens=None,
                        cu_seqlens_host=None, output_final_state=True, ht=None, stream=None):
    """Token-by-token recurrence (decoding; short segments).  Returns (o, ht).

    Same tensors as comba_chunk_fwd (fp32 inputs also allow d = 128) and no
    workspace.  ``ht`` may be passed as the output state buffer; passing the
    ``h0`` tensor itself updates the states in place."""
    import torch

    lib = load_library()
    shp, (B, T, H, dk, dv, N) = _prepare(q, k, v, g, beta, d, h0, cu_seqlens,
                                         extra=_beta_tilde(beta_tilde, beta),
                                         cu_seqlens_host=cu_seqlens_host)
    o = torch.empty((B, T, H, dv), dtype=torch.float32, device=q.device)
    if ht is not None:
        if ht.dtype != torch.float32 or tuple(ht.shape) != (N, H, dk, dv) \
                or not ht.is_contiguous() or ht.device != q.device:
            raise CombaError("comba: ht must be contiguous float32 [N,H,dk,dv] on the device")
    elif output_final_state:
        ht = torch.empty((N, H, dk, dv), dtype=torch.float32, device=q.device)
    st = torch.cuda.current_stream(q.device).cuda_stream if stream is None else stream
    _check(lib.comba_recurrent_fwd(ctypes.byref(shp), _ptr(q), _ptr(k), _ptr(v), _ptr(g),
                                   _ptr(beta), _ptr(beta_tilde), _ptr(d), _ptr(h0), _ptr(o),
                                   _ptr(ht), ctypes.c_void_p(st)))
    return o, ht


def _prologue_shape(xq, xk, xv, wq, wk, wv, cu_seqlens, extra=(), cu_seqlens_host=None):
    import torch

    if not xq.is_cuda:
        raise CombaError("comba: tensors must be on a GPU device")
    if xq.dtype not in (torch.bfloat16, torch.float32) or xk.dtype != xq.dtype \
            or xv.dtype != xq.dtype:
        raise CombaError("comba: xq, xk, xv must share one dtype (bfloat16 or float32)")
    B, T, H, dk = xq.shape
    dv = xv.shape[-1]
    if xk.shape != xq.shape or tuple(xv.shape[:3]) != (B, T, H) or \
            tuple(wq.shape) != (H, dk, 4) or tuple(wk.shape) != (H, dk, 4) or \
            tuple(wv.shape) != (H, dv, 4):
        raise CombaError("comba: inconsistent prologue shapes")
    for t in (xq, xk, xv, wq, wk, wv) + tuple(extra):
        if not t.is_contiguous() or t.device != xq.device:
            raise CombaError("comba: all tensors must be contiguous and on one device")
    for t in (wq, wk, wv) + tuple(extra):
        if t.dtype != torch.float32:
            raise CombaError("comba: taps and gradients must be float32")
    if cu_seqlens is not None:
        if cu_seqlens.dtype != torch.int32 or B != 1:
            raise CombaError("comba: cu_seqlens must be int32 on the device, B == 1")
        N = cu_seqlens.numel() - 1
    else:
        if cu_seqlens_host is not None:
            raise CombaError("comba: cu_seqlens_host needs cu_seqlens")
        N = B
    code = COMBA_BF16 if xq.dtype == torch.bfloat16 else COMBA_F32
    return _make_shape(B, T, H, dk, dv, N, _ptr(cu_seqlens), code,
                       cu_host=_host_offsets(cu_seqlens_host, N + 1))


def comba_prologue_fwd(xq, xk, xv, wq, wk, wv, *, cu_seqlens=None, cu_seqlens_host=None,
                       stream=None):
    """Layer input prologue: causal short conv (4 taps), SiLU, L2 norm of q and k.
    Returns (q, k, v) in the dtype of x."""
    import torch

    lib = load_library()
    shp = _prologue_shape(xq, xk, xv, wq, wk, wv, cu_seqlens, cu_seqlens_host=cu_seqlens_host)
    q, k, v = torch.empty_like(xq), torch.empty_like(xk), torch.empty_like(xv)
    st = torch.cuda.current_stream(xq.device).cuda_stream if stream is None else stream
    _check(lib.comba_prologue_fwd(ctypes.byref(shp), _ptr(xq), _ptr(xk), _ptr(xv), _ptr(wq),
                                  _ptr(wk), _ptr(wv), _ptr(q), _ptr(k), _ptr(v),
                                  ctypes.c_void_p(st)))
    return q, k, v


def comba_prologue_bwd(xq, xk, xv, wq, wk, wv, gq, gk, gv, *, cu_seqlens=None,
                       cu_seqlens_host=None, workspace=None, stream=None):
    """Backward of the prologue from the fp32 gradients of q, k, v.  Returns dict
    dxq, dxk, dxv, dwq, dwk, dwv (fp32)."""
    import torch

    lib = load_library()
    shp = _prologue_shape(xq, xk, xv, wq, wk, wv, cu_seqlens, extra=(gq, gk, gv),
                          cu_seqlens_host=cu_seqlens_host)
    if gq.shape != xq.shape or gk.shape != xk.shape or gv.shape != xv.shape:
        raise CombaError("comba: gradients must have the shapes of q, k, v")
    f32 = torch.float32
    out = {"dxq": torch.empty(xq.shape, dtype=f32, device=xq.device),
           "dxk": torch.empty(xk.shape, dtype=f32, device=xq.device),
           "dxv": torch.empty(xv.shape, dtype=f32, device=xq.device),
           "dwq": torch.empty_like(wq), "dwk": torch.empty_like(wk), "dwv": torch.empty_like(wv)}
    nbytes = lib.comba_prologue_workspace_bytes(ctypes.byref(shp))
    if nbytes == 0:
        _check(2)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=xq.device)
    st = torch.cuda.current_stream(xq.device).cuda_stream if stream is None else stream
    _check(lib.comba_prologue_bwd(ctypes.byref(shp), _ptr(xq), _ptr(xk), _ptr(xv), _ptr(wq),
                                  _ptr(wk), _ptr(wv), _ptr(gq), _ptr(gk), _ptr(gv),
                                  _ptr(out["dxq"]), _ptr(out["dxk"]), _ptr(out["dxv"]),
                                  _ptr(out["dwq"]), _ptr(out["dwk"]), _ptr(out["dwv"]),
                                  _ptr(workspace), ctypes.c_size_t(workspace.numel()),
                                  ctypes.c_void_p(st)))
    return out


def _gate_shape(o, z):
    import torch

    if not o.is_cuda or o.dtype != torch.float32 or z.shape != o.shape or not o.is_contiguous() \
            or not z.is_contiguous() or z.device != o.device or \
            z.dtype not in (torch.bfloat16, torch.float32):
        raise CombaError("comba: gate takes o (float32) and z (bfloat16 or float32) of one shape")
    B, T, H, dv = o.shape
    code = COMBA_BF16 if z.dtype == torch.bfloat16 else COMBA_F32
    return _make_shape(B, T, H, 64 if dv == 64 else 128, dv, B, None, code)


def comba_gate_fwd(o, z, *, stream=None):
    """Output gate y = o * sigmoid(z); y in the dtype of z."""
    import torch

    shp = _gate_shape(o, z)
    y = torch.empty_like(z)
    st = torch.cuda.current_stream(o.device).cuda_stream if stream is None else stream
    _check(load_library().comba_gate_fwd(ctypes.byref(shp), _ptr(o), _ptr(z), _ptr(y),
                                         ctypes.c_void_p(st)))
    return y


def comba_gate_bwd(o, z, dy, *, stream=None):
    """Backward of the output gate from dy (float32).  Returns (do, dz), float32."""
    import torch

    shp = _gate_shape(o, z)
    if dy.shape != o.shape or dy.dtype != torch.float32 or not dy.is_contiguous():
        raise CombaError("comba: dy must be contiguous float32 of the shape of o")
    do, dz = torch.empty_like(o), torch.empty(o.shape, dtype=torch.float32, device=o.device)
    st = torch.cuda.current_stream(o.device).cuda_stream if stream is None else stream
    _check(load_library().comba_gate_bwd(ctypes.byref(shp), _ptr(o), _ptr(z), _ptr(dy), _ptr(do),
                                         _ptr(dz), ctypes.c_void_p(st)))
    return do, dz


def _bwd(saved, q, k, v, g, beta, d, h0, dO, dht, cu_seqlens, need_dh0, workspace, stream,
         beta_tilde, cu_seqlens_host=None):
    import torch

    lib = load_library()
    shp, (B, T, H, dk, dv, N) = _prepare(q, k, v, g, beta, d, h0, cu_seqlens,
                                         extra=(("dO", dO),) + _beta_tilde(beta_tilde, beta),
                                         cu_seqlens_host=cu_seqlens_host)
    if dht is not None and (dht.dtype != torch.float32 or tuple(dht.shape) != (N, H, dk, dv)
                            or not dht.is_contiguous()):
        raise CombaError("comba: dht must be contiguous float32 [N,H,dk,dv]")
    if tuple(dO.shape) != (B, T, H, dv):
        raise CombaError("comba: dO must be [B,T,H,dv]")
    dev = q.device
    f32 = torch.float32
    out = {
        "dq": torch.empty((B, T, H, dk), dtype=f32, device=dev),
        "dk": torch.empty((B, T, H, dk), dtype=f32, device=dev),
        "dv": torch.empty((B, T, H, dv), dtype=f32, device=dev),
        "dg": torch.empty((B, T, H), dtype=f32, device=dev),
        "dbeta": torch.empty((B, T, H), dtype=f32, device=dev),
        "dbeta_tilde": None if beta_tilde is None else torch.empty((B, T, H), dtype=f32,
                                                                   device=dev),
        "dd": torch.empty((H,), dtype=f32, device=dev),
        "dh0": torch.empty((N, H, dk, dv), dtype=f32, device=dev) if need_dh0 else None,
    }
    nbytes = lib.comba_bwd_workspace_bytes(ctypes.byref(shp))
    if nbytes == 0:
        _check(2)
    if workspace is None or workspace.numel() < nbytes:
        if saved:
            raise CombaError("comba: comba_chunk_bwd_saved needs the workspace filled by "
                             "comba_chunk_fwd_save")
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    st = torch.cuda.current_stream(dev).cuda_stream if stream is None else stream
    fn = lib.comba_chunk_bwd_saved if saved else lib.comba_chunk_bwd
    _check(fn(ctypes.byref(shp), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
              _ptr(beta_tilde), _ptr(d), _ptr(h0), _ptr(dO), _ptr(dht), _ptr(out["dq"]),
              _ptr(out["dk"]), _ptr(out["dv"]), _ptr(out["dg"]), _ptr(out["dbeta"]),
              _ptr(out["dbeta_tilde"]), _ptr(out["dd"]), _ptr(out["dh0"]), _ptr(workspace),
              ctypes.c_size_t(workspace.numel()), ctypes.c_void_p(st)))
    if beta_tilde is None:
        del out["dbeta_tilde"]
    return out


def comba_chunk_bwd(q, k, v, g, beta, d, h0, dO, dht=None, *, beta_tilde=None, cu_seqlens=None,
                    cu_seqlens_host=None, need_dh0=True, workspace=None, stream=None):
    """Chunk-wise backward (recomputes the forward).  Returns dict dq, dk, dv, dg, dbeta, dd,
    dh0 (fp32), and dbeta_tilde when beta_tilde is given (dbeta is then the derivative
    through the write strength only; otherwise it is the total derivative)."""
    return _bwd(False, q, k, v, g, beta, d, h0, dO, dht, cu_seqlens, need_dh0, workspace, stream,
                beta_tilde, cu_seqlens_host)


def comba_chunk_bwd_saved(q, k, v, g, beta, d, h0, dO, dht=None, *, workspace, beta_tilde=None,
                          cu_seqlens=None, cu_seqlens_host=None, need_dh0=True, stream=None):
    """Backward reusing the state left by comba_chunk_fwd_save in `workspace`."""
    return _bwd(True, q, k, v, g, beta, d, h0, dO, dht, cu_seqlens, need_dh0, workspace, stream,
                beta_tilde, cu_seqlens_host)


def _autograd_function():
    import torch

    class _ChunkComba(torch.autograd.Function):
        """The training pair as one differentiable op: comba_chunk_fwd_save in
        the forward (its workspace kept for the backward), comba_chunk_bwd_saved
        in the backward.  Gradients come back in the inputs' dtypes; the
        upstream gradient of o is rounded to the inputs' dtype (the kernels
        take dO in in_dtype)."""

        @staticmethod
        def forward(ctx, q, k, v, g, beta, d, h0, beta_tilde, cu_seqlens, cu_seqlens_host):
            ctx.set_materialize_grads(False)  # an unused output's gradient arrives as None
            o, ht, ws = comba_chunk_fwd_save(q, k, v, g, beta, d, h0, beta_tilde=beta_tilde,
                                             cu_seqlens=cu_seqlens,
                                             cu_seqlens_host=cu_seqlens_host)
            ctx.save_for_backward(q, k, v, g, beta, d, h0, beta_tilde, cu_seqlens, ws)
            ctx.cu_seqlens_host = cu_seqlens_host
            return o, ht

        @staticmethod
        def backward(ctx, do, dht):
            q, k, v, g, beta, d, h0, beta_tilde, cu_seqlens, ws = ctx.saved_tensors
            if do is None:
                do = torch.zeros(q.shape[:3] + (v.shape[-1],), dtype=torch.float32,
                                 device=q.device)
            need = ctx.needs_input_grad
            gr = comba_chunk_bwd_saved(q, k, v, g, beta, d, h0,
                                       do.to(q.dtype).contiguous(),
                                       None if dht is None else dht.float().contiguous(),
                                       workspace=ws, beta_tilde=beta_tilde,
                                       cu_seqlens=cu_seqlens,
                                       cu_seqlens_host=ctx.cu_seqlens_host,
                                       need_dh0=h0 is not None and need[6])

            def cast(x, like, i):
                return None if (x is None or not need[i]) else x.to(like.dtype)

            return (cast(gr["dq"], q, 0), cast(gr["dk"], k, 1), cast(gr["dv"], v, 2),
                    cast(gr["dg"], g, 3), cast(gr["dbeta"], beta, 4), cast(gr["dd"], d, 5),
                    None if h0 is None else cast(gr["dh0"], h0, 6),
                    None if beta_tilde is None else cast(gr["dbeta_tilde"], beta_tilde, 7),
                    None, None)

    return _ChunkComba


_CHUNK_FN = None


def comba_chunk(q, k, v, g, beta, d, h0=None, *, beta_tilde=None, cu_seqlens=None,
                cu_seqlens_host=None):
    """Differentiable chunk-wise Comba (torch.autograd): returns (o [B,T,H,dv]
    fp32, ht [N,H,dk,dv] fp32); gradients flow to q, k, v, g, beta, d, h0 and
    beta~ through the library's training pair.  Each call keeps its
    backward-sized workspace until the backward has run."""
    global _CHUNK_FN
    if _CHUNK_FN is None:
        _CHUNK_FN = _autograd_function()
    return _CHUNK_FN.apply(q, k, v, g, beta, d, h0, beta_tilde, cu_seqlens, cu_seqlens_host)
