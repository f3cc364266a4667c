"""comba_chunk_fwd_noalloc (workspace in the library's static device scratch)
against comba_chunk_fwd (caller workspace), through the C ABI.

Both run the same kernels, so their outputs must be bitwise equal; the small
case is also held to the oracle at the bf16 bar (2e-3).  Two calls in a row,
the second smaller than the first, show that what the first call leaves in the
shared scratch does not leak into the second.  A shape beyond the scratch is
rejected before any launch (its output buffer stays untouched)."""
import ctypes

import numpy as np
import pytest

from comba_inputs import random_case
from gpu_helpers import maxrel, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _call_noalloc(w, a):
    """comba_chunk_fwd_noalloc through ctypes with caller-made outputs."""
    import torch
    import paper_2506_02475_amd as comba

    lib = comba.load_library()
    N = w.nseq
    shp = comba._make_shape(w.B, w.T, w.H, w.dk, w.dv, N,
                            None if a["cu_seqlens"] is None
                            else ctypes.c_void_p(a["cu_seqlens"].data_ptr()),
                            comba.COMBA_BF16, cu_host=w.cu_seqlens)
    o = torch.full((w.B, w.T, w.H, w.dv), 7.0, dtype=torch.float32, device="cuda")
    ht = torch.full((N, w.H, w.dk, w.dv), 7.0, dtype=torch.float32, device="cuda")
    P = ctypes.c_void_p
    st = torch.cuda.current_stream().cuda_stream
    args = [a[n] for n in ("q", "k", "v", "g", "beta", "beta_tilde", "d", "h0")]
    rc = lib.comba_chunk_fwd_noalloc(ctypes.byref(shp),
                                     *[None if t is None else P(t.data_ptr()) for t in args],
                                     P(o.data_ptr()), P(ht.data_ptr()), P(st))
    torch.cuda.synchronize()
    return rc, o, ht


def _reference(w, a):
    import torch
    import paper_2506_02475_amd as comba

    o, ht = comba.comba_chunk_fwd(a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"], a["h0"],
                                  beta_tilde=a["beta_tilde"], cu_seqlens=a["cu_seqlens"])
    torch.cuda.synchronize()
    return o, ht


CASES = [
    # (first call, second smaller call)
    (dict(B=2, T=700, H=4, dk=128, dv=128, seed=61),
     dict(B=1, T=130, H=2, dk=128, dv=128, seed=62)),
    (dict(T=0, H=3, dk=128, dv=128, seed=63, seqlens=[300, 0, 65, 640]),
     dict(T=0, H=2, dk=128, dv=128, seed=64, seqlens=[1, 70])),
    (dict(B=1, T=520, H=2, dk=256, dv=256, seed=65),
     dict(B=1, T=64, H=1, dk=256, dv=256, seed=66)),
]


@pytest.mark.parametrize("first,second", CASES, ids=["fixed", "varlen", "d256"])
def test_noalloc_matches_workspace_forward(first, second):
    import oracle
    import paper_2506_02475_amd as comba

    for kw in (first, second):
        w = random_case(in_dtype="bf16", grad=False, **kw)
        need = comba.fwd_workspace_bytes(w.B, w.T, w.H, w.dk, w.dv, num_seqs=w.nseq,
                                         varlen=w.cu_seqlens is not None)
        assert 0 < need <= comba.noalloc_scratch_bytes()
        a = to_device(w)
        rc, o, ht = _call_noalloc(w, a)
        assert rc == 0, comba.load_library().comba_status_string(rc)
        ro, rht = _reference(w, a)
        assert np.array_equal(o.cpu().numpy(), ro.cpu().numpy())
        assert np.array_equal(ht.cpu().numpy(), rht.cpu().numpy())
        if kw is second:
            so, sht = oracle.workload_fwd(w)
            assert maxrel(o.cpu().numpy(), so) <= 2e-3
            assert maxrel(ht.cpu().numpy(), sht) <= 2e-3


def test_noalloc_binding_and_the_headline_shape_fits():
    import paper_2506_02475_amd as comba

    # the 1.3B layer's forward (B4 T4096 H16 d128) fits the scratch
    assert comba.fwd_workspace_bytes(4, 4096, 16, 128, 128) <= comba.noalloc_scratch_bytes()
    w = random_case(B=1, T=200, H=2, dk=128, dv=128, in_dtype="bf16", grad=False, seed=67)
    a = to_device(w)
    o, ht = comba.comba_chunk_fwd_noalloc(a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"],
                                          a["h0"])
    ro, rht = _reference(w, a)
    assert np.array_equal(o.cpu().numpy(), ro.cpu().numpy())
    assert np.array_equal(ht.cpu().numpy(), rht.cpu().numpy())


def test_noalloc_rejects_shapes_beyond_the_scratch():
    import torch
    import paper_2506_02475_amd as comba

    lib = comba.load_library()
    # B4 T8192 H16 d128 needs about twice the scratch: rejected before any
    # launch (the pointers are never dereferenced; the output keeps its fill)
    shp = comba._make_shape(4, 8192, 16, 128, 128, 4, None, comba.COMBA_BF16)
    assert lib.comba_fwd_workspace_bytes(ctypes.byref(shp)) > comba.noalloc_scratch_bytes()
    o = torch.full((16,), 3.0, device="cuda")
    P = ctypes.c_void_p
    fake = P(o.data_ptr())
    rc = lib.comba_chunk_fwd_noalloc(ctypes.byref(shp), *([fake] * 10), None)
    torch.cuda.synchronize()
    assert rc == 7 and b"scratch" in lib.comba_status_string(rc)
    assert torch.all(o == 3.0)
    # an invalid shape is a shape error, not a scratch error
    bad = comba._make_shape(1, 64, 1, 96, 128, 1, None, comba.COMBA_BF16)
    assert lib.comba_chunk_fwd_noalloc(ctypes.byref(bad), *([fake] * 10), None) == 2
