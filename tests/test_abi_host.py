"""Host-side checks of the C ABI: the library loads, exports every symbol that
include/comba.h declares, sizes workspaces, and rejects bad arguments before
any kernel launch (these calls never reach the GPU, so they run without one)."""
import ctypes
import os
import subprocess

import pytest

import paper_2506_02475_amd as comba

pytestmark = pytest.mark.skipif(not os.path.exists(comba.library_path()),
                                reason="libcomba.so not built")

OK, ENULL, ESHAPE, EDTYPE, EALIGN, EWS = 0, 1, 2, 3, 4, 5
FAKE = 0x100000  # aligned, never dereferenced: validation fails before any launch


def shape(B=1, T=128, H=2, dk=128, dv=128, chunk=64, N=None, cu=None, dtype=comba.COMBA_BF16,
          cu_host=None):
    """The C shape struct; ``cu_host`` is a list of host offsets (kept alive on it)."""
    hp = None
    if cu_host is not None:
        cu_host = (ctypes.c_int32 * len(cu_host))(*cu_host)
        hp = ctypes.cast(cu_host, ctypes.c_void_p)
    s = comba.CombaShape(B, T, H, dk, dv, chunk, B if N is None else N,
                         None if cu is None else ctypes.c_void_p(cu), hp, dtype)
    s._keep = cu_host
    return s


def fwd(shp, ptrs=None, ws_bytes=1 << 40, **over):
    lib = comba.load_library()
    p = dict(q=FAKE, k=FAKE, v=FAKE, g=FAKE, beta=FAKE, beta_tilde=None, d=FAKE, h0=None, o=FAKE,
             ht=None, ws=FAKE)
    p.update(over)
    P = ctypes.c_void_p
    return lib.comba_chunk_fwd(ctypes.byref(shp), P(p["q"]), P(p["k"]), P(p["v"]), P(p["g"]),
                               P(p["beta"]), P(p["beta_tilde"]), P(p["d"]), P(p["h0"]),
                               P(p["o"]), P(p["ht"]), P(p["ws"]), ctypes.c_size_t(ws_bytes), None)


def bwd(shp, ws_bytes=1 << 40, **over):
    lib = comba.load_library()
    names = ["q", "k", "v", "g", "beta", "beta_tilde", "d", "h0", "dO", "dht", "dq", "dk", "dv",
             "dg", "dbeta", "dbeta_tilde", "dd", "dh0", "ws"]
    p = {n: FAKE for n in names}
    p.update(beta_tilde=None, dbeta_tilde=None, h0=None, dht=None, dh0=None)
    p.update(over)
    P = ctypes.c_void_p
    args = [P(p[n]) for n in names]
    return lib.comba_chunk_bwd(ctypes.byref(shp), *args[:-1], args[-1],
                               ctypes.c_size_t(ws_bytes), None)


def test_library_exports_every_declared_symbol():
    declared = comba.exported_symbols()
    assert set(declared) == {"comba_fwd_workspace_bytes", "comba_bwd_workspace_bytes",
                             "comba_chunk_fwd", "comba_chunk_bwd", "comba_status_string",
                             "comba_profile_enable", "comba_profile_read",
                             "comba_profile_select",
                             "comba_chunk_fwd_save", "comba_chunk_bwd_saved",
                             "comba_recurrent_fwd", "comba_prologue_fwd", "comba_prologue_bwd",
                             "comba_prologue_workspace_bytes", "comba_gate_fwd", "comba_gate_bwd",
                             "comba_chunk_fwd_noalloc", "comba_noalloc_scratch_bytes"}
    out = subprocess.run(["nm", "-D", "--defined-only", comba.library_path()],
                         capture_output=True, text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for name in declared:
        assert name in exported, name
        assert hasattr(comba.load_library(), name)


def test_profile_read_without_calls_is_empty():
    comba.profile_enable(True)
    assert comba.profile_read() == []


def test_profile_select_sets_and_clears_without_a_device():
    # selecting a stage touches no device; a session with a selection and no
    # calls records nothing
    comba.profile_select("intra_bwd")
    comba.profile_enable(True)
    assert comba.profile_read() == []
    comba.profile_enable(False)
    comba.profile_select(None)
    comba.profile_enable(False)


def test_status_strings():
    lib = comba.load_library()
    for code in range(8):
        assert lib.comba_status_string(code)
    assert lib.comba_status_string(99) == b"unknown status"


def test_workspace_sizes_grow_with_problem():
    small = comba.fwd_workspace_bytes(1, 64, 1, 64, 64)
    big = comba.fwd_workspace_bytes(4, 4096, 16, 128, 128)
    assert 0 < small < big
    assert comba.bwd_workspace_bytes(4, 4096, 16, 128, 128) > big
    # variable-length: each sequence may add one partial chunk
    assert comba.fwd_workspace_bytes(1, 1000, 2, 128, 128, num_seqs=16, varlen=True) > \
        comba.fwd_workspace_bytes(1, 1000, 2, 128, 128)
    # fixed-length rows with a ragged tail each hold their own partial chunk
    assert comba.fwd_workspace_bytes(3, 1, 2, 64, 64) > comba.fwd_workspace_bytes(1, 3, 2, 64, 64)
    lib = comba.load_library()
    assert lib.comba_fwd_workspace_bytes(ctypes.byref(shape(chunk=32))) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(chunk=32), ESHAPE),
    (dict(dk=96), ESHAPE),
    (dict(dv=512), ESHAPE),
    (dict(dk=64, dv=256), ESHAPE),
    (dict(dk=128, dtype=comba.COMBA_F32), ESHAPE),   # fp32 path supports d = 64 only
    (dict(H=0), ESHAPE),
    (dict(T=-1), ESHAPE),
    (dict(B=2, N=3), ESHAPE),                         # fixed-length: N must equal B
    (dict(B=2, cu=FAKE, N=2), ESHAPE),                # varlen needs B == 1
    (dict(dtype=7), EDTYPE),
])
def test_rejects_bad_shapes(kw, code):
    assert fwd(shape(**kw)) == code
    assert bwd(shape(**kw)) == code


def test_rejects_null_and_misaligned_pointers():
    s = shape()
    for name in ("q", "k", "v", "g", "beta", "d", "o", "ws"):
        assert fwd(s, **{name: None}) == ENULL, name
    for name in ("q", "dO", "dq", "dk", "dv", "dg", "dbeta", "dd", "ws"):
        assert bwd(s, **{name: None}) == ENULL, name
    assert fwd(s, q=FAKE + 8) == EALIGN
    assert fwd(s, ws=FAKE + 16) == EALIGN
    assert fwd(s, o=FAKE + 2) == EALIGN
    assert bwd(s, dO=FAKE + 4) == EALIGN
    # fp32 tensors with a dk / dv last dimension are written 16 bytes at a time
    for name in ("o", "h0", "ht"):
        assert fwd(s, **{name: FAKE + 4}) == EALIGN, name
    for name in ("dq", "dk", "dv", "h0", "dht", "dh0"):
        assert bwd(s, **{name: FAKE + 8}) == EALIGN, name
    # per-token / per-head fp32 tensors need only 4 bytes: with a too-small
    # workspace the next check fails instead (and nothing is launched)
    for name in ("g", "d"):
        assert fwd(s, ws_bytes=1, **{name: FAKE + 4}) == EWS, name
    for name in ("dg", "dbeta", "dd"):
        assert bwd(s, ws_bytes=1, **{name: FAKE + 4}) == EWS, name
    lib = comba.load_library()
    assert lib.comba_chunk_fwd(None, *[ctypes.c_void_p(FAKE)] * 10, ctypes.c_void_p(FAKE),
                               ctypes.c_size_t(1 << 40), None) == ENULL


def test_beta_tilde_arguments():
    # beta_tilde is optional (NULL: tied to beta); when it is given, its
    # gradient dbeta_tilde is required.  dbeta_tilde alone is allowed (the
    # derivative split by role).  A one-byte workspace stops every call that
    # passes validation before any launch.
    s = shape()
    assert fwd(s, ws_bytes=1, beta_tilde=FAKE) == EWS
    assert bwd(s, ws_bytes=1, beta_tilde=FAKE, dbeta_tilde=FAKE) == EWS
    assert bwd(s, ws_bytes=1, dbeta_tilde=FAKE) == EWS
    assert bwd(s, ws_bytes=1, beta_tilde=FAKE) == ENULL
    # element alignment: bf16 beta_tilde 2 bytes, fp32 dbeta_tilde 4 bytes
    assert fwd(s, ws_bytes=1, beta_tilde=FAKE + 1) == EALIGN
    assert fwd(s, ws_bytes=1, beta_tilde=FAKE + 2) == EWS
    assert fwd(shape(dk=64, dv=64, dtype=comba.COMBA_F32), ws_bytes=1,
               beta_tilde=FAKE + 2) == EALIGN
    assert bwd(s, ws_bytes=1, beta_tilde=FAKE, dbeta_tilde=FAKE + 2) == EALIGN
    assert bwd(s, ws_bytes=1, beta_tilde=FAKE, dbeta_tilde=FAKE + 4) == EWS
    # without tokens both may be NULL
    assert bwd(shape(T=0), ws_bytes=1, beta_tilde=FAKE) == EWS


def test_token_free_calls_accept_null_token_tensors():
    # no tokens (T == 0 or B == 0): the per-token tensors may be NULL and the
    # states pass through; d, dd and the workspace stay required.  A one-byte
    # workspace makes the next check fail, so nothing is launched.
    token_fwd = ("q", "k", "v", "g", "beta", "o")
    token_bwd = ("q", "k", "v", "g", "beta", "dO", "dq", "dk", "dv", "dg", "dbeta")
    for s in (shape(T=0), shape(B=0), shape(T=0, cu=FAKE, N=3)):
        assert fwd(s, ws_bytes=1, **{n: None for n in token_fwd}) == EWS
        assert bwd(s, ws_bytes=1, **{n: None for n in token_bwd}) == EWS
        assert fwd(s, ws_bytes=1, d=None) == ENULL
        assert fwd(s, ws_bytes=1, ws=None) == ENULL
        assert bwd(s, ws_bytes=1, dd=None) == ENULL
    # with tokens they are required as before
    assert fwd(shape(T=1), ws_bytes=1, q=None) == ENULL
    assert bwd(shape(T=1), ws_bytes=1, dbeta=None) == ENULL


def rec(shp, **over):
    lib = comba.load_library()
    p = dict(q=FAKE, k=FAKE, v=FAKE, g=FAKE, beta=FAKE, beta_tilde=None, d=FAKE, h0=None, o=FAKE,
             ht=None)
    p.update(over)
    P = ctypes.c_void_p
    names = ("q", "k", "v", "g", "beta", "beta_tilde", "d", "h0", "o", "ht")
    return lib.comba_recurrent_fwd(ctypes.byref(shp), *[P(p[n]) for n in names], None)


def test_recurrent_validates_before_launch():
    # every call below stops at a check (a misaligned o or ht marks the ones
    # whose shape passed), so nothing is launched
    assert rec(shape(dk=96)) == ESHAPE
    assert rec(shape(dv=512)) == ESHAPE
    assert rec(shape(B=2, N=3)) == ESHAPE
    assert rec(shape(dtype=7)) == EDTYPE
    # the chunk length is not used; fp32 inputs allow d = 128 here
    assert rec(shape(chunk=32), o=FAKE + 4) == EALIGN
    assert rec(shape(dk=128, dv=128, dtype=comba.COMBA_F32), o=FAKE + 4) == EALIGN
    # head dim 256 (the paper's models): with 128 or 256 on the other side
    for dk, dv in ((256, 256), (128, 256), (256, 128)):
        assert rec(shape(dk=dk, dv=dv), o=FAKE + 4) == EALIGN, (dk, dv)
    assert rec(shape(dk=64, dv=256)) == ESHAPE
    assert rec(shape(dk=256, dv=64)) == ESHAPE
    for name in ("q", "k", "v", "g", "beta", "d", "o"):
        assert rec(shape(), **{name: None}) == ENULL, name
    assert rec(shape(), beta_tilde=FAKE + 1) == EALIGN
    assert rec(shape(), h0=FAKE + 8) == EALIGN
    assert rec(shape(), ht=FAKE + 8) == EALIGN
    # without tokens the token tensors may be NULL (d stays required)
    none = {n: None for n in ("q", "k", "v", "g", "beta", "o")}
    assert rec(shape(T=0), ht=FAKE + 8, **none) == EALIGN
    assert rec(shape(T=0), d=None, **none) == ENULL


def test_head256_accepted_by_every_chunk_call():
    # head dim 256 (bf16): every chunk entry point accepts it (a misaligned
    # output shows the shape passed; nothing is launched)
    for dk, dv in ((256, 256), (128, 256), (256, 128)):
        s = shape(dk=dk, dv=dv)
        assert comba.fwd_workspace_bytes(1, 128, 2, dk, dv) > 0
        assert comba.bwd_workspace_bytes(1, 128, 2, dk, dv) > 0
        assert fwd(s, o=FAKE + 4) == EALIGN
        assert bwd(s, dq=FAKE + 4) == EALIGN
        lib = comba.load_library()
        P = ctypes.c_void_p
        args = [P(FAKE)] * 10
        args[8] = P(FAKE + 4)  # o
        assert lib.comba_chunk_fwd_save(ctypes.byref(s), *args, P(FAKE),
                                        ctypes.c_size_t(1 << 40), None) == EALIGN
    assert fwd(shape(dk=64, dv=256)) == ESHAPE
    assert fwd(shape(dk=256, dv=256, dtype=comba.COMBA_F32)) == ESHAPE


def pro(shp, bwd=False, ws_bytes=1 << 40, **over):
    lib = comba.load_library()
    P = ctypes.c_void_p
    if not bwd:
        names = ("xq", "xk", "xv", "wq", "wk", "wv", "q", "k", "v")
        p = {n: FAKE for n in names}
        p.update(over)
        return lib.comba_prologue_fwd(ctypes.byref(shp), *[P(p[n]) for n in names], None)
    names = ("xq", "xk", "xv", "wq", "wk", "wv", "gq", "gk", "gv", "dxq", "dxk", "dxv",
             "dwq", "dwk", "dwv", "ws")
    p = {n: FAKE for n in names}
    p.update(over)
    return lib.comba_prologue_bwd(ctypes.byref(shp), *[P(p[n]) for n in names],
                                  ctypes.c_size_t(ws_bytes), None)


def test_prologue_validates_before_launch():
    lib = comba.load_library()
    s = shape(B=2, T=130, H=3, dk=128, dv=64)
    need = lib.comba_prologue_workspace_bytes(ctypes.byref(s))
    # 3 runs x 3 heads x (2 x 128 + 64) channels x 4 taps of fp32 partials
    assert need >= 3 * 3 * 320 * 4 * 4
    assert pro(shape(dk=96)) == ESHAPE and pro(shape(dk=64, dv=256), bwd=True) == ESHAPE
    assert pro(shape(dtype=7)) == EDTYPE
    assert pro(shape(cu=FAKE, N=0)) == ESHAPE  # tokens without sequences
    for name in ("xq", "xk", "xv", "wq", "wk", "wv", "q", "k", "v"):
        assert pro(s, **{name: None}) == ENULL, name
    for name in ("gq", "dxv", "dwk", "ws"):
        assert pro(s, bwd=True, **{name: None}) == ENULL, name
    assert pro(s, xq=FAKE + 8) == EALIGN
    assert pro(s, bwd=True, dwq=FAKE + 2) == EALIGN
    assert pro(s, bwd=True, ws_bytes=need - 1) == EWS
    # the chunk length is not used; head dim 256 is accepted (stopped by the alignment check)
    assert pro(shape(chunk=32, dk=256, dv=256), q=FAKE + 8) == EALIGN


def test_gate_validates_before_launch():
    lib = comba.load_library()
    P = ctypes.c_void_p
    s = shape()
    assert lib.comba_gate_fwd(ctypes.byref(s), P(FAKE), None, P(FAKE), None) == ENULL
    assert lib.comba_gate_fwd(ctypes.byref(s), P(FAKE), P(FAKE), P(FAKE + 4), None) == EALIGN
    assert lib.comba_gate_bwd(ctypes.byref(s), P(FAKE), P(FAKE), None, P(FAKE), P(FAKE),
                              None) == ENULL
    assert lib.comba_gate_bwd(ctypes.byref(s), P(FAKE), P(FAKE), P(FAKE), P(FAKE + 8), P(FAKE),
                              None) == EALIGN
    assert lib.comba_gate_fwd(ctypes.byref(shape(dv=96)), P(FAKE), P(FAKE), P(FAKE), None) == ESHAPE


def test_saved_pair_validates_like_the_plain_calls():
    lib = comba.load_library()
    P = ctypes.c_void_p
    s = shape(chunk=32)
    args = [P(FAKE)] * 10
    assert lib.comba_chunk_fwd_save(ctypes.byref(s), *args, P(FAKE), ctypes.c_size_t(1 << 40),
                                    None) == ESHAPE
    s = shape()
    # the forward-with-save needs the backward-sized workspace
    need_f = lib.comba_fwd_workspace_bytes(ctypes.byref(s))
    need_b = lib.comba_bwd_workspace_bytes(ctypes.byref(s))
    assert need_b > need_f
    assert lib.comba_chunk_fwd_save(ctypes.byref(s), *args, P(FAKE), ctypes.c_size_t(need_f),
                                    None) == EWS
    bargs = [P(FAKE)] * 18
    assert lib.comba_chunk_bwd_saved(ctypes.byref(s), *bargs, P(FAKE),
                                     ctypes.c_size_t(need_b - 1), None) == EWS
    bargs[8] = None  # dO
    assert lib.comba_chunk_bwd_saved(ctypes.byref(s), *bargs, P(FAKE),
                                     ctypes.c_size_t(need_b), None) == ENULL


def test_rejects_small_workspace():
    s = shape(B=2, T=256, H=4)
    need = comba.load_library().comba_fwd_workspace_bytes(ctypes.byref(s))
    assert fwd(s, ws_bytes=need - 1) == EWS
    needb = comba.load_library().comba_bwd_workspace_bytes(ctypes.byref(s))
    assert bwd(s, ws_bytes=needb - 1) == EWS


@pytest.mark.parametrize("cu_host,ok", [
    ([0, 40, 40, 128], True),
    ([0, 128], True),
    ([0, 0, 0, 128], True),
    ([1, 40, 90, 128], False),     # cu[0] != 0
    ([0, 40, 90, 127], False),     # cu[N] != T
    ([0, 90, 40, 128], False),     # not monotone
    ([0, 40, -5, 128], False),
])
def test_host_offsets_are_validated_before_any_launch(cu_host, ok):
    # with a host copy of the offsets every entry point rejects a malformed
    # table with a shape error; a well-formed one passes on to the next check
    # (here the one-byte workspace, resp. a misaligned output), so nothing is
    # launched either way
    n = len(cu_host) - 1
    s = shape(T=128, cu=FAKE, N=n, cu_host=cu_host)
    assert fwd(s, ws_bytes=1) == (EWS if ok else ESHAPE)
    assert bwd(s, ws_bytes=1) == (EWS if ok else ESHAPE)
    assert rec(s, o=FAKE + 4) == (EALIGN if ok else ESHAPE)
    assert pro(s, q=FAKE + 8) == (EALIGN if ok else ESHAPE)
    lib = comba.load_library()
    P = ctypes.c_void_p
    args = [P(FAKE)] * 10
    assert lib.comba_chunk_fwd_save(ctypes.byref(s), *args, P(FAKE), ctypes.c_size_t(1),
                                    None) == (EWS if ok else ESHAPE)


def test_host_offsets_need_a_packed_batch():
    assert fwd(shape(B=2, T=64, cu_host=[0, 64, 128]), ws_bytes=1) == ESHAPE


def test_binding_checks_host_offsets():
    import numpy as np

    with pytest.raises(comba.CombaError):
        comba._host_offsets(np.array([0, 5, 9], dtype=np.int64), 4)
    a = comba._host_offsets([0, 5, 9], 3)
    assert a.dtype == np.int32 and a.flags.c_contiguous
    shp = comba._make_shape(1, 9, 1, 64, 64, 2, ctypes.c_void_p(FAKE), comba.COMBA_BF16,
                            cu_host=a)
    assert shp.cu_seqlens_host == a.ctypes.data


@pytest.fixture
def seg_env():
    old = os.environ.get("COMBA_SCAN_SEGMENTS")
    yield
    if old is None:
        os.environ.pop("COMBA_SCAN_SEGMENTS", None)
    else:
        os.environ["COMBA_SCAN_SEGMENTS"] = old


@pytest.mark.parametrize("dk,dv", [(128, 128), (128, 64), (256, 256)])
def test_segmented_workspace_holds_the_per_segment_states(seg_env, dk, dv):
    # a forced segment count P: the forward's workspace adds the virtual rows'
    # table (16 bytes per segment) and four per-segment states (F, X0, HT:
    # dk x dv; Phi: dk x dk, fp32), the backward-sized one three more (G, Y0,
    # DH0), each rounded up to 256 bytes
    lib = comba.load_library()
    s = shape(B=2, T=64 * 32, H=3, dk=dk, dv=dv)
    rnd = lambda x: (x + 255) // 256 * 256
    os.environ["COMBA_SCAN_SEGMENTS"] = "1"
    f1, b1 = lib.comba_fwd_workspace_bytes(ctypes.byref(s)), lib.comba_bwd_workspace_bytes(ctypes.byref(s))
    for P in (2, 4, 8, 16, 32):
        os.environ["COMBA_SCAN_SEGMENTS"] = str(P)
        nvr = 2 * P * 3
        sdv, sdk, tab = rnd(nvr * dk * dv * 4), rnd(nvr * dk * dk * 4), rnd(2 * P * 16)
        assert lib.comba_fwd_workspace_bytes(ctypes.byref(s)) == f1 + tab + 3 * sdv + sdk
        assert lib.comba_bwd_workspace_bytes(ctypes.byref(s)) == b1 + tab + 6 * sdv + sdk


@pytest.mark.parametrize("T,env", [
    (64 * 12, "8"),      # 12 chunks: 8 does not divide them
    (64 * 32 - 1, "2"),  # a partial last chunk
    (64 * 32, "0"),      # the automatic choice, which needs a device (none here)
    (64 * 32, "65"),     # beyond the largest count
])
def test_segments_not_taken_when_they_do_not_fit_the_rows(seg_env, T, env):
    lib = comba.load_library()
    s = shape(B=1, T=T, H=2)
    os.environ["COMBA_SCAN_SEGMENTS"] = "1"
    plain = lib.comba_fwd_workspace_bytes(ctypes.byref(s))
    os.environ["COMBA_SCAN_SEGMENTS"] = env
    assert lib.comba_fwd_workspace_bytes(ctypes.byref(s)) == plain


def test_packed_batches_are_segmented_and_fp32_inputs_are_not(seg_env):
    # packed sequences take any forced count (a sequence's segments are
    # ceil(n / P) chunks, the last ones shorter or empty); fp32 inputs never
    lib = comba.load_library()
    packed = shape(B=1, T=64 * 30 + 5, H=2, N=2, cu=FAKE)
    f32 = shape(B=1, T=64 * 32, H=2, dk=64, dv=64, dtype=comba.COMBA_F32)
    for s, grows in ((packed, True), (f32, False)):
        os.environ["COMBA_SCAN_SEGMENTS"] = "1"
        plain = lib.comba_fwd_workspace_bytes(ctypes.byref(s))
        os.environ["COMBA_SCAN_SEGMENTS"] = "4"
        assert (lib.comba_fwd_workspace_bytes(ctypes.byref(s)) > plain) == grows
