"""GPU parity of the segmented scans (few long rows).

When fixed-length rows give the state scan fewer chains than the chip has CUs
(for example one long sequence), comba_chunk_fwd cuts each row into P
segments: every segment's final state from a zero start and its transition
product are scanned side by side, the true state entering each segment follows
from the affine dependence on the initial state (X_{p+1} = Phi_p X_p + F_p),
and the outputs of all segments are then scanned in parallel.  The result is
the recurrence of Eq. comba-S, compared here with the fp64 oracle (bar 2e-3 for
bf16 inputs) and with the unsegmented scan (COMBA_SCAN_SEGMENTS=1).  The
backward (stateless and training pair) is segmented the same way: every
segment's state gradient at its start from a zero end, the gradient leaving
each segment from Y_{p-1} = Phi_p^T Y_p + G_p, and the reverse scan of all
segments in parallel.

The gates are weak (log-gates scaled by 0.002, about 25% of a state surviving
a 1024-token segment) so that every segment's outputs depend strongly on the
state carried in from the segments before it; `_carry` checks that on the
oracle, so a wrong boundary state could not pass unnoticed.
"""
import ctypes
import os

import numpy as np
import pytest

import oracle
from comba_inputs import random_case
from gpu_helpers import check_fwd, gpu_fwd, maxrel

pytestmark = pytest.mark.gpu

ENV = "COMBA_SCAN_SEGMENTS"


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    old = os.environ.get(ENV)
    yield
    if old is None:
        os.environ.pop(ENV, None)
    else:
        os.environ[ENV] = old


def _case(B, T, H, dk, dv, seed, h0=True):
    print("segmented case: B%d T%d H%d dk%d dv%d seed %d" % (B, T, H, dk, dv, seed), flush=True)
    w = random_case(B=B, T=T, H=H, dk=dk, dv=dv, in_dtype="bf16", seed=seed, h0=h0, grad=False)
    w.g = (w.g * np.float32(0.002)).astype(np.float32)
    return w


def _carry(w, P, heads):
    """Relative change of the oracle's outputs when every segment of P starts
    from a zero state instead of the state carried in: how much a wrong
    boundary state would show."""
    B, T, H = w.q.shape[:3]
    sel = list(heads)
    ro, _ = oracle.step_fwd(w.q[:, :, sel], w.k[:, :, sel], w.v[:, :, sel], w.g[:, :, sel],
                            w.beta[:, :, sel], w.d[sel], None if w.h0 is None else w.h0[:, sel])
    Tp = T // P
    cut = lambda x: np.ascontiguousarray(x.reshape((B * P, Tp) + x.shape[2:]))
    rz, _ = oracle.step_fwd(cut(w.q[:, :, sel]), cut(w.k[:, :, sel]), cut(w.v[:, :, sel]),
                            cut(w.g[:, :, sel]), cut(w.beta[:, :, sel]), w.d[sel], None)
    return maxrel(rz.reshape(ro.shape), ro)


def _plain_and_segmented(w, P):
    os.environ[ENV] = "1"
    o1, h1 = gpu_fwd(w)
    os.environ[ENV] = str(P)
    o2, h2 = gpu_fwd(w)
    return (o1, h1), (o2, h2)


@pytest.mark.parametrize("B,T,H,dk,dv,P", [
    (1, 8192, 2, 128, 128, 8),     # 8 segments of 16 chunks
    (2, 4096, 1, 128, 64, 4),      # dk != dv: the transition product is dk x dk
    (1, 4096, 2, 64, 128, 2),
    (1, 8192, 1, 256, 256, 4),     # head dim 256
])
def test_forced_segments_match_the_oracle_and_the_plain_scan(B, T, H, dk, dv, P):
    w = _case(B, T, H, dk, dv, seed=900 + P + dk)
    carry = _carry(w, P, range(H))
    assert carry > 0.1, carry                      # the boundary states matter
    (o1, h1), (o2, h2) = _plain_and_segmented(w, P)
    os.environ[ENV] = str(P)
    errs = check_fwd(w)
    print("forced P=%d: %s, carry %.2f" % (P, {k: "%.2e" % v for k, v in errs.items()}, carry),
          flush=True)
    # the two scans reach the same result up to rounding
    assert maxrel(o2, o1) <= 2e-4 and maxrel(h2, h1) <= 2e-4, (maxrel(o2, o1), maxrel(h2, h1))


def test_auto_segments_on_one_long_sequence():
    import torch

    import paper_2506_02475_amd as comba

    os.environ.pop(ENV, None)
    w = _case(1, 65536, 2, 128, 128, seed=77)
    a = {n: torch.from_numpy(np.ascontiguousarray(x)).cuda() for n, x in
         (("q", w.q), ("k", w.k), ("v", w.v), ("g", w.g), ("beta", w.beta), ("d", w.d),
          ("h0", w.h0))}
    bf = torch.bfloat16
    comba.profile_enable(True)
    o, ht = comba.comba_chunk_fwd(a["q"].to(bf), a["k"].to(bf), a["v"].to(bf), a["g"],
                                  a["beta"].to(bf), a["d"], a["h0"])
    torch.cuda.synchronize()
    stages = [n for n, _ in comba.profile_read()]
    comba.profile_enable(False)
    # 2 heads x 4 slices = 8 chains on a 256-CU chip: the segmented scan runs
    assert "scan_seg_state" in stages and "scan_seg_phi" in stages, stages
    errs = check_fwd(w)
    print("auto: %s" % {k: "%.2e" % v for k, v in errs.items()}, flush=True)
    # deterministic
    o_again, ht_again = comba.comba_chunk_fwd(a["q"].to(bf), a["k"].to(bf), a["v"].to(bf), a["g"],
                                              a["beta"].to(bf), a["d"], a["h0"])
    assert torch.equal(o, o_again) and torch.equal(ht, ht_again)


def test_without_initial_or_final_state():
    import torch

    import paper_2506_02475_amd as comba

    w = _case(1, 4096, 1, 128, 128, seed=31, h0=False)
    os.environ[ENV] = "4"
    bf = torch.bfloat16
    t = lambda x, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(x)).cuda().to(dt)
    o, ht = comba.comba_chunk_fwd(t(w.q, bf), t(w.k, bf), t(w.v, bf), t(w.g), t(w.beta, bf),
                                  t(w.d), None, output_final_state=False)
    torch.cuda.synchronize()
    assert ht is None
    ro, _ = oracle.step_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, None)
    assert maxrel(o.cpu().numpy(), ro) <= 2e-3


def test_a_workspace_without_the_segment_buffers_runs_the_plain_scan():
    import torch

    import paper_2506_02475_amd as comba

    w = _case(1, 8192, 1, 128, 128, seed=5)
    lib = comba.load_library()
    bf = torch.bfloat16
    t = lambda x, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(x)).cuda().to(dt)
    q, k, v, g, beta, d, h0 = (t(w.q, bf), t(w.k, bf), t(w.v, bf), t(w.g), t(w.beta, bf),
                               t(w.d), t(w.h0))
    shp, (B, T, H, dk, dv, N) = comba._prepare(q, k, v, g, beta, d, h0, None)
    os.environ[ENV] = "1"
    plain = lib.comba_fwd_workspace_bytes(ctypes.byref(shp))
    os.environ[ENV] = "8"
    seg = lib.comba_fwd_workspace_bytes(ctypes.byref(shp))
    assert seg > plain > 0
    outs = []
    for env, nbytes in (("1", plain), ("8", plain), ("8", seg)):
        os.environ[ENV] = env
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        o = torch.empty((B, T, H, dv), dtype=torch.float32, device="cuda")
        ht = torch.empty((N, H, dk, dv), dtype=torch.float32, device="cuda")
        st = torch.cuda.current_stream().cuda_stream
        P = ctypes.c_void_p
        rc = lib.comba_chunk_fwd(ctypes.byref(shp), P(q.data_ptr()), P(k.data_ptr()),
                                 P(v.data_ptr()), P(g.data_ptr()), P(beta.data_ptr()), None,
                                 P(d.data_ptr()), P(h0.data_ptr()), P(o.data_ptr()),
                                 P(ht.data_ptr()), P(ws.data_ptr()), ctypes.c_size_t(nbytes),
                                 P(st))
        assert rc == 0
        torch.cuda.synchronize()
        outs.append((o.cpu().numpy(), ht.cpu().numpy()))
    # the segmented request with the plain-sized workspace ran the plain scan
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
    # with its buffers it ran the segmented one (same result up to rounding)
    assert not np.array_equal(outs[0][0], outs[2][0])
    assert maxrel(outs[2][0], outs[0][0]) <= 2e-4


def _grad_case(B, T, H, dk, dv, seed):
    print("segmented backward case: B%d T%d H%d dk%d dv%d seed %d" % (B, T, H, dk, dv, seed),
          flush=True)
    w = random_case(B=B, T=T, H=H, dk=dk, dv=dv, in_dtype="bf16", seed=seed, grad=True, dht=True)
    w.g = (w.g * np.float32(0.002)).astype(np.float32)
    return w


GRAD_NAMES = ("dq", "dk", "dv", "dg", "dbeta", "dd", "dh0")


@pytest.mark.parametrize("B,T,H,dk,dv,P", [
    (1, 8192, 2, 128, 128, 8),
    (2, 4096, 1, 128, 64, 4),
    (1, 8192, 1, 256, 256, 4),
])
def test_segmented_backward_matches_the_oracle_and_the_plain_scans(B, T, H, dk, dv, P):
    from gpu_helpers import check_bwd, gpu_bwd

    w = _grad_case(B, T, H, dk, dv, seed=700 + P + dk)
    os.environ[ENV] = "1"
    plain = gpu_bwd(w)
    os.environ[ENV] = str(P)
    errs = check_bwd(w)                                # stateless backward, segmented
    print("backward P=%d: %s" % (P, {k: "%.2e" % v for k, v in errs.items()}), flush=True)
    seg = gpu_bwd(w)
    for name in GRAD_NAMES:
        assert maxrel(seg[name], plain[name]) <= 5e-4, (name, maxrel(seg[name], plain[name]))


@pytest.mark.parametrize("P", [4, 8])
def test_segmented_training_pair_equals_the_stateless_pair(P):
    import torch

    import paper_2506_02475_amd as comba
    from gpu_helpers import to_device

    w = _grad_case(1, 8192, 2, 128, 128, seed=61 + P)
    os.environ[ENV] = str(P)
    a = to_device(w)
    args = (a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"], a["h0"])
    o_s, ht_s = comba.comba_chunk_fwd(*args)
    g_s = comba.comba_chunk_bwd(*args, a["dO"], a["dht"])
    comba.profile_enable(True)
    o_p, ht_p, ws = comba.comba_chunk_fwd_save(*args)
    g_p = comba.comba_chunk_bwd_saved(*args, a["dO"], a["dht"], workspace=ws)
    torch.cuda.synchronize()
    stages = [n for n, _ in comba.profile_read()]
    comba.profile_enable(False)
    assert "scan_seg_phi" in stages and "scan_seg_grad" in stages, stages
    # the same arithmetic in both pairs: bitwise equal
    assert torch.equal(o_s, o_p) and torch.equal(ht_s, ht_p)
    for name in GRAD_NAMES:
        assert torch.equal(g_s[name], g_p[name]), name


def test_segmented_pair_with_separate_feedback_strength_and_no_final_gradient():
    """beta~ given on its own (dbeta and dbeta~ split) and dht = 0, P = 8."""
    from comba_inputs import attach_beta_tilde
    from gpu_helpers import check_bwd, gpu_bwd

    print("segmented case: beta~ independent, no dht, B1 T8192 H2 d128", flush=True)
    w = random_case(B=1, T=8192, H=2, dk=128, dv=128, in_dtype="bf16", seed=404, grad=True,
                    dht=False)
    w.g = (w.g * np.float32(0.002)).astype(np.float32)
    attach_beta_tilde(w, "independent", seed=405)
    os.environ[ENV] = "1"
    plain_o, plain_ht = gpu_fwd(w)
    plain = gpu_bwd(w)
    os.environ[ENV] = "8"
    ferrs = check_fwd(w)
    berrs = check_bwd(w)
    print("beta~ P=8: fwd %s bwd %s" % ({k: "%.2e" % v for k, v in ferrs.items()},
                                        {k: "%.2e" % v for k, v in berrs.items()}), flush=True)
    seg = gpu_bwd(w)
    assert "dbeta_tilde" in seg and seg["dbeta_tilde"] is not None
    for name in GRAD_NAMES + ("dbeta_tilde",):
        assert maxrel(seg[name], plain[name]) <= 5e-4, (name, maxrel(seg[name], plain[name]))


def _packed_case(seqlens, H, seed, grad):
    print("segmented packed case: lengths %s H%d seed %d" % (seqlens, H, seed), flush=True)
    w = random_case(B=1, T=0, H=H, dk=128, dv=128, in_dtype="bf16", seed=seed, seqlens=seqlens,
                    grad=grad, dht=grad)
    w.g = (w.g * np.float32(0.002)).astype(np.float32)
    return w


@pytest.mark.parametrize("seqlens,P", [
    ([5000, 64, 0, 12345], 8),    # short and empty sequences: empty segments
    ([3000, 2999], 4),
])
def test_packed_segments_match_the_oracle_and_the_plain_scans(seqlens, P):
    from gpu_helpers import check_bwd, gpu_bwd

    w = _packed_case(seqlens, 2, seed=31 + P, grad=True)
    os.environ[ENV] = "1"
    po, pht = gpu_fwd(w)
    pg = gpu_bwd(w)
    os.environ[ENV] = str(P)
    ferrs = check_fwd(w)
    berrs = check_bwd(w)
    print("packed P=%d: fwd %s bwd %s" % (P, {k: "%.2e" % v for k, v in ferrs.items()},
                                          {k: "%.2e" % v for k, v in berrs.items()}), flush=True)
    so, sht = gpu_fwd(w)
    sg = gpu_bwd(w)
    assert maxrel(so, po) <= 2e-4 and maxrel(sht, pht) <= 2e-4
    for name in GRAD_NAMES:
        assert maxrel(sg[name], pg[name]) <= 5e-4, (name, maxrel(sg[name], pg[name]))


def test_packed_auto_segments_and_training_pair():
    import torch

    import paper_2506_02475_amd as comba
    from gpu_helpers import to_device

    os.environ.pop(ENV, None)
    w = _packed_case([40000, 30001], 2, seed=12, grad=True)
    a = to_device(w)
    cuh = w.cu_seqlens.astype(np.int32)
    args = (a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"], a["h0"])
    kw = dict(cu_seqlens=a["cu_seqlens"], cu_seqlens_host=cuh)
    comba.profile_enable(True)
    o_s, ht_s = comba.comba_chunk_fwd(*args, **kw)
    g_s = comba.comba_chunk_bwd(*args, a["dO"], a["dht"], **kw)
    o_p, ht_p, ws = comba.comba_chunk_fwd_save(*args, **kw)
    g_p = comba.comba_chunk_bwd_saved(*args, a["dO"], a["dht"], workspace=ws, **kw)
    torch.cuda.synchronize()
    stages = [n for n, _ in comba.profile_read()]
    comba.profile_enable(False)
    # 2 sequences x 2 heads x 4 slices = 16 chains: the host offsets let the
    # library cut them
    assert "scan_seg_state" in stages and "scan_seg_grad" in stages, stages
    ro, rht = oracle.step_fwd(w.q, w.k, w.v, w.g, w.beta, w.d, w.h0, cu_seqlens=w.cu_seqlens)
    assert maxrel(o_s.cpu().numpy(), ro) <= 2e-3 and maxrel(ht_s.cpu().numpy(), rht) <= 2e-3
    assert torch.equal(o_s, o_p) and torch.equal(ht_s, ht_p)
    for name in GRAD_NAMES:
        assert torch.equal(g_s[name], g_p[name]), name
