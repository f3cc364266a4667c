"""The differentiable op (comba_chunk, torch.autograd) over the training pair.

Its gradients must be exactly those of comba_chunk_fwd_save +
comba_chunk_bwd_saved called directly with the same upstream gradients (cast
to the inputs' dtypes), whichever outputs the loss uses; the direct calls
themselves are held against the fp64 oracle by the parity tests."""
import numpy as np
import pytest

from comba_inputs import random_case

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _inputs(w, dt, packed=False):
    import torch

    t = lambda x, d=torch.float32: torch.from_numpy(np.ascontiguousarray(x)).cuda().to(d)
    leaves = dict(q=t(w.q, dt), k=t(w.k, dt), v=t(w.v, dt), g=t(w.g), beta=t(w.beta, dt),
                  d=t(w.d), h0=t(w.h0))
    for x in leaves.values():
        x.requires_grad_(True)
    return leaves


@pytest.mark.parametrize("case,use", [
    ("bf16", "both"), ("bf16", "o"), ("bf16", "ht"), ("f32", "both"), ("packed", "both"),
])
def test_autograd_gradients_equal_the_direct_training_pair(case, use):
    import torch

    import paper_2506_02475_amd as comba

    print("autograd case: %s, loss on %s" % (case, use), flush=True)
    if case == "f32":
        w = random_case(B=2, T=150, H=2, dk=64, dv=64, in_dtype="f32", seed=11, grad=True)
        dt = torch.float32
    elif case == "packed":
        w = random_case(T=0, H=2, dk=128, dv=128, in_dtype="bf16", seed=12, grad=True,
                        seqlens=[100, 0, 333])
        dt = torch.bfloat16
    else:
        w = random_case(B=2, T=150, H=2, dk=128, dv=128, in_dtype="bf16", seed=13, grad=True)
        dt = torch.bfloat16
    x = _inputs(w, dt)
    cu = None if w.cu_seqlens is None else torch.from_numpy(w.cu_seqlens.astype(np.int32)).cuda()
    o, ht = comba.comba_chunk(x["q"], x["k"], x["v"], x["g"], x["beta"], x["d"], x["h0"],
                              cu_seqlens=cu)
    gen = torch.Generator(device="cpu").manual_seed(5)
    # upstream gradients representable in the inputs' dtype (the op rounds dO to it)
    W = torch.randn(o.shape, generator=gen).to(dt).float().cuda()
    V = torch.randn(ht.shape, generator=gen).cuda()
    loss = 0
    if use in ("both", "o"):
        loss = loss + (o * W).sum()
    if use in ("both", "ht"):
        loss = loss + (ht * V).sum()
    loss.backward()
    torch.cuda.synchronize()
    # the same pair called directly
    det = {n: t.detach() for n, t in x.items()}
    args = (det["q"], det["k"], det["v"], det["g"], det["beta"], det["d"], det["h0"])
    o2, ht2, ws = comba.comba_chunk_fwd_save(*args, cu_seqlens=cu)
    dO = (W if use in ("both", "o") else torch.zeros_like(W)).to(dt).contiguous()
    dht = V if use in ("both", "ht") else None
    gr = comba.comba_chunk_bwd_saved(*args, dO, dht, workspace=ws, cu_seqlens=cu)
    torch.cuda.synchronize()
    assert torch.equal(o.detach(), o2) and torch.equal(ht.detach(), ht2)
    for name, key in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("g", "dg"), ("beta", "dbeta"),
                      ("d", "dd"), ("h0", "dh0")):
        ref = gr[key].to(x[name].dtype)
        assert x[name].grad is not None and x[name].grad.dtype == x[name].dtype, name
        assert torch.equal(x[name].grad, ref), name


def test_autograd_with_separate_feedback_strength():
    import torch

    import paper_2506_02475_amd as comba
    from comba_inputs import attach_beta_tilde

    w = random_case(B=1, T=200, H=2, dk=128, dv=128, in_dtype="bf16", seed=14, grad=True)
    attach_beta_tilde(w, "b_beta", seed=15)
    x = _inputs(w, torch.bfloat16)
    bt = torch.from_numpy(np.ascontiguousarray(w.extra["beta_tilde"])).cuda().to(torch.bfloat16)
    bt.requires_grad_(True)
    o, ht = comba.comba_chunk(x["q"], x["k"], x["v"], x["g"], x["beta"], x["d"], x["h0"],
                              beta_tilde=bt)
    o.float().square().sum().backward()
    torch.cuda.synchronize()
    det = {n: t.detach() for n, t in x.items()}
    args = (det["q"], det["k"], det["v"], det["g"], det["beta"], det["d"], det["h0"])
    o2, ht2, ws = comba.comba_chunk_fwd_save(*args, beta_tilde=bt.detach())
    gr = comba.comba_chunk_bwd_saved(*args, (2 * o2).to(torch.bfloat16), None, workspace=ws,
                                     beta_tilde=bt.detach())
    assert torch.equal(bt.grad, gr["dbeta_tilde"].to(torch.bfloat16))
    assert torch.equal(x["beta"].grad, gr["dbeta"].to(torch.bfloat16))


def test_autograd_over_segmented_scans():
    """One long row cut into 4 segments (forced): the op's gradients equal the
    directly called pair's under the same setting."""
    import os

    import torch

    import paper_2506_02475_amd as comba

    w = random_case(B=1, T=4096, H=2, dk=128, dv=128, in_dtype="bf16", seed=16, grad=True)
    old = os.environ.get("COMBA_SCAN_SEGMENTS")
    os.environ["COMBA_SCAN_SEGMENTS"] = "4"
    try:
        x = _inputs(w, torch.bfloat16)
        comba.profile_enable(True)
        o, ht = comba.comba_chunk(x["q"], x["k"], x["v"], x["g"], x["beta"], x["d"], x["h0"])
        (o.sum() + ht.square().sum()).backward()
        torch.cuda.synchronize()
        stages = [n for n, _ in comba.profile_read()]
        comba.profile_enable(False)
        # the forward's stages (the session is per host thread; autograd runs
        # the backward on its own device thread, which records nothing)
        assert "scan_seg_state" in stages and "seg_combine" in stages, stages
        det = {n: t.detach() for n, t in x.items()}
        args = (det["q"], det["k"], det["v"], det["g"], det["beta"], det["d"], det["h0"])
        o2, ht2, ws = comba.comba_chunk_fwd_save(*args)
        gr = comba.comba_chunk_bwd_saved(*args, torch.ones_like(o2).to(torch.bfloat16), 2 * ht2,
                                         workspace=ws)
        torch.cuda.synchronize()
    finally:
        if old is None:
            os.environ.pop("COMBA_SCAN_SEGMENTS", None)
        else:
            os.environ["COMBA_SCAN_SEGMENTS"] = old
    assert torch.equal(o.detach(), o2) and torch.equal(ht.detach(), ht2)
    for name, key in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("g", "dg"), ("beta", "dbeta"),
                      ("d", "dd"), ("h0", "dh0")):
        assert torch.equal(x[name].grad, gr[key].to(x[name].dtype)), name
