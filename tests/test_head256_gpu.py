"""GPU parity of the chunk-wise path at head dimension 256.

The paper's models keep the head dimension at 256 (Section 2, to match the
state size of Mamba2).  Covered here: the stateless forward (prefill), the
backward (pass-wise intra-chunk kernel), the saved training pair with a
separate beta~, mixed 128/256 head sizes, packed sequences, and the
B4 T4096 H8 d256 layer on sampled heads; the token-by-token decoding step at
d = 256 is covered with the other recurrent tests.  Compared element by
element with the fp64 oracle at the bf16 bar (2e-3, norm-wise max relative
error)."""
import zlib

import numpy as np
import pytest

import oracle
from comba_inputs import random_case
from gpu_helpers import check_fwd, maxrel, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _log(msg):
    print(msg, flush=True)


CASES = [
    ("d256_T200", dict(B=1, T=200, H=2, dk=256, dv=256)),
    ("d256_B2_T63", dict(B=2, T=63, H=2, dk=256, dv=256)),
    ("dk128_dv256", dict(B=1, T=150, H=2, dk=128, dv=256)),
    ("dk256_dv128", dict(B=2, T=129, H=1, dk=256, dv=128)),
    ("d256_varlen", dict(T=0, H=2, dk=256, dv=256, seqlens=[1, 64, 0, 130, 5])),
]


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_forward_head256(name, kw):
    w = random_case(seed=zlib.crc32(name.encode()) % 1000 + 17, grad=False, in_dtype="bf16", **kw)
    _log("head256 fwd %s %s" % (name, check_fwd(w)))


def test_forward_head256_agrees_with_recurrent():
    import torch
    import paper_2506_02475_amd as comba

    w = random_case(seed=61, B=2, T=100, H=2, dk=256, dv=256, in_dtype="bf16", grad=False)
    a = to_device(w)
    args = (a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"], a["h0"])
    o_c, h_c = comba.comba_chunk_fwd(*args)
    o_r, h_r = comba.comba_recurrent_fwd(*args)
    torch.cuda.synchronize()
    assert maxrel(o_c.cpu().numpy(), o_r.cpu().numpy()) <= 2e-3
    assert maxrel(h_c.cpu().numpy(), h_r.cpu().numpy()) <= 2e-3


BWD_CASES = [
    ("d256_T200", dict(B=1, T=200, H=2, dk=256, dv=256)),
    ("dk128_dv256", dict(B=2, T=130, H=1, dk=128, dv=256)),
    ("dk256_dv128", dict(B=1, T=129, H=2, dk=256, dv=128)),
    ("d256_varlen", dict(T=0, H=2, dk=256, dv=256, seqlens=[1, 64, 0, 70])),
]


@pytest.mark.parametrize("name,kw", BWD_CASES, ids=[c[0] for c in BWD_CASES])
def test_backward_head256(name, kw):
    from gpu_helpers import check_bwd

    w = random_case(seed=zlib.crc32(name.encode()) % 1000 + 19, dht=True, in_dtype="bf16", **kw)
    _log("head256 bwd %s %s" % (name, check_bwd(w)))


def test_head256_saved_pair_and_beta_tilde():
    import torch
    import paper_2506_02475_amd as comba
    from comba_inputs import attach_beta_tilde

    w = attach_beta_tilde(random_case(seed=62, B=2, T=150, H=2, dk=256, dv=256,
                                      in_dtype="bf16", dht=True), "b_beta", seed=3)
    a = to_device(w)
    args = (a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"], a["h0"])
    o_s, ht_s, ws = comba.comba_chunk_fwd_save(*args, beta_tilde=a["beta_tilde"])
    gr_s = comba.comba_chunk_bwd_saved(*args, a["dO"], a["dht"], workspace=ws,
                                       beta_tilde=a["beta_tilde"])
    gr = comba.comba_chunk_bwd(*args, a["dO"], a["dht"], beta_tilde=a["beta_tilde"])
    torch.cuda.synchronize()
    for key in gr:
        assert torch.equal(gr_s[key], gr[key]), key
    ref = oracle.workload_bwd(w)
    for key in ("dq", "dk", "dv", "dg", "dbeta", "dbeta_tilde", "dd", "dh0"):
        assert maxrel(gr_s[key].cpu().numpy(), ref[key]) <= 2e-3, key


def test_prefill_head256_layer_shape():
    # a 1.3B-model layer at head dim 256 (8 heads of 256 instead of 16 of 128):
    # B4 T4096, sampled heads against the oracle
    import torch
    import paper_2506_02475_amd as comba

    w = random_case(seed=63, B=4, T=4096, H=8, dk=256, dv=256, in_dtype="bf16", grad=False)
    a = to_device(w)
    o, ht = comba.comba_chunk_fwd(a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"], a["h0"])
    torch.cuda.synchronize()
    heads = [1, 6]
    ro, rht = oracle.workload_fwd(w, heads=heads)
    errs = {"o": maxrel(o.cpu().numpy()[:, :, heads], ro),
            "ht": maxrel(ht.cpu().numpy()[:, heads], rht)}
    _log("prefill B4 T4096 H8 d256 %s" % errs)
    assert max(errs.values()) <= 2e-3


def test_train_head256_layer_shape():
    # the training pair at B4 T4096 H8 d256 (the bench's d = 256 leg), sampled
    # heads against the oracle
    import torch
    import paper_2506_02475_amd as comba

    w = random_case(seed=64, B=4, T=4096, H=8, dk=256, dv=256, in_dtype="bf16", dht=True)
    a = to_device(w)
    args = (a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"], a["h0"])
    o, ht, ws = comba.comba_chunk_fwd_save(*args)
    gr = comba.comba_chunk_bwd_saved(*args, a["dO"], a["dht"], workspace=ws)
    torch.cuda.synchronize()
    heads = [2, 5]
    ref = oracle.workload_bwd(w, heads=heads)
    errs = {n: maxrel(gr[n].cpu().numpy()[:, :, heads], ref[n])
            for n in ("dq", "dk", "dv", "dg", "dbeta")}
    errs["dd"] = maxrel(gr["dd"].cpu().numpy()[heads], ref["dd"])
    errs["dh0"] = maxrel(gr["dh0"].cpu().numpy()[:, heads], ref["dh0"])
    _log("train B4 T4096 H8 d256 %s" % errs)
    assert max(errs.values()) <= 2e-3
