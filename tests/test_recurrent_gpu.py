"""GPU parity of the token-by-token recurrence (comba_recurrent_fwd).

The kernel evaluates Eq. comba-S one token at a time in fp32 on inputs that are
exact in their storage dtype, so it is held to the fp32 bar (norm-wise max
relative error <= 1e-5 against the fp64 oracle) for bf16 inputs too.  Covered:
decoding (T = 1, in place), short multi-token segments, every head-size pair,
fp32 and bf16 inputs, packed sequences with empty ones, a separate feedback
strength, missing initial / final states, and agreement with the chunk-wise
path."""
import zlib

import numpy as np
import pytest

import oracle
from comba_inputs import attach_beta_tilde, random_case
from gpu_helpers import gpu_fwd, maxrel, to_device

pytestmark = pytest.mark.gpu

TOL = 1e-5


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _log(msg):
    print(msg, flush=True)


def gpu_rec(w, **kw):
    import torch
    import paper_2506_02475_amd as comba

    a = to_device(w)
    o, ht = comba.comba_recurrent_fwd(a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"], a["h0"],
                                      beta_tilde=a["beta_tilde"], cu_seqlens=a["cu_seqlens"],
                                      **kw)
    torch.cuda.synchronize()
    return o.cpu().numpy(), (None if ht is None else ht.cpu().numpy())


def check_rec(w, tol=TOL):
    o, ht = gpu_rec(w)
    ro, rht = oracle.workload_fwd(w)
    errs = {"o": maxrel(o, ro), "ht": maxrel(ht, rht)}
    for name, e in errs.items():
        assert np.isfinite(e) and e <= tol, (name, e, tol)
    return errs


CASES = [
    ("decode_bf16_B64", dict(B=64, T=1, H=4, dk=128, dv=128, in_dtype="bf16")),
    ("decode_f32_d64", dict(B=8, T=1, H=2, dk=64, dv=64, in_dtype="f32")),
    ("decode_f32_d128", dict(B=8, T=1, H=2, dk=128, dv=128, in_dtype="f32")),
    ("bf16_T37_dv64", dict(B=2, T=37, H=2, dk=128, dv=64, in_dtype="bf16")),
    ("bf16_T70_dk64", dict(B=1, T=70, H=3, dk=64, dv=128, in_dtype="bf16")),
    ("f32_T130", dict(B=1, T=130, H=2, dk=64, dv=64, in_dtype="f32")),
    ("f32_T65_d128", dict(B=2, T=65, H=1, dk=128, dv=128, in_dtype="f32")),
    ("bf16_varlen", dict(T=0, H=2, dk=128, dv=128, in_dtype="bf16", seqlens=[1, 0, 5, 64, 3])),
    ("f32_varlen", dict(T=0, H=2, dk=64, dv=64, in_dtype="f32", seqlens=[0, 9, 1, 0])),
    # head dim 256, the paper's model setting: two 128-column workgroups of 8 waves
    ("decode_bf16_d256", dict(B=16, T=1, H=4, dk=256, dv=256, in_dtype="bf16")),
    ("bf16_T45_d256", dict(B=2, T=45, H=2, dk=256, dv=256, in_dtype="bf16")),
    ("f32_T20_dk128_dv256", dict(B=2, T=20, H=2, dk=128, dv=256, in_dtype="f32")),
    ("bf16_varlen_dk256_dv128", dict(T=0, H=2, dk=256, dv=128, in_dtype="bf16",
                                     seqlens=[3, 0, 40])),
    # at least 1024 state slices: the full-width launch (fewer: 32-column slices)
    ("decode_f32_d64_wide", dict(B=64, T=1, H=16, dk=64, dv=64, in_dtype="f32")),
    ("decode_bf16_d256_wide", dict(B=32, T=1, H=16, dk=256, dv=256, in_dtype="bf16")),
    ("decode_bf16_dk128_dv256_wide", dict(B=32, T=1, H=16, dk=128, dv=256, in_dtype="bf16")),
]


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_recurrent_parity(name, kw):
    w = random_case(seed=zlib.crc32(name.encode()) % 1000 + 11, grad=False, **kw)
    _log("recurrent %s %s" % (name, check_rec(w)))


@pytest.mark.parametrize("form", ["b_beta", "independent", "iplr"])
def test_recurrent_beta_tilde(form):
    w = random_case(seed=41, B=3, T=50, H=2, dk=128, dv=128, in_dtype="bf16", grad=False)
    attach_beta_tilde(w, form, seed=42)
    _log("recurrent beta~ %s %s" % (form, check_rec(w)))


def test_recurrent_without_states():
    w = random_case(seed=43, B=2, T=20, H=2, dk=128, dv=128, in_dtype="bf16", grad=False,
                    h0=False)
    o, ht = gpu_rec(w, output_final_state=False)
    assert ht is None
    ro, _ = oracle.workload_fwd(w)
    assert maxrel(o, ro) <= TOL


def test_recurrent_token_free_passes_states_through():
    w = random_case(seed=44, B=3, T=0, H=2, dk=128, dv=128, in_dtype="bf16", grad=False)
    o, ht = gpu_rec(w)
    assert o.size == 0 and np.array_equal(ht, w.h0)
    w.h0 = None
    _, ht = gpu_rec(w)
    assert np.all(ht == 0)


def test_decode_steps_in_place_equal_one_call():
    # T calls of one token each, updating the states in place (ht is h0), give
    # bitwise the outputs and final states of one call over the T tokens
    import torch
    import paper_2506_02475_amd as comba

    w = random_case(seed=45, B=4, T=12, H=2, dk=128, dv=128, in_dtype="bf16", grad=False)
    a = to_device(w)
    o_all, ht_all = comba.comba_recurrent_fwd(a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"],
                                              a["h0"])
    state = a["h0"].clone()
    outs = []
    for t in range(w.T):
        sl = [x[:, t:t + 1].contiguous() for x in (a["q"], a["k"], a["v"], a["g"], a["beta"])]
        o_t, ht_t = comba.comba_recurrent_fwd(*sl, a["d"], state, ht=state)
        assert ht_t.data_ptr() == state.data_ptr()
        outs.append(o_t)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat(outs, dim=1), o_all)
    assert torch.equal(state, ht_all)


def test_recurrent_agrees_with_chunk_path():
    # two different algorithms for the same recurrence: each against the oracle
    # at its own bar, and with each other at the chunk path's bar
    w = random_case(seed=46, B=2, T=200, H=2, dk=128, dv=128, in_dtype="bf16", grad=False)
    o_r, h_r = gpu_rec(w)
    o_c, h_c = gpu_fwd(w)
    ro, rht = oracle.workload_fwd(w)
    assert maxrel(o_r, ro) <= TOL and maxrel(h_r, rht) <= TOL
    assert maxrel(o_c, o_r) <= 2e-3 and maxrel(h_c, h_r) <= 2e-3


def test_decode_full_layer_shape():
    # the decoding step the benchmark times: 64 sequences, 16 heads, d = 128,
    # bf16 inputs, one token, states updated in place
    import torch
    import paper_2506_02475_amd as comba

    w = random_case(seed=47, B=64, T=1, H=16, dk=128, dv=128, in_dtype="bf16", grad=False)
    a = to_device(w)
    state = a["h0"].clone()
    o, _ = comba.comba_recurrent_fwd(a["q"], a["k"], a["v"], a["g"], a["beta"], a["d"], state,
                                     ht=state)
    torch.cuda.synchronize()
    ro, rht = oracle.workload_fwd(w)
    errs = {"o": maxrel(o.cpu().numpy(), ro), "ht": maxrel(state.cpu().numpy(), rht)}
    _log("decode B64 H16 d128 %s" % errs)
    assert max(errs.values()) <= TOL
