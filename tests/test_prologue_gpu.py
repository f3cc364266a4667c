"""GPU parity of the layer prologue (short causal conv, SiLU, L2 norm of q, k)
against the fp64 oracle in oracle/prologue.py.

The kernels compute in fp32 on inputs exact in their storage dtype.  Forward
outputs in bf16 are rounded to nearest, so they are held to one bf16 unit in the
last place of the oracle value (plus 1e-5 of the tensor's largest value for
values near zero, where the fp32 sum of four products has no relative bound);
fp32 outputs and every gradient (fp32) to a norm-wise max relative error of
1e-5."""
import zlib

import numpy as np
import pytest

from comba_inputs import prologue_case
from gpu_helpers import maxrel
from oracle.prologue import prologue_bwd, prologue_fwd

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _log(msg):
    print(msg, flush=True)


def run_gpu(c):
    import torch
    import paper_2506_02475_amd as comba

    dt = torch.bfloat16 if c["in_dtype"] == "bf16" else torch.float32
    t = lambda x, d=torch.float32: torch.from_numpy(np.ascontiguousarray(x)).to("cuda", d)
    xs = [t(c[n], dt) for n in ("xq", "xk", "xv")]
    ws = [t(c[n]) for n in ("wq", "wk", "wv")]
    gs = [t(c[n]) for n in ("gq", "gk", "gv")]
    cu = None if c["cu_seqlens"] is None else t(c["cu_seqlens"], torch.int32)
    q, k, v = comba.comba_prologue_fwd(*xs, *ws, cu_seqlens=cu)
    gr = comba.comba_prologue_bwd(*xs, *ws, *gs, cu_seqlens=cu)
    torch.cuda.synchronize()
    return [x.float().cpu().numpy() for x in (q, k, v)], {n: x.cpu().numpy() for n, x in gr.items()}


def check(c):
    ys, gr = run_gpu(c)
    cu = c["cu_seqlens"]
    errs = {}
    for i, (n, norm) in enumerate((("q", True), ("k", True), ("v", False))):
        x, w, g = c["x" + n], c["w" + n], c["g" + n]
        ref = prologue_fwd(x, w, norm, cu_seqlens=cu)
        y = ys[i]
        if c["in_dtype"] == "bf16":
            bound = 2.0 ** -8 * np.abs(ref) + 1e-5 * np.max(np.abs(ref))
            assert np.all(np.abs(y - ref) <= bound), n
            errs[n] = float(np.max(np.abs(y - ref) / (np.abs(ref) + 1e-30)))
        else:
            errs[n] = maxrel(y, ref)
            assert errs[n] <= 1e-5, (n, errs[n])
        dx, dw = prologue_bwd(x, w, norm, g, cu_seqlens=cu)
        errs["dx" + n] = maxrel(gr["dx" + n], dx)
        errs["dw" + n] = maxrel(gr["dw" + n], dw)
        assert errs["dx" + n] <= 1e-5 and errs["dw" + n] <= 1e-5, errs
    return errs


CASES = [
    ("bf16_d128", dict(B=2, T=200, H=2, dk=128, dv=128, in_dtype="bf16")),
    ("bf16_dk64_dv128", dict(B=1, T=130, H=3, dk=64, dv=128, in_dtype="bf16")),
    ("bf16_d256", dict(B=1, T=150, H=2, dk=256, dv=256, in_dtype="bf16")),
    ("f32_d64", dict(B=2, T=70, H=2, dk=64, dv=64, in_dtype="f32")),
    ("f32_dk128_dv256", dict(B=1, T=66, H=1, dk=128, dv=256, in_dtype="f32")),
    ("bf16_T3", dict(B=3, T=3, H=2, dk=128, dv=128, in_dtype="bf16")),
    # head counts that leave the forward's last group of heads partly empty
    ("bf16_d128_H5", dict(B=2, T=333, H=5, dk=128, dv=128, in_dtype="bf16")),
    ("bf16_d256_H3", dict(B=1, T=517, H=3, dk=256, dv=256, in_dtype="bf16")),
    # packed sequences: empty ones, sequences shorter than the taps, boundaries
    # inside a run and exactly at run edges
    ("bf16_varlen", dict(H=2, dk=128, dv=128, in_dtype="bf16",
                         seqlens=[1, 0, 2, 61, 64, 3, 0, 130, 5])),
    ("f32_varlen", dict(H=1, dk=64, dv=64, in_dtype="f32", seqlens=[63, 1, 66, 0, 2])),
    # enough tokens that the forward's runs (sized to the device's wave slots)
    # are tens of tokens long and cross sequence boundaries inside a run
    ("bf16_varlen_mid", dict(H=16, dk=128, dv=128, in_dtype="bf16",
                             seqlens=[700, 1, 1333, 0, 95, 2100, 64, 513])),
]


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_prologue_parity(name, kw):
    c = prologue_case(seed=zlib.crc32(name.encode()) % 1000 + 5, **kw)
    _log("prologue %s %s" % (name, check(c)))


def test_prologue_layer_shape():
    # the 1.3B layer's q, k, v (B4 T4096 H16 d128 bf16), checked on every
    # token of two sampled heads
    c = prologue_case(seed=71, B=4, T=4096, H=16, dk=128, dv=128, in_dtype="bf16")
    ys, gr = run_gpu(c)
    heads = [3, 12]
    for i, (n, norm) in enumerate((("q", True), ("k", True), ("v", False))):
        x, w, g = (c["x" + n][:, :, heads], c["w" + n][heads], c["g" + n][:, :, heads])
        ref = prologue_fwd(x, w, norm)
        y = ys[i][:, :, heads]
        assert np.all(np.abs(y - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-5 * np.max(np.abs(ref))), n
        dx, dw = prologue_bwd(x, w, norm, g)
        assert maxrel(gr["dx" + n][:, :, heads], dx) <= 1e-5, n
        assert maxrel(gr["dw" + n][heads], dw) <= 1e-5, n


@pytest.mark.parametrize("in_dtype,dv,shape", [("bf16", 128, (2, 100, 3)), ("f32", 256, (1, 70, 2)),
                                               ("bf16", 64, (3, 5, 1)), ("bf16", 128, (4, 4096, 16))],
                         ids=["bf16_d128", "f32_d256", "bf16_d64_T5", "bf16_layer"])
def test_gate_parity(in_dtype, dv, shape):
    import torch
    import paper_2506_02475_amd as comba
    from comba_inputs import bf16_round
    from oracle.prologue import gate_bwd, gate_fwd

    rng = np.random.default_rng(dv + shape[1])
    B, T, H = shape
    o = rng.standard_normal((B, T, H, dv), dtype=np.float32)
    z = 2.0 * rng.standard_normal((B, T, H, dv), dtype=np.float32)
    dy = rng.standard_normal((B, T, H, dv), dtype=np.float32)
    if in_dtype == "bf16":
        z = bf16_round(z)
    dt = torch.bfloat16 if in_dtype == "bf16" else torch.float32
    t = lambda x, d=torch.float32: torch.from_numpy(np.ascontiguousarray(x)).to("cuda", d)
    y = comba.comba_gate_fwd(t(o), t(z, dt))
    do, dz = comba.comba_gate_bwd(t(o), t(z, dt), t(dy))
    torch.cuda.synchronize()
    ref = gate_fwd(o, z)
    y = y.float().cpu().numpy()
    if in_dtype == "bf16":
        assert np.all(np.abs(y - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-6 * np.max(np.abs(ref)))
    else:
        assert maxrel(y, ref) <= 1e-5
    rdo, rdz = gate_bwd(o, z, dy)
    assert maxrel(do.cpu().numpy(), rdo) <= 1e-5 and maxrel(dz.cpu().numpy(), rdz) <= 1e-5


def test_prologue_and_gate_without_tokens():
    # T = 0: nothing to convolve; the tap gradients are exact zeros
    import torch
    import paper_2506_02475_amd as comba

    c = prologue_case(seed=81, B=2, T=0, H=2, dk=128, dv=128, in_dtype="bf16")
    t = lambda x, d=torch.float32: torch.from_numpy(np.ascontiguousarray(x)).to("cuda", d)
    xs = [t(c[n], torch.bfloat16) for n in ("xq", "xk", "xv")]
    ws = [t(c[n]) for n in ("wq", "wk", "wv")]
    gs = [t(c[n]) for n in ("gq", "gk", "gv")]
    q, k, v = comba.comba_prologue_fwd(*xs, *ws)
    gr = comba.comba_prologue_bwd(*xs, *ws, *gs)
    o = torch.zeros((2, 0, 2, 128), device="cuda")
    y = comba.comba_gate_fwd(o, o.to(torch.bfloat16))
    do, dz = comba.comba_gate_bwd(o, o.to(torch.bfloat16), o)
    torch.cuda.synchronize()
    assert q.numel() == 0 and y.numel() == 0 and do.numel() == 0
    for n in ("dwq", "dwk", "dwv"):
        assert torch.count_nonzero(gr[n]).item() == 0, n


def test_prologue_deterministic():
    c = prologue_case(seed=82, B=1, T=300, H=2, dk=128, dv=128, in_dtype="bf16",
                      seqlens=None)
    a = run_gpu(c)
    b = run_gpu(c)
    for x, y in zip(a[0], b[0]):
        assert np.array_equal(x, y)
    for n in a[1]:
        assert np.array_equal(a[1][n], b[1][n]), n
