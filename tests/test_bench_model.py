"""The benchmark's algorithmic byte / flop models (the roofline numerators)
against per-unit figures worked out by hand for the measured shapes."""
import importlib.util
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
bench = importlib.util.module_from_spec(spec)
spec.loader.exec_module(bench)

MiB = 2.0 ** 20


def test_method_model_at_the_headline_shape():
    # the method's minimal bytes per chunk-head (C = 64, d = 128, bf16 in, fp32 out):
    # forward q, k, v 3 x 16 KiB + o 32 KiB + one fp32 state 64 KiB = 144 KiB;
    # backward q, k, v, dO 4 x 16 KiB + the state 64 KiB + dq, dk, dv 3 x 32 KiB =
    # 224 KiB; 4096 chunk-heads
    fl_f, by_f = bench.method_model("fwd_save", 4, 4096, 16, 128, 128)
    fl_b, by_b = bench.method_model("bwd", 4, 4096, 16, 128, 128)
    assert by_f == 144 * 1024 * 4096 == 603979776
    assert by_b == 224 * 1024 * 4096 == 939524096
    assert by_f + by_b == 1543503872
    # inference forward: no states kept
    assert bench.method_model("fwd", 4, 4096, 16, 128, 128)[1] == 80 * 1024 * 4096
    # flops per chunk-head: forward 2 C^2 (3 dk + 2 dv) + 6 C dk dv = 11.53 M,
    # backward 12 C^2 dk + 8 C^2 dv + 12 C dk dv + 4 C^3 = 24.12 M; 146.0 GFLOP per step
    assert fl_f == (2 * 64 * 64 * (5 * 128) + 6 * 64 * 128 * 128) * 4096
    assert fl_b == (12 * 4096 * 128 + 8 * 4096 * 128 + 12 * 64 * 128 * 128 + 4 * 64 ** 3) * 4096
    assert abs((fl_f + fl_b) / 1e9 - 146.03) < 0.01
    assert fl_f + fl_b == bench.op_flops(4, 4096, 16, 128, 128)


def test_method_model_of_packed_sequences():
    # partial chunks count their own tokens: 70 tokens = chunks of 64 and 6
    cu = [0, 70, 70, 134]
    assert bench.chunk_lengths(134, cu_seqlens=cu) == [64, 6, 64]
    fl, by = bench.method_model("fwd", 1, 134, 2, 128, 128, cu_seqlens=cu)
    assert by == 134 * 2 * (3 * 128 * 2 + 128 * 4)
    per = lambda L: 2 * L * L * 640 + 6 * L * 128 * 128
    assert fl == 2 * (2 * per(64) + per(6))
    fl, by = bench.method_model("bwd", 1, 134, 2, 128, 128, cu_seqlens=cu)
    assert by == 134 * 2 * (4 * 128 * 2 + 3 * 128 * 4) + 3 * 2 * 128 * 128 * 4


def test_roofline_credits_the_direction_of_the_kernel():
    assert bench.stage_direction("intra_bwd") == "bwd"
    assert bench.stage_direction("scan_fwd_save") == "fwd_save"
    assert bench.stage_direction("scan_fwd", saved=False) == "fwd"
    m = bench.method_model("bwd", 4, 4096, 16, 128, 128)
    r = bench.kernel_roofline("intra_bwd", 0.285, m,
                              design=bench.stage_model("intra_bwd", 4, 4096, 16, 128, 128))
    assert r["bound"] == "hbm" and r["algorithmic_bytes"] == 939524096
    assert abs(r["frac"] - 939524096 / 0.285e-3 / 8e12) < 1e-4
    assert r["design_bytes"] > r["algorithmic_bytes"]


def test_intra_bwd_design_bytes_at_the_headline_shape():
    # per chunk-head (C = 64, d = 128, bf16 in): q, k, v, dO 4 x 16 KiB; X, Y int16
    # 2 x (32 KiB + 2 KiB scales); D, dR int16 2 x (16 KiB + 1 KiB); G, beta 384 B;
    # dq, dk, dv fp32 3 x 32 KiB; dg, dbeta 512 B  ->  262.9 KiB; 4096 chunk-heads
    fl, by = bench.stage_model("intra_bwd", 4, 4096, 16, 128, 128)
    per = 4 * 16384 + 2 * (32768 + 2048) + 2 * (16384 + 1024) + 64 * 6 + 3 * 32768 + 2 * 256
    assert by == per * 4096
    assert abs(by / MiB - 1051.5) < 0.1
    assert fl == (6 * 64 * 128 * 128 + 4 * 64 * 64 * 128 + 10 * 64 * 64 * 128) * 4096


def test_separate_beta_tilde_adds_its_read_and_gradient():
    _, base = bench.stage_model("intra_bwd", 4, 4096, 16, 128, 128)
    _, sep = bench.stage_model("intra_bwd", 4, 4096, 16, 128, 128, sep_bt=True)
    assert sep - base == 64 * (2 + 4) * 4096
    _, base = bench.stage_model("scan_fwd_save", 4, 4096, 16, 128, 128)
    _, sep = bench.stage_model("scan_fwd_save", 4, 4096, 16, 128, 128, sep_bt=True)
    assert sep - base == 64 * 2 * 4096


def test_decode_bytes():
    # per head: state read + write 2 x 64 KiB, q, k, v 3 x 256 B, g 4 B, beta 2 B, o 512 B
    assert bench.decode_bytes(64, 16, 128, 128) == 1024 * (131072 + 768 + 6 + 512)


@pytest.mark.parametrize("stage,per", [("prologue_fwd", 2 * 2), ("prologue_bwd", 2 + 8)])
def test_prologue_bytes(stage, per):
    assert bench.prologue_bytes(stage, 4, 4096, 16, 128, 128) == 4 * 4096 * 16 * 384 * per


def test_only_one_gpu():
    import subprocess
    import sys

    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr
