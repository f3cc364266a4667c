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


def test_intra_bwd_bytes_at_the_headline_shape():
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
