#!/usr/bin/env python3
"""Benchmark of the chunk-wise Comba forward + backward on one MI355X.

One step = one pass of the whole hot path over one batch, as a training step
runs it: comba_chunk_fwd_save (chunk tables, gates/score matrix/UT inverse,
state scan fused with the output, keeping the chunk states for the backward)
followed by comba_chunk_bwd_saved (reverse state scan and intra-chunk
gradients).  The stateless pair comba_chunk_fwd + comba_chunk_bwd (whose
backward recomputes the forward) is timed as well and reported beside it.  Workload: the 1.3B-model
layer shape, B=4, H=16, T=4096, dk=dv=128, chunk 64, bf16 inputs, fp32 state and
outputs, seeded synthetic inputs (comba_inputs, PCG64).

Prints one JSON line with the whole-job throughput in tokens/s, the roofline of
the dominant kernel and the fp64 CPU oracle timed on this host's cores on a
bounded sample of the same workload.  The roofline credits the dominant kernel
with the method's minimal HBM bytes (and flops) of its direction: the
backward's q, k, v, dO and one fp32 state per chunk in, fp32 dq, dk, dv out
(method_model), divided by the kernel's average launch time (HIP events
recorded by the library on its launch stream over the timed region, right
before and after that kernel only, on every fourth step: timing every stage
there would add about 3% to the step); the per-stage breakdown comes from a separate pass before the
timed region (timed_steps); the bytes this design's own intermediates add are
reported beside them ("design_bytes"), and "step_roofline" holds the whole
step's method bytes and flops over the step time.  Separate forward and backward times, per-kernel MFMA
use (algorithmic, and counted by rocprofv3 where the committed counters match
the kernel source) are reported too.  Further legs timed after the headline
region under "variants": the training pair with a separate state-feedback
strength beta~ = b * beta (Section 3.2, one b per head), decoding, the
long-context packed forward, head dim 256 and the layer prologue.
"""
from __future__ import annotations

import argparse
import copy
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X published peaks
PEAK_HBM_GBS = 8000.0          # HBM3E, GB/s
PEAK_BF16_TFLOPS = 2500.0      # dense bf16 MFMA
RIDGE = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)   # flop / byte
WORKLOAD_INDEX = 3             # l1p3b_fwdbwd


def stage_model(name, B, T, H, dk, dv, C=64, in_bytes=2, sep_bt=False):
    """Algorithmic (flops, bytes) of one launch of a kernel stage.

    Per chunk-head (C tokens of one head): the dense products the stage performs
    (2 m n k flops each) and the HBM bytes it must move at minimum (each operand
    read once, each result written once; L2 re-reads excluded).  M and A count
    2 bytes per element plus one 4-byte scale per row (M) or column (A), the
    chunk states X, Y and pseudo-values D, dR handed from the scans to the
    backward gradient kernel 2 bytes per element plus one 4-byte scale per 32
    elements (their int16 storage).  The reverse scan transposes M, A and K on
    chip; the Q^T copy made by the prep stage of the training pair is counted
    where it is written and read.
    ``sep_bt``: a separate feedback strength beta~ (read where beta and beta~
    both act: the forward scan and the gradient kernel, which also writes
    dbeta~; the prep and reverse scan read beta~ in place of beta).
    """
    nch = B * math.ceil(T / C) * H
    f4 = 4
    qk = C * dk * in_bytes          # one of q, k (or its transpose)
    vv = C * dv * in_bytes          # one of v, dO
    gb = C * (f4 + in_bytes)        # g (or G) and beta
    cc = C * C * 2 + C * f4         # one stored C x C matrix (int16 + row / column scales)
    st = dk * dv * 2 + dk * (dv // 32) * f4     # one stored state (int16 + scales)
    cd = C * dv * 2 + C * (dv // 32) * f4       # one stored C x dv matrix
    if name in ("prep", "prep_save"):    # K K^T, Q K^T; q, k, g, beta -> M, A, G
        fl = 4 * C * C * dk
        by = 2 * qk + gb + 2 * cc + C * f4
        if name == "prep_save":           # + Q^T for the backward
            by += qk
    elif name in ("scan_fwd", "scan_fwd_save"):  # K X, Q X, M R, A D, K^T D
        fl = 6 * C * dk * dv + 4 * C * C * dv
        by = 2 * qk + vv + 2 * cc + gb + C * dv * f4   # q, k, v, M, A, g, beta -> o (fp32)
        if name == "scan_fwd_save":       # + chunk states X and D for the backward
            by += st + cd
        if sep_bt:
            by += C * in_bytes
    elif name == "scan_fwd_store":  # K X, M R, K^T D; -> X, D
        fl = 4 * C * dk * dv + 2 * C * C * dv
        by = qk + vv + cc + gb + st + cd
    elif name == "scan_bwd":      # K Y, A^T dO, M^T dD, Q^T Pg, K^T W2; -> Y, dR
        fl = 6 * C * dk * dv + 4 * C * C * dv
        by = 2 * qk + vv + 2 * cc + gb + st + cd      # k, Q^T, dO, M, A, g, beta
    elif name == "scans":         # the stateless backward's two scans, side by side
        f1, b1 = stage_model("scan_fwd_store", B, T, H, dk, dv, C, in_bytes, sep_bt)
        f2, b2 = stage_model("scan_bwd", B, T, H, dk, dv, C, in_bytes, sep_bt)
        return f1 + f2, b1 + b2
    elif name == "intra_bwd":     # 3 C x dk x dv, 2 C x C x dv, 5 C x C x dk products
        fl = 6 * C * dk * dv + 4 * C * C * dv + 10 * C * C * dk
        by = (2 * qk + 2 * vv + 2 * st + 2 * cd + gb          # q,k,v,dO,X,Y,D,dR
              + C * (2 * dk + dv) * f4 + 2 * C * f4)           # dq, dk, dv, dg, dbeta
        if sep_bt:
            by += C * (in_bytes + f4)                           # beta~ in, dbeta~ out
    else:
        return 0.0, 0.0
    return float(fl * nch), float(by * nch)


def op_flops(B, T, H, dk, dv, C=64):
    """Algorithmic fwd+bwd flops of the chunk-wise method (no recomputation)."""
    nch = B * math.ceil(T / C) * H
    fwd = 2 * C * C * (3 * dk + 2 * dv) + 6 * C * dk * dv
    bwd = 12 * C * C * dk + 8 * C * C * dv + 12 * C * dk * dv + 4 * C ** 3
    return float((fwd + bwd) * nch)


# Stages of the forward and of the backward direction (the names the library's
# stage timing records)
FWD_STAGES = ("chunk_map", "prep", "prep_save", "scan_fwd", "scan_fwd_save")
BWD_STAGES = ("scan_fwd_store", "scan_bwd", "scans", "intra_bwd", "reduce_dd")


def chunk_lengths(T, B=1, cu_seqlens=None, C=64):
    """Token counts of every chunk of every sequence (one head)."""
    import numpy as np

    if cu_seqlens is None:
        lens = [T] * B
    else:
        cu = np.asarray(cu_seqlens, dtype=np.int64)
        lens = list(cu[1:] - cu[:-1])
    out = []
    for n in lens:
        n = int(n)
        out += [C] * (n // C) + ([n % C] if n % C else [])
    return out


def method_model(direction, B, T, H, dk, dv, C=64, in_bytes=2, cu_seqlens=None):
    """Algorithmic (flops, bytes) of the chunk-wise method itself for one
    direction over the whole batch, independent of how the kernels are split.

    Bytes (minimal HBM traffic, fp32 outputs): the forward reads q, k, v and
    writes o ("fwd", inference); "fwd_save" also writes one fp32 dk x dv state
    per chunk for the backward; "bwd" reads q, k, v, dO and the per-chunk
    states and writes dq, dk, dv.  Gates, beta and the gradients of per-token
    scalars (4-6 bytes per token-head) and the h0/ht/dht/dh0 states of each
    sequence are left out (below 0.3% at the 1.3B layer shape).
    Flops, per chunk of L tokens (the dense products of the chunk form): forward
    2 L^2 (3 dk + 2 dv) + 6 L dk dv (K K^T, Q K^T, W, U, the masked score
    product; W H, Q H and the state update); backward 12 L^2 dk + 8 L^2 dv +
    12 L dk dv + 4 L^3.
    """
    lens = chunk_lengths(T, B, cu_seqlens, C)
    tok = sum(lens) * H
    nch = len(lens) * H
    if direction in ("fwd", "fwd_save"):
        by = tok * ((2 * dk + dv) * in_bytes + dv * 4)
        if direction == "fwd_save":
            by += nch * dk * dv * 4
        fl = sum(2 * L * L * (3 * dk + 2 * dv) + 6 * L * dk * dv for L in lens) * H
    elif direction == "bwd":
        by = tok * ((2 * dk + 2 * dv) * in_bytes + (2 * dk + dv) * 4) + nch * dk * dv * 4
        fl = sum(12 * L * L * dk + 8 * L * L * dv + 12 * L * dk * dv + 4 * L ** 3
                 for L in lens) * H
    else:
        raise ValueError(direction)
    return float(fl), float(by)


def stage_direction(name, saved=True):
    if name in BWD_STAGES:
        return "bwd"
    if name in FWD_STAGES:
        return "fwd_save" if saved else "fwd"
    raise ValueError(name)


def kernel_roofline(kernel, avg_ms, method, design=None, traffic=None, mfma_counted=None):
    """Roofline of one kernel: the method's (flops, bytes) of the direction the
    kernel belongs to, divided by the kernel's average launch time (each
    launch covers the whole batch), against the MI355X peak of the bound it
    falls under.  ``design`` (flops, bytes) are what the kernel itself moves and
    computes in this design (its own intermediates included), kept beside the
    method figures; ``traffic`` the HBM bytes per launch measured by counters."""
    fl, by = method
    sec = avg_ms * 1e-3
    if fl / by < RIDGE:
        ach = by / sec / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(ach / PEAK_HBM_GBS, 4)}
    else:
        ach = fl / sec / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4)}
    roof.update({"traffic": traffic, "kernel": kernel, "avg_launch_ms": round(avg_ms, 4),
                 "algorithmic_bytes": by, "algorithmic_flops": fl})
    if design is not None:
        dfl, dby = design
        roof["design_bytes"] = dby
        roof["design_flops"] = dfl
        roof["design_frac_hbm"] = round(dby / sec / 1e9 / PEAK_HBM_GBS, 4)
        roof["mfma_pct_algorithmic"] = round(100.0 * dfl / sec / (PEAK_BF16_TFLOPS * 1e12), 3)
    if mfma_counted is not None:
        roof["mfma_pct_counted"] = round(100.0 * mfma_counted / sec / (PEAK_BF16_TFLOPS * 1e12), 3)
    return roof


def kernel_source_sha(files=("comba_kernels.hip", "comba_device.hpp")):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2506_02475_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


DECODE_SOURCES = ("comba_recurrent.hip", "comba_device.hpp")


def measured_traffic(kernel, summary="traffic_counters_l1p3b_fwdbwd.md",
                     sources=("comba_kernels.hip", "comba_device.hpp")):
    """HBM bytes per launch of a kernel stage from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary (scaled by a plain copy of known size), if
    the counters were taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", summary)
    try:
        with open(path) as f:
            text = f.read()
        rec = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    except (OSError, ValueError, IndexError):
        return None
    if rec.get("source_sha") != kernel_source_sha(sources):
        return None
    k = rec.get("kernels", {}).get(kernel)
    if not k:
        return None
    return round(float(k["bytes_per_launch"]))


def measured_mfma(kernel, summary="mfma_counters_l1p3b_fwdbwd.md",
                  sources=("comba_kernels.hip", "comba_device.hpp")):
    """MFMA flops per launch of a kernel stage counted by rocprofv3
    (SQ_INSTS_VALU_MFMA_MOPS_*, every MFMA the kernel issues, split products
    and recomputation included), from the committed summary, if it was taken
    on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", summary)
    try:
        with open(path) as f:
            text = f.read()
        rec = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    except (OSError, ValueError, IndexError):
        return None
    if rec.get("source_sha") != kernel_source_sha(sources):
        return None
    k = rec.get("kernels", {}).get(kernel)
    return None if not k else float(k["mfma_flops_per_launch"])


DECODE = dict(B=64, H=16, dk=128, dv=128, layers=8, seed=47)


def decode_bytes(B, H, dk, dv, in_bytes=2):
    """Algorithmic HBM bytes of one decoding call (T = 1, states updated in place):
    every state read and written once (fp32), q, k, v, g, beta read, o written."""
    per_head = 2 * dk * dv * 4 + (2 * dk + dv) * in_bytes + 4 + in_bytes + dv * 4
    return float(B * H * per_head)


def time_decode(comba, torch, steps, warmup, threads=None, with_cpu=False):
    """Decoding step of one layer: one token for each of B sequences through
    comba_recurrent_fwd, states updated in place.  The timed loop cycles over
    the states of DECODE['layers'] layers (512 MiB at the default shape, more
    than the 256 MB on-die cache), as a model's layers would."""
    import numpy as np
    import oracle
    from comba_inputs import random_case

    c = DECODE
    w = random_case(seed=c["seed"], B=c["B"], T=1, H=c["H"], dk=c["dk"], dv=c["dv"],
                    in_dtype="bf16", grad=False)
    dev = torch.device("cuda:0")
    bf = torch.bfloat16

    def t(x, dt=torch.float32):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev, dt)

    q, k, v, g, beta, d = t(w.q, bf), t(w.k, bf), t(w.v, bf), t(w.g), t(w.beta, bf), t(w.d)
    h0 = t(w.h0)
    states = [h0.clone() for _ in range(c["layers"])]

    def call(st):
        return comba.comba_recurrent_fwd(q, k, v, g, beta, d, st, ht=st)

    for _ in range(warmup):
        for st in states:
            call(st)
    torch.cuda.synchronize()
    # the timed calls go straight through the C ABI with their arguments
    # marshalled beforehand: a decoding call is shorter than the binding's
    # per-call checks, which would otherwise leave the GPU waiting between calls
    import ctypes
    lib = comba.load_library()
    shp = comba.CombaShape(c["B"], 1, c["H"], c["dk"], c["dv"], comba.CHUNK, c["B"], None, None,
                           comba.COMBA_BF16)
    o = torch.empty((c["B"], 1, c["H"], c["dv"]), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    P = ctypes.c_void_p
    fixed = [P(x.data_ptr()) for x in (q, k, v, g, beta)] + [None, P(d.data_ptr())]
    argv = [[ctypes.byref(shp)] + fixed + [P(st.data_ptr()), P(o.data_ptr()), P(st.data_ptr()),
                                            P(stream.cuda_stream)] for st in states]
    fn = lib.comba_recurrent_fwd
    for a in argv:
        assert fn(*a) == 0
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        for a in argv:
            fn(*a)
    e1.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ncalls = steps * len(states)
    ms_call = (t1 - t0) * 1e3 / ncalls
    # average launch duration: HIP events on the launch stream around the
    # back-to-back calls (each launch is one kernel)
    kms = e0.elapsed_time(e1) / ncalls
    by = decode_bytes(c["B"], c["H"], c["dk"], c["dv"])
    achieved = by / (kms * 1e-3) / 1e9
    res = {"value": round(c["B"] / (ms_call * 1e-3), 1), "unit": "tokens/s (one layer)",
           "ms_per_call": round(ms_call, 5), "config": {k_: c[k_] for k_ in ("B", "H", "dk", "dv",
                                                                             "layers")},
           "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                        "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                        "traffic": measured_traffic("recurrent",
                                                    "traffic_counters_decode_b64_h16_d128.md",
                                                    DECODE_SOURCES),
                        "kernel": "recurrent", "avg_launch_ms": round(kms, 5),
                        "algorithmic_bytes": by}}
    if with_cpu:
        reps = 0
        t0 = time.perf_counter()
        while True:
            oracle.workload_fwd(w, nthreads=threads)
            reps += 1
            if time.perf_counter() - t0 > 2.0:
                break
        dt = (time.perf_counter() - t0) / reps
        res["cpu_baseline"] = {"value": c["B"] / dt, "unit": "tokens/s (one layer)",
                               "cores": threads, "kind": "oracle",
                               "sample": "fp64 step recurrence on the whole decoding call "
                                         "(%d sequences x %d heads, T = 1), %d repetitions"
                                         % (c["B"], c["H"], reps)}
    return res


PREFILL256 = dict(B=4, T=4096, H=8, dk=256, dv=256, seed=63)


def timed_steps(comba, torch, step, steps, sample_every=4):
    """The timing protocol of every leg (after its warm-up).  First a stage
    pass: `steps` steps with a HIP event on the launch stream before every
    kernel stage, which gives each stage's average launch duration and picks
    the dominant stage (largest time per step); its step time is not reported.
    Then the timed region: `steps` steps bracketed by device synchronisations,
    in which every `sample_every`-th step records events right before and right
    after the dominant stage only (comba_profile_select; the other steps record
    none), so the stages run back to back as they do without timing, and the
    dominant stage's duration is still measured live over the timed region.
    (An event pair costs the step about 9 us of idle GPU, 1.2% at the 1.3B
    shape; every stage marked costs 3%.)"""
    torch.cuda.synchronize()
    comba.profile_select(None)
    comba.profile_enable(True)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    marks = comba.profile_read()
    comba.profile_enable(False)
    tot, cnt = {}, {}
    for name, ms in marks:
        tot[name] = tot.get(name, 0.0) + ms
        cnt[name] = cnt.get(name, 0) + 1
    dom = max(tot, key=tot.get)
    comba.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        # a name no stage has: that step records nothing
        comba.profile_select(dom if i % sample_every == 0 else "-")
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    live = [ms for name, ms in comba.profile_read() if name == dom]
    comba.profile_enable(False)
    comba.profile_select(None)
    return {"ms_per_step": (t1 - t0) * 1e3 / steps,
            "stages_ms": {n: x / steps for n, x in tot.items()},
            "stage_avg_ms": {n: tot[n] / cnt[n] for n in tot},
            "dominant": dom, "dom_avg_ms": sum(live) / len(live), "dom_launches_timed": len(live)}


def time_train256(comba, torch, steps, warmup):
    """Training pair (comba_chunk_fwd_save + comba_chunk_bwd_saved) at head dim 256:
    B4 T4096 H8 d256 bf16.  Per-stage live timing; roofline of the dominant stage."""
    import numpy as np
    from comba_inputs import random_case

    c = PREFILL256
    w = random_case(seed=c["seed"] + 1, B=c["B"], T=c["T"], H=c["H"], dk=c["dk"], dv=c["dv"],
                    in_dtype="bf16", grad=True)
    dev = torch.device("cuda:0")
    bf = torch.bfloat16

    def t(x, dt=torch.float32):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev, dt)

    q, k, v, g, beta, d, h0, dO = (t(w.q, bf), t(w.k, bf), t(w.v, bf), t(w.g), t(w.beta, bf),
                                   t(w.d), t(w.h0), t(w.dO, bf))
    B, T, H, dk, dv = c["B"], c["T"], c["H"], c["dk"], c["dv"]
    ws = torch.empty(comba.bwd_workspace_bytes(B, T, H, dk, dv), dtype=torch.uint8, device=dev)

    def step():
        comba.comba_chunk_fwd_save(q, k, v, g, beta, d, h0, workspace=ws)
        return comba.comba_chunk_bwd_saved(q, k, v, g, beta, d, h0, dO, None, workspace=ws)

    for _ in range(warmup):
        step()
    tm = timed_steps(comba, torch, step, steps)
    dom, ms_step, tot = tm["dominant"], tm["ms_per_step"], tm["stages_ms"]
    roof = kernel_roofline(dom, tm["dom_avg_ms"],
                           method_model(stage_direction(dom), B, T, H, dk, dv),
                           design=stage_model(dom, B, T, H, dk, dv),
                           traffic=measured_traffic(dom, TRAIN256_TRAFFIC))
    return {"value": round(B * T / (ms_step * 1e-3), 1), "unit": "tokens/s",
            "ms_per_step": round(ms_step, 4),
            "ms_fwd": round(sum(x for n, x in tot.items() if n in FWD_STAGES), 4),
            "ms_bwd": round(sum(x for n, x in tot.items() if n in BWD_STAGES), 4),
            "config": {k_: c[k_] for k_ in ("B", "T", "H", "dk", "dv")},
            "stages_ms": {n: round(x, 4) for n, x in tot.items()},
            "roofline": roof}


TRAIN256_TRAFFIC = "traffic_counters_train_b4_t4096_h8_d256.md"
PREFILL256_TRAFFIC = "traffic_counters_prefill_b4_t4096_h8_d256.md"


def time_prefill256(comba, torch, steps, warmup):
    """Inference prefill at head dim 256 (the paper's models): the stateless
    comba_chunk_fwd over B4 T4096 with 8 heads of 256 (a 1.3B-model layer with
    the heads of 128 merged pairwise).  Per-stage live timing as in the
    headline; the roofline is that of the dominant stage."""
    import numpy as np
    from comba_inputs import random_case

    c = PREFILL256
    w = random_case(seed=c["seed"], B=c["B"], T=c["T"], H=c["H"], dk=c["dk"], dv=c["dv"],
                    in_dtype="bf16", grad=False)
    dev = torch.device("cuda:0")
    bf = torch.bfloat16

    def t(x, dt=torch.float32):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev, dt)

    q, k, v, g, beta, d, h0 = (t(w.q, bf), t(w.k, bf), t(w.v, bf), t(w.g), t(w.beta, bf),
                               t(w.d), t(w.h0))
    B, T, H, dk, dv = c["B"], c["T"], c["H"], c["dk"], c["dv"]
    ws = torch.empty(comba.fwd_workspace_bytes(B, T, H, dk, dv), dtype=torch.uint8, device=dev)
    def call():
        return comba.comba_chunk_fwd(q, k, v, g, beta, d, h0, workspace=ws)

    for _ in range(warmup):
        call()
    tm = timed_steps(comba, torch, call, steps)
    dom, ms_step, tot = tm["dominant"], tm["ms_per_step"], tm["stages_ms"]
    roof = kernel_roofline(dom, tm["dom_avg_ms"],
                           method_model(stage_direction(dom, saved=False), B, T, H, dk, dv),
                           design=stage_model(dom, B, T, H, dk, dv),
                           traffic=measured_traffic(dom, PREFILL256_TRAFFIC))
    return {"value": round(B * T / (ms_step * 1e-3), 1), "unit": "tokens/s",
            "ms_per_step": round(ms_step, 4),
            "config": {k_: c[k_] for k_ in ("B", "T", "H", "dk", "dv")},
            "stages_ms": {n: round(x, 4) for n, x in tot.items()},
            "roofline": roof}


VARLEN_TRAFFIC = "traffic_counters_varlen_512k_fwd.md"


def time_varlen(comba, torch, steps, warmup):
    """Long-context packed forward: 16 sequences of U[1024, 65536] tokens
    (525,868 in total) x 16 heads x d = 128, bf16 inputs, per-sequence fp32
    initial and final states, through the stateless comba_chunk_fwd (the
    inference form: no chunk states are kept).  Per-stage live timing; the
    roofline is that of the dominant stage, credited the forward's method
    bytes (q, k, v in, o out)."""
    import numpy as np
    from comba_inputs import WORKLOADS, generate

    spec = WORKLOADS[4]
    w = generate(4)
    dev = torch.device("cuda:0")
    bf = torch.bfloat16

    def t(x, dt=torch.float32):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev, dt)

    q, k, v = t(w.q, bf), t(w.k, bf), t(w.v, bf)
    g, beta, d, h0 = t(w.g), t(w.beta, bf), t(w.d), t(w.h0)
    cu = torch.from_numpy(w.cu_seqlens.astype(np.int32)).to(dev)
    cu_host = w.cu_seqlens.astype(np.int32)
    N, T, H, dk, dv = w.nseq, w.T, w.H, w.dk, w.dv
    del w
    ws = torch.empty(comba.fwd_workspace_bytes(1, T, H, dk, dv, num_seqs=N, varlen=True),
                     dtype=torch.uint8, device=dev)

    def call():
        return comba.comba_chunk_fwd(q, k, v, g, beta, d, h0, cu_seqlens=cu,
                                     cu_seqlens_host=cu_host, workspace=ws)

    for _ in range(warmup):
        call()
    tm = timed_steps(comba, torch, call, steps)
    dom, ms_step, tot = tm["dominant"], tm["ms_per_step"], tm["stages_ms"]
    fwd = method_model("fwd", 1, T, H, dk, dv, cu_seqlens=cu_host)
    roof = kernel_roofline(dom, tm["dom_avg_ms"], fwd,
                           traffic=measured_traffic(dom, VARLEN_TRAFFIC))
    lens = np.diff(cu_host)
    return {"value": round(T / (ms_step * 1e-3), 1), "unit": "tokens/s",
            "ms_per_step": round(ms_step, 4),
            "config": {"N": int(N), "T_total": int(T), "H": H, "dk": dk, "dv": dv,
                       "longest": int(lens.max()), "shortest": int(lens.min())},
            "workload": spec.name,
            "stages_ms": {n: round(x, 4) for n, x in tot.items()},
            "step_roofline": {"method_bytes": fwd[1],
                              "frac_hbm": round(fwd[1] / (ms_step * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                              "method_flops": fwd[0],
                              "mfma_pct": round(100.0 * fwd[0] / (ms_step * 1e-3) /
                                                (PEAK_BF16_TFLOPS * 1e12), 3)},
            "roofline": roof}


def time_long1(comba, torch, steps, warmup):
    """One long sequence: the long-context workload's tokens (config 4's 16
    packed sequences, 525,868 tokens, H16 d128 bf16) cut to 525,824 tokens (a
    whole number of chunks) and run as ONE sequence through the stateless
    comba_chunk_fwd with its initial state.  The scan then has only H x dv/32 =
    64 chains for 256 CUs, so the forward cuts the sequence into segments
    (segmented scan, COMBA_SCAN_SEGMENTS unset); the same call with
    COMBA_SCAN_SEGMENTS=1 (one chain per slice over the whole sequence) is
    timed beside it.  The roofline credits the dominant stage with the
    forward's method bytes."""
    import numpy as np
    from comba_inputs import generate

    w = generate(4)
    dev = torch.device("cuda:0")
    bf = torch.bfloat16
    T = (w.T // 512) * 512       # whole chunks, divisible into up to 8 segments
    H, dk, dv = w.H, w.dk, w.dv

    def t(x, dt=torch.float32):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev, dt)

    q, k, v = t(w.q[:, :T], bf), t(w.k[:, :T], bf), t(w.v[:, :T], bf)
    g, beta, d = t(w.g[:, :T]), t(w.beta[:, :T], bf), t(w.d)
    h0 = t(w.h0[:1])
    del w
    old = os.environ.get("COMBA_SCAN_SEGMENTS")
    out = {}
    try:
        for mode, env in (("segmented", None), ("plain", "1")):
            if env is None:
                os.environ.pop("COMBA_SCAN_SEGMENTS", None)
            else:
                os.environ["COMBA_SCAN_SEGMENTS"] = env
            ws = torch.empty(comba.fwd_workspace_bytes(1, T, H, dk, dv), dtype=torch.uint8,
                             device=dev)

            def call():
                return comba.comba_chunk_fwd(q, k, v, g, beta, d, h0, workspace=ws)

            for _ in range(warmup):
                call()
            out[mode] = timed_steps(comba, torch, call, steps)
            del ws
    finally:
        if old is None:
            os.environ.pop("COMBA_SCAN_SEGMENTS", None)
        else:
            os.environ["COMBA_SCAN_SEGMENTS"] = old
    tm = out["segmented"]
    fwd = method_model("fwd", 1, T, H, dk, dv)
    roof = kernel_roofline(tm["dominant"], tm["dom_avg_ms"], fwd)
    ms = tm["ms_per_step"]
    return {"value": round(T / (ms * 1e-3), 1), "unit": "tokens/s", "ms_per_step": round(ms, 4),
            "config": {"B": 1, "T": T, "H": H, "dk": dk, "dv": dv},
            "stages_ms": {n: round(x, 4) for n, x in tm["stages_ms"].items()},
            "plain_ms_per_step": round(out["plain"]["ms_per_step"], 4),
            "plain_stages_ms": {n: round(x, 4) for n, x in out["plain"]["stages_ms"].items()},
            "speedup_vs_plain": round(out["plain"]["ms_per_step"] / ms, 3),
            "step_roofline": {"method_bytes": fwd[1],
                              "frac_hbm": round(fwd[1] / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)},
            "roofline": roof}


def time_long1_train(comba, torch, steps, warmup):
    """Training pair (comba_chunk_fwd_save + comba_chunk_bwd_saved) on one long
    sequence: B1 T65536 H16 d128 bf16 (the 1.3B layer's heads, its input
    distributions), with the segmented scans (both scans of the pair cut into
    segments; 64 chains otherwise) and, timed beside it, with
    COMBA_SCAN_SEGMENTS=1."""
    import numpy as np
    from comba_inputs import random_case

    B, T, H, dk, dv = 1, 65536, 16, 128, 128
    w = random_case(seed=83, B=B, T=T, H=H, dk=dk, dv=dv, in_dtype="bf16", grad=True)
    dev = torch.device("cuda:0")
    bf = torch.bfloat16

    def t(x, dt=torch.float32):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev, dt)

    q, k, v, g, beta, d, h0, dO = (t(w.q, bf), t(w.k, bf), t(w.v, bf), t(w.g), t(w.beta, bf),
                                   t(w.d), t(w.h0), t(w.dO, bf))
    del w
    old = os.environ.get("COMBA_SCAN_SEGMENTS")
    out = {}
    try:
        for mode, env in (("segmented", None), ("plain", "1")):
            if env is None:
                os.environ.pop("COMBA_SCAN_SEGMENTS", None)
            else:
                os.environ["COMBA_SCAN_SEGMENTS"] = env
            ws = torch.empty(comba.bwd_workspace_bytes(B, T, H, dk, dv), dtype=torch.uint8,
                             device=dev)

            def step():
                comba.comba_chunk_fwd_save(q, k, v, g, beta, d, h0, workspace=ws)
                return comba.comba_chunk_bwd_saved(q, k, v, g, beta, d, h0, dO, None,
                                                   workspace=ws)

            for _ in range(warmup):
                step()
            out[mode] = timed_steps(comba, torch, step, steps)
            del ws
    finally:
        if old is None:
            os.environ.pop("COMBA_SCAN_SEGMENTS", None)
        else:
            os.environ["COMBA_SCAN_SEGMENTS"] = old
    tm = out["segmented"]
    ms = tm["ms_per_step"]
    return {"value": round(B * T / (ms * 1e-3), 1), "unit": "tokens/s", "ms_per_step": round(ms, 4),
            "config": {"B": B, "T": T, "H": H, "dk": dk, "dv": dv},
            "step": "comba_chunk_fwd_save + comba_chunk_bwd_saved",
            "stages_ms": {n: round(x, 4) for n, x in tm["stages_ms"].items()},
            "plain_ms_per_step": round(out["plain"]["ms_per_step"], 4),
            "plain_stages_ms": {n: round(x, 4) for n, x in out["plain"]["stages_ms"].items()},
            "speedup_vs_plain": round(out["plain"]["ms_per_step"] / ms, 3)}


PROLOGUE = dict(B=4, T=4096, H=16, dk=128, dv=128, seed=71)
PROLOGUE_SOURCES = ("comba_prologue.hip", "comba_device.hpp")
PROLOGUE_TRAFFIC = "traffic_counters_prologue_b4_t4096_h16_d128.md"


def prologue_bytes(stage, B, T, H, dk, dv, in_bytes=2):
    """Algorithmic HBM bytes of one prologue launch: the forward reads x and
    writes q, k, v (in_dtype); the backward reads x (in_dtype) and the fp32
    gradients of q, k, v and writes fp32 dx (taps and dw are negligible)."""
    n = B * T * H * (2 * dk + dv)
    return float(n * 2 * in_bytes if stage == "prologue_fwd" else n * (in_bytes + 8))


def time_prologue(comba, torch, steps, warmup):
    """Layer input prologue (short conv, SiLU, L2 norm) forward + backward on the
    1.3B layer's q, k, v (B4 T4096 H16 d128 bf16)."""
    import numpy as np
    from comba_inputs import prologue_case

    c = PROLOGUE
    pc = prologue_case(seed=c["seed"], B=c["B"], T=c["T"], H=c["H"], dk=c["dk"], dv=c["dv"],
                       in_dtype="bf16")
    dev = torch.device("cuda:0")

    def t(x, dt=torch.float32):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev, dt)

    xs = [t(pc[n], torch.bfloat16) for n in ("xq", "xk", "xv")]
    ws = [t(pc[n]) for n in ("wq", "wk", "wv")]
    gs = [t(pc[n]) for n in ("gq", "gk", "gv")]
    wsp = None

    def step():
        nonlocal wsp
        comba.comba_prologue_fwd(*xs, *ws)
        out = comba.comba_prologue_bwd(*xs, *ws, *gs, workspace=wsp)
        return out

    for _ in range(warmup):
        step()
    tm = timed_steps(comba, torch, step, steps)
    ms_step, tot = tm["ms_per_step"], tm["stages_ms"]
    roof = {}
    for st in ("prologue_fwd", "prologue_bwd"):
        # the dominant stage live over the timed region, the other from the stage pass
        avg = tm["dom_avg_ms"] if st == tm["dominant"] else tm["stage_avg_ms"][st]
        by = prologue_bytes(st, c["B"], c["T"], c["H"], c["dk"], c["dv"])
        ach = by / (avg * 1e-3) / 1e9
        roof[st] = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
                    "traffic": measured_traffic(st, PROLOGUE_TRAFFIC, PROLOGUE_SOURCES),
                    "kernel": st, "avg_launch_ms": round(avg, 4), "algorithmic_bytes": by}
    # the output gate on the operator's output shape (o fp32, z bf16): stream
    # events around back-to-back calls
    n = c["B"] * c["T"] * c["H"] * c["dv"]
    o = torch.randn(c["B"], c["T"], c["H"], c["dv"], device=dev)
    z = torch.randn(c["B"], c["T"], c["H"], c["dv"], device=dev).to(torch.bfloat16)
    dy = torch.randn_like(o)
    gate = {}
    for name, fn, by in (("gate_fwd", lambda: comba.comba_gate_fwd(o, z), n * 8.0),
                         ("gate_bwd", lambda: comba.comba_gate_bwd(o, z, dy), n * 18.0)):
        for _ in range(warmup):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        gate[name] = {"ms": round(ms, 4), "achieved_GBs": round(by / (ms * 1e-3) / 1e9, 1),
                      "frac": round(by / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4), "bytes": by}
    return {"value": round(c["B"] * c["T"] / (ms_step * 1e-3), 1), "unit": "tokens/s",
            "ms_per_step": round(ms_step, 4),
            "config": {k_: c[k_] for k_ in ("B", "T", "H", "dk", "dv")},
            "stages_ms": {n_: round(x, 4) for n_, x in tot.items()},
            "roofline": roof["prologue_bwd"], "roofline_fwd": roof["prologue_fwd"], "gate": gate}


def calibration_copy(torch, nbytes):
    """One plain device-to-device copy of ``nbytes`` (its HBM traffic counters
    calibrate those of the kernels in the same profiled run); returns the size."""
    n = nbytes // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    return n * 4


def cpu_baseline(w, heads_sample, threads):
    import oracle

    t0 = time.perf_counter()
    oracle.workload_fwd(w, heads=heads_sample, nthreads=threads)
    oracle.workload_bwd(w, heads=heads_sample, nthreads=threads)
    dt = time.perf_counter() - t0
    tokens = w.B * w.T * len(heads_sample) / w.H   # layer-equivalent tokens
    return {"value": tokens / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": "fp64 step recurrence fwd+bwd on %d of %d heads x all %d rows x T=%d "
                      "(%.1f s wall), scaled to the full layer" % (len(heads_sample), w.H, w.B,
                                                                  w.T, dt)}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--skip-stateless", action="store_true",
                    help="time only the training pair (profiling runs: one stage per kernel)")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the timed variant legs (separate feedback strength beta~)")
    ap.add_argument("--beta-tilde", action="store_true",
                    help="time the workload with beta~ = b * beta as the headline (profiling "
                         "runs of that variant; implies --no-variants)")
    ap.add_argument("--decode", action="store_true",
                    help="time the decoding step (comba_recurrent_fwd, T = 1, B = 64, H = 16, "
                         "d = 128, in place) as the headline instead of the training pair")
    ap.add_argument("--varlen", action="store_true",
                    help="time the long-context packed forward (16 sequences, 525,868 tokens, "
                         "H16 d128, comba_chunk_fwd) as the headline")
    ap.add_argument("--prefill256", action="store_true",
                    help="time the inference prefill at head dim 256 (comba_chunk_fwd, B4 T4096 "
                         "H8 d256) as the headline")
    ap.add_argument("--train256", action="store_true",
                    help="time the training pair at head dim 256 (B4 T4096 H8 d256) as the headline")
    ap.add_argument("--long1", action="store_true",
                    help="time one long sequence (the long-context workload's 525,824 tokens as "
                         "one row, H16 d128, comba_chunk_fwd, segmented scan vs plain) as the "
                         "headline")
    ap.add_argument("--prologue", action="store_true",
                    help="time the layer input prologue (short conv, SiLU, L2 norm; fwd + bwd) "
                         "on the 1.3B layer's q, k, v as the headline")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="after the timed steps, run one plain device-to-device copy of this "
                         "many bytes (calibrates HBM traffic counters against a known size)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this benchmark runs on exactly one GPU (the operator is measured "
              "on one MI355X); got --gpus %d, WORLD_SIZE %d" % (args.gpus, world),
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2506_02475_amd as comba
    from comba_inputs import WORKLOADS, attach_beta_tilde, generate

    try:
        threads = len(os.sched_getaffinity(0))
    except Exception:
        threads = os.cpu_count() or 1
    if args.train256:
        torch.cuda.set_device(0)
        r = time_train256(comba, torch, args.steps, args.warmup)
        result = {
            "metric": "Comba fwd+bwd tokens/s at B=4,T=4096,H=8,d=256 bf16 (training pair)",
            "value": r["value"], "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": r["ms_per_step"], "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded PCG64, comba_inputs.random_case)",
            "config": {"workload": "train_b4_t4096_h8_d256", **r["config"]},
            "step": "comba_chunk_fwd_save + comba_chunk_bwd_saved", "stages_ms": r["stages_ms"],
            "roofline": r["roofline"], "cpu_baseline": None}
        if args.copy_bytes > 0:
            result["copy_bytes"] = calibration_copy(torch, args.copy_bytes)
        print(json.dumps(result), flush=True)
        return
    if args.prologue:
        torch.cuda.set_device(0)
        r = time_prologue(comba, torch, args.steps, args.warmup)
        result = {
            "metric": "Comba layer prologue (conv4, SiLU, L2 norm) fwd+bwd tokens/s at "
                      "B=4,T=4096,H=16,d=128 bf16",
            "value": r["value"], "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": r["ms_per_step"], "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded PCG64, comba_inputs.prologue_case)",
            "config": {"workload": "prologue_b4_t4096_h16_d128", **r["config"]},
            "step": "comba_prologue_fwd + comba_prologue_bwd", "stages_ms": r["stages_ms"],
            "roofline": r["roofline"], "roofline_fwd": r["roofline_fwd"], "gate": r["gate"],
            "cpu_baseline": None}
        if args.copy_bytes > 0:
            result["copy_bytes"] = calibration_copy(torch, args.copy_bytes)
        print(json.dumps(result), flush=True)
        return
    if args.long1:
        torch.cuda.set_device(0)
        r = time_long1(comba, torch, args.steps, args.warmup)
        r["train"] = time_long1_train(comba, torch, args.steps, args.warmup)
        result = {
            "metric": "Comba forward tokens/s on one long sequence (525,824 tokens, H=16, d=128 "
                      "bf16; segmented scan)",
            "value": r["value"], "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": r["ms_per_step"], "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded PCG64, comba_inputs.generate(4) as one sequence)",
            "config": {"workload": "long1_525k_fwd", **r["config"]}, "step": "comba_chunk_fwd",
            "stages_ms": r["stages_ms"], "plain_ms_per_step": r["plain_ms_per_step"],
            "speedup_vs_plain": r["speedup_vs_plain"], "roofline": r["roofline"],
            "step_roofline": r["step_roofline"], "train_65k": r["train"], "cpu_baseline": None}
        if args.copy_bytes > 0:
            result["copy_bytes"] = calibration_copy(torch, args.copy_bytes)
        print(json.dumps(result), flush=True)
        return
    if args.varlen:
        torch.cuda.set_device(0)
        r = time_varlen(comba, torch, args.steps, args.warmup)
        result = {
            "metric": "Comba long-context packed forward tokens/s (16 sequences, 525,868 tokens, "
                      "H=16, d=128 bf16)",
            "value": r["value"], "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": r["ms_per_step"], "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded PCG64, comba_inputs.generate(4))",
            "config": {"workload": r["workload"], **r["config"]}, "step": "comba_chunk_fwd",
            "stages_ms": r["stages_ms"], "roofline": r["roofline"],
            "step_roofline": r["step_roofline"], "cpu_baseline": None}
        if args.copy_bytes > 0:
            result["copy_bytes"] = calibration_copy(torch, args.copy_bytes)
        print(json.dumps(result), flush=True)
        return
    if args.prefill256:
        torch.cuda.set_device(0)
        r = time_prefill256(comba, torch, args.steps, args.warmup)
        result = {
            "metric": "Comba prefill tokens/s (stateless forward) at B=4,T=4096,H=8,d=256 bf16",
            "value": r["value"], "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": r["ms_per_step"], "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded PCG64, comba_inputs.random_case)",
            "config": {"workload": "prefill_b4_t4096_h8_d256", **r["config"]},
            "step": "comba_chunk_fwd", "stages_ms": r["stages_ms"], "roofline": r["roofline"],
            "cpu_baseline": None}
        if args.copy_bytes > 0:
            result["copy_bytes"] = calibration_copy(torch, args.copy_bytes)
        print(json.dumps(result), flush=True)
        return
    if args.decode:
        torch.cuda.set_device(0)
        r = time_decode(comba, torch, args.steps, args.warmup, threads,
                        with_cpu=not args.no_cpu_baseline)
        c = DECODE
        result = {
            "metric": "Comba decoding tokens/s per layer (T=1, states in place) at B=64,H=16,d=128 "
                      "bf16",
            "value": r["value"], "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(r["ms_per_call"] * c["layers"], 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded PCG64, comba_inputs.random_case)",
            "config": {"workload": "decode_b64_h16_d128", **r["config"]},
            "step": "comba_recurrent_fwd on each of %d layers' states" % c["layers"],
            "ms_per_call": r["ms_per_call"], "roofline": r["roofline"],
            "cpu_baseline": r.get("cpu_baseline")}
        if args.copy_bytes > 0:
            result["copy_bytes"] = calibration_copy(torch, args.copy_bytes)
        print(json.dumps(result), flush=True)
        return

    spec = WORKLOADS[WORKLOAD_INDEX]
    w = generate(WORKLOAD_INDEX)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    bf = torch.bfloat16

    def t(x, dt=torch.float32):
        return None if x is None else torch.from_numpy(np.ascontiguousarray(x)).to(dev, dt)

    q, k, v = t(w.q, bf), t(w.k, bf), t(w.v, bf)
    g, beta, d, h0 = t(w.g), t(w.beta, bf), t(w.d), t(w.h0)
    dO = t(w.dO, bf)
    B, T, H, dk, dv = w.B, w.T, w.H, w.dk, w.dv
    ws_f = torch.empty(comba.fwd_workspace_bytes(B, T, H, dk, dv), dtype=torch.uint8, device=dev)
    ws_b = torch.empty(comba.bwd_workspace_bytes(B, T, H, dk, dv), dtype=torch.uint8, device=dev)
    # the paper's separate feedback strength beta~ = b * beta (one b per head)
    w_bt = copy.copy(w)
    w_bt.extra = {}
    attach_beta_tilde(w_bt, "b_beta", seed=31)
    bt_var = t(w_bt.extra["beta_tilde"], bf)
    bt_main = bt_var if args.beta_tilde else None

    def step(bt=bt_main):
        # training pair: the forward leaves the backward's state in ws_b
        o, ht, _ = comba.comba_chunk_fwd_save(q, k, v, g, beta, d, h0, beta_tilde=bt,
                                              workspace=ws_b)
        gr = comba.comba_chunk_bwd_saved(q, k, v, g, beta, d, h0, dO, None, beta_tilde=bt,
                                         workspace=ws_b)
        return o, gr

    def step_stateless():
        o, ht = comba.comba_chunk_fwd(q, k, v, g, beta, d, h0, beta_tilde=bt_main, workspace=ws_f)
        gr = comba.comba_chunk_bwd(q, k, v, g, beta, d, h0, dO, None, beta_tilde=bt_main,
                                   workspace=ws_b)
        return o, gr

    ms_stateless = ms_fwd_stateless = ms_bwd_stateless = None
    if not args.skip_stateless:
        for _ in range(args.warmup):
            step_stateless()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            step_stateless()
        torch.cuda.synchronize()
        ms_stateless = round((time.perf_counter() - t0) * 1e3 / args.steps, 4)
        # the operator's forward and backward calls on their own
        for name, call in (("fwd", lambda: comba.comba_chunk_fwd(
                q, k, v, g, beta, d, h0, beta_tilde=bt_main, workspace=ws_f)),
                           ("bwd", lambda: comba.comba_chunk_bwd(
                q, k, v, g, beta, d, h0, dO, None, beta_tilde=bt_main, workspace=ws_b))):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(args.steps):
                call()
            torch.cuda.synchronize()
            ms = round((time.perf_counter() - t0) * 1e3 / args.steps, 4)
            if name == "fwd":
                ms_fwd_stateless = ms
            else:
                ms_bwd_stateless = ms

    for _ in range(args.warmup):
        step()
    tm = timed_steps(comba, torch, step, args.steps)
    ms_per_step = tm["ms_per_step"]
    tokens = B * T
    value = tokens / (ms_per_step * 1e-3)
    # per-stage average launch durations (ms) from the stage pass; the dominant
    # stage's is its live average over the timed region
    dom, tot = tm["dominant"], tm["stages_ms"]
    avg = dict(tm["stage_avg_ms"])
    avg[dom] = tm["dom_avg_ms"]
    models = {dr: method_model(dr, B, T, H, dk, dv) for dr in ("fwd_save", "bwd")}
    # the committed counters cover the headline workload only
    roof = kernel_roofline(dom, avg[dom], models[stage_direction(dom)],
                           design=stage_model(dom, B, T, H, dk, dv, sep_bt=args.beta_tilde),
                           traffic=None if args.beta_tilde else measured_traffic(dom),
                           mfma_counted=None if args.beta_tilde else measured_mfma(dom))
    roof["launches_timed"] = tm["dom_launches_timed"]
    mfma_by_kernel = {}
    for n in tot:
        dfl, _ = stage_model(n, B, T, H, dk, dv, sep_bt=args.beta_tilde)
        if dfl > 0:
            cnt = None if args.beta_tilde else measured_mfma(n)
            mfma_by_kernel[n] = {
                "avg_launch_ms": round(avg[n], 4),
                "algorithmic_pct": round(100.0 * dfl / (avg[n] * 1e-3) /
                                         (PEAK_BF16_TFLOPS * 1e12), 3),
                "counted_pct": None if cnt is None else
                round(100.0 * cnt / (avg[n] * 1e-3) / (PEAK_BF16_TFLOPS * 1e12), 3)}
    ms_fwd = sum(x for n, x in tot.items() if n in FWD_STAGES)
    ms_bwd = sum(x for n, x in tot.items() if n in BWD_STAGES)
    step_fl = models["fwd_save"][0] + models["bwd"][0]
    step_by = models["fwd_save"][1] + models["bwd"][1]
    step_sec = ms_per_step * 1e-3
    step_roof = {"method_bytes": step_by, "achieved_GBs": round(step_by / step_sec / 1e9, 1),
                 "frac_hbm": round(step_by / step_sec / 1e9 / PEAK_HBM_GBS, 4),
                 "method_flops": step_fl,
                 "mfma_pct": round(100.0 * step_fl / step_sec / (PEAK_BF16_TFLOPS * 1e12), 3),
                 "fwd_method_bytes": models["fwd_save"][1], "bwd_method_bytes": models["bwd"][1]}
    op_fl = op_flops(B, T, H, dk, dv)
    mfma_frac_op = op_fl / (ms_per_step * 1e-3) / (PEAK_BF16_TFLOPS * 1e12)

    result = {
        "metric": "Comba fwd+bwd tokens/sec at H=16,T=4096,d=128 bf16; % MFMA peak",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded PCG64; q,k L2-normalised, log alpha=-softplus(N(0,1)), "
                "beta=sigmoid(N(0,1)), d~U(0,1)%s)" % (
                    "; beta~=b*beta, b=sigmoid(N(0,1)) per head" if args.beta_tilde else ""),
        "config": {"workload": spec.name + ("_beta_tilde" if args.beta_tilde else ""),
                   "B": B, "T": T, "H": H, "dk": dk, "dv": dv,
                   "chunk": 64, "in_dtype": "bf16", "out_dtype": "f32"},
        "step": "comba_chunk_fwd_save + comba_chunk_bwd_saved",
        "ms_per_step_stateless": ms_stateless,
        "ms_fwd": round(ms_fwd, 4),
        "ms_bwd": round(ms_bwd, 4),
        "ms_fwd_stateless": ms_fwd_stateless,
        "ms_bwd_stateless": ms_bwd_stateless,
        "mfma_pct_peak_op": round(100.0 * mfma_frac_op, 3),
        "op_algorithmic_tflops": round(op_fl / (ms_per_step * 1e-3) / 1e12, 2),
        "stages_ms": {n: round(x, 4) for n, x in tot.items()},
        "roofline": roof,
        "step_roofline": step_roof,
        "mfma_by_kernel": mfma_by_kernel,
    }
    if not (args.no_variants or args.beta_tilde):
        # the same training pair with beta~ = b * beta, timed after the headline region
        for _ in range(args.warmup):
            step(bt_var)
        tm_bt = timed_steps(comba, torch, lambda: step(bt_var), args.steps)
        result["variants"] = {"beta_tilde_b_beta": {
            "value": round(tokens / (tm_bt["ms_per_step"] * 1e-3), 1), "unit": "tokens/s",
            "ms_per_step": round(tm_bt["ms_per_step"], 4),
            "stages_ms": {n: round(x, 4) for n, x in tm_bt["stages_ms"].items()}}}
        result["variants"]["decode_b64_h16_d128"] = time_decode(comba, torch, args.steps,
                                                                args.warmup)
        result["variants"]["prefill_b4_t4096_h8_d256"] = time_prefill256(comba, torch,
                                                                         args.steps, args.warmup)
        result["variants"]["prologue_b4_t4096_h16_d128"] = time_prologue(comba, torch,
                                                                         args.steps, args.warmup)
        result["variants"]["varlen_512k_fwd"] = time_varlen(comba, torch, args.steps,
                                                           args.warmup)
        result["variants"]["long1_525k_fwd"] = time_long1(comba, torch, args.steps, args.warmup)
        result["variants"]["long1_train_65k"] = time_long1_train(comba, torch, args.steps,
                                                                 args.warmup)
        result["variants"]["train_b4_t4096_h8_d256"] = time_train256(comba, torch, args.steps,
                                                                     args.warmup)
    if args.copy_bytes > 0:
        result["copy_bytes"] = calibration_copy(torch, args.copy_bytes)
    if not args.no_cpu_baseline:
        nh = min(H, max(1, math.ceil(2 * threads / B)))
        heads = list(range(0, H, max(1, H // nh)))[:nh]
        result["cpu_baseline"] = cpu_baseline(w_bt if args.beta_tilde else w, heads, threads)
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
