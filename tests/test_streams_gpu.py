"""The stateless backward's two scans run side by side (the reverse scan on a
helper stream of the library, joined back before the gradient kernel).

Checks that the stage record shows the combined stage, and that calls from two
host threads on streams of their own, each with its own workspace, give
gradients bitwise equal to a single call (the helper stream and its events are
shared under a lock)."""
import threading

import numpy as np
import pytest

from comba_inputs import random_case

pytestmark = pytest.mark.gpu

GRADS = ("dq", "dk", "dv", "dg", "dbeta", "dd", "dh0")


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _args():
    import torch

    print("streams case: B2 T1000 H2 d128 bf16 stateless backward", flush=True)
    w = random_case(B=2, T=1000, H=2, dk=128, dv=128, in_dtype="bf16", seed=909, grad=True)
    bf = torch.bfloat16

    def t(x, dt=torch.float32):
        return torch.from_numpy(np.ascontiguousarray(x)).cuda().to(dt)

    args = (t(w.q, bf), t(w.k, bf), t(w.v, bf), t(w.g), t(w.beta, bf), t(w.d), t(w.h0))
    dht = np.random.default_rng(910).standard_normal(w.h0.shape).astype(np.float32)
    return args, t(w.dO, bf), t(dht)


def test_stateless_backward_records_the_side_by_side_scans():
    import torch

    import paper_2506_02475_amd as comba

    args, dO, dht = _args()
    comba.profile_enable(True)
    comba.comba_chunk_bwd(*args, dO, dht)
    torch.cuda.synchronize()
    stages = [n for n, _ in comba.profile_read()]
    comba.profile_enable(False)
    assert "scans" in stages and "intra_bwd" in stages, stages
    assert "scan_bwd" not in stages and "scan_fwd_store" not in stages, stages


def test_stateless_backward_from_two_threads_matches_one_call():
    import torch

    import paper_2506_02475_amd as comba

    args, dO, dht = _args()
    ref = comba.comba_chunk_bwd(*args, dO, dht)
    torch.cuda.synchronize()
    results = [[], []]
    errors = []

    def work(i):
        try:
            s = torch.cuda.Stream()  # default priority
            s.wait_stream(torch.cuda.default_stream())
            with torch.cuda.stream(s):
                for _ in range(6):
                    results[i].append(comba.comba_chunk_bwd(*args, dO, dht))
            s.synchronize()
        except Exception as e:  # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(i,)) for i in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for res in results:
        assert len(res) == 6
        for gr in res:
            for name in GRADS:
                assert torch.equal(gr[name], ref[name]), name


def test_stateless_backward_replays_from_a_captured_graph():
    """The fork to the helper stream and the join back are captured with the
    kernels (the helper exists from an eager call before the capture); every
    replay, with eager calls and synchronisations between them, equals the
    eager result."""
    import torch

    import paper_2506_02475_amd as comba

    args, dO, dht = _args()
    ref = comba.comba_chunk_bwd(*args, dO, dht)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        comba.comba_chunk_bwd(*args, dO, dht)  # warm-up on a side stream, as capture expects
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        out = comba.comba_chunk_bwd(*args, dO, dht)
    torch.cuda.synchronize()
    for i in range(3):
        print("graph replay %d" % i, flush=True)
        graph.replay()
        torch.cuda.synchronize()
        for name in GRADS:
            assert torch.equal(out[name], ref[name]), (i, name)
        again = comba.comba_chunk_bwd(*args, dO, dht)
        torch.cuda.synchronize()
        for name in GRADS:
            assert torch.equal(again[name], ref[name]), (i, name)
