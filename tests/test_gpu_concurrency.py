"""Concurrent execution of the step's independent ops on several streams and
its capture into a HIP graph: both must give exactly the tensors of the
one-stream program order (every kernel is deterministic and every edge of the
op graph is honoured, so equality is bitwise).

Graph replays are checked several times, each after an eager restore of the
Variables, unrelated eager work and a synchronisation, against the eager
step; the capture contains only the library's kernel launches and the
executor's event edges (no memset nodes)."""

import gc

import numpy as np
import pytest
import torch

from paper_1603_04467_amd import workloads
from paper_1603_04467_amd.step import DenseStep, fused_below

pytestmark = pytest.mark.gpu

CASES = [
    ("dense784x100", None, None),
    ("mlp784-1024-1024-10", None, None),
    ("mlp784-1024-1024-10-xent", None, None),
    ("wide4096x4-f32", 520, (136, 256, 512, 264, 128)),
    ("wide4096x4-bf16", 1032, (512, 768, 512, 256, 512)),
    ("wide4096x4-bf16-trunc", 600, (256, 384, 264, 128, 200)),
    ("tall512x32768-bf16", 264, (96, 4104)),
]


def _workload(name, batch, dims):
    w = workloads.workload(name)
    return w if batch is None else w.scaled(batch=batch, dims=dims)


def _state(s):
    # the input gradients the step stores (with fusion, only those not folded
    # into the ReluGrad of the layer below)
    dx = [s.dx[l] for l in range(s.w.layers) if not fused_below(s.w, l, s.fuse)]
    ts = list(s.h[1:]) + [s.g] + [t for t in s.dy if t is not None] + dx + list(s.dw) + list(s.db)
    ts += list(s.variables()) + [s.loss]
    return [t.clone() for t in ts]


def _same_bits(x, y):
    return x.shape == y.shape and torch.equal(x.contiguous().view(torch.uint8), y.contiguous().view(torch.uint8))


def _assert_same(a, b, what):
    assert len(a) == len(b)
    for i, (x, y) in enumerate(zip(a, b)):
        assert _same_bits(x, y), f"{what}: tensor {i} differs"


@pytest.mark.parametrize("name,batch,dims", CASES)
@pytest.mark.parametrize("num_streams", [2, 3, 4])
def test_concurrent_step_equals_program_order(name, batch, dims, num_streams):
    w = _workload(name, batch, dims)
    s = DenseStep(w, workloads.generate(w, seed=1))
    s.run()
    torch.cuda.synchronize()
    want = _state(s)
    for _ in range(2):
        s.restore()
        s.run_concurrent(num_streams)
        torch.cuda.synchronize()
        _assert_same(_state(s), want, f"{w.name} on {num_streams} streams")


@pytest.mark.parametrize("name,batch,dims", CASES)
@pytest.mark.parametrize("concurrent", [False, True])
def test_graph_replays_equal_eager_step(name, batch, dims, concurrent):
    w = _workload(name, batch, dims)
    s = DenseStep(w, workloads.generate(w, seed=2))
    s.run()
    torch.cuda.synchronize()
    want = _state(s)
    g = s.capture(concurrent=concurrent)
    junk = torch.randn(1 << 20, device="cuda")
    for r in range(4):
        s.restore()
        junk = junk * 1.5 + 1.0                      # unrelated eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _assert_same(_state(s), want, f"{w.name} replay {r}")
    # an eager step after the replays still agrees
    s.restore()
    s.run()
    torch.cuda.synchronize()
    _assert_same(_state(s), want, f"{w.name} eager after replays")
    del g


def test_repeated_concurrent_steps_chain_correctly():
    """Back-to-back steps without restores: step k+1 reads what step k wrote
    (the updated Variables), so the fork/join must order them."""
    w = workloads.workload("mlp784-1024-1024-10")
    inp = workloads.generate(w, seed=4)
    a = DenseStep(w, inp)
    b = DenseStep(w, inp)
    for _ in range(3):
        a.run()
        b.run_concurrent(3)
    torch.cuda.synchronize()
    _assert_same(_state(a), _state(b), "three chained steps")
    assert np.isfinite(a.loss.item())


@pytest.mark.parametrize("name,batch,dims", CASES)
@pytest.mark.parametrize("mode", ["streams", "graph", "graph_streams"])
def test_concurrent_and_graph_outputs_match_the_oracle(name, batch, dims, mode):
    """The multi-stream step and the graph replays checked against the oracle
    directly (not only against the serial step): the whole chain from the
    seeded inputs, and every op teacher-forced on the GPU's own operands."""
    from tests.teacher import check_step
    from tests.test_gpu_step import _compare_full

    w = _workload(name, batch, dims)
    inp = workloads.generate(w, seed=3)
    s = DenseStep(w, inp)
    g = None
    if mode != "streams":
        g = s.capture(concurrent=mode == "graph_streams", num_streams=3)
    for rep in range(2):
        s.restore()
        if g is None:
            s.run_concurrent(3)
        else:
            g.replay()
        torch.cuda.synchronize()
        _compare_full(w, inp, s)
        check_step(s)
    del g


def test_capture_with_dead_steps_holding_graphs():
    """capture() while dead object cycles hold other steps' HIP graphs and the
    cyclic collector is set to run at almost every allocation: the steps are
    collected before the capture, never inside it (a graph destroyed while a
    stream is being captured aborts the process), and the captured graph
    replays the eager step bit for bit."""
    w = workloads.workload("dense784x100")
    for seed in range(3):
        dead = DenseStep(w, workloads.generate(w, seed=seed))
        dead._held = dead.capture(concurrent=False)
        dead._self = dead                       # a cycle the collector must break
        del dead
    old = gc.get_threshold()
    s = DenseStep(w, workloads.generate(w, seed=5))
    gc.set_threshold(1, 1, 1)
    try:
        graphs = [s.capture(concurrent=False), s.capture(concurrent=True)]
    finally:
        gc.set_threshold(*old)
    s.restore()
    s.run()
    torch.cuda.synchronize()
    want = [t.clone() for t in list(s.h[1:]) + list(s.variables()) + [s.loss]]
    for g in graphs:
        s.restore()
        g.replay()
        torch.cuda.synchronize()
        got = list(s.h[1:]) + list(s.variables()) + [s.loss]
        for a, b in zip(got, want):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))
