"""The one-kernel training step (tfd_mlp_step) against the oracle.

The persistent kernel computes the same step as the per-op launches (forward
MatMul + BiasAdd + Relu, the cost head, ReluGrad, the two transposed MatMuls,
BiasAddGrad, the SGD update; section 2 and section 4.1) with its own tile
schedule, so it is checked against the oracle directly: the whole chain from
the seeded inputs (mask flips only inside the rounding band, row-local
gradients on untouched rows, reductions within their bounds) and every op
teacher-forced on the operands the kernel read. Also: bitwise reproducible,
the barrier words are left at zero, steps chain through the updated
Variables, and shapes that are not multiples of the 32 x 32 tile or of the
16-byte loads are handled."""

import numpy as np
import pytest
import torch

from paper_1603_04467_amd import workloads
from paper_1603_04467_amd.step import DenseStep
from tests.teacher import check_step
from tests.test_gpu_step import _compare_full

pytestmark = pytest.mark.gpu

CASES = [
    ("dense784x100", None, None),
    ("mlp784-1024-1024-10", None, None),
    ("mlp784-1024-1024-10-xent", None, None),
    ("dense784x100", 33, (97, 65)),                          # ragged everything, odd leading dimensions
    ("mlp784-1024-1024-10", 130, (100, 257, 66, 10)),
    ("mlp784-1024-1024-10-xent", 200, (784, 1024, 1024, 1000)),
    ("mlp784-1024-1024-10", 1024, (784, 2048, 2048, 10)),
    ("mlp784-1024-1024-10", 1, (784, 1024, 1024, 10)),      # one row
]


def _workload(name, batch, dims):
    w = workloads.workload(name)
    return w if batch is None else w.scaled(batch=batch, dims=dims)


def _outputs(s):
    ts = list(s.h[1:]) + [s.g, s.dx[0]] + [t for t in s.dy if t is not None] + list(s.dw) + list(s.db)
    return [t.clone() for t in ts + list(s.variables()) + [s.loss]]


@pytest.mark.parametrize("persistent", [True, False])
@pytest.mark.parametrize("name,batch,dims", CASES)
def test_fused_step_matches_the_oracle(name, batch, dims, persistent):
    w = _workload(name, batch, dims)
    inp = workloads.generate(w, seed=11)
    s = DenseStep(w, inp)
    assert s.fusable()
    s.run_fused(persistent=persistent)
    torch.cuda.synchronize()
    assert s.fused_barrier_error() == 0
    ctl = s._fws[:4096].view(torch.int32).cpu().numpy()
    assert ctl[0] == 0, "barrier error word set"
    assert not np.any(np.delete(ctl, 64)), "barrier counters not left at zero"
    assert ctl[64] == (2 * w.layers + 1 if persistent else 0), ctl[64]   # one generation per barrier
    flips = _compare_full(w, inp, s)
    tf = check_step(s)
    print(f"{w.name}: {flips} rows with in-band mask differences, {tf} teacher-forced flips")


@pytest.mark.parametrize("name,batch,dims", CASES[:3])
def test_fused_step_is_reproducible_and_chains(name, batch, dims):
    """Both launch forms store the same bits (same work items, same orders),
    run after run."""
    w = _workload(name, batch, dims)
    inp = workloads.generate(w, seed=12)
    s = DenseStep(w, inp)
    s.run_fused()
    torch.cuda.synchronize()
    want = _outputs(s)
    for r in range(4):
        s.restore()
        s.run_fused(persistent=r % 2 == 1)
        torch.cuda.synchronize()
        got = _outputs(s)
        for i, (a, b) in enumerate(zip(got, want)):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"output {i} differs between runs"
    # three chained steps (no restore) track the per-op program within the
    # parity bounds of one step each: compare the loss sequence
    a, b = DenseStep(w, inp), DenseStep(w, inp)
    la, lb = [], []
    for i in range(3):
        a.run()
        b.run_fused(persistent=i == 1)
        torch.cuda.synchronize()
        la.append(a.loss.item())
        lb.append(b.loss.item())
    assert np.allclose(la, lb, rtol=1e-4, atol=0), (la, lb)


def test_default_launch_mode():
    """Small steps pick the measured fastest launch mode on their first
    step() (Variables left as they were) and then write exactly what that
    mode writes when run explicitly; large ones run in program order."""
    for name in ("dense784x100", "mlp784-1024-1024-10", "mlp784-1024-1024-10-xent"):
        w = workloads.workload(name)
        inp = workloads.generate(w, seed=1)
        s, ref = DenseStep(w, inp), DenseStep(w, inp)
        assert s.launch_mode == "auto"
        before = [t.clone() for t in s.variables()]
        times = s.autotune_launch_mode()
        for a, b in zip(s.variables(), before):
            assert torch.equal(a, b), "autotuning changed the Variables"
        assert set(times) == {"serial", "graph", "fused"} and s.launch_mode == min(times, key=times.get)
        print(name, s.launch_mode, {k: round(v, 4) for k, v in times.items()})
        for _ in range(2):
            s.restore()
            s.step()
            ref.restore()
            if s.launch_mode == "fused":
                ref.run_fused()
            else:
                ref.run()
            torch.cuda.synchronize()
            for a, b in zip(_outputs(s), _outputs(ref)):
                assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))
    w = workloads.workload("wide4096x4-f32").scaled(batch=2048)
    s = DenseStep(w, workloads.generate(w, seed=1))
    assert s.launch_mode == "serial" and s.fusable() and not s.small()
    w = workloads.workload("wide4096x4-bf16").scaled(batch=256, dims=(256, 256, 256, 256, 256))
    s = DenseStep(w, workloads.generate(w, seed=1))
    assert not s.fusable()
    with pytest.raises(ValueError):
        s.run_fused()
