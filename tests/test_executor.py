"""Host logic of the dependency-count executor (section 3.1's ready counts,
section 2's control dependencies): edge derivation, transitive reduction and
the stream schedule, on abstract graphs and on every workload's step graph."""

import itertools

import pytest

from paper_1603_04467_amd import executor, workloads
from paper_1603_04467_amd.step import fused_below, fused_top, op_graph


class _N:
    def __init__(self, name, reads=(), writes=()):
        self.name, self.reads, self.writes = name, reads, writes


def _ancestors(deps):
    anc = []
    for i, d in enumerate(deps):
        a = set()
        for p in d:
            a |= anc[p] | {p}
        anc.append(a)
    return anc


def test_edges_from_read_write_sets():
    nodes = [_N("w1", writes=("a",)), _N("r1", reads=("a",)), _N("r2", reads=("a",)),
             _N("w2", writes=("a",)), _N("r3", reads=("a", "b")), _N("wb", writes=("b",))]
    deps = executor.dependencies(nodes)
    assert deps[1] == {0} and deps[2] == {0}          # read after write
    assert deps[3] == {0, 1, 2}                       # write after write and after both reads
    assert deps[4] == {3}                             # reads the second value of a; b never written before
    assert deps[5] == {4}                             # write after read of b
    red = executor.transitive_reduction(deps)
    assert red[3] == {1, 2}                           # 0 is implied through 1 and 2


def test_schedule_is_topological_and_complete():
    deps = [set(), {0}, {0}, {1, 2}, {0}, {3, 4}]
    for k in (1, 2, 3, 5):
        plan = executor.schedule(deps, k)
        assert sorted(i for i, _ in plan) == list(range(6))
        pos = {i: n for n, (i, _) in enumerate(plan)}
        assert all(pos[p] < pos[i] for i, d in enumerate(deps) for p in d)
        assert all(0 <= s < k for _, s in plan)
    plan = dict(executor.schedule(deps, 3))
    assert len({plan[1], plan[2], plan[4]}) == 3      # three independent successors of node 0


@pytest.mark.parametrize("masks", [False, True])
@pytest.mark.parametrize("fuse", [False, True])
@pytest.mark.parametrize("name", sorted(workloads.WORKLOADS))
def test_step_graph_orders_updates_after_reads(name, fuse, masks):
    w = workloads.workload(name)
    ops = op_graph(w, fuse, masks)
    names = [o[0] for o in ops]
    deps = executor.transitive_reduction(executor.dependencies([_N(*o) for o in ops]))
    anc = _ancestors(deps)
    idx = {n: i for i, n in enumerate(names)}
    L = w.layers

    def dy_producer(l):   # the op that writes layer l's masked gradient and db
        if l == L and fused_top(w, fuse):
            return f"fwd{L}"
        return f"dx{l + 1}" if fused_below(w, l, fuse) else f"relugrad{l}"

    for l in range(1, L + 1):
        if w.update:
            s = idx[f"sgd{l}"]
            # the update of W_l and b_l waits for every reader of the old values
            for r in (f"fwd{l}", f"dx{l}", f"dw{l}", dy_producer(l)):
                assert idx[r] in anc[s], (r, f"sgd{l}")
        # dX_l and dW_l are independent of each other (concurrent)
        dx, dw = idx[f"dx{l}"], idx[f"dw{l}"]
        assert dx not in anc[dw] and dw not in anc[dx]
        # both need the masked gradient, which needs the gradient from above
        if w.relus[l - 1]:
            assert idx[dy_producer(l)] in anc[dx] and idx[dy_producer(l)] in anc[dw]
        if l < L and not fused_below(w, l, fuse):
            assert idx[f"dx{l + 1}"] in anc[idx[f"relugrad{l}"]]
    # fused: one op per layer above a Relu layer replaces the relugrad op,
    # and the output layer's MatMul also runs the squared-error head
    assert ("relugrad1" in names) == (not fused_below(w, 1, fuse) and not (L == 1 and fused_top(w, fuse)))
    assert ("loss" in names) == (w.cost != "upstream" and not fused_top(w, fuse))
    # the forward chain precedes the cost and all of the backward pass
    first_bwd = min(i for i, n in enumerate(names) if not n.startswith("fwd") and n != "loss")
    assert idx[f"fwd{L}"] in anc[first_bwd]
    plan = dict(executor.schedule(deps, 3))
    for l in range(1, L + 1):
        assert plan[idx[f"dx{l}"]] != plan[idx[f"dw{l}"]]
    # with masks, each Relu layer's ReluGrad reads the mask its forward op wrote
    for l in range(L):
        key = f"m{l}"
        writers = [n for n, _, wr in ops if key in wr]
        readers = [n for n, rd, _ in ops if key in rd]
        if masks and w.relus[l]:
            assert writers == [f"fwd{l + 1}"] and len(readers) == 1
            assert idx[writers[0]] in anc[idx[readers[0]]]
            assert readers[0] == dy_producer(l + 1)
        else:
            assert not writers and not readers


def test_schedule_of_one_stream_is_program_order_for_the_step():
    w = workloads.workload("mlp784-1024-1024-10")
    ops = op_graph(w)
    deps = executor.transitive_reduction(executor.dependencies([_N(*o) for o in ops]))
    plan = executor.schedule(deps, 1)
    assert all(s == 0 for _, s in plan)
    # every permutation the schedule makes still respects the edges
    pos = {i: n for n, (i, _) in enumerate(plan)}
    assert all(pos[p] < pos[i] for i, d in enumerate(deps) for p in d)
    assert len(list(itertools.islice(plan, 100))) == len(ops)
