"""Dependency-count execution of a step's op graph on several HIP streams.

Section 3.1 of the paper runs a graph by keeping, for every node, the count
of its inputs not yet produced; a node whose count reaches zero enters a
ready queue, and finishing a node decrements the counts of its successors.
Section 2's control dependencies add edges that order a Variable's readers
before its writer. Here the same bookkeeping runs once on the host while the
nodes are *enqueued*: each ready node is placed on one of a few streams and
made to wait (with a HIP event) for every predecessor that sits on another
stream, so independent nodes (e.g. a layer's input gradient, weight gradient
and bias update) execute concurrently on the GPU. The result is identical to
the one-stream order because every edge of the graph is honoured.

The edges are derived from what each node reads and writes, in program
order: read-after-write (data), write-after-read and write-after-write (the
control dependencies that keep an update after every read of the old value).

Enqueueing from a fork/join on an origin stream makes the whole schedule
capturable into one HIP graph (torch.cuda.CUDAGraph on ROCm).
"""

from __future__ import annotations

import collections
import dataclasses
from typing import Callable, List, Sequence

import torch


@dataclasses.dataclass
class Node:
    name: str
    launch: Callable[[torch.cuda.Stream], None]   # enqueues the node's kernels on the given stream
    reads: Sequence[str] = ()
    writes: Sequence[str] = ()


def dependencies(nodes: Sequence[Node]) -> List[set]:
    """Predecessor sets from the read/write sets in program order."""
    deps = [set() for _ in nodes]
    last_writer = {}
    readers = collections.defaultdict(set)
    for i, n in enumerate(nodes):
        for k in n.reads:
            if k in last_writer:
                deps[i].add(last_writer[k])              # read after write
        for k in n.writes:
            if k in last_writer:
                deps[i].add(last_writer[k])              # write after write
            deps[i] |= readers[k]                        # write after read
        for k in n.reads:
            readers[k].add(i)
        for k in n.writes:
            last_writer[k] = i
            readers[k] = set()
        deps[i].discard(i)
    return deps


def transitive_reduction(deps: List[set]) -> List[set]:
    """Drop edges implied by other paths (fewer event waits)."""
    n = len(deps)
    reach = [set() for _ in range(n)]          # all ancestors of i
    for i in range(n):                          # program order is a topological order
        for p in deps[i]:
            reach[i] |= reach[p] | {p}
    out = []
    for i in range(n):
        keep = set(deps[i])
        for p in deps[i]:
            for q in deps[i]:
                if q != p and p in reach[q]:
                    keep.discard(p)
                    break
        out.append(keep)
    return out


def schedule(deps: List[set], num_streams: int):
    """(node, stream) pairs in ready-queue order: the host-side bookkeeping
    of the dependency counts. A node continues the stream of a predecessor
    that is that stream's last node when there is one; otherwise it takes the
    stream used least recently."""
    n = len(deps)
    succ = [[] for _ in range(n)]
    for i, d in enumerate(deps):
        for p in d:
            succ[p].append(i)
    pending = [len(d) for d in deps]
    ready = collections.deque(i for i, c in enumerate(pending) if c == 0)
    tail = [None] * num_streams
    last_use = [-1] * num_streams
    order = []
    while ready:
        i = ready.popleft()
        own = [s for s in range(num_streams) if tail[s] is not None and tail[s] in deps[i]]
        s = min(own) if own else min(range(num_streams), key=lambda q: last_use[q])
        tail[s] = i
        last_use[s] = len(order)
        order.append((i, s))
        for j in succ[i]:
            pending[j] -= 1
            if pending[j] == 0:
                ready.append(j)
    if len(order) != n:
        raise RuntimeError("the op graph has a cycle")
    return order


class StreamExecutor:
    """Enqueues `nodes` on `num_streams` streams following the ready-count
    algorithm; the origin stream (the caller's current stream) forks to the
    others at the start and joins them at the end."""

    def __init__(self, nodes: Sequence[Node], num_streams: int = 3, device=None):
        self.nodes = list(nodes)
        self.deps = transitive_reduction(dependencies(self.nodes))
        self.side = [torch.cuda.Stream(device=device) for _ in range(num_streams - 1)]
        self.done = [torch.cuda.Event() for _ in self.nodes]
        self.fork = torch.cuda.Event()
        self.plan = schedule(self.deps, num_streams)

    def streams_used(self):
        return sorted({s for _, s in self.plan})

    def enqueue(self, origin: torch.cuda.Stream = None):
        origin = origin or torch.cuda.current_stream()
        streams = [origin] + self.side
        self.fork.record(origin)
        forked = set()
        stream_of = {}
        for i, s in self.plan:
            st = streams[s]
            if s != 0 and s not in forked:
                st.wait_event(self.fork)
                forked.add(s)
            for p in self.deps[i]:
                if stream_of[p] != s:
                    st.wait_event(self.done[p])
            self.nodes[i].launch(st)
            self.done[i].record(st)
            stream_of[i] = s
        # join: the origin waits for the last node of every side stream
        last = {}
        for i, s in self.plan:
            last[s] = i
        for s, i in last.items():
            if s != 0:
                origin.wait_event(self.done[i])
