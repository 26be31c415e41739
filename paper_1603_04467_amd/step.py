"""One training step of a stack of dense layers, as a fixed sequence of
libtfdense calls on one HIP stream.

The order is the one a dependency-respecting executor of the paper's graph
would take (section 3.1 runs a node once its inputs are ready; section 2's
control dependencies order a Variable's readers before its writer):

  forward  l = 1..L : H_l = Relu(H_{l-1} W_l + b_l)   (identity on the output layer)
  cost              : G = H_L - T, L = 1/2 |G|^2     (squared error), or
                      G = softmax(H_L) - onehot(y), L = cross-entropy (class labels y),
                      or a given upstream gradient
  backward l = L..1 : dY_l, db_l = ReluGrad + BiasAddGrad(G_l, H_l)
                      G_{l-1} = dX_l = dY_l W_l^T          (reads the old W_l)
                      dW_l = H_{l-1}^T dY_l
                      W_l -= lr dW_l ; b_l -= lr db_l      (after both reads of W_l)

Stream order is the only synchronisation; nothing waits on the host inside a
step. All tensors stay resident in device memory between steps.
"""

from __future__ import annotations

from typing import Optional

import gc
import numpy as np
import torch

from . import tfdense as T
from .workloads import Workload


def _to_device(a: np.ndarray, act: str, device) -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def fused_below(w: Workload, l: int, fuse: bool) -> bool:
    """Whether layer l's input-gradient MatMul also applies the ReluGrad and
    BiasAddGrad of layer l - 1 (one fused call instead of two)."""
    return fuse and 1 <= l < w.layers and w.relus[l - 1]


def fused_top(w: Workload, fuse: bool) -> bool:
    """Whether the output layer's MatMul also computes the squared-error cost,
    its gradient and the output layer's BiasAddGrad (one fused call instead
    of three; only for an identity output layer)."""
    return fuse and w.cost in ("sq_err", "half_sq") and not w.relus[-1]


def default_masks(w: Workload) -> bool:
    """Whether the step keeps ReLU masks (one bit per element of H > 0) for
    its ReluGrads by default: with 16-bit activations, where the forward
    MatMul writes the mask in its epilogue and the backward pass then reads
    1 bit instead of 16 per element."""
    return w.act == "bf16"


def op_graph(w: Workload, fuse: bool = True, masks: bool = False):
    """(name, reads, writes) of every op of one step of ``w``, in program
    order. Keys name buffers: h<l> activations (h0 = x), g the cost gradient,
    dy<l>/dx<l>/dw<l>/db<l> the gradients of layer l, W<l>/b<l> its Variables
    (all copies of the weights), m<l> the ReLU mask of layer l's output, ws
    the shared reduction workspace. With ``fuse``, the input-gradient MatMul
    of a layer above a Relu layer also produces that layer's dY and db (no
    separate relugrad op, no stored dX). With ``masks``, a Relu layer's
    forward MatMul also writes its mask and its ReluGrad reads the mask
    instead of the layer's output."""
    L = w.layers
    mk = lambda l: masks and w.relus[l]  # noqa: E731
    ops = [(f"fwd{l + 1}", (f"h{l}", f"W{l}", f"b{l}"), (f"h{l + 1}",) + ((f"m{l}",) if mk(l) else ()))
           for l in range(L)]
    if fused_top(w, fuse):
        ops[-1] = (f"fwd{L}", (f"h{L - 1}", f"W{L - 1}", f"b{L - 1}", "target"),
                   (f"h{L}", "g", "loss", f"db{L - 1}", "ws"))
    elif w.cost != "upstream":
        ops.append(("loss", (f"h{L}", "target"), ("g", "loss", "ws")))
    gkey = "g"
    for l in reversed(range(L)):
        dykey = f"dy{l}" if w.relus[l] else gkey
        if not fused_below(w, l + 1, fuse) and not (l == L - 1 and fused_top(w, fuse)):
            rg_writes = (f"dy{l}", f"db{l}", "ws") if w.relus[l] else (f"db{l}", "ws")
            ops.append((f"relugrad{l + 1}", (gkey, f"m{l}" if mk(l) else f"h{l + 1}"), rg_writes))
        if fused_below(w, l, fuse):
            ops.append((f"dx{l + 1}", (dykey, f"W{l}", f"m{l - 1}" if mk(l - 1) else f"h{l}"),
                        (f"dy{l - 1}", f"db{l - 1}", "ws")))
        else:
            # the plain input-gradient MatMul may split its k range through the
            # shared workspace
            ops.append((f"dx{l + 1}", (dykey, f"W{l}"), (f"dx{l}", "ws")))
        ops.append((f"dw{l + 1}", (f"h{l}", dykey), (f"dw{l}",)))
        if w.update:
            ops.append((f"sgd{l + 1}", (f"dw{l}", f"db{l}"), (f"W{l}", f"b{l}")))
        gkey = f"dx{l}"
    return ops


class DenseStep:
    """Device state and launch sequence of one step of workload ``w``."""

    def __init__(self, w: Workload, inputs: dict, device="cuda", fuse: bool = True, masks: Optional[bool] = None):
        self.w = w
        self.fuse = fuse
        self.use_masks = default_masks(w) if masks is None else bool(masks)
        self.device = torch.device(device)
        self.act = torch.bfloat16 if w.act == "bf16" else torch.float32
        dev = self.device
        L, N = w.layers, w.batch
        self.x = _to_device(inputs["x"], w.act, dev)
        self.weights = [_to_device(a, w.act, dev) for a in inputs["weights"]]
        self.masters = None if inputs["masters"] is None else [_to_device(a, "f32", dev) for a in inputs["masters"]]
        self.biases = [_to_device(a, "f32", dev) for a in inputs["biases"]]
        # 16-bit weights over a short k range (a layer with fan_in under 2048,
        # whose forward MatMul runs the 8-wave kernel) are kept twice: W
        # [fan_in, fan_out] for the input-gradient MatMul and W^T [fan_out,
        # fan_in] so that the forward MatMul reads its weight operand
        # k-contiguous (transpose_b). With fp32 masters both copies are
        # refreshed by the update kernel; weights that are never updated (a
        # given layer) get the transposed copy once. Over long k ranges the
        # forward reads W itself (the 4-wave kernel is as fast on it), and the
        # update writes one 16-bit copy instead of two.
        self.weights_t = None
        short_k = w.act == "bf16" and min(w.dims[:-1]) < 2048
        if short_k and (self.masters is not None or not w.update):
            self.weights_t = [torch.empty(w.dims[l + 1], w.dims[l], dtype=self.act, device=dev) for l in range(L)]
        # layout of the forward MatMul ("NN": H W; "NT": H (W^T)^T)
        self.forward_layout = "NT" if self.weights_t is not None else "NN"
        self.target = None if inputs["target"] is None else _to_device(inputs["target"], w.act, dev)
        self.upstream = None if inputs["upstream"] is None else _to_device(inputs["upstream"], w.act, dev)
        labels = inputs.get("labels")
        self.labels = None if labels is None else torch.from_numpy(np.ascontiguousarray(labels, np.int32)).to(dev)

        self.h = [self.x] + [torch.empty(N, w.dims[l + 1], dtype=self.act, device=dev) for l in range(L)]
        self.g = self.upstream if self.upstream is not None else torch.empty(N, w.dims[-1], dtype=self.act, device=dev)
        self.dy = [torch.empty(N, w.dims[l + 1], dtype=self.act, device=dev) if w.relus[l] else None
                   for l in range(L)]
        self.dx = [torch.empty(N, w.dims[l], dtype=self.act, device=dev) for l in range(L)]
        self.dw = [torch.empty(w.dims[l], w.dims[l + 1], dtype=torch.float32, device=dev) for l in range(L)]
        # ReLU masks of the Relu layers' outputs (uint32 words in int32 tensors)
        self.masks = [T.new_relu_mask(N, w.dims[l + 1], dev) if self.use_masks and w.relus[l] else None
                      for l in range(L)]
        self.db = [torch.empty(w.dims[l + 1], dtype=torch.float32, device=dev) for l in range(L)]
        self.loss = torch.zeros(1, dtype=torch.float64, device=dev)

        need = [T.tfd_reduction_workspace_size(N, w.dims[l + 1], self.act) for l in range(L)]
        need.append(T.tfd_loss_workspace_size(N * w.dims[-1], self.act))
        need.append(T.tfd_softmax_xent_workspace_size(N))
        need += [T.tfd_matmul_relu_grad_workspace_size(N, w.dims[l], self.act) for l in range(1, L)]
        need.append(T.tfd_matmul_l2_loss_grad_workspace_size(N, w.dims[-1], self.act))
        need += [T.tfd_matmul_workspace_size(N, w.dims[l], w.dims[l + 1], self.act, self.act, transpose_b=True)
                 for l in range(L)]
        self.workspace = torch.empty(max(need), dtype=torch.uint8, device=dev)

        if self.weights_t is not None or self.masters is not None:
            # derive the 16-bit W (and W^T) with the update kernel (alpha = 0)
            # from the masters under the workload's rounding, or W^T from the
            # exact fp32 value of a given 16-bit W (which it reproduces bit for
            # bit)
            for l in range(L):
                self.dw[l].zero_()
                if self.masters is not None:
                    T.tfd_apply_gradient_descent_matrix(
                        self.masters[l], 0.0, self.dw[l], var_bf16=self.weights[l],
                        var_bf16_t=None if self.weights_t is None else self.weights_t[l], rounding=w.rounding)
                else:
                    wf = torch.empty(w.dims[l], w.dims[l + 1], dtype=torch.float32, device=dev)
                    T.tfd_convert_bf16_to_f32(self.weights[l], wf)
                    T.tfd_apply_gradient_descent_matrix(wf, 0.0, self.dw[l], var_bf16_t=self.weights_t[l])

        # pristine copies of the Variables, to restart from the same state
        self._saved = [t.clone() for t in self.variables()]

    def variables(self):
        out = list(self.weights) + list(self.biases)
        if self.masters is not None:
            out += list(self.masters)
        if self.weights_t is not None:
            out += list(self.weights_t)
        return out

    def restore(self):
        """Reset the Variables to their initial values (stream-ordered copies)."""
        for t, s in zip(self.variables(), self._saved):
            t.copy_(s)

    def nodes(self):
        """The step's op nodes in program order (op_graph), each with the
        launch of its kernels on a given stream (built once: the buffers they
        launch on are fixed at construction)."""
        if "_nodes" not in self.__dict__:
            self._nodes = self._build_nodes()
        return self._nodes

    def _build_nodes(self):
        from .executor import Node

        w, L = self.w, self.w.layers
        ws = self.workspace
        launches = {}

        def fwd(l):
            epi = "bias_relu" if w.relus[l] else "bias"

            def launch(st):
                if self.masks[l] is not None:
                    wt = self.weights_t is not None
                    T.tfd_matmul_relu_mask(self.h[l], self.weights_t[l] if wt else self.weights[l], self.biases[l],
                                           self.h[l + 1], self.masks[l], transpose_b=wt, rounding=w.rounding,
                                           stream=st)
                elif self.weights_t is not None:
                    T.tfd_matmul(self.h[l], self.weights_t[l], self.h[l + 1], transpose_b=True, bias=self.biases[l],
                                 epilogue=epi, rounding=w.rounding, stream=st)
                else:
                    T.tfd_matmul(self.h[l], self.weights[l], self.h[l + 1], bias=self.biases[l], epilogue=epi,
                                 rounding=w.rounding, stream=st)
            return launch

        for l in range(L):
            launches[f"fwd{l + 1}"] = fwd(l)
        if fused_top(w, self.fuse):
            top = L - 1
            src = self.weights_t[top] if self.weights_t is not None else self.weights[top]

            def fwd_loss(st):
                T.tfd_matmul_l2_loss_grad(self.h[top], src, self.biases[top], self.h[L], self.target, self.g,
                                          self.loss, self.db[top], transpose_b=self.weights_t is not None,
                                          rounding=w.rounding, workspace=ws, stream=st)
            launches[f"fwd{L}"] = fwd_loss

        def loss(st):
            if self.labels is not None:
                T.tfd_softmax_cross_entropy_grad(self.h[L], self.labels, self.g, self.loss, workspace=ws, stream=st)
            else:
                T.tfd_l2_loss_grad(self.h[L], self.target, self.g, self.loss, workspace=ws, stream=st)
        launches["loss"] = loss

        def backward(l, grad):
            dyl = self.dy[l] if w.relus[l] else grad

            def relugrad(st):
                if self.masks[l] is not None:
                    T.tfd_relu_mask_grad_bias_add_grad(grad, self.masks[l], self.dy[l], self.db[l], workspace=ws,
                                                       stream=st)
                elif w.relus[l]:
                    T.tfd_relu_grad_bias_add_grad(grad, self.h[l + 1], self.dy[l], self.db[l], workspace=ws, stream=st)
                else:
                    T.tfd_bias_add_grad(grad, self.db[l], workspace=ws, stream=st)

            def dx(st):
                if fused_below(w, l, self.fuse) and self.masks[l - 1] is not None:
                    T.tfd_matmul_relu_mask_grad_bias_add_grad(dyl, self.weights[l], self.masks[l - 1], self.dy[l - 1],
                                                              self.db[l - 1], transpose_b=True, rounding=w.rounding,
                                                              workspace=ws, stream=st)
                elif fused_below(w, l, self.fuse):
                    T.tfd_matmul_relu_grad_bias_add_grad(dyl, self.weights[l], self.h[l], self.dy[l - 1], self.db[l - 1],
                                                         transpose_b=True, rounding=w.rounding, workspace=ws,
                                                         stream=st)
                else:
                    T.tfd_matmul(dyl, self.weights[l], self.dx[l], transpose_b=True, rounding=w.rounding, workspace=ws,
                                 stream=st)

            def dw(st):
                T.tfd_matmul(self.h[l], dyl, self.dw[l], transpose_a=True, stream=st)

            def sgd(st):
                if self.masters is not None:
                    T.tfd_apply_gradient_descent_matrix(self.masters[l], w.lr, self.dw[l], var_bf16=self.weights[l],
                                                        var_bf16_t=None if self.weights_t is None else self.weights_t[l],
                                                        rounding=w.rounding, stream=st)
                else:
                    T.tfd_apply_gradient_descent(self.weights[l], w.lr, self.dw[l], stream=st)
                T.tfd_apply_gradient_descent(self.biases[l], w.lr, self.db[l], stream=st)

            launches.update({f"relugrad{l + 1}": relugrad, f"dx{l + 1}": dx, f"dw{l + 1}": dw, f"sgd{l + 1}": sgd})

        grad = self.g
        for l in reversed(range(L)):
            backward(l, grad)
            grad = self.dx[l]
        return [Node(name, launches[name], reads, writes)
                for name, reads, writes in op_graph(w, self.fuse, self.use_masks)]

    def run(self, mark=None, stream=None):
        """Enqueue one step in program order on one stream (the current one
        by default). ``mark(name)`` (optional) is called between launches,
        e.g. to record timing events."""
        st = stream or torch.cuda.current_stream()
        for n in self.nodes():
            if mark:
                mark(n.name)
            n.launch(st)
        if mark:
            mark("end")

    def executor(self, num_streams=3):
        """A StreamExecutor over this step's op graph (cached per stream count)."""
        from .executor import StreamExecutor

        cache = self.__dict__.setdefault("_executors", {})
        if num_streams not in cache:
            cache[num_streams] = StreamExecutor(self.nodes(), num_streams=num_streams, device=self.device)
        return cache[num_streams]

    def run_concurrent(self, num_streams=3):
        """Enqueue one step with independent ops on separate streams, forked
        from and joined back to the current stream."""
        self.executor(num_streams).enqueue(torch.cuda.current_stream())

    def fusable(self) -> bool:
        """Whether the whole step can run as one tfd_mlp_step kernel: fp32,
        at most four layers, a Relu on every hidden layer, a squared-error or
        softmax cost head, the fused program (dX of a layer above a Relu folded
        into the ReluGrad below it), no masks."""
        w = self.w
        return (w.act == "f32" and w.layers <= T.MLP_MAX_LAYERS and all(w.relus[:-1]) and self.fuse
                and not self.use_masks and w.cost in ("sq_err", "half_sq", "xent") and self.upstream is None)

    def _fused_desc(self):
        if "_fdesc" not in self.__dict__:
            w, L = self.w, self.w.layers
            layers = [{"weights": self.weights[l], "bias": self.biases[l], "activations": self.h[l + 1],
                       "backprop": self.dy[l], "weight_grad": self.dw[l], "bias_grad": self.db[l],
                       "relu": w.relus[l]} for l in range(L)]
            cost = "softmax_xent" if w.cost == "xent" else "sq_err"
            self._fdesc = T.mlp_step_desc(self.x, layers, cost, self.g, self.loss, target=self.target,
                                          labels=self.labels, input_grad=self.dx[0], learning_rate=w.lr,
                                          update=w.update)
            # the first 4096 bytes (the kernel's grid barrier) start at zero;
            # every completed step leaves its counters and error word at zero
            self._fws = torch.zeros(T.tfd_mlp_step_workspace_size(self._fdesc), dtype=torch.uint8, device=self.device)
        return self._fdesc

    def run_fused(self, stream=None, persistent=False):
        """Enqueue the whole step through tfd_mlp_step: one launch per phase
        (2 L + 2 launches), or with ``persistent`` one cooperative kernel with
        grid barriers between the phases; the same tensors as run() are
        written."""
        if not self.fusable():
            raise ValueError(f"{self.w.name}: the fused step needs fp32, <= {T.MLP_MAX_LAYERS} layers, "
                             "Relu hidden layers, a squared-error or softmax cost and the fused program")
        d = self._fused_desc()
        d.persistent = 1 if persistent else 0
        T.tfd_mlp_step(d, self._fws, stream=stream)

    def fused_barrier_error(self) -> int:
        """The fused kernel's barrier error word (nonzero: a wait timed out)."""
        if "_fws" not in self.__dict__:
            return 0
        return int(self._fws[0:4].view(torch.int32).item())

    def small(self) -> bool:
        """Whether the step's MatMuls are too small to fill the GPU one at a
        time (every activation under 2^22 elements): its time is launch
        latency more than arithmetic."""
        w = self.w
        return w.batch * max(w.dims) <= (1 << 22)

    def autotune_launch_mode(self, steps: int = 5):
        """Time the launch modes that apply (program order; the program
        captured into a HIP graph; tfd_mlp_step with one launch per phase) on
        `steps` chained steps each, keep the fastest as this step's default,
        and put the Variables back as they were. Returns the mean ms per mode."""
        saved = [t.clone() for t in self.variables()]
        if "_graph" not in self.__dict__:
            self._graph = self.capture(concurrent=False)
        modes = {"serial": self.run, "graph": self._graph.replay}
        if self.fusable():
            modes["fused"] = self.run_fused
        times = {}
        st = torch.cuda.current_stream()
        for mode, fn in modes.items():
            for _ in range(2):
                fn()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(st)
            for _ in range(steps):
                fn()
            b.record(st)
            torch.cuda.synchronize()
            times[mode] = a.elapsed_time(b) / steps
            for t, v in zip(self.variables(), saved):
                t.copy_(v)
        torch.cuda.synchronize()
        self._launch_mode = min(times, key=times.get)
        self.launch_times = times
        return times

    @property
    def launch_mode(self) -> str:
        """This step's default launch mode: the measured fastest of
        autotune_launch_mode for small steps (run on the first step()), the
        kernels in program order otherwise. On MI355X the small steps pick
        tfd_mlp_step with one launch per phase: 784x100 0.026 ms (graph replay
        0.041, program order 0.050), the 784-1024-1024-10 MLP 0.098 ms
        (program order 0.13, graph replay 0.137)."""
        if "_launch_mode" in self.__dict__:
            return self._launch_mode
        return "auto" if self.small() else "serial"

    def step(self, stream=None):
        """One step in this step's default launch mode (launch_mode)."""
        mode = self.launch_mode
        if mode == "auto":
            self.autotune_launch_mode()
            mode = self._launch_mode
        if mode == "serial":
            self.run(stream=stream)
        elif mode == "fused":
            self.run_fused(stream=stream)
        else:
            st = stream or torch.cuda.current_stream()
            with torch.cuda.stream(st):
                self._graph.replay()

    def capture(self, concurrent=True, num_streams=3):
        """Record one step into a HIP graph (torch.cuda.CUDAGraph); replaying
        it runs the same kernels on the same buffers. The library's calls
        only launch kernels (no allocation, no memset), so they capture.

        Python's cyclic garbage collector stays off during the capture, after
        a collection beforehand: a dead object cycle that holds GPU objects
        (a step's own HIP graph, events, tensors; DenseStep's launch closures
        refer back to the step) would otherwise be destroyed in the middle of
        the capture, and destructors that call the runtime while a stream is
        being captured abort the process."""
        g = torch.cuda.CUDAGraph()
        if concurrent:
            ex = self.executor(num_streams)
        torch.cuda.synchronize()
        gc.collect()
        was_enabled = gc.isenabled()
        gc.disable()
        try:
            with torch.cuda.graph(g):
                if concurrent:
                    ex.enqueue(torch.cuda.current_stream())
                else:
                    self.run()
        finally:
            if was_enabled:
                gc.enable()
        torch.cuda.synchronize()
        return g

    def dy_of(self, l: int) -> torch.Tensor:
        """dY of layer l (0-based): the masked gradient, or the incoming
        gradient itself on an identity layer."""
        if self.w.relus[l]:
            return self.dy[l]
        return self.g if l == self.w.layers - 1 else self.dx[l + 1]
