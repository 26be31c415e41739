"""Benchmark of one dense-layer training step (forward, gradient subgraph,
SGD update) through libtfdense on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

Prints ONE JSON line. The headline workload is the 4-layer, 4096-wide MLP
with 16-bit activations/weights, fp32 accumulation and fp32 master weights,
batch 16384 ("wide4096x4-bf16"); its fp32 twin at batch 8192
("wide4096x4-f32"), the truncating 16-bit variant, the tall 512 -> 32768 layer
and the MNIST-shaped steps are timed in the same run and reported under
"also"; the per-replica GEMM shapes of an 8-way batch split under
"per_replica".

Timing. Inputs are generated once and stay resident in HBM. Every step
starts from the same Variables (a stream-ordered restore before the step's
start event), so each timed step is exactly the computation the parity tests
check. Per workload:
  1. W warm-up steps;
  2. a per-op pass (K steps, a HIP event between every two launches) that
     gives the per-op breakdown and picks the dominant kernel: the GEMM
     kernel variant (layout, fused epilogue, shape) with the most time per
     step;
  3. the timed pass (K steps): HIP events at the step boundaries and around
     each launch of the dominant kernel only, on the launch stream.
     ms_per_step is the mean step interval, value = GEMM FLOPs per step
     (sum of 2 m n k) / ms_per_step; roofline.achieved = the dominant
     kernel's FLOPs per launch / its mean launch interval in this pass.
The MNIST-shaped steps are launch-bound: their value comes from the fastest
unmarked launch mode (one stream, several streams, HIP graph replay of
either, the one-kernel step).

The cpu_baseline leg times the oracle (float64 numpy) on bounded row samples
of every workload on the host cores, and compares the oracle's row-local
outputs (H, G, dY, dX) on those rows with the GPU's from the timed pass
(parity ratios max|err| / D, ReLU decisions inside the rounding band).
"""

from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "TFLOP/s per dense-layer fwd+bwd+SGD step; % of MI355X MFMA peak"
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2516.6}   # dense MFMA peaks (256 CUs x 2.4 GHz)
HBM_PEAK_GBS = 8000.0
PRIMARY = "wide4096x4-bf16"
# steps too small to fill the GPU with one kernel at a time: also timed with
# concurrent streams and HIP graph replay
LAUNCH_BOUND = ("mlp784-1024-1024-10-xent", "mlp784-1024-1024-10", "dense784x100")
SECONDARY = ("wide4096x4-f32", "wide4096x4-bf16-trunc", "tall512x32768-bf16", "mlp784-1024-1024-10-xent",
             "mlp784-1024-1024-10", "dense784x100")
# oracle samples (batch rows) per workload: bounded CPU work, about 15 s in all
CPU_ROWS = {"wide4096x4-bf16": 4096, "wide4096x4-f32": 2048, "tall512x32768-bf16": 2048,
            "mlp784-1024-1024-10": None, "dense784x100": None}
KERNEL_SOURCES = {"bf16": "paper_1603_04467_amd/csrc/gemm_bf16.hip", "f32": "paper_1603_04467_amd/csrc/gemm.hip"}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.md")


# ----------------------------------------------------------------- kernels

def _op_kind(name: str) -> str:
    for p in ("fwd", "dx", "dw", "relugrad", "sgd", "loss"):
        if name.startswith(p):
            return p
    return name


def op_info(s, tag):
    """What the launch of op `tag` computes: for GEMMs the layout, fused
    epilogue, shape and FLOPs (and a kernel id shared by every launch of the
    same kernel variant), for the memory-bound ops their compulsory bytes."""
    from paper_1603_04467_amd import tfdense as T
    from paper_1603_04467_amd.step import fused_below, fused_top

    w = s.w
    kind = _op_kind(tag)
    l = int(tag[len(kind):]) - 1 if tag[len(kind):].isdigit() else None
    eb = 2 if w.act == "bf16" else 4
    N, L = w.batch, w.layers
    d = {"kind": kind}
    if kind in ("fwd", "dx", "dw"):
        if kind == "fwd":
            m, n, k, lay = N, w.dims[l + 1], w.dims[l], s.forward_layout
            if l == L - 1 and fused_top(w, s.fuse):
                epi = "bias+sq_err+colsum"
            elif s.masks[l] is not None:
                epi = "bias_relu+mask"
            else:
                epi = "bias_relu" if w.relus[l] else "bias"
        elif kind == "dx":
            m, n, k, lay = N, w.dims[l], w.dims[l + 1], "NT"
            if fused_below(w, l, s.fuse):
                epi = "relugrad_mask+colsum" if s.masks[l - 1] is not None else "relugrad+colsum"
            else:
                split = T.tfd_matmul_workspace_size(m, n, k, s.act, s.act, transpose_b=True) > 0
                epi = "splitk" if split else "none"
        else:
            m, n, k, lay = w.dims[l], w.dims[l + 1], N, "TN"
            epi = "none"
        out = "f32" if kind == "dw" else w.act
        ob = 4 if out == "f32" else eb
        # operands in, product out, plus what the fused epilogue reads and writes
        extra = {"bias_relu+mask": m * n // 8 + 4 * n, "bias_relu": 4 * n, "bias": 4 * n,
                 "bias+sq_err+colsum": 2 * m * n * eb + 4 * n + 4 * n * (m // 256),
                 "relugrad_mask+colsum": m * n // 8 + 4 * n * (m // 256),
                 "relugrad+colsum": m * n * eb + 4 * n * (m // 256)}.get(epi, 0)
        d.update(layout=lay, epi=epi, shape=[m, n, k], flops=2 * m * n * k,
                 kernel=f"gemm {w.act} {lay} {epi} {m}x{n}x{k} -> {out}",
                 algorithmic_bytes=m * k * eb + k * n * eb + m * n * ob + extra)
    elif kind == "relugrad":
        M = w.dims[l + 1]
        if not w.relus[l]:
            byt = N * M * eb + 4 * M                 # BiasAddGrad alone
        elif s.use_masks:
            byt = 2 * N * M * eb + N * M // 8 + 4 * M  # gradient and 1-bit mask in, dY out
        else:
            byt = 3 * N * M * eb + 4 * M             # gradient and features in, dY out
        d["bytes"] = byt
    elif kind == "sgd":
        K, M = w.dims[l], w.dims[l + 1]
        d["bytes"] = K * M * (12 + (4 if w.masters else 0)) + 12 * M
    elif kind == "loss":
        d["bytes"] = 3 * N * w.dims[-1] * eb if w.cost != "xent" else 2 * N * w.dims[-1] * eb + 4 * N
    return d


# ----------------------------------------------------------------- clock

def _clock_probe_mhz(counters):
    c = counters.cpu().numpy()
    return [100.0 * float(r[0]) / float(r[1]) for r in c if r[1] > 0]


CLOCK_PROBES = 8


def sample_clock(s, probes: int = CLOCK_PROBES, iterations: int = 50_000):
    """Engine clock in MHz, from tfd_clock_probe (shader clock cycles over
    100 MHz real-time ticks in one wave, about 1 ms): `probes` probes each
    enqueued right behind a step (restored Variables, as in the timed pass),
    so that it runs at the clock the step left the GPU at, and as many with
    the GPU idle before. The probe runs on the launch stream, never beside a
    step: a wave of its own on one compute unit would keep a workgroup of the
    whole-tile GEMMs (one per compute unit, one round over the chip) off that
    unit and stretch the GEMM it overlaps."""
    import torch

    from paper_1603_04467_amd import tfdense as T

    after = torch.zeros(probes, 3, dtype=torch.int64, device="cuda")
    idle = torch.zeros(probes, 3, dtype=torch.int64, device="cuda")
    torch.cuda.synchronize()
    for i in range(probes):
        T.tfd_clock_probe(idle[i], iterations)
        torch.cuda.synchronize()
        time.sleep(0.01)
    for i in range(probes):
        s.restore()
        s.run()
        T.tfd_clock_probe(after[i], iterations)
    torch.cuda.synchronize()

    def stats(v):
        return {"median": round(float(np.median(v)), 1), "min": round(float(np.min(v)), 1),
                "max": round(float(np.max(v)), 1), "probes": len(v)} if v else None
    return {"after_step": stats(_clock_probe_mhz(after)), "idle": stats(_clock_probe_mhz(idle)),
            "source": "tfd_clock_probe: 100 * s_memtime cycles / s_memrealtime ticks of one wave over about 1 ms; "
                      "after_step: enqueued right behind a step on the launch stream"}


# ----------------------------------------------------------------- timing

def _event():
    import torch
    return torch.cuda.Event(enable_timing=True)


def time_workload(name: str, steps: int, warmup: int, keep_rows: int = 0, clock: bool = False):
    import torch

    from paper_1603_04467_amd import workloads
    from paper_1603_04467_amd.step import DenseStep

    w = workloads.workload(name)
    inp = workloads.generate(w, seed=0)
    s = DenseStep(w, inp)
    stream = torch.cuda.current_stream()
    tags = [n.name for n in s.nodes()]
    info = {t: op_info(s, t) for t in tags}

    for _ in range(warmup):
        s.restore()
        s.run()
    torch.cuda.synchronize()

    # per-op pass: an event between every two launches
    op_ev = []
    for _ in range(steps):
        s.restore()
        marks = []

        def mark(tag, marks=marks):
            e = _event()
            e.record(stream)
            marks.append((tag, e))

        s.run(mark=mark)
        op_ev.append(marks)
    torch.cuda.synchronize()
    per_op = {}
    for marks in op_ev:
        for (tag, e0), (_, e1) in zip(marks[:-1], marks[1:]):
            per_op.setdefault(tag, []).append(e0.elapsed_time(e1))
    ops = {}
    for tag in tags:
        d = dict(info[tag])
        d["ms"] = float(np.mean(per_op[tag]))
        if "flops" in d:
            d["tflops"] = d["flops"] / (d["ms"] * 1e-3) / 1e12
        if "bytes" in d:
            d["gbs"] = d["bytes"] / (d["ms"] * 1e-3) / 1e9
        ops[tag] = d

    # dominant kernel: the GEMM kernel variant with the most time per step
    by_kernel = {}
    for tag, d in ops.items():
        if "kernel" in d:
            by_kernel.setdefault(d["kernel"], []).append(tag)
    dom_kernel, dom_tags = max(by_kernel.items(), key=lambda kv: sum(ops[t]["ms"] for t in kv[1]))

    # timed pass: step boundaries and the dominant kernel's launches only
    step_ev, dom_ev = [], []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        s.restore()
        open_ = []

        def mark(tag, open_=open_):
            if open_:
                e = _event()
                e.record(stream)
                dom_ev.append((open_.pop(), e))
            if tag in dom_tags:
                e = _event()
                e.record(stream)
                open_.append(e)

        a, b = _event(), _event()
        a.record(stream)
        s.run(mark=mark)
        b.record(stream)
        step_ev.append((a, b))
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps * 1e3
    step_ms = [a.elapsed_time(b) for a, b in step_ev]
    dom_ms = [a.elapsed_time(b) for a, b in dom_ev]
    ms = float(np.mean(step_ms))
    pct = {f"p{q}": round(float(np.percentile(step_ms, q)), 4) for q in (10, 50, 90)}
    tflops = w.flops() / (ms * 1e-3) / 1e12
    dom = info[dom_tags[0]]
    dom_mean = float(np.mean(dom_ms))
    achieved = dom["flops"] / (dom_mean * 1e-3) / 1e12
    peak = PEAK_TFLOPS[w.act]
    traffic = lookup_traffic(dom_kernel, w.act)
    out = {
        "workload": w,
        "ms": ms,
        "ms_percentiles": pct,
        "wall_ms": wall,
        "tflops": tflops,
        "pct_peak": 100.0 * tflops / peak,
        "ops": ops,
        "clock": sample_clock(s) if clock else None,
        "roofline": {
            "bound": "mfma",
            "kernel": dom_kernel,
            "launches_per_step": len(dom_tags),
            # the dominant kernel's launches in this workload's leg, in order:
            # warm-up, per-op pass, timed pass, clock-probe pass
            "launches_in_leg": len(dom_tags) * (warmup + 2 * steps + (CLOCK_PROBES if clock else 0)),
            "timed_launches": [len(dom_tags) * (warmup + steps), len(dom_tags) * (warmup + 2 * steps)],
            "ms_per_launch": round(dom_mean, 5),
            "achieved": round(achieved, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": None if traffic is None else traffic["bytes"],
            "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE x2 + WRITE_SIZE x1, calibrated)",
            "algorithmic_bytes": dom["algorithmic_bytes"],
            "flops_per_launch": dom["flops"],
            "src": KERNEL_SOURCES[w.act],
        },
        "loss": float(s.loss.item()),
        "invariants": invariants(s),
    }
    if keep_rows:
        out["gpu_rows"] = _gpu_rows(s, keep_rows)
    if name in LAUNCH_BOUND:
        out["launch_modes"] = time_modes(s, steps, warmup)
    del s
    torch.cuda.empty_cache()
    return out


def invariants(s):
    """Identities the step's own tensors (from the timed pass) must satisfy,
    counted on the GPU in full (measurement only): ReLU masks equal the signs
    of the stored activations; a ReluGrad output is +0 wherever its layer's
    activation is not > 0; each bias gradient equals the column sums of its dY within the fp32 sum
    bound 2 N 2^-24 sum|dY| (reported as the largest ratio to that bound)."""
    import torch

    w, L = s.w, s.w.layers
    out = {"mask_bit_mismatches": 0, "relugrad_nonzero_where_inactive": 0}
    for l in range(L):
        h = s.h[l + 1]
        if s.masks[l] is not None and h.shape[1] % 32 == 0:
            bits = (h > 0).view(h.shape[0], -1, 32).to(torch.int64)
            words = (bits << torch.arange(32, device=h.device)).sum(dim=2)
            got = s.masks[l][:, :words.shape[1]].to(torch.int64) & 0xFFFFFFFF
            out["mask_bit_mismatches"] += int((got != words).sum().item())
        if w.relus[l] and s.dy[l] is not None:
            dy = s.dy_of(l)
            bad = (h <= 0) & ((dy != 0) | torch.signbit(dy))
            out["relugrad_nonzero_where_inactive"] += int(bad.sum().item())
    worst = 0.0
    for l in range(L):
        dy = s.dy_of(l).double()
        col = dy.sum(dim=0)
        bound = 2.0 * w.batch * 2.0 ** -24 * dy.abs().sum(dim=0) + 2.0 ** -24 * col.abs()
        r = ((s.db[l].double() - col).abs() / bound.clamp_min(1e-300)).max().item()
        worst = max(worst, r)
    out["db_colsum_ratio_to_bound"] = round(worst, 4)
    return out


def _gpu_rows(s, rows):
    """Host copies of the step's row-local outputs on batch rows 0..rows-1
    (the oracle's sample), for the parity ratios."""
    from paper_1603_04467_amd.step import fused_below

    def f64(t):
        return t[:rows].float().cpu().numpy().astype(np.float64)
    L = s.w.layers
    return {
        "h": [f64(t) for t in s.h],
        "g": f64(s.g),
        "dy": [f64(s.dy_of(l)) for l in range(L)],
        "dx": [None if fused_below(s.w, l, s.fuse) else f64(s.dx[l]) for l in range(L)],
    }


def time_modes(s, steps: int, warmup: int, num_streams: int = 3):
    """Step time under the launch modes, without per-op events: one stream
    in program order ("serial"), independent ops on `num_streams` streams
    ("streams"), both captured into a HIP graph and replayed ("graph",
    "graph_streams"), and, where the step qualifies, the step through
    tfd_mlp_step: one launch per phase ("fused") or one persistent kernel
    ("fused_persistent"). Every step starts from the
    same Variables (restore outside the timed interval); times are HIP-event
    means in ms."""
    import torch

    stream = torch.cuda.current_stream()
    graphs = {"graph": s.capture(concurrent=False),
              "graph_streams": s.capture(concurrent=True, num_streams=num_streams)}
    modes = {
        "serial": s.run,
        "streams": lambda: s.run_concurrent(num_streams),
        "graph": graphs["graph"].replay,
        "graph_streams": graphs["graph_streams"].replay,
    }
    if s.fusable():
        modes["fused"] = s.run_fused
        modes["fused_persistent"] = lambda: s.run_fused(persistent=True)
    out = {}
    for mode, fn in modes.items():
        for _ in range(warmup):
            s.restore()
            fn()
        ev = []
        for _ in range(steps):
            s.restore()
            a, b = _event(), _event()
            a.record(stream)
            fn()
            b.record(stream)
            ev.append((a, b))
        torch.cuda.synchronize()
        out[mode] = round(float(np.mean([a.elapsed_time(b) for a, b in ev])), 4)
    best = min(out, key=out.get)
    return {"ms_per_step": out, "best": best, "tflops_best": round(s.w.flops() / (out[best] * 1e-3) / 1e12, 3)}


def time_per_replica(reps: int = 20, replicas: int = 8):
    """GEMMs of one 4096-wide layer at the per-replica batch of a `replicas`-way
    data-parallel split (the part of the synchronous data-parallel step one
    GPU can show): forward, input gradient and weight gradient, fp32 at
    8192 / replicas rows and 16-bit at 16384 / replicas rows."""
    import torch

    from paper_1603_04467_amd import tfdense as T

    stream = torch.cuda.current_stream()
    out = {}
    for dt, batch in (("f32", 8192), ("bf16", 16384)):
        tdt = torch.bfloat16 if dt == "bf16" else torch.float32
        n = batch // replicas
        x = torch.randn(n, 4096, device="cuda").to(tdt)
        wt = (torch.randn(4096, 4096, device="cuda") / 64).to(tdt)
        dy = torch.randn(n, 4096, device="cuda").to(tdt)
        bias = torch.zeros(4096, device="cuda")
        y = torch.empty(n, 4096, dtype=tdt, device="cuda")
        dw = torch.empty(4096, 4096, device="cuda")
        calls = {
            f"fwd {n}x4096x4096 NT": lambda: T.tfd_matmul(x, wt, y, transpose_b=True, bias=bias, epilogue="bias_relu"),
            f"dx {n}x4096x4096 NT": lambda: T.tfd_matmul(dy, wt, y, transpose_b=True),
            f"dw 4096x4096x{n} TN": lambda: T.tfd_matmul(x, dy, dw, transpose_a=True),
        }
        res = {}
        for name, fn in calls.items():
            for _ in range(3):
                fn()
            ev = [_event() for _ in range(reps + 1)]
            ev[0].record(stream)
            for i in range(reps):
                fn()
                ev[i + 1].record(stream)
            torch.cuda.synchronize()
            ms = float(np.mean([ev[i].elapsed_time(ev[i + 1]) for i in range(reps)]))
            f = 2 * n * 4096 * 4096
            res[name] = {"ms": round(ms, 4), "tflops": round(f / (ms * 1e-3) / 1e12, 1),
                         "frac": round(f / (ms * 1e-3) / 1e12 / PEAK_TFLOPS[dt], 3)}
        out[f"{dt} batch {batch}/{replicas}"] = res
    return out


def time_conversions(count: int = 1 << 26, reps: int = 20):
    """The 32 <-> 16-bit conversion ops of section 5.5 on `count` elements
    (fp32 -> 16 truncating and nearest even, 16 -> fp32), resident in HBM:
    mean launch time from HIP events and GB/s of compulsory traffic."""
    import torch

    from paper_1603_04467_amd import tfdense as T

    stream = torch.cuda.current_stream()
    src = torch.randn(count, device="cuda")
    h = torch.empty(count, dtype=torch.bfloat16, device="cuda")
    back = torch.empty(count, device="cuda")
    calls = {
        "f32_to_bf16_truncate": (lambda: T.tfd_convert_f32_to_bf16(src, h, rounding="truncate"), 6 * count),
        "f32_to_bf16_nearest": (lambda: T.tfd_convert_f32_to_bf16(src, h, rounding="nearest"), 6 * count),
        "bf16_to_f32": (lambda: T.tfd_convert_bf16_to_f32(h, back), 6 * count),
    }
    out = {}
    for name, (fn, byt) in calls.items():
        for _ in range(3):
            fn()
        ev = [_event() for _ in range(reps + 1)]
        ev[0].record(stream)
        for i in range(reps):
            fn()
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        ms = float(np.mean([ev[i].elapsed_time(ev[i + 1]) for i in range(reps)]))
        out[name] = {"elements": count, "ms": round(ms, 4), "gbs": round(byt / (ms * 1e-3) / 1e9, 1),
                     "frac_hbm": round(byt / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 3)}
    return out


# ----------------------------------------------------------------- records

def _sha256(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def lookup_traffic(kernel: str, dtype: str):
    """Bytes per launch (FETCH_SIZE and WRITE_SIZE, each scaled by its
    calibration factor) recorded for `kernel` in profiles/traffic.md, or None.
    A record applies only while the kernel's source file is unchanged (its
    sha256 is part of the record)."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    src = _sha256(os.path.join(ROOT, KERNEL_SOURCES[dtype]))
    for line in open(TRAFFIC_FILE):
        if not line.startswith("record "):
            continue
        kv = dict(item.split("=", 1) for item in line[len("record "):].strip().split(" ; "))
        if kv.get("kernel") == kernel and kv.get("src_sha256") == src:
            fetch = float(kv["fetch_kib"]) * float(kv["fetch_scale"]) * 1024
            write = float(kv["write_kib"]) * float(kv["write_scale"]) * 1024
            return {"bytes": fetch + write, "fetch_bytes": fetch, "write_bytes": write}
    return None


def revision():
    """git revision of the tree when .git is present, and a hash of the
    library sources either way."""
    rev = None
    try:
        r = subprocess.run(["git", "-C", ROOT, "rev-parse", "--short=12", "HEAD"], capture_output=True, text=True,
                           timeout=10)
        if r.returncode == 0:
            rev = r.stdout.strip()
    except (OSError, subprocess.TimeoutExpired):
        pass
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(ROOT, "paper_1603_04467_amd", "csrc", "*"))):
        h.update(os.path.basename(p).encode())
        h.update(open(p, "rb").read())
    return {"git": rev, "csrc_sha256": h.hexdigest()[:16]}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


# ----------------------------------------------------------------- oracle leg

def _oracle_inputs(w, rows):
    import oracle
    from paper_1603_04467_amd import workloads

    inp = workloads.generate(w, seed=0)
    conv = oracle.bf16_bits_to_f64 if w.act == "bf16" else (lambda a: a.astype(np.float64))
    sl = slice(0, rows)
    return {
        "x": conv(inp["x"])[sl],
        "weights": [conv(a) for a in inp["weights"]],
        "biases": [a.astype(np.float64) for a in inp["biases"]],
        "masters": None if inp["masters"] is None else [a.astype(np.float64) for a in inp["masters"]],
        "target": None if inp["target"] is None else conv(inp["target"])[sl],
        "upstream": None if inp["upstream"] is None else conv(inp["upstream"])[sl],
        "labels": None if inp.get("labels") is None else inp["labels"][sl],
    }


def _run_oracle(w, hi):
    import oracle
    return oracle.dense_step(hi["x"], hi["weights"], hi["biases"], list(w.relus), act=w.act, target=hi["target"],
                             upstream_grad=hi["upstream"], lr=w.lr, masters=hi["masters"], update=w.update,
                             labels=hi["labels"], rounding=w.rounding)


def _parity(w, hi, ref, gpu, tau):
    """Normalised errors max|err| / D of the GPU's row-local outputs against
    the oracle's chain on the same rows (D as in the parity tests), and the
    ReLU decisions: how many differ from the sign of the oracle's
    pre-activation, all of which must lie in the band |y| <= tau D."""
    import oracle

    def ne(got, want, D):
        return float(np.max(np.abs(got - want)) / D) if got.size and D > 0 else 0.0

    out, flips, band = {}, 0, 0
    amax = lambda a: float(np.max(np.abs(a))) if np.size(a) else 0.0  # noqa: E731
    D_fwd = []
    for l in range(w.layers):
        D = w.dims[l] * amax(ref["h"][l]) * amax(hi["weights"][l]) + amax(hi["biases"][l])
        D_fwd.append(D)
        out[f"H{l + 1}"] = ne(gpu["h"][l + 1], ref["h"][l + 1], D)
        if w.relus[l]:
            y = oracle.matmul(ref["h"][l], hi["weights"][l], out="f64", bias=hi["biases"][l])
            inb = np.abs(y) <= tau * D
            diff = (gpu["h"][l + 1] > 0) != (y > 0)
            band += int(inb.sum())
            flips += int(diff.sum())
            out[f"relu{l + 1}_flips_outside_band"] = int((diff & ~inb).sum())
    D_g = D_fwd[-1] + amax(ref["g"]) if w.cost != "upstream" else amax(ref["g"])
    out["G"] = ne(gpu["g"], ref["g"], D_g)
    # row-local gradients on rows no ReLU flip touched
    touched = np.zeros(gpu["g"].shape[0], dtype=bool)
    for l in range(w.layers):
        if w.relus[l]:
            touched |= np.any((gpu["h"][l + 1] > 0) != (ref["h"][l + 1] > 0), axis=1)
    keep = ~touched
    for l in reversed(range(w.layers)):
        md = amax(ref["dy"][l])
        out[f"dY{l + 1}"] = ne(gpu["dy"][l][keep], ref["dy"][l][keep], D_g)
        D_g = w.dims[l + 1] * md * amax(hi["weights"][l])
        if gpu["dx"][l] is not None:
            out[f"dX{l + 1}"] = ne(gpu["dx"][l][keep], ref["dx"][l][keep], D_g)
    return {"max_err_over_D": {k: (round(v, 8) if isinstance(v, float) else v) for k, v in out.items()},
            "relu_flips": flips, "mask_band_count": band, "rows_compared": int(keep.sum()), "tau": tau}


def cpu_baseline(results, threads):
    """The oracle's full step on bounded row samples of every workload, on
    the host cores; C1 and C2 whole (median of 5, and with one thread).
    Returns the headline workload's figure with the others beside it."""
    from threadpoolctl import threadpool_limits

    from paper_1603_04467_amd import workloads

    tau = {"f32": 1e-5, "bf16": 1e-2}
    per = {}
    for name, rows in CPU_ROWS.items():
        w = workloads.workload(name)
        rows = rows or w.batch
        hi = _oracle_inputs(w, rows)
        reps = 5 if rows == w.batch else 1
        times = []
        with threadpool_limits(limits=threads):
            for _ in range(reps):
                t0 = time.perf_counter()
                ref = _run_oracle(w, hi)
                times.append(time.perf_counter() - t0)
        dt = float(np.median(times))
        flops = w.scaled(batch=rows).flops()
        d = {"rows": rows, "of_batch": w.batch, "step_s": round(dt, 4), "tflops": round(flops / dt / 1e12, 5),
             "repeats": reps}
        if rows == w.batch:
            t1 = []
            with threadpool_limits(limits=1):
                for _ in range(reps):
                    t0 = time.perf_counter()
                    _run_oracle(w, hi)
                    t1.append(time.perf_counter() - t0)
            d["step_s_one_thread"] = round(float(np.median(t1)), 4)
        r = results.get(name)
        if r is not None and r.get("gpu_rows") is not None:
            g = {k: v for k, v in r["gpu_rows"].items()}
            g = {"h": [a[:rows] for a in g["h"]], "g": g["g"][:rows], "dy": [a[:rows] for a in g["dy"]],
                 "dx": [None if a is None else a[:rows] for a in g["dx"]]}
            d["parity"] = _parity(w, hi, ref, g, tau[w.act])
        per[name] = d
    head = per[PRIMARY]
    return {
        "value": head["tflops"],
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{PRIMARY}: one full step (forward, gradients, update) on batch rows 0..{head['rows'] - 1} of "
                  f"{head['of_batch']}, float64 numpy, in {head['step_s']} s",
        "cpu_model": cpu_model(),
        "workloads": per,
    }


# ----------------------------------------------------------------- main

def _per_op(ops):
    out = {}
    for k, v in ops.items():
        d = {"ms": round(v["ms"], 4)}
        if "tflops" in v:
            d["tflops"] = round(v["tflops"], 1)
            d["kernel"] = v["kernel"]
            d["algorithmic_bytes"] = v["algorithmic_bytes"]
            t = lookup_traffic(v["kernel"], v["kernel"].split()[1])
            if t is not None:
                d["traffic_bytes"] = round(t["bytes"])
        if "gbs" in v:
            d["gbs"] = round(v["gbs"], 1)
        out[k] = d
    return out


def _entry(name, r):
    e = {
        "workload": name,
        "value": round(r["tflops"], 3),
        "unit": "TFLOP/s",
        "ms_per_step": round(r["ms"], 4),
        "ms_per_step_percentiles": r["ms_percentiles"],
        "pct_mfma_peak": round(r["pct_peak"], 2),
        "roofline": r["roofline"],
        "per_op": _per_op(r["ops"]),
        "loss": r["loss"],
        "invariants": r["invariants"],
    }
    if "launch_modes" in r:
        lm = r["launch_modes"]
        best = lm["ms_per_step"][lm["best"]]
        e["launch_modes"] = lm
        e["ms_per_step_marked"] = e["ms_per_step"]
        e["ms_per_step"] = best
        e["value"] = round(r["workload"].flops() / (best * 1e-3) / 1e12, 3)
        e["pct_mfma_peak"] = round(100 * e["value"] / PEAK_TFLOPS[r["workload"].act], 3)
        e["value_source"] = f"fastest unmarked launch mode ({lm['best']})"
    return e


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=PRIMARY)
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(the data-parallel sharding is a design note only).", file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "no GPU visible"
    torch.cuda.set_device(0)
    want_rows = not args.no_cpu_baseline

    print(f"bench: timing {args.workload} ({args.steps} steps, {args.warmup} warm-up)", file=sys.stderr, flush=True)
    results = {}
    keep = (CPU_ROWS.get(args.workload) or workloads_batch(args.workload)) if want_rows else 0
    r = time_workload(args.workload, args.steps, args.warmup, keep_rows=keep, clock=True)
    results[args.workload] = r
    w = r["workload"]
    out = {
        "metric": METRIC,
        "value": round(r["tflops"], 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms"], 4),
        "ms_per_step_percentiles": r["ms_percentiles"],
        "wall_ms_per_step": round(r["wall_ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.act,
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "batch": w.batch,
            "dims": list(w.dims),
            "relus": list(w.relus),
            "storage": w.act,
            "accumulate": "f32",
            "master_weights": "f32" if (w.masters or w.act == "f32") else None,
            "lr": w.lr,
            "gemm_flops_per_step": w.flops(),
        },
        "pct_mfma_peak": round(r["pct_peak"], 2),
        "roofline": r["roofline"],
        "per_op": _per_op(r["ops"]),
        "sclk_mhz": r["clock"],
        "loss": r["loss"],
        "invariants": r["invariants"],
        "revision": revision(),
    }
    if not args.no_secondary and args.workload == PRIMARY:
        out["also"] = []
        for name in SECONDARY:
            print(f"bench: timing {name}", file=sys.stderr, flush=True)
            keep = (CPU_ROWS.get(name) or workloads_batch(name)) if (want_rows and name in CPU_ROWS) else 0
            r2 = time_workload(name, args.steps, args.warmup, keep_rows=keep)
            results[name] = r2
            out["also"].append(_entry(name, r2))
        print("bench: timing the per-replica GEMM shapes", file=sys.stderr, flush=True)
        out["per_replica"] = time_per_replica()
        print("bench: timing the 32 <-> 16-bit conversions", file=sys.stderr, flush=True)
        out["conversions"] = time_conversions()
    if want_rows:
        threads = len(os.sched_getaffinity(0))
        print(f"bench: timing the oracle on {threads} host threads", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(results, threads)
    print(json.dumps(out), flush=True)


def workloads_batch(name):
    from paper_1603_04467_amd import workloads
    return workloads.workload(name).batch


if __name__ == "__main__":
    main()
