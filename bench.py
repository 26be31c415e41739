"""Benchmark of one dense-layer training step (forward, gradient subgraph,
SGD update) through libtfdense on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

Prints ONE JSON line. The headline workload is the 4-layer, 4096-wide MLP
with 16-bit activations/weights, fp32 accumulation and fp32 master weights,
batch 16384 ("wide4096x4-bf16"); its fp32 twin at batch 8192
("wide4096x4-f32"), the truncating 16-bit variant, the tall 512 -> 32768 layer
and the MNIST-shaped steps are timed in the same run and reported under "also".

Timing: every step starts from the same Variables (a stream-ordered restore
before the step's start event), so each timed step is exactly the computation
the parity tests check. ms_per_step is the mean of the per-step HIP event
intervals on the launch stream; the host-side bracket (synchronize on both
sides of the K steps, restores included) is reported as wall_ms_per_step.
Throughput counts the step's GEMM FLOPs, sum of 2*m*n*k.
The cpu_baseline leg times the oracle (float64 numpy) on a row slice of the
same workload on the host cores.
"""

from __future__ import annotations

import argparse
import json
import os
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
# timed in the same run and reported under "also": the fp32 twin, the truncating
# 16-bit variant, the tall 512 -> 32768 layer (given upstream gradient, no update),
# then the MNIST-shaped steps (classifier head and squared-error head) and the single layer
SECONDARY = ("wide4096x4-f32", "wide4096x4-bf16-trunc", "tall512x32768-bf16", "mlp784-1024-1024-10-xent",
             "mlp784-1024-1024-10", "dense784x100")


def _gemm_bytes(shape, layout, eb):
    """Compulsory HBM bytes of one GEMM: read A and B once, write C once
    (the weight gradient is written in fp32)."""
    m, n, k = shape
    out = 4 if layout == "TN" else eb
    return m * k * eb + k * n * eb + m * n * out


def _op_kind(name: str) -> str:
    for p in ("fwd", "dx", "dw", "relugrad", "sgd", "loss"):
        if name.startswith(p):
            return p
    return name


def time_workload(name: str, steps: int, warmup: int):
    import torch

    from paper_1603_04467_amd import workloads
    from paper_1603_04467_amd.step import DenseStep

    w = workloads.workload(name)
    inp = workloads.generate(w, seed=0)
    s = DenseStep(w, inp)
    stream = torch.cuda.current_stream()

    for _ in range(warmup):
        s.restore()
        s.run()
    torch.cuda.synchronize()

    # per-step and per-op events, recorded on the launch stream
    step_ev = []
    op_ev = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        s.restore()
        marks = []

        def mark(tag, marks=marks):
            e = torch.cuda.Event(enable_timing=True)
            e.record(stream)
            marks.append((tag, e))

        s.run(mark=mark)
        step_ev.append((marks[0][1], marks[-1][1]))
        op_ev.append(marks)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps * 1e3

    step_ms = [a.elapsed_time(b) for a, b in step_ev]
    per_op = {}
    for marks in op_ev:
        for (tag, e0), (_, e1) in zip(marks[:-1], marks[1:]):
            per_op.setdefault(tag, []).append(e0.elapsed_time(e1))
    ms = float(np.mean(step_ms))
    pct = {f"p{q}": round(float(np.percentile(step_ms, q)), 4) for q in (10, 50, 90)}
    flops = w.flops()
    tflops = flops / (ms * 1e-3) / 1e12

    # per-op summary: mean ms, and FLOP/s or bytes/s against the roofline
    gemm_shapes = w.gemm_shapes()
    L = w.layers
    eb = 2 if w.act == "bf16" else 4
    N = w.batch
    ops = {}
    for tag, v in per_op.items():
        kind = _op_kind(tag)
        l = int(tag[len(kind):]) if tag[len(kind):].isdigit() else None
        d = {"ms": float(np.mean(v))}
        if kind in ("fwd", "dx", "dw"):
            if kind == "fwd":
                m, n, k, lay = gemm_shapes[l - 1]
                lay = s.forward_layout
            else:
                idx = L + 2 * (L - l) + (0 if kind == "dx" else 1)
                m, n, k, lay = gemm_shapes[idx]
            f = 2 * m * n * k
            d.update(layout=lay, shape=[m, n, k], flops=f, tflops=f / (d["ms"] * 1e-3) / 1e12)
        elif kind == "relugrad":
            M = w.dims[l]
            if not w.relus[l - 1]:
                byt = N * M * eb + 4 * M                 # BiasAddGrad alone
            elif s.use_masks:
                byt = 2 * N * M * eb + N * M // 8 + 4 * M  # gradient and 1-bit mask in, dY out
            else:
                byt = 3 * N * M * eb + 4 * M             # gradient and features in, dY out
            d.update(bytes=byt, gbs=byt / (d["ms"] * 1e-3) / 1e9)
        elif kind == "sgd":
            K, M = w.dims[l - 1], w.dims[l]
            # fp32 var and delta read, var written; with fp32 masters also the
            # 16-bit copy and its transpose (2 + 2 bytes); the bias update
            byt = K * M * (12 + (4 if w.masters else 0)) + 12 * M
            d.update(bytes=byt, gbs=byt / (d["ms"] * 1e-3) / 1e9)
        elif kind == "loss":
            # squared error: output and target read, gradient written;
            # cross-entropy: logits read, gradient written, one label per row
            byt = 3 * N * w.dims[-1] * eb if w.cost != "xent" else 2 * N * w.dims[-1] * eb + 4 * N
            d.update(bytes=byt, gbs=byt / (d["ms"] * 1e-3) / 1e9)
        ops[tag] = d

    # dominant kernel: the GEMM layout with the most total time
    by_layout = {}
    for tag, d in ops.items():
        if "layout" in d:
            by_layout.setdefault(d["layout"], []).append(d)
    dom_layout, dom = max(by_layout.items(), key=lambda kv: sum(x["ms"] for x in kv[1]))
    dom_ms = float(np.mean([x["ms"] for x in dom]))
    dom_flops = dom[0]["flops"]
    achieved = dom_flops / (dom_ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[w.act]
    kernel_name = f"gemm_{dom_layout}_{w.act}"
    traffic = lookup_traffic(kernel_name, dom[0]["shape"], w.act)
    return {
        "workload": w,
        "ms": ms,
        "ms_percentiles": pct,
        "wall_ms": wall,
        "tflops": tflops,
        "pct_peak": 100.0 * tflops / peak,
        "ops": ops,
        "roofline": {
            "bound": "mfma",
            "kernel": kernel_name,
            "shape": dom[0]["shape"],
            "achieved": achieved,
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": achieved / peak,
            "traffic": None if traffic is None else traffic["bytes"],
            "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, calibrated)",
            "algorithmic_bytes": _gemm_bytes(dom[0]["shape"], dom_layout, eb),
            "src": KERNEL_SOURCES[w.act],
        },
        "loss": float(s.loss.item()),
    }


# HBM traffic of the dominant kernel, from rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE
# runs summarised under profiles/. A record applies only while the kernel's
# source file is unchanged (its sha256 is part of the record).
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.md")
KERNEL_SOURCES = {"bf16": "paper_1603_04467_amd/csrc/gemm_bf16.hip", "f32": "paper_1603_04467_amd/csrc/gemm.hip"}


def _sha256(path):
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def lookup_traffic(kernel: str, shape, dtype: str):
    """Bytes per launch (FETCH_SIZE and WRITE_SIZE, each scaled by its
    calibration factor) recorded for `kernel` at `shape`, or None."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    src = _sha256(os.path.join(ROOT, KERNEL_SOURCES[dtype]))
    want = f"{shape[0]}x{shape[1]}x{shape[2]}"
    for line in open(TRAFFIC_FILE):
        if not line.startswith("record "):
            continue
        kv = dict(item.split("=", 1) for item in line.split()[1:])
        if kv.get("kernel") == kernel and kv.get("shape") == want and kv.get("src_sha256") == src:
            fetch = float(kv["fetch_kib"]) * float(kv["fetch_scale"]) * 1024
            write = float(kv["write_kib"]) * float(kv["write_scale"]) * 1024
            return {"bytes": fetch + write, "fetch_bytes": fetch, "write_bytes": write}
    return None


def cpu_baseline(name: str, rows: int):
    """Time the oracle's step on the first `rows` batch rows of the workload."""
    import oracle
    from paper_1603_04467_amd import workloads

    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    w = workloads.workload(name)
    inp = workloads.generate(w, seed=0)
    conv = oracle.bf16_bits_to_f64 if w.act == "bf16" else (lambda a: a.astype(np.float64))
    x = conv(inp["x"])[:rows]
    t = None if inp["target"] is None else conv(inp["target"])[:rows]
    up = None if inp["upstream"] is None else conv(inp["upstream"])[:rows]
    lab = None if inp.get("labels") is None else inp["labels"][:rows]
    ws = [conv(a) for a in inp["weights"]]
    ms_ = None if inp["masters"] is None else [a.astype(np.float64) for a in inp["masters"]]
    bs = [a.astype(np.float64) for a in inp["biases"]]
    t0 = time.perf_counter()
    oracle.dense_step(x, ws, bs, list(w.relus), act=w.act, target=t, upstream_grad=up, lr=w.lr, masters=ms_,
                      update=w.update, labels=lab)
    dt = time.perf_counter() - t0
    flops = w.scaled(batch=rows).flops()
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"{name}: one full step on batch rows 0..{rows - 1} of {w.batch} "
                  f"({flops / 1e12:.3f} TFLOP in {dt:.1f} s, float64 numpy)",
    }


def time_modes(name: str, steps: int, warmup: int, num_streams: int = 3):
    """Step time of one workload under four launch modes: one stream in
    program order ("serial"), independent ops on `num_streams` streams
    ("streams"), and both captured into a HIP graph and replayed ("graph",
    "graph_streams"). Every step starts from the same Variables (restore
    outside the timed interval); times are HIP-event means in ms."""
    import torch

    from paper_1603_04467_amd import workloads
    from paper_1603_04467_amd.step import DenseStep

    w = workloads.workload(name)
    s = DenseStep(w, workloads.generate(w, seed=0))
    stream = torch.cuda.current_stream()
    graphs = {"graph": s.capture(concurrent=False), "graph_streams": s.capture(concurrent=True,
                                                                               num_streams=num_streams)}
    modes = {
        "serial": s.run,
        "streams": lambda: s.run_concurrent(num_streams),
        "graph": graphs["graph"].replay,
        "graph_streams": graphs["graph_streams"].replay,
    }
    out = {}
    for mode, fn in modes.items():
        for _ in range(warmup):
            s.restore()
            fn()
        ev = []
        for _ in range(steps):
            s.restore()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            ev.append((a, b))
        torch.cuda.synchronize()
        out[mode] = round(float(np.mean([a.elapsed_time(b) for a, b in ev])), 4)
    best = min(out, key=out.get)
    return {"ms_per_step": out, "best": best, "tflops_best": round(w.flops() / (out[best] * 1e-3) / 1e12, 3)}


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
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        ev[0].record(stream)
        for i in range(reps):
            fn()
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        ms = float(np.mean([ev[i].elapsed_time(ev[i + 1]) for i in range(reps)]))
        out[name] = {"elements": count, "ms": round(ms, 4), "gbs": round(byt / (ms * 1e-3) / 1e9, 1),
                     "frac_hbm": round(byt / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 3)}
    return out


def _per_op(ops):
    """Mean ms per op, with TFLOP/s (GEMMs) or GB/s (memory-bound ops)."""
    out = {}
    for k, v in ops.items():
        d = {"ms": round(v["ms"], 4)}
        if "tflops" in v:
            d["tflops"] = round(v["tflops"], 1)
        if "gbs" in v:
            d["gbs"] = round(v["gbs"], 1)
        out[k] = d
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=PRIMARY)
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=16384)
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(the data-parallel sharding is a design note only).", file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "no GPU visible"
    torch.cuda.set_device(0)

    print(f"bench: timing {args.workload} ({args.steps} steps, {args.warmup} warm-up)", file=sys.stderr, flush=True)
    r = time_workload(args.workload, args.steps, args.warmup)
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
        "loss": r["loss"],
    }
    if not args.no_secondary and args.workload == PRIMARY:
        out["also"] = []
        for name in SECONDARY:
            print(f"bench: timing {name}", file=sys.stderr, flush=True)
            r2 = time_workload(name, args.steps, args.warmup)
            out["also"].append({
                "workload": name,
                "value": round(r2["tflops"], 3),
                "unit": "TFLOP/s",
                "ms_per_step": round(r2["ms"], 4),
                "ms_per_step_percentiles": r2["ms_percentiles"],
                "pct_mfma_peak": round(r2["pct_peak"], 2),
                "roofline": r2["roofline"],
                "per_op": _per_op(r2["ops"]),
                "loss": r2["loss"],
            })
            if name in LAUNCH_BOUND:
                out["also"][-1]["launch_modes"] = time_modes(name, args.steps, args.warmup)
    if not args.no_secondary and args.workload == PRIMARY:
        print("bench: timing the 32 <-> 16-bit conversions", file=sys.stderr, flush=True)
        out["conversions"] = time_conversions()
    if not args.no_cpu_baseline:
        print(f"bench: timing the oracle on {args.cpu_rows} rows", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(args.workload, args.cpu_rows)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
