"""Summaries of rocprofv3 runs of bench.py, for the records under profiles/.

    python -m paper_1603_04467_amd.profiling trace DIR BENCH_JSON
    python -m paper_1603_04467_amd.profiling traffic FETCH_DIR WRITE_DIR BENCH_JSON
    python -m paper_1603_04467_amd.profiling phases DIR
    python -m paper_1603_04467_amd.profiling counters PMC_DIR [PMC_DIR ...]

DIR, FETCH_DIR and WRITE_DIR are rocprofv3 output directories written with
`--output-format csv -o run` (run_kernel_stats.csv, run_kernel_trace.csv,
run_counter_collection.csv); BENCH_JSON holds the JSON line that the same
bench.py run printed.

`trace` prints the kernel-time table of the run and checks the bench line's
roofline against it: the dominant kernel's launches are found in the kernel
trace by their compiled symbol (layout, output type, waves, epilogue) and
grid, and their mean duration gives the achieved TFLOP/s and the fraction of
peak, beside the figures bench.py measured with HIP events.

`phases` prints the per-phase kernel times of the fused small step
(tfd_mlp_step, one launch per phase) found in a kernel trace.

`counters` prints the MFMA and LDS counters of the 16-bit GEMM kernels per
variant from `rocprofv3 --pmc` runs.

`traffic` prints, per GEMM kernel of the bench line's per-op table, the mean
FETCH_SIZE and WRITE_SIZE per launch (KiB), each scaled by what the same
counter reads for the run's 64 MiB device-to-device copies (the restores of
the fp32 Variables), beside the kernel's algorithmic bytes (operands, output
and what its fused epilogue reads and writes, from the bench line), and as
`record` lines that bench.py looks up.
"""

from __future__ import annotations

import csv
import hashlib
import json
import os
import re
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KERNEL_SOURCES = {"bf16": "paper_1603_04467_amd/csrc/gemm_bf16.hip", "f32": "paper_1603_04467_amd/csrc/gemm.hip"}
COPY_BYTES = 64 << 20   # one restore of a 4096 x 4096 fp32 Variable

# epilogue of a bench kernel id -> template EP of the 16-bit whole-tile kernel
_EP_OF = {"none": 0, "bias": 0, "bias_relu": 0, "splitk": 0, "relugrad+colsum": 1, "bias+sq_err+colsum": 2,
          "relugrad_mask+colsum": 3, "bias_relu+mask": 4}
_EP_NAME = {0: "plain", 1: "ReluGrad(features)", 2: "squared error", 3: "ReluGrad(mask)", 4: "ReLU mask out"}


def parse_kernel_id(kid: str) -> dict:
    """'gemm bf16 NT bias_relu+mask 16384x4096x4096 -> bf16' -> its fields."""
    m = re.match(r"gemm (\w+) (NN|NT|TN) (\S+) (\d+)x(\d+)x(\d+) -> (\w+)$", kid)
    if not m:
        raise ValueError(f"not a GEMM kernel id: {kid}")
    act, lay, epi, mm, nn, kk, out = m.groups()
    return {"act": act, "layout": lay, "epi": epi, "m": int(mm), "n": int(nn), "k": int(kk), "out": out}


def symbol_fields(name: str):
    """Template arguments of a 16-bit whole-tile GEMM symbol (mangled or
    demangled), or None for any other kernel."""
    m = re.search(r"gemm_bf16_256ILb(\d)ELb(\d)E(DF16b|f)Li(\d)ELi(\d)ELi(\d)E", name)
    if m:
        a, b, o, wm, wn, ep = m.groups()
        return {"a_kc": a == "1", "b_kc": b == "1", "out": "bf16" if o == "DF16b" else "f32", "waves": (int(wm), int(wn)),
                "ep": int(ep)}
    m = re.search(r"gemm_bf16_256<(\w+), (\w+), (\w+|__bf16), (\d+), (\d+)(?:, (\d+))?>", name)
    if m:
        a, b, o, wm, wn, ep = m.groups()
        return {"a_kc": a == "true", "b_kc": b == "true", "out": "f32" if o == "float" else "bf16",
                "waves": (int(wm), int(wn)), "ep": int(ep or 0)}
    return None


def _layout(f):
    return {(True, True): "NT", (True, False): "NN", (False, False): "TN"}[(f["a_kc"], f["b_kc"])]


def matches(kid: dict, name: str, grid_threads=None, waves=None) -> bool:
    """Whether kernel symbol `name` (launched with `grid_threads` work-items)
    is the 16-bit whole-tile kernel of bench kernel id `kid`. The library picks
    the waves per workgroup by layout, epilogue and k range; the grid (one
    workgroup of 64 x waves work-items per 256 x 256 tile) must agree with the
    symbol's, and with `waves` when given."""
    f = symbol_fields(name)
    if f is None or kid["act"] != "bf16" or kid["epi"] == "splitk":
        return False
    wm, wn = f["waves"]
    if waves is not None and tuple(waves) != (wm, wn):
        return False
    if _layout(f) != kid["layout"] or f["out"] != kid["out"] or f["ep"] != _EP_OF[kid["epi"]]:
        return False
    if grid_threads is not None:
        tiles = (kid["m"] // 256) * (kid["n"] // 256)
        if int(grid_threads) != tiles * 64 * wm * wn:
            return False
    return True


def readable(name: str) -> str:
    f = symbol_fields(name)
    if f:
        return (f"gemm_bf16_256 {_layout(f)} -> {f['out']}, {f['waves'][0] * f['waves'][1]} waves, "
                f"epilogue {_EP_NAME[f['ep']]}")
    n = re.sub(r"^void ", "", name).replace("tfd::(anonymous namespace)::", "")
    return re.sub(r"\(.*$", "", n)[:100]


def _rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _grid(r):
    return r.get("Grid_Size_X") or r.get("Grid_Size")


def _bench(path):
    with open(path) as f:
        lines = [ln for ln in f.read().splitlines() if ln.strip().startswith("{")]
    return json.loads(lines[-1])


def trace(outdir: str, bench_json: str) -> str:
    stats = _rows(os.path.join(outdir, "run_kernel_stats.csv"))
    tr = _rows(os.path.join(outdir, "run_kernel_trace.csv"))
    b = _bench(bench_json)
    rl = b["roofline"]
    kid = parse_kernel_id(rl["kernel"])
    hits = [r for r in tr if matches(kid, r["Kernel_Name"], _grid(r))]
    launches = sorted((int(r["Start_Timestamp"]), (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-6)
                      for r in hits)
    symbols = sorted({readable(r["Kernel_Name"]) for r in hits})
    # the bench line's own leg comes first in the run (the headline workload
    # is timed before any other): its launches are the first launches_in_leg,
    # and the timed pass is the slice timed_launches of them
    if "launches_in_leg" in rl:
        launches = launches[:rl["launches_in_leg"]]
    durs = [d for _, d in launches]
    timed = None
    if "timed_launches" in rl and len(launches) >= rl["timed_launches"][1]:
        t0, t1 = rl["timed_launches"]
        timed = [d for _, d in launches[t0:t1]]
    out = ["| kernel | calls | mean us | min us | max us | % of GPU time |", "|---|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"]))[:16]:
        out.append(f"| {readable(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                   f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | {float(r['Percentage']):.2f} |")
    if not durs:
        out.append(f"\nno launch of {rl['kernel']} found in the trace")
        return "\n".join(out)
    def row(label, d):
        mean = sum(d) / len(d)
        ach = rl["flops_per_launch"] / (mean * 1e-3) / 1e12
        return f"| {label} | {len(d)} | {mean:.5f} | {ach:.1f} | {ach / rl['peak']:.4f} |", ach / rl["peak"]

    out += ["", f"Dominant kernel of the bench line: `{rl['kernel']}` ({'; '.join(symbols)}, "
            f"grid {(kid['m'] // 256) * (kid['n'] // 256)} workgroups)", "",
            "| source | launches | mean ms per launch | achieved TFLOP/s | frac of peak |", "|---|---|---|---|---|"]
    line, frac = row("rocprofv3 kernel trace, every launch of the leg", durs)
    out.append(line)
    if timed:
        line, frac = row("rocprofv3 kernel trace, the timed pass", timed)
        out.append(line)
    out += [f"| bench.py HIP events (timed pass) | {rl['launches_per_step']} x {b['steps']} | {rl['ms_per_launch']:.5f} "
            f"| {rl['achieved']:.1f} | {rl['frac']:.4f} |",
            "", f"difference of the fractions (bench line vs trace{', timed pass' if timed else ''}): "
            f"{100 * (rl['frac'] - frac) / frac:+.2f}%"]
    return "\n".join(out)


def _counter(outdir, counter):
    rows = [r for r in _rows(os.path.join(outdir, "run_counter_collection.csv")) if r["Counter_Name"] == counter]
    return rows


def _scale(rows, counter):
    """COPY_BYTES / (KiB the counter reads for one 64 MiB copy dispatch)."""
    vals = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
    if not vals:
        raise ValueError(f"{counter}: no copy dispatch to calibrate on")
    # the 64 MiB restores are the largest copies of the run
    big = max(vals)
    sel = [v for v in vals if abs(v - big) <= 0.01 * big]
    kib = sum(sel) / len(sel)
    return COPY_BYTES / 1024 / kib, kib


def _sha256(rel):
    with open(os.path.join(ROOT, rel), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def traffic(fetch_dir: str, write_dir: str, bench_json: str) -> str:
    b = _bench(bench_json)
    fe, wr = _counter(fetch_dir, "FETCH_SIZE"), _counter(write_dir, "WRITE_SIZE")
    fs, fkib = _scale(fe, "FETCH_SIZE")
    ws, wkib = _scale(wr, "WRITE_SIZE")
    kids = sorted({v["kernel"] for v in b["per_op"].values() if "kernel" in v})
    alg_of = {v["kernel"]: v.get("algorithmic_bytes") for v in b["per_op"].values() if "kernel" in v}
    out = [f"calibration: a 64 MiB copy reads FETCH_SIZE {fkib:.0f} KiB -> x {fs:.4f}, "
           f"WRITE_SIZE {wkib:.0f} KiB -> x {ws:.4f}", "",
           "| kernel | launches | FETCH_SIZE KiB/launch | WRITE_SIZE KiB/launch | scaled bytes/launch | algorithmic bytes "
           "| ratio |", "|---|---|---|---|---|---|---|"]
    recs = []
    for k in kids:
        kid = parse_kernel_id(k)
        f = [float(r["Counter_Value"]) for r in fe if matches(kid, r["Kernel_Name"], _grid(r))]
        w = [float(r["Counter_Value"]) for r in wr if matches(kid, r["Kernel_Name"], _grid(r))]
        if not f or not w:
            continue
        fk, wk = sum(f) / len(f), sum(w) / len(w)
        eb = 2 if kid["act"] == "bf16" else 4
        alg = alg_of.get(k) or (kid["m"] * kid["k"] * eb + kid["k"] * kid["n"] * eb +
                                kid["m"] * kid["n"] * (4 if kid["out"] == "f32" else eb))
        byt = fk * 1024 * fs + wk * 1024 * ws
        out.append(f"| {k} | {len(f)} | {fk:.0f} | {wk:.0f} | {byt:.4g} | {alg:.4g} | {byt / alg:.2f} |")
        recs.append(f"record kernel={k} ; src_sha256={_sha256(KERNEL_SOURCES[kid['act']])} ; fetch_kib={fk:.1f} ; "
                    f"write_kib={wk:.1f} ; fetch_scale={fs:.4f} ; write_scale={ws:.4f}")
    return "\n".join(out + [""] + recs)


def phases(outdir: str, name: str = "mlp_step_kernel") -> str:
    """Per-phase kernel times of the fused step launched one kernel per phase:
    the launches of kernel `name` in time order, grouped into steps by the
    period of their grid sizes (the longest stretch in which every launch has
    the grid of the launch one period later, taken at the smallest period of
    at least two with at least three whole steps and more than one distinct
    grid, which leaves out runs of the one-kernel persistent form); per
    phase the median duration over the steps, and per step the median span
    from the first phase's start to the last phase's end."""
    tr = _rows(os.path.join(outdir, "run_kernel_trace.csv"))
    ks = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), int(_grid(r))) for r in tr if name in r["Kernel_Name"])
    grids = [g for _, _, g in ks]
    found = None
    for per in range(2, 17):
        best, run = (0, 0), 0
        for i in range(len(grids) - per):
            run = run + 1 if grids[i] == grids[i + per] else 0
            if run > best[0]:
                best = (run, i - run + 1)
        steps = (best[0] + per) // per
        if steps >= 3 and len(set(grids[best[1]:best[1] + per])) > 1:
            found = (per, best[1], steps)
            break
    if found is None:
        return f"no periodic run of {name} launches found"
    per, s0, steps = found
    med = lambda v: sorted(v)[len(v) // 2]
    out = [f"{steps} steps of {per} launches of {name}", "",
           "| phase | workgroups | median us |", "|---|---|---|"]
    tot = 0.0
    for k in range(per):
        d = [(ks[s0 + k + m * per][1] - ks[s0 + k + m * per][0]) * 1e-3 for m in range(steps)]
        tot += med(d)
        out.append(f"| {k} | {grids[s0 + k] // 256} | {med(d):.1f} |")
    span = [(ks[s0 + m * per + per - 1][1] - ks[s0 + m * per][0]) * 1e-3 for m in range(steps)]
    out += ["", f"sum of the phase medians {tot:.1f} us; median step span (first start to last end) {med(span):.1f} us"]
    return "\n".join(out)


def counters(dirs, flops: float = 2.0 * 16384 * 4096 * 4096) -> str:
    """MFMA and LDS counters of the 16-bit whole-tile GEMM launches in one or
    more `rocprofv3 --pmc` output directories (one counter set each), per
    kernel variant (layout, output type, waves, epilogue), averaged over its
    launches: duration from the dispatch timestamps; engine clock =
    GRBM_GUI_ACTIVE / 8 XCDs / duration; TF/s = `flops` / duration; MFMA busy =
    SQ_VALU_MFMA_BUSY_CYCLES / (clock cycles x 1024 SIMDs); LDS-issue waits =
    mean SQ_WAIT_INST_LDS / mean SQ_WAVE_CYCLES (from different passes)."""
    disp, meta = {}, {}
    for i, d in enumerate(dirs):
        for r in _rows(os.path.join(d, "run_counter_collection.csv")):
            f = symbol_fields(r["Kernel_Name"])
            if f is None:
                continue
            lab = (f"{_layout(f)} {f['out']} out, {f['waves'][0] * f['waves'][1]} waves"
                   + (f", epilogue {_EP_NAME[f['ep']]}" if f["out"] == "bf16" else ""))
            key = (i, r["Dispatch_Id"])
            disp.setdefault(key, {})[r["Counter_Name"]] = float(r["Counter_Value"])
            meta[key] = (lab, (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    agg = {}
    for key, c in disp.items():
        lab, dur = meta[key]
        a = agg.setdefault(lab, {})
        put = lambda k, v: a.setdefault(k, []).append(v)  # noqa: E731
        cyc = c.get("GRBM_GUI_ACTIVE", float("nan")) / 8.0
        put("dur", dur * 1e6)
        put("clock", cyc / dur / 1e9)
        if "SQ_VALU_MFMA_BUSY_CYCLES" in c:
            put("tflops", flops / dur / 1e12)
            put("busy", c["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * 1024))
            put("mfma", c.get("SQ_INSTS_MFMA", float("nan")))
        for k in ("SQ_WAVE_CYCLES", "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_WAIT_INST_LDS"):
            if k in c:
                put(k, c[k])
    mean = lambda v: sum(v) / len(v) if v else float("nan")  # noqa: E731
    out = ["| kernel | launches | µs (under counters) | engine clock GHz | TF/s | % of 2516.6 | MFMA busy (of SIMD "
           "cycles) | MFMA insts | LDS insts | LDS bank-conflict cycles | LDS-issue waits / wave cycles |",
           "|---|---|---|---|---|---|---|---|---|---|---|"]
    for lab in sorted(agg):
        a = agg[lab]
        tf = mean(a.get("tflops", []))
        wl = mean(a.get("SQ_WAIT_INST_LDS", [])) / mean(a.get("SQ_WAVE_CYCLES", []))
        out.append(f"| {lab} | {len(a.get('busy', []))} | {mean(a['dur']):.0f} | {mean(a['clock']):.2f} | {tf:.0f} | "
                   f"{100 * tf / 2516.6:.1f} | {100 * mean(a.get('busy', [])):.1f} % | {mean(a.get('mfma', [])):.4g} | "
                   f"{mean(a.get('SQ_INSTS_LDS', [])):.4g} | {mean(a.get('SQ_LDS_BANK_CONFLICT', [])):.3g} | "
                   f"{100 * wl:.1f} % |")
    return "\n".join(out)


def main(argv):
    if len(argv) == 3 and argv[0] == "trace":
        print(trace(argv[1], argv[2]))
    elif len(argv) == 4 and argv[0] == "traffic":
        print(traffic(argv[1], argv[2], argv[3]))
    elif len(argv) == 2 and argv[0] == "phases":
        print(phases(argv[1]))
    elif len(argv) >= 2 and argv[0] == "counters":
        print(counters(argv[1:]))
    else:
        print(__doc__, file=sys.stderr)
        return 2
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
