"""The rocprofv3 summariser (paper_1603_04467_amd/profiling.py) on small
synthetic outputs: kernel ids map to the compiled symbols, the roofline
check reproduces a known fraction, traffic records scale by the copy
calibration and round-trip through bench.py's lookup."""

import csv
import json
import os
import re

import pytest

from paper_1603_04467_amd import profiling as P

TN = "_ZN3tfd12_GLOBAL__N_113gemm_bf16_256ILb0ELb0EfLi4ELi4ELi0EEEvNS0_6ParamsE"
NT_MASK = "_ZN3tfd12_GLOBAL__N_113gemm_bf16_256ILb1ELb1EDF16bLi2ELi4ELi4EEEvNS0_6ParamsE"
NT_PLAIN = "_ZN3tfd12_GLOBAL__N_113gemm_bf16_256ILb1ELb1EDF16bLi2ELi4ELi0EEEvNS0_6ParamsE"
COPY = "__amd_rocclr_copyBuffer"
TN_ID = "gemm bf16 TN none 4096x4096x16384 -> f32"
NT_ID = "gemm bf16 NT bias_relu+mask 16384x4096x4096 -> bf16"


def test_kernel_ids_and_symbols():
    kid = P.parse_kernel_id(TN_ID)
    assert (kid["layout"], kid["out"], kid["m"], kid["k"]) == ("TN", "f32", 4096, 16384)
    assert P.matches(kid, TN, 256 * 1024)
    assert not P.matches(kid, TN, 512 * 1024)           # other grid: another shape
    assert not P.matches(kid, NT_PLAIN, 256 * 1024)
    nt = P.parse_kernel_id(NT_ID)
    assert P.matches(nt, NT_MASK, 1024 * 512)
    assert not P.matches(nt, NT_PLAIN, 1024 * 512)      # epilogue differs
    assert P.symbol_fields("void tfd::(anonymous namespace)::gemm_bf16_256<true, true, __bf16, 2, 4, 4>(Params)") == \
        {"a_kc": True, "b_kc": True, "out": "bf16", "waves": (2, 4), "ep": 4}
    with pytest.raises(ValueError):
        P.parse_kernel_id("sgd")


def _write(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0]))
        w.writeheader()
        w.writerows(rows)


def _bench(path, frac=0.5):
    peak = 2516.6
    flops = 2 * 4096 * 4096 * 16384
    ms = flops / (frac * peak * 1e12) * 1e3
    line = {"steps": 20, "roofline": {"kernel": TN_ID, "launches_per_step": 4, "ms_per_launch": ms,
                                      "achieved": frac * peak, "peak": peak, "frac": frac, "flops_per_launch": flops},
            "per_op": {"dw1": {"ms": ms, "kernel": TN_ID}, "fwd1": {"ms": 0.5, "kernel": NT_ID}, "sgd1": {"ms": 0.05}}}
    with open(path, "w") as f:
        f.write("noise\n" + json.dumps(line) + "\n")
    return ms


def test_trace_reproduces_the_fraction(tmp_path):
    ms = _bench(tmp_path / "b.json", frac=0.5)
    ns = int(ms * 1e6)
    trace = [{"Kernel_Name": TN, "Grid_Size_X": 256 * 1024, "Start_Timestamp": 1000 * i, "End_Timestamp": 1000 * i + ns}
             for i in range(8)]
    trace.append({"Kernel_Name": NT_MASK, "Grid_Size_X": 1024 * 512, "Start_Timestamp": 0, "End_Timestamp": 5})
    _write(tmp_path / "run_kernel_trace.csv", trace)
    _write(tmp_path / "run_kernel_stats.csv", [
        {"Name": TN, "Calls": 8, "TotalDurationNs": 8 * ns, "AverageNs": ns, "Percentage": 99.0, "MinNs": ns,
         "MaxNs": ns}])
    text = P.trace(str(tmp_path), str(tmp_path / "b.json"))
    assert "| rocprofv3 kernel trace, every launch of the leg | 8 |" in text
    assert "0.5000 |" in text and re.search(r"difference of the fractions \(bench line vs trace\): [+-]0\.00%", text)


def test_trace_selects_the_leg_and_its_timed_pass(tmp_path):
    """Launches after the bench line's own leg (later workloads reusing the
    kernel at another k) and outside its timed pass are left out."""
    ms = _bench(tmp_path / "b.json", frac=0.5)
    b = json.loads(open(tmp_path / "b.json").read().splitlines()[-1])
    b["roofline"].update(launches_in_leg=12, timed_launches=[4, 8])
    open(tmp_path / "b.json", "w").write(json.dumps(b) + "\n")
    ns = int(ms * 1e6)
    durs = [3 * ns] * 4 + [ns] * 4 + [2 * ns] * 4 + [ns // 8] * 10    # warm-up, timed, clock pass, another leg
    trace = [{"Kernel_Name": TN, "Grid_Size_X": 256 * 1024, "Start_Timestamp": 10 ** 7 * i,
              "End_Timestamp": 10 ** 7 * i + d} for i, d in enumerate(durs)]
    _write(tmp_path / "run_kernel_trace.csv", trace)
    _write(tmp_path / "run_kernel_stats.csv", [
        {"Name": TN, "Calls": len(durs), "TotalDurationNs": sum(durs), "AverageNs": sum(durs) / len(durs),
         "Percentage": 99.0, "MinNs": min(durs), "MaxNs": max(durs)}])
    text = P.trace(str(tmp_path), str(tmp_path / "b.json"))
    assert "| rocprofv3 kernel trace, every launch of the leg | 12 |" in text
    assert "| rocprofv3 kernel trace, the timed pass | 4 |" in text
    assert re.search(r"\(bench line vs trace, timed pass\): [+-]0\.00%", text)


def test_traffic_records_round_trip(tmp_path, monkeypatch):
    _bench(tmp_path / "b.json")
    os.makedirs(tmp_path / "f")
    os.makedirs(tmp_path / "w")
    # the counters read half the bytes of a copy for FETCH_SIZE, all of them for WRITE_SIZE
    base = {"Grid_Size_X": 256 * 1024}
    _write(tmp_path / "f" / "run_counter_collection.csv", [
        dict(base, Kernel_Name=COPY, Counter_Name="FETCH_SIZE", Counter_Value=32768.0),
        dict(base, Kernel_Name=COPY, Counter_Name="FETCH_SIZE", Counter_Value=100.0),
        dict(base, Kernel_Name=TN, Counter_Name="FETCH_SIZE", Counter_Value=400000.0),
        dict(base, Kernel_Name=TN, Counter_Name="FETCH_SIZE", Counter_Value=402000.0)])
    _write(tmp_path / "w" / "run_counter_collection.csv", [
        dict(base, Kernel_Name=COPY, Counter_Name="WRITE_SIZE", Counter_Value=65536.0),
        dict(base, Kernel_Name=TN, Counter_Name="WRITE_SIZE", Counter_Value=65600.0),
        dict(base, Kernel_Name=TN, Counter_Name="WRITE_SIZE", Counter_Value=65600.0)])
    text = P.traffic(str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "b.json"))
    assert "x 2.0000" in text and "x 1.0000" in text
    rec = [ln for ln in text.splitlines() if ln.startswith("record ")]
    assert len(rec) == 1 and f"kernel={TN_ID} ;" in rec[0]
    # bench.py reads the record back while the kernel source is unchanged
    import bench
    tf = tmp_path / "traffic.md"
    tf.write_text("\n".join(rec) + "\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tf))
    got = bench.lookup_traffic(TN_ID, "bf16")
    want = 401000.0 * 1024 * 2.0 + 65600.0 * 1024 * 1.0
    assert got is not None and abs(got["bytes"] - want) <= 1e-6 * want


def test_phases_groups_the_fused_steps(tmp_path):
    """Launches of the fused step (3 phases of 4, 2 and 9 workgroups, 5 steps,
    copies between the steps) followed by persistent launches: the phases
    are found by the period of the grids, their durations are medians."""
    rows, t = [], 0
    for step in range(5):
        rows.append({"Kernel_Name": COPY, "Grid_Size_X": 1024, "Start_Timestamp": t, "End_Timestamp": t + 500})
        t += 1000
        for k, (wg, dur) in enumerate(((4, 3000), (2, 2000), (9, 7000 + step))):
            rows.append({"Kernel_Name": "tfd::(anonymous namespace)::mlp_step_kernel(StepArgs)", "Grid_Size_X": wg * 256,
                         "Start_Timestamp": t, "End_Timestamp": t + dur})
            t += dur + 100
    for _ in range(4):
        rows.append({"Kernel_Name": "tfd::(anonymous namespace)::mlp_step_kernel(StepArgs)", "Grid_Size_X": 512 * 256,
                     "Start_Timestamp": t, "End_Timestamp": t + 40000})
        t += 41000
    _write(tmp_path / "run_kernel_trace.csv", rows)
    out = P.phases(str(tmp_path))
    assert "5 steps of 3 launches" in out, out
    assert "| 0 | 4 | 3.0 |" in out and "| 1 | 2 | 2.0 |" in out and "| 2 | 9 | 7.0 |" in out, out
    assert "sum of the phase medians 12.0 us" in out and "median step span (first start to last end) 12.2 us" in out, out


def test_counters_per_variant(tmp_path):
    """Two counter passes over two launches of one kernel: clock, TF/s, MFMA
    busy and the LDS-wait share follow from the counters as documented."""
    d1, d2 = tmp_path / "p1", tmp_path / "p2"
    d1.mkdir(), d2.mkdir()
    rows1, rows2 = [], []
    for disp in (1, 2):
        base = {"Kernel_Name": TN, "Dispatch_Id": disp, "Start_Timestamp": 0, "End_Timestamp": 400_000}  # 400 us
        for name, val in (("GRBM_GUI_ACTIVE", 8 * 800_000), ("SQ_VALU_MFMA_BUSY_CYCLES", 0.5 * 800_000 * 1024),
                          ("SQ_INSTS_MFMA", 100.0), ("SQ_WAVE_CYCLES", 1000.0)):
            rows1.append(dict(base, Counter_Name=name, Counter_Value=val))
        for name, val in (("GRBM_GUI_ACTIVE", 8 * 800_000), ("SQ_INSTS_LDS", 7.0), ("SQ_LDS_BANK_CONFLICT", 0.0),
                          ("SQ_WAIT_INST_LDS", 50.0)):
            rows2.append(dict(base, Counter_Name=name, Counter_Value=val))
    _write(d1 / "run_counter_collection.csv", rows1)
    _write(d2 / "run_counter_collection.csv", rows2)
    out = P.counters([str(d1), str(d2)], flops=2.0 * 4096 * 4096 * 16384)
    # 800k cycles in 400 us: 2.00 GHz; 5.5e11 / 400 us = 1374 TF/s; busy 50 %; LDS waits 50 / 1000
    assert "| TN f32 out, 16 waves | 2 | 400 | 2.00 | 1374 | 54.6 | 50.0 % | 100 | 7 | 0 | 5.0 % |" in out, out
