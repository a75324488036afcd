#!/usr/bin/env python3
"""Throughput of the MBE editing-pass hot path on one MI355X.

One step = one pass of the whole path over one batch: editing-window
attention (paged prefix + bidirectional window) followed by edit selection
over the vocabulary logits, both through libmbe's C ABI.  Inputs are seeded
synthetic tensors (synth/) already resident in HBM.

Default workload: 64 sequences, prefixes 32*U{128..1024} (4096..32768),
window of k = 4 blocks of 32 (128 queries), 16 query / 4 KV heads, head_dim
128, 16-token pages, edit selection over 8192 rows x 131072 vocabulary.

Prints one JSON line.  `value` is the step's fraction of MI355X speed of
light, 100 * (attention FLOP / MFMA peak + edit-select bytes / HBM peak) /
step time, with the attention TFLOP/s and edit-select GB/s alongside.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6      # MI355X dense bf16 MFMA (256 CU x 4096 flop/clk x 2.4 GHz; "2.5 PFLOP/s")
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
DEFAULT_WORKLOAD = "long_context_b64_p4096to32768_k4"
METRIC = "edit-window attention TFLOP/s (bf16) + edit-select GB/s, % of MI355X peak"
def traffic_file(workload):
    """profiles/hbm_traffic_<workload>.txt (workload tag, with _k<k> for the span sweep)."""
    return os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.txt")
CALIB_COPY_BYTES = 256 << 20     # the plain device copy bench.py runs once, for counter calibration


def attention_work(case):
    """Algorithmic FLOPs and bytes of one window-attention call (bidirectional):
    4*D per visible (query, key) pair per query head; K/V read once per KV head,
    Q read and O written once."""
    P = case.prefix_lens.numpy().astype(np.int64)
    W = case.window_lens.numpy().astype(np.int64)
    D, Hq, Hkv = case.head_dim, case.num_q_heads, case.num_kv_heads
    flops = 4 * D * Hq * int(np.sum(W * (P + W)))
    kv_bytes = int(np.sum(P + W)) * Hkv * D * 2 * 2
    qo_bytes = int(W.sum()) * Hq * D * 2 * 2
    return flops, kv_bytes + qo_bytes


RIDGE_FLOP_PER_BYTE = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)   # ~315


def attention_kernel_name(case, mode=0, v_token_major=False, kv_split_tokens=0):
    """The window_attention_kernel<D, MODE, KS, VT, PIPE> instantiation a call
    on this case runs (bounds and host lengths as the bench passes them), from
    the library's own launch plan (mbe_window_attention_plan)."""
    import paper_2607_22663_amd as mbe
    kp = case.k_pages
    vp = kp if v_token_major else kp.transpose(2, 3)       # only the shape is read
    plan = mbe.window_attention_plan(case.num_q_heads, kp, vp, case.page_table, case.batch, int(case.q.shape[0]),
                                     max_prefix_len=int(case.prefix_lens.max()),
                                     max_window_len=int(case.window_lens.max()), mask_mode=mode,
                                     kv_split_tokens=kv_split_tokens, host_prefix_lens=case.prefix_lens,
                                     host_window_lens=case.window_lens)
    return plan["kernel"]


def attention_roofline(flops, nbytes, seconds, kernel, traffic=None):
    """Roofline entry of one attention call: MFMA-bound (TFLOP/s against the
    bf16 peak) when its intensity exceeds the ridge point, else HBM-bound
    (algorithmic GB/s against 8 TB/s)."""
    if flops / nbytes >= RIDGE_FLOP_PER_BYTE:
        ach, peak, unit, bound = flops / seconds / 1e12, PEAK_BF16_TFLOPS, "TFLOP/s", "mfma"
    else:
        ach, peak, unit, bound = nbytes / seconds / 1e9, PEAK_HBM_GBS, "GB/s", "hbm"
    return {"kernel": kernel, "bound": bound, "achieved": round(ach, 2), "peak": peak, "unit": unit,
            "frac": round(ach / peak, 4), "traffic": traffic["bytes_per_launch"] if traffic else None,
            "traffic_detail": traffic, "algorithmic_bytes": nbytes, "algorithmic_flops": flops}


def edit_bytes(rows, vocab):
    """bf16 logits read once; current token read; new token, confidence and
    changed flag written (4 + 4 + 4 + 1 bytes per row)."""
    return rows * vocab * 2 + rows * 13


def kernel_source_hash():
    """Hash of the code of the timed kernels' sources: comments, trailing
    blanks and empty lines are dropped first, so that an edit of a comment
    keeps counters taken on the same code valid."""
    h = hashlib.sha256()
    for f in ("attn_window.hip", "edit_select.hip", "internal.h"):
        with open(os.path.join(ROOT, "paper_2607_22663_amd", "csrc", f)) as fh:
            src = fh.read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        src = re.sub(r"//[^\n]*", "", src)
        h.update("\n".join(ln.rstrip() for ln in src.splitlines() if ln.strip()).encode())
    return h.hexdigest()[:16]


def read_traffic_file(workload):
    """The traffic summary of a workload: one `key=value ...` line per kernel."""
    out = {}
    try:
        with open(traffic_file(workload)) as f:
            for line in f:
                if line.startswith("#") or "=" not in line:
                    continue
                kv = dict(tok.split("=", 1) for tok in line.split())
                out[(kv["kernel"], kv.get("variant"))] = kv
                out.setdefault(kv["kernel"], kv)
    except OSError:
        pass
    return out


def measured_traffic(kernel, workload, variant=None):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary
    (profiles/hbm_traffic_<workload>.txt), if it was taken on the current
    kernel sources, this workload and (when given) this kernel instantiation;
    else None."""
    tf = read_traffic_file(workload)
    e = tf.get((kernel, variant)) if variant is not None else tf.get(kernel)
    if not e or e.get("kernel_sha") != kernel_source_hash() or e.get("workload") != workload:
        return None
    out = {"read_bytes": int(float(e["read_bytes"])), "write_bytes": int(float(e["write_bytes"])),
           "bytes_per_launch": int(float(e["read_bytes"]) + float(e["write_bytes"])),
           "calibration": e.get("calibration")}
    if "req_read_bytes" in e:
        out["read_bytes_by_request_size"] = int(float(e["req_read_bytes"]))
    return out


def _counter_rows(path):
    import csv
    import glob
    files = glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True)
    rows = []
    for f in files:
        with open(f) as fh:
            rows.extend(csv.DictReader(fh))
    return rows


_KERNELS = {"window_attention_kernel": "window_attention", "window_attention_merge_kernel": "window_attention_merge",
            "edit_select_kernel": "edit_select", "edit_select_finalize_kernel": "edit_select_finalize",
            "threshold_block_kernel": "threshold_update_blocks", "kv_write_kernel": "kv_write",
            "tail_entropy_kernel": "tail_entropy_scores", "select_start_kernel": "select_start_block",
            "refresh_kernel": "refresh_blocks"}


def _kernel_key(name):
    # "window_attention_kernel<" also prefixes the merge kernel's name: match on the full token
    if "edit_select_kernel<" in name and name.split("edit_select_kernel<")[1].startswith(("true, true", "false, true")):
        return "threshold_update_rows"      # the row pass with the entropy accumulator
    for k in sorted(_KERNELS, key=len, reverse=True):
        if k + "<" in name or k + "(" in name:
            return _KERNELS[k]
    return None


def _variant(name):
    """'window_attention_kernel<128,0,1,0>' from a demangled kernel name."""
    m = re.search(r"(\w+_kernel<[^>]*>)", name)
    return m.group(1).replace(" ", "") if m else None


def summarize_pmc(dirs, workload, bench_cmd=""):
    """Writes the HBM traffic summary (profiles/hbm_traffic_<workload>.txt) from
    rocprofv3 --pmc runs of this script:
    FETCH_SIZE, then WRITE_SIZE, then optionally TCC_EA0_RDREQ_{32B,64B,128B}_sum
    plus TCC_EA0_RDREQ_sum.  FETCH_SIZE and WRITE_SIZE are each scaled by what
    the counter reads for the plain device copy of CALIB_COPY_BYTES that
    bench.py runs before timing (the copy reads and writes that many bytes).
    The request-size pass counts read bytes directly (32, 64 or 128 bytes per
    request), which the copy scaling cannot do when a kernel's mix of request
    sizes differs from the copy's."""
    fetch_dir, write_dir = dirs[0], dirs[1]
    req_dir = dirs[2] if len(dirs) > 2 else None
    cmd = bench_cmd or "python3 -u bench.py --steps 3 --warmup 1 --no-cpu-baseline --no-next --no-others"
    lines = ["# HBM traffic per launch from rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE (KiB per dispatch),",
             "# each scaled by the same counter's reading for a plain 256 MiB device copy;",
             "# req_read_bytes = 32*RDREQ_32B + 64*RDREQ_64B + 128*RDREQ_128B (TCC to memory read requests).",
             f"# workload {workload}; kernel_sha = hash of the code (comments and blank lines dropped) of the "
             "kernel sources the counters were taken on",
             "# commands (one MI355X, repository root), then python3 bench.py --summarize-pmc <the three folders>:",
             f"#   rocprofv3 --pmc FETCH_SIZE -d {fetch_dir} -o run --output-format csv -- {cmd}",
             f"#   rocprofv3 --pmc WRITE_SIZE -d {write_dir} -o run --output-format csv -- {cmd}",
             f"#   rocprofv3 --pmc TCC_EA0_RDREQ_32B_sum TCC_EA0_RDREQ_64B_sum TCC_EA0_RDREQ_128B_sum TCC_EA0_RDREQ_sum "
             f"-d {req_dir} -o run --output-format csv -- {cmd}"]
    scale = {}
    per_kernel = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = [r for r in _counter_rows(d) if r["Counter_Name"] == counter]
        copies = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        scale[counter] = CALIB_COPY_BYTES / (max(copies) * 1024.0)   # the 256 MiB copy is the largest
        for r in rows:
            k = _kernel_key(r["Kernel_Name"])
            if k:
                key = (k, _variant(r["Kernel_Name"]))
                per_kernel.setdefault(key, {}).setdefault(counter, []).append(float(r["Counter_Value"]))
    if req_dir:
        for r in _counter_rows(req_dir):
            k = _kernel_key(r["Kernel_Name"])
            if k:
                key = (k, _variant(r["Kernel_Name"]))
                per_kernel.setdefault(key, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    sha = kernel_source_hash()

    def avg(v, c):
        x = v.get(c)
        return sum(x) / len(x) if x else None

    for (k, var), v in sorted(per_kernel.items(), key=lambda kv: (kv[0][0], kv[0][1] or "")):
        f, w = avg(v, "FETCH_SIZE"), avg(v, "WRITE_SIZE")
        if f is None or w is None:
            continue
        line = (f"kernel={k} variant={var} workload={workload} kernel_sha={sha} fetch_kib={f:.1f} write_kib={w:.1f} "
                f"read_bytes={f * 1024 * scale['FETCH_SIZE']:.0f} write_bytes={w * 1024 * scale['WRITE_SIZE']:.0f} "
                f"calibration=fetch_x{scale['FETCH_SIZE']:.3f},write_x{scale['WRITE_SIZE']:.3f}")
        n32, n64, n128 = (avg(v, f"TCC_EA0_RDREQ_{b}_sum") for b in ("32B", "64B", "128B"))
        if n32 is not None and n64 is not None and n128 is not None:
            line += (f" rdreq_32b={n32:.0f} rdreq_64b={n64:.0f} rdreq_128b={n128:.0f} "
                     f"rdreq_all={avg(v, 'TCC_EA0_RDREQ_sum') or 0:.0f} "
                     f"req_read_bytes={32 * n32 + 64 * n64 + 128 * n128:.0f}")
        lines.append(line)
    with open(traffic_file(workload), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


MFMA_COUNTERS = ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_MFMA", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CYCLES",
                 "GRBM_GUI_ACTIVE")


def _by_variant(rows):
    """Counter averages per dispatch of each kernel variant in the rows
    (variant -> (dispatches, {counter: average})), in order of appearance."""
    per = {}
    for r in rows:
        per.setdefault(_variant(r["Kernel_Name"]), {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    out = {}
    for var, cs in per.items():
        out[var] = (max(len(v) for v in cs.values()), {k: sum(v) / len(v) for k, v in cs.items()})
    return out


def summarize_mfma(pmc_dir, bench_stdout, out_path, command, workload):
    """Markdown summary of one rocprofv3 --pmc pass of MFMA counters over the
    attention kernel, one section per kernel variant the run launched (the
    timed layout's and the other V layout's): the bf16 MFMA work the hardware
    counted (MOPS, units of 512 flops) against the algorithmic FLOPs, and the
    MFMA-busy share."""
    rows = [r for r in _counter_rows(pmc_dir) if _kernel_key(r["Kernel_Name"]) == "window_attention"]
    line = None
    with open(bench_stdout) as f:
        for ln in f:
            if ln.startswith("{"):
                line = json.loads(ln)
    gflop = line["attention"]["gflop"] if line else float("nan")
    timed = line["attention"].get("kernel") if line else None
    lines = ["# window attention: MFMA counters", "", f"Workload {workload}, one rocprofv3 --pmc pass, average per "
             "dispatch of each kernel variant the run launched.", "", "Command:", "", "```", command, "```"]
    groups = _by_variant(rows)
    for var in sorted(groups, key=lambda v: v != timed):
        n, avg = groups[var]
        counted = avg.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) * 512 / 1e9
        mfma_insts = avg.get("SQ_INSTS_MFMA", 0.0)
        role = "the timed call" if var == timed else "the other V layout"
        lines += ["", f"## `{var}` ({role}, {n} dispatches)", "", "| counter | value per dispatch |", "|---|---|"]
        for k in MFMA_COUNTERS:
            if k in avg:
                lines.append(f"| {k} | {avg[k]:.4g} |")
        lines += ["", f"- bf16 MFMA work counted: {counted:.1f} GFLOP (MOPS x 512) against {gflop:.1f} GFLOP algorithmic "
                  f"(ratio {counted / gflop:.4f}; the extra is the masked keys of each sequence's last 64-key tile).",
                  f"- MFMA instructions: {mfma_insts:.4g} (32x32x16 bf16, 32768 flops each: "
                  f"{mfma_insts * 32768 / 1e9:.1f} GFLOP)."]
        if "SQ_VALU_MFMA_BUSY_CYCLES" in avg and "GRBM_GUI_ACTIVE" in avg:
            busy = avg["SQ_VALU_MFMA_BUSY_CYCLES"] / (4 * 256 * avg["GRBM_GUI_ACTIVE"] / 8)
            lines.append(f"- MFMA busy share: {100 * busy:.1f}% = SQ_VALU_MFMA_BUSY_CYCLES / (4 SIMDs x 256 CUs x "
                         "GRBM_GUI_ACTIVE / 8), reading GRBM_GUI_ACTIVE as summed over the 8 XCDs.")
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_counters(pmc_dir, kernel, out_path, command, workload):
    """Markdown table of one rocprofv3 --pmc pass: each counter's average per
    dispatch of one kernel (a key of _KERNELS), one section per kernel variant
    the run launched, with the LDS bank-conflict share and the VALU issue
    share when their counters are there."""
    rows = [r for r in _counter_rows(pmc_dir) if _kernel_key(r["Kernel_Name"]) == kernel]
    lines = [f"# {kernel}: rocprofv3 counters", "", f"Workload {workload}, one rocprofv3 --pmc pass, average per "
             "dispatch of each kernel variant the run launched.", "", "Command:", "", "```", command, "```"]
    groups = _by_variant(rows)
    for var in groups:
        n, avg = groups[var]
        lines += ["", f"## `{var}` ({n} dispatches)", "", "| counter | value per dispatch |", "|---|---|"]
        for k in sorted(avg):
            lines.append(f"| {k} | {avg[k]:.4g} |")
        lines.append("")
        if "SQ_LDS_BANK_CONFLICT" in avg and avg.get("SQ_LDS_IDX_ACTIVE"):
            lines.append(f"- LDS bank-conflict cycles per LDS-active cycle: "
                         f"{avg['SQ_LDS_BANK_CONFLICT'] / avg['SQ_LDS_IDX_ACTIVE']:.2e} "
                         "(SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE).")
        if "SQ_ACTIVE_INST_VALU" in avg and avg.get("SQ_WAVE_CYCLES"):
            lines.append(f"- VALU issue share of wave cycles: {100 * avg['SQ_ACTIVE_INST_VALU'] / avg['SQ_WAVE_CYCLES']:.1f}% "
                         "(SQ_ACTIVE_INST_VALU / SQ_WAVE_CYCLES).")
        if "SQ_WAIT_INST_ANY" in avg and avg.get("SQ_WAVE_CYCLES"):
            lines.append(f"- Waiting for any instruction's inputs: {100 * avg['SQ_WAIT_INST_ANY'] / avg['SQ_WAVE_CYCLES']:.1f}% "
                         "of wave cycles (SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES).")
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_stats(stats_dir, bench_stdout, out_path, command):
    """Writes a short markdown summary of a rocprofv3 --kernel-trace --stats run
    of this script: rocprofv3's per-kernel statistics, the average over the
    timed dispatches from the kernel trace, and the JSON line that the same
    profiled run printed (its event-timed kernel durations)."""
    import csv
    import glob

    def read(pattern):
        rows = []
        for f in glob.glob(os.path.join(stats_dir, "**", pattern), recursive=True):
            with open(f) as fh:
                rows.extend(csv.DictReader(fh))
        return rows

    stats, trace = read("*kernel_stats.csv"), read("*kernel_trace.csv")
    line = None
    with open(bench_stdout) as f:
        for ln in f:
            if ln.startswith("{"):
                line = json.loads(ln)
    lines = ["# rocprofv3 kernel statistics", "", "Command (run from the repository root on one MI355X):", "",
             "```", command, "```", "",
             "| kernel | calls | average (us) | min (us) | max (us) | share of GPU time |", "|---|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: -float(r.get("TotalDurationNs", 0))):
        lines.append(f"| `{r['Name'][:90]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.1f}% |")
    nxt = (line or {}).get("next_rows") or {}
    if line and nxt:
        lines += ["", "This run also times the calls outside the step (`next_rows` of the JSON line, at several "
                      "shapes, including the graph-pool passes); the table above aggregates all their dispatches, "
                      "and their HIP-event times per call are in the JSON line below."]
    if trace and line and not nxt:
        steps = int(line["steps"])
        lines += ["", f"Average over the {steps} timed dispatches (the last {steps} of each kernel in the trace) "
                  "next to the same run's HIP-event timing:", "",
                  "| kernel | rocprofv3 trace average (us) | bench.py event average (us) |", "|---|---|---|"]
        ev = {"window_attention": line["attention"]["ms"] * 1e3,
              "edit_select": (line.get("edit_select") or {}).get("ms", 0) * 1e3}
        # the timed attention variant only: the other V layout's calls come
        # after the timed steps and are reported on their own line
        timed_var = line["attention"].get("kernel")
        by, other = {}, {}
        for r in sorted(trace, key=lambda r: int(r["Start_Timestamp"])):
            k = _kernel_key(r["Kernel_Name"])
            if not k:
                continue
            d_us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            var = _variant(r["Kernel_Name"])
            if k == "window_attention" and timed_var and var != timed_var:
                other.setdefault(var, []).append(d_us)
            else:
                by.setdefault(k, []).append(d_us)
        for k, d in sorted(by.items()):
            d = d[-steps:]
            name = f"{k} (`{timed_var}`)" if k == "window_attention" and timed_var else k
            lines.append(f"| {name} | {sum(d) / len(d):.2f} | {ev[k]:.2f} |" if k in ev else
                         f"| {name} | {sum(d) / len(d):.2f} | (part of a call timed as a whole) |")
        for var, d in other.items():
            ov = (line.get("attention_other_v_layout") or {})
            ev_o = f"{ov['ms'] * 1e3:.2f}" if ov.get("kernel") == var and "ms" in ov else "—"
            lines.append(f"| window_attention, other V layout (`{var}`, {len(d)} calls) | {sum(d) / len(d):.2f} | {ev_o} |")
        if "window_attention_merge" in by and "window_attention" in by:
            a, m = by["window_attention"][-steps:], by["window_attention_merge"][-steps:]
            lines += ["", f"The attention call is the main kernel plus the split merge: "
                          f"{sum(a) / len(a) + sum(m) / len(m):.2f} us of kernel time per call by the trace, "
                          f"{ev['window_attention']:.2f} us by HIP events. The events span the whole call; under "
                          "rocprofv3 every dispatch carries extra launch overhead, which shows in short calls."]
    if line:
        lines += ["", "JSON line printed by the profiled run:", "", "```", json.dumps(line), "```"]
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _time_events(fn, n):
    import torch
    stream = torch.cuda.current_stream()
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record(stream)
    for _ in range(n):
        fn()
    ev[1].record(stream)
    torch.cuda.synchronize()
    return ev[0].elapsed_time(ev[1]) / n / 1e3


def _time_cold(fn, n, flush):
    """Mean and median time of fn over n calls, each after a read of `flush`
    (a 512 MiB buffer, so no input is served from the infinity cache), with
    HIP events around the call alone on the current stream."""
    import torch
    stream = torch.cuda.current_stream()
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    d = []
    for _ in range(n):
        flush.view(torch.float32).sum()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        d.append(e0.elapsed_time(e1) / 1e3)
    return float(np.mean(d)), float(np.median(d))


def _time_cold_pair(fa, fb, n, flush):
    """_time_cold of two calls taken in turn (a, b, a, b, ...), so that both
    run under the same clock and power state; returns ((mean, median) of a,
    (mean, median) of b)."""
    import torch
    stream = torch.cuda.current_stream()
    for _ in range(3):
        fa()
        fb()
    torch.cuda.synchronize()
    d = ([], [])
    for _ in range(n):
        for fn, out in ((fa, d[0]), (fb, d[1])):
            flush.view(torch.float32).sum()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            out.append(e0.elapsed_time(e1) / 1e3)
    return tuple((float(np.mean(x)), float(np.median(x))) for x in d)


def _host_issue_time(fn, n):
    """Host time to issue one call of fn (mean over n calls queued behind a
    GPU spin, so that the queue never waits on the GPU), synchronised after."""
    import torch
    fn()
    torch.cuda.synchronize()
    torch.cuda._sleep(2_000_000)            # about a millisecond of GPU work ahead of the calls
    t0 = time.perf_counter()
    for _ in range(n):
        fn()
    t = (time.perf_counter() - t0) / n
    torch.cuda.synchronize()
    return t


def bench_next_rows(mbe, attn_case, c, logits, cur, R, V, steps, edit_case):
    """Times the calls outside the timed step: the full threshold update with
    entropy on the step's logits (every 32 rows a block, 40% of rows masked),
    the K/V write-back of the window (all sequences, every window token), and
    tail-entropy scores plus start-block choice for every sequence."""
    import torch
    dev = logits.device
    B = 32
    g = torch.Generator(device="cpu").manual_seed(5)
    cur_m = cur.clone()
    masked = torch.rand(R, generator=g) < 0.4
    cur_m[masked.to(dev)] = V - 1
    out = mbe.threshold_update(logits, cur_m, V - 1, B, 0.5, 0.0, with_entropy=True)

    def update():
        mbe.threshold_update(logits, cur_m, V - 1, B, 0.5, 0.0, with_entropy=True, out=out)
    t_upd = _time_events(update, steps)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    flush.fill_(1)
    t_upd_cold, _ = _time_cold(update, steps, flush)
    del flush
    upd_bytes = R * V * 2 + R * (4 + 4 + 4 + 1 + 4) + R // B
    # refresh write-back of every window token (k blocks per sequence)
    P = attn_case.prefix_lens.to(dev)
    W = attn_case.window_lens.to(dev)
    Hkv, D = attn_case.num_kv_heads, attn_case.head_dim
    T = int(attn_case.window_lens.sum())
    kn = torch.randn(T, Hkv, D, generator=g).to(torch.bfloat16).to(dev)
    vn = torch.randn(T, Hkv, D, generator=g).to(torch.bfloat16).to(dev)
    kp, vp = c.k_pages.clone(), c.v_pages.clone()       # keep the step's pools intact
    max_w = int(attn_case.window_lens.max())
    t_kv = _time_events(lambda: mbe.kv_write(kp, vp, c.page_table, P, W, kn, vn, max_len=max_w), steps)
    del kp, vp
    kv_bytes = 2 * 2 * T * Hkv * D * 2
    # tail scores of the step's rows and one start block per sequence
    ent = out["entropy"]
    scores = mbe.tail_entropy_scores(ent, B, 0.25)
    nb = scores.shape[0] // attn_case.batch
    sc2 = scores[: nb * attn_case.batch].view(attn_case.batch, nb)
    jcur = torch.full((attn_case.batch,), nb, dtype=torch.int32, device=dev)
    t_tail = _time_events(lambda: mbe.tail_entropy_scores(ent, B, 0.25, out=scores), steps)
    t_sel = _time_events(lambda: mbe.select_start_block(sc2, jcur, 4), steps)
    # one editing pass (attention + threshold update with entropy) at small
    # shapes, launched eagerly through the binding vs replayed from the
    # multi-shape graph pool: GPU time per pass (events) and host time to
    # issue one pass
    from paper_2607_22663_amd.graphs import EditPassGraphs
    pool_rows = {}
    max_p = int(attn_case.prefix_lens.max())
    pool = EditPassGraphs(k_pages=c.k_pages, v_pages=c.v_pages, max_batch=8, max_window=64, block_size=B,
                          num_q_heads=attn_case.num_q_heads, max_pages_per_seq=c.page_table.shape[1],
                          max_prefix_len=max_p, vocab=V, mask_id=V - 1)
    for nb, win in ((1, 32), (1, 64), (8, 64)):
        n = nb * win
        pool.capture(nb, win)
        inp = pool.inputs(nb, win)
        inp["q"].copy_(c.q[:n])
        inp["page_table"].copy_(c.page_table[:nb])
        inp["prefix_lens"].copy_(P[:nb])
        inp["logits"].copy_(logits[:n])
        inp["cur_tokens"].copy_(cur_m[:n])
        qv, ptv, pv = c.q[:n], c.page_table[:nb].contiguous(), P[:nb]
        wv = torch.full((nb,), win, dtype=torch.int32, device=dev)
        lv, cv = logits[:n], cur_m[:n]
        o_att = torch.empty_like(qv)
        o_upd = mbe.threshold_update(lv, cv, V - 1, B, 0.5, 0.0, with_entropy=True)

        def eager():
            mbe.window_attention(qv, c.k_pages, c.v_pages, ptv, pv, wv, B, out=o_att, max_prefix_len=max_p,
                                 max_window_len=win)
            mbe.threshold_update(lv, cv, V - 1, B, 0.5, 0.0, with_entropy=True, out=o_upd)
        t_e = _time_events(eager, steps)
        t_g = _time_events(lambda: pool.replay(nb, win), steps)
        pool_rows[f"{nb}x{win}"] = {"eager_ms": round(t_e * 1e3, 4), "graph_ms": round(t_g * 1e3, 4),
                                    "eager_host_us": round(_host_issue_time(eager, steps) * 1e6, 1),
                                    "graph_host_us": round(_host_issue_time(lambda: pool.replay(nb, win), steps)
                                                           * 1e6, 1)}
    del pool
    loop = bench_pass_loop(mbe, attn_case, c, logits, edit_case, V, steps)
    return {
        "graph_pool_edit_pass": pool_rows,
        "pass_loop_graph": loop,
        "threshold_update": {"ms": round(t_upd * 1e3, 4), "rows": R, "vocab": V, "block": B,
                             "with_entropy": True, "algorithmic_mb": round(upd_bytes / 1e6, 1),
                             "gbs": round(upd_bytes / t_upd / 1e9, 1),
                             "pct_hbm_peak": round(100 * upd_bytes / t_upd / 1e9 / PEAK_HBM_GBS, 2),
                             "timing": "back to back",
                             "cold": {"ms": round(t_upd_cold * 1e3, 4),
                                      "gbs": round(upd_bytes / t_upd_cold / 1e9, 1),
                                      "pct_hbm_peak": round(100 * upd_bytes / t_upd_cold / 1e9 / PEAK_HBM_GBS, 2),
                                      "timing": "512 MiB read before each call, as the step's edit selection"}},
        "kv_write": {"ms": round(t_kv * 1e3, 4), "tokens": T, "kv_heads": Hkv, "head_dim": D,
                     "algorithmic_mb": round(kv_bytes / 1e6, 2), "gbs": round(kv_bytes / t_kv / 1e9, 1)},
        "tail_entropy_scores": {"ms": round(t_tail * 1e3, 4), "blocks": int(scores.shape[0])},
        "select_start_block": {"ms": round(t_sel * 1e3, 4), "sequences": attn_case.batch},
    }


def _amdsmi_sample():
    """(socket power W, [gfx clock MHz of each XCD]) from one
    `amd-smi metric --power --clock --json`, or None."""
    import subprocess
    try:
        r = subprocess.run(["amd-smi", "metric", "--power", "--clock", "--json"], capture_output=True, text=True,
                           timeout=10)
        g = json.loads(r.stdout)["gpu_data"][0]
        pw = float(g["power"]["socket_power"]["value"])
        clk = [float(v["clk"]["value"]) for k, v in g["clock"].items()
               if k.startswith("gfx_") and isinstance(v, dict) and isinstance(v.get("clk"), dict)]
        return pw, clk
    except Exception:
        return None


def sample_power(fn, seconds):
    """Runs fn back to back for `seconds` while a host thread reads socket
    power and the gfx clocks with amd-smi (about two readings a second); the
    first half second, while the clocks settle, is left out.  Returns the
    readings' summary (None fields when amd-smi gave nothing)."""
    import threading
    import torch
    samples = []
    stop = threading.Event()
    t_start = time.perf_counter()

    def poll():
        while not stop.is_set():
            r = _amdsmi_sample()
            if r is not None:
                samples.append((time.perf_counter() - t_start, r[0], r[1]))
    th = threading.Thread(target=poll, daemon=True)
    th.start()
    calls = 0
    while time.perf_counter() - t_start < seconds:
        for _ in range(10):
            fn()
        calls += 10
        torch.cuda.synchronize()
    stop.set()
    th.join(timeout=15)
    use = [x for x in samples if x[0] >= 0.5]
    if not use:
        return {"samples": 0, "calls": calls}
    pw = [x[1] for x in use]
    clk = [float(np.mean(x[2])) for x in use if x[2]]
    return {"samples": len(use), "calls": calls, "seconds": seconds,
            "socket_power_w": {"mean": round(float(np.mean(pw)), 1), "min": min(pw), "max": max(pw)},
            "gfx_clock_mhz": ({"mean": round(float(np.mean(clk)), 1), "min": round(min(clk), 1),
                               "max": round(max(clk), 1)} if clk else None)}


def gemm_ceiling(n, seconds, steps):
    """Dense bf16 GEMM ceiling of this part as a function of the operand
    values: torch.mm (the vendor GEMM library) on n x n x n with operands
    all zero, all one, N(0,1) x N(0,1) (the Q.K^T case) and U(0,1) x N(0,1)
    (the P.V case), each timed with HIP events over `steps` back-to-back
    calls and then run for `seconds` while socket power and gfx clocks are
    read.  At the board's power limit the clock, and with it the rate,
    depends on how much the multiplied bits toggle."""
    import torch
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    flops = 2.0 * n ** 3

    def operands(kind):
        if kind == "zeros":
            return (torch.zeros(n, n, dtype=torch.bfloat16, device=dev),) * 2
        if kind == "ones":
            return (torch.ones(n, n, dtype=torch.bfloat16, device=dev),) * 2
        b = torch.randn(n, n, generator=g, device=dev).to(torch.bfloat16).contiguous()
        if kind == "normal_x_normal":
            a = torch.randn(n, n, generator=g, device=dev).to(torch.bfloat16)
        else:
            a = torch.rand(n, n, generator=g, device=dev).to(torch.bfloat16)
        return a, b

    res = {"shape": [n, n, n], "library": "torch.mm (bf16 in, bf16 out, fp32 accumulation)"}
    for kind in ("zeros", "ones", "normal_x_normal", "uniform_x_normal"):
        a, b = operands(kind)
        c = torch.empty(n, n, dtype=torch.bfloat16, device=dev)

        def mm():
            torch.mm(a, b, out=c)
        for _ in range(10):
            mm()
        torch.cuda.synchronize()
        t = _time_events(mm, steps)
        tf = flops / t / 1e12
        pw = sample_power(mm, seconds) if seconds > 0 else None
        res[kind] = {"ms": round(t * 1e3, 4), "tflops": round(tf, 1),
                     "pct_bf16_peak": round(100 * tf / PEAK_BF16_TFLOPS, 2), "power_clock": pw}
        print(f"[gemm] {kind}: {t * 1e3:.3f} ms, {tf:.0f} TFLOP/s", file=sys.stderr, flush=True)
        del a, b, c
    return res


def attention_timeline(mbe, lib, names, repeats=3):
    """Per-workgroup phase timeline of single attention calls (profiling build
    libmbe_timeline.so).  Each workload is called after a read of 512 MiB
    ("cold": inputs and kernel code evicted from the caches) and right after
    another call ("warm"), one call per record.  Phases per workgroup: lengths
    read (entry -> 1), first tile in LDS (-> 2), key loop (-> 3), epilogue
    until its stores completed (-> 4).  The GPU is kept busy (the read, or a
    spin after the warm-up call) while the host queues the timed call, so
    that the events do not time the host.  `outside_us` is the HIP-event time of
    the call minus the span from the first workgroup's start to the last
    one's end: launch latency, the split merge kernel and the gap before it."""
    import ctypes
    import torch
    import synth
    dev = torch.device("cuda:0")
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev).fill_(1)
    n_wg = 8192
    res = {}
    for name in names:
        k, base = None, name
        if name not in synth.WORKLOADS:
            base, ks = name.rsplit("_k", 1)
            k = int(ks)
        case = synth.workload_attention(base, k_blocks=k)
        c = case.to(dev)
        out = torch.empty_like(c.q)
        mp, mw = int(case.prefix_lens.max()), int(case.window_lens.max())

        def call():
            mbe.window_attention(c.q, c.k_pages, c.v_pages, c.page_table, c.prefix_lens, c.window_lens,
                                 case.block_size, out=out, max_prefix_len=mp, max_window_len=mw,
                                 host_prefix_lens=case.prefix_lens, host_window_lens=case.window_lens)
        for _ in range(5):
            call()
        torch.cuda.synchronize()
        recs = []
        for mode in ["cold"] * repeats + ["warm"] * repeats:
            if lib.mbe_timeline_clear() != 0:
                raise RuntimeError("mbe_timeline_clear failed")
            torch.cuda.synchronize()
            if mode == "cold":
                flush.view(torch.float32).sum()
            else:
                call()
                torch.cuda._sleep(200000)       # keeps the GPU busy while the timed call is queued
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            call()
            e1.record()
            torch.cuda.synchronize()
            buf = np.zeros(n_wg * 8, dtype=np.uint64)
            if lib.mbe_timeline_read(buf.ctypes.data_as(ctypes.c_void_p), ctypes.c_size_t(buf.nbytes)) != 0:
                raise RuntimeError("mbe_timeline_read failed")
            t = buf.reshape(n_wg, 8).astype(np.int64)
            t = t[t[:, 4] > 0]                      # workgroups that ran to the end
            rel = (t[:, :5] - t[:, 0].min()) * 0.01  # 100 MHz ticks -> us
            span = float(rel[:, 4].max())
            ev = e0.elapsed_time(e1) * 1e3
            ph = rel[:, 1:5] - rel[:, 0:4]
            cyc = (t[:, 7] - t[:, 6]) / ((t[:, 4] - t[:, 0]) * 10.0)   # shader cycles per ns
            recs.append({"mode": mode, "event_us": round(ev, 2), "workgroups": int(t.shape[0]),
                         "start_spread_us": round(float(rel[:, 0].max()), 2),
                         "phase_mean_us": [round(float(x), 2) for x in ph.mean(axis=0)],
                         "phase_max_us": [round(float(x), 2) for x in ph.max(axis=0)],
                         "span_us": round(span, 2), "outside_us": round(ev - span, 2),
                         "clock_ghz": round(float(np.mean(cyc)), 3)})
            print(f"[timeline] {name} {mode}: {json.dumps(recs[-1])}", file=sys.stderr, flush=True)
        res[name] = recs
        del c, out
    return res


def bench_pass_loop(mbe, attn_case, c, logits, edit_case, V, steps):
    """N_MBE = 5 editing passes (window attention + threshold update) of 8
    sequences x 2 blocks captured as one graph, each pass after the first
    gated on the previous pass's changed count.  Pass 0 edits (rows with a
    +8 peak, omega_edit 0.5), pass 1 changes nothing (flat rows: confidence
    1/V), passes 2-4 would edit: the replay runs two passes and skips three
    on the device.  Timed against the two passes launched
    eagerly, so (graph - eager) / 3 is the cost of a skipped pass."""
    import torch
    from paper_2607_22663_amd.graphs import PassLoopGraph
    dev = logits.device
    B, nb, win, n_pass = 32, 8, 64, 5
    T = nb * win
    planted = np.zeros(logits.shape[0], dtype=bool)
    planted[edit_case.planted_rows] = True
    rows_peak = torch.from_numpy(np.nonzero(planted)[0][:T]).to(dev)
    g = PassLoopGraph(k_pages=c.k_pages, v_pages=c.v_pages, batch=nb, window=win, block_size=B,
                      num_q_heads=attn_case.num_q_heads, max_pages_per_seq=c.page_table.shape[1],
                      max_prefix_len=int(attn_case.prefix_lens.max()), vocab=V, mask_id=V - 1, n_passes=n_pass,
                      omega_mask=0.5, omega_edit=0.5)
    g.page_table.copy_(c.page_table[:nb])
    g.prefix_lens.copy_(attn_case.prefix_lens[:nb].to(dev))
    for i in range(n_pass):
        g.q[i].copy_(c.q[i * T:(i + 1) * T])
        if i == 1:
            g.logits[i].zero_()          # flat rows: confidence 1/V, nothing to edit
        else:
            g.logits[i].copy_(logits[rows_peak])
    tok0 = edit_case.cur_tokens.to(dev)[rows_peak]
    g.capture()

    def replay():
        g.tokens.copy_(tok0)
        g.replay()

    def eager2():
        g.tokens.copy_(tok0)
        g.run_eager(0)
        g.run_eager(1)
    replay()
    torch.cuda.synchronize()
    ran = [int(x) for x in g.counts.cpu()]
    t_graph = _time_events(replay, steps)
    t_eager = _time_events(eager2, steps)
    del g
    return {"passes": n_pass, "changed_per_pass": ran, "graph_ms": round(t_graph * 1e3, 4),
            "eager_two_passes_ms": round(t_eager * 1e3, 4),
            "skipped_pass_ms": round((t_graph - t_eager) / 3 * 1e3, 4),
            "shape": f"{nb} sequences x {win} rows, vocab {V}"}


def bench_other_workloads(mbe, headline, steps):
    """The other configurations, each timed like the headline step (inputs in
    HBM, 512 MiB read before every timed call, HIP events on the launch
    stream): attention, and edit selection where the configuration has one.
    Figures are per call; the attention share is against its own roofline."""
    import torch
    import synth
    dev = torch.device("cuda:0")
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    flush.fill_(1)

    def timed(fn):
        return _time_cold(fn, steps, flush)

    res = {}
    for name, wl in synth.WORKLOADS.items():
        ks = synth.SPAN_SWEEP_K if name.startswith("span_sweep") else (None,)
        for k in ks:
            if name == headline and k is None:
                continue
            tag = name if k is None else f"{name}_k{k}"
            case = synth.workload_attention(name, k_blocks=k)
            c = case.to(dev)
            out = torch.empty_like(c.q)
            mp, mw = int(case.prefix_lens.max()), int(case.window_lens.max())
            flops, nbytes = attention_work(case)
            roof = min(PEAK_BF16_TFLOPS, flops / nbytes * PEAK_HBM_GBS / 1e3)
            r = {}
            # both V layouts, their calls taken in turn
            layouts = ((False, c.v_pages), (True, c.v_pages.transpose(2, 3).contiguous()))
            calls = [lambda vp=vp: mbe.window_attention(
                c.q, c.k_pages, vp, c.page_table, c.prefix_lens, c.window_lens, case.block_size, out=out,
                max_prefix_len=mp, max_window_len=mw, host_prefix_lens=case.prefix_lens,
                host_window_lens=case.window_lens) for _, vp in layouts]
            times = _time_cold_pair(calls[0], calls[1], steps, flush)
            for (vt, _), (t, tm) in zip(layouts, times):
                tf = flops / t / 1e12
                r["attention" if not vt else "attention_v_token_major"] = {
                    "ms": round(t * 1e3, 4), "ms_median": round(tm * 1e3, 4), "tflops": round(tf, 2),
                    "pct_mfma_peak": round(100 * tf / PEAK_BF16_TFLOPS, 2),
                    "roofline_tflops": round(roof, 1), "pct_of_roofline": round(100 * tf / roof, 2),
                    "gbs": round(nbytes / t / 1e9, 1),
                    "roofline": attention_roofline(flops, nbytes, t, attention_kernel_name(case, 0, vt))}
            del layouts, calls
            del c, out
            if wl.edit is not None and k is None:
                ec = synth.workload_edit(name)
                L, cur = ec.logits.to(dev), ec.cur_tokens.to(dev)
                R, V = L.shape
                eo = (torch.empty(R, dtype=torch.int32, device=dev), torch.empty(R, dtype=torch.float32, device=dev),
                      torch.empty(R, dtype=torch.uint8, device=dev))
                t, tm = timed(lambda: mbe.edit_select(L, cur, ec.threshold, out=eo))
                gbs = edit_bytes(R, V) / t / 1e9
                r["edit_select"] = {"ms": round(t * 1e3, 4), "ms_median": round(tm * 1e3, 4), "rows": R, "vocab": V,
                                    "gbs": round(gbs, 1), "pct_hbm_peak": round(100 * gbs / PEAK_HBM_GBS, 2)}
                del L, cur, eo
            res[tag] = r
            print(f"[bench] {tag}: attention {r['attention']['ms']:.4f} ms (token-major V "
                  f"{r['attention_v_token_major']['ms']:.4f} ms)", file=sys.stderr, flush=True)
    # the floor under any call: one and two back-to-back launches of a
    # one-element fill, timed the same way
    tiny = torch.zeros(1, dtype=torch.int32, device=dev)
    t1, _ = timed(lambda: tiny.fill_(1))
    t2, _ = timed(lambda: (tiny.fill_(1), tiny.fill_(2)))
    res["launch_floor"] = {"one_kernel_us": round(t1 * 1e6, 2), "two_kernels_us": round(t2 * 1e6, 2),
                           "what": "one-element torch fill_ (one or two launches), 512 MiB read before each"}
    del flush
    return res


def cpu_baseline(wl, attn_case, edit_case, flops_total, edit_bytes_total, attn_sample, edit_sample):
    """Times the fp64 oracle (as it stands) on a bounded sample of the same
    workload on the host cores, scaled to the whole step."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # threadpoolctl missing: numpy elementwise work is single-threaded
        cores = 1
    c = attn_case
    cu = c.cu_q
    nb = min(attn_sample, c.batch)
    rows = slice(0, int(cu[nb]))
    sub_flops = 4 * c.head_dim * c.num_q_heads * int(np.sum(
        c.window_lens.numpy()[:nb].astype(np.int64) *
        (c.prefix_lens.numpy()[:nb].astype(np.int64) + c.window_lens.numpy()[:nb])))
    t0 = time.perf_counter()
    oracle.window_attention(c.q[rows], c.k_pages, c.v_pages, c.page_table[:nb], c.prefix_lens[:nb],
                            c.window_lens[:nb], c.block_size)
    t_attn = time.perf_counter() - t0
    attn_rate = sub_flops / t_attn                        # flop/s
    er = min(edit_sample, edit_case.logits.shape[0])
    t0 = time.perf_counter()
    oracle.edit_select(edit_case.logits[:er], edit_case.cur_tokens[:er], edit_case.threshold)
    t_edit = time.perf_counter() - t0
    edit_rate = edit_bytes(er, edit_case.logits.shape[1]) / t_edit   # byte/s
    t_step = flops_total / attn_rate + edit_bytes_total / edit_rate
    sol = flops_total / (PEAK_BF16_TFLOPS * 1e12) + edit_bytes_total / (PEAK_HBM_GBS * 1e9)
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {
        "value": 100.0 * sol / t_step,
        "unit": "% of MI355X peak (speed-of-light step time / oracle step time)",
        "cores": int(cores),
        "cpu": model,
        "kind": "oracle",
        "sample": (f"fp64 numpy oracle: window attention of the first {nb} of {c.batch} sequences "
                   f"({sub_flops / 1e9:.1f} GFLOP, {t_attn:.1f} s) and edit selection of the first {er} "
                   f"of {edit_case.logits.shape[0]} rows ({edit_bytes(er, edit_case.logits.shape[1]) / 1e6:.0f} MB, "
                   f"{t_edit:.1f} s), scaled to the full step"),
        "attention_gflops": attn_rate / 1e9,
        "edit_select_gbs": edit_rate / 1e9,
        "step_s": t_step,
    }


def workload_tag(args):
    return args.workload if args.k is None else f"{args.workload}_k{args.k}"


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--k", type=int, default=None, help="window blocks (span sweep workload)")
    ap.add_argument("--kv-split-tokens", type=int, default=0)
    ap.add_argument("--v-layout", choices=("minor", "major"), default="minor",
                    help="V page layout of the timed step: token-minor [D][16] or token-major [16][D] (like K); "
                         "the other layout is timed too and reported beside it")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-next", action="store_true", help="skip timing the refresh/update/selection calls")
    ap.add_argument("--no-flush", action="store_true", help="do not flush the infinity cache before each step")
    ap.add_argument("--no-others", action="store_true", help="skip timing the other configurations")
    ap.add_argument("--power-sample", type=float, default=0.0, metavar="SECONDS",
                    help="after timing, run the attention and then the edit selection back to back for SECONDS each "
                         "while amd-smi reads socket power and gfx clocks (reported under power_clock)")
    ap.add_argument("--gemm-ceiling", type=int, default=0, metavar="N",
                    help="only measure the bf16 GEMM ceiling (N x N x N) for several operand distributions "
                         "(with --power-sample seconds of power and clock readings each) and exit")
    ap.add_argument("--timeline", nargs="+", metavar="WORKLOAD",
                    help="only record the attention's per-workgroup phase timeline on these workloads "
                         "(span sweep as <name>_k<k>) with the profiling build libmbe_timeline.so, and exit")
    ap.add_argument("--attn-sample", type=int, default=28, help="sequences the CPU oracle times")
    ap.add_argument("--edit-sample", type=int, default=8192, help="edit rows the CPU oracle times")
    ap.add_argument("--summarize-pmc", nargs="+", metavar="PMC_DIR",
                    help="write profiles/hbm_traffic_<workload>.txt from rocprofv3 --pmc output folders (FETCH_SIZE, "
                         "WRITE_SIZE, optionally the TCC_EA0_RDREQ_* request-size pass) and exit")
    ap.add_argument("--summarize-stats", nargs=4, metavar=("STATS_DIR", "BENCH_STDOUT", "OUT_MD", "COMMAND"),
                    help="write a markdown summary of a rocprofv3 --kernel-trace --stats run and exit")
    ap.add_argument("--summarize-counters", nargs=3, metavar=("PMC_DIR", "KERNEL", "OUT_MD"),
                    help="write OUT_MD from a rocprofv3 --pmc pass over one kernel (the command is --counter-command)")
    ap.add_argument("--counter-command", default="")
    ap.add_argument("--summarize-mfma", nargs=4, metavar=("PMC_DIR", "BENCH_STDOUT", "OUT_MD", "COMMAND"),
                    help="write a markdown summary of a rocprofv3 --pmc pass of MFMA counters and exit")
    args = ap.parse_args()
    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc, workload_tag(args), args.counter_command)
        return
    if args.summarize_stats:
        summarize_stats(*args.summarize_stats)
        return
    if args.summarize_mfma:
        summarize_mfma(*args.summarize_mfma, workload_tag(args))
        return
    if args.summarize_counters:
        pmc_dir, kernel, out_md = args.summarize_counters
        summarize_counters(pmc_dir, kernel, out_md, args.counter_command, workload_tag(args))
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus} GPUs, WORLD_SIZE={world}); "
              "this library has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    import paper_2607_22663_amd as mbe

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.gemm_ceiling:
        res = gemm_ceiling(args.gemm_ceiling, args.power_sample, max(args.steps, 20))
        print(json.dumps({"gemm_ceiling": res}), flush=True)
        return
    if args.timeline:
        from paper_2607_22663_amd.build import TIMELINE_LIB
        lib = mbe.load(TIMELINE_LIB)
        lib.mbe_timeline_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t]
        lib.mbe_timeline_clear.argtypes = []
        print(json.dumps({"attention_timeline": attention_timeline(mbe, lib, args.timeline)}), flush=True)
        return
    mbe.load()

    wl = synth.WORKLOADS[args.workload]
    print(f"[bench] generating {args.workload} (seed {wl.seed})", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    vt = args.v_layout == "major"
    attn_case = synth.workload_attention(args.workload, k_blocks=args.k, v_token_major=vt)
    edit_case = synth.workload_edit(args.workload) if wl.edit is not None else None
    print(f"[bench] generated in {time.perf_counter() - t0:.1f} s", file=sys.stderr, flush=True)

    c = attn_case.to(dev)
    max_p = int(attn_case.prefix_lens.max())
    max_w = int(attn_case.window_lens.max())
    hp, hw = attn_case.prefix_lens, attn_case.window_lens      # host copies of the lengths
    out = torch.empty_like(c.q)
    R = V = 0
    if edit_case is not None:
        logits = edit_case.logits.to(dev)
        cur = edit_case.cur_tokens.to(dev)
        R, V = logits.shape
        eo = (torch.empty(R, dtype=torch.int32, device=dev), torch.empty(R, dtype=torch.float32, device=dev),
              torch.empty(R, dtype=torch.uint8, device=dev))
    torch.cuda.synchronize()

    # A plain copy of known size, outside the timed region: its rocprofv3 counter
    # readings calibrate the HBM byte counters of the other kernels.
    calib = torch.empty(CALIB_COPY_BYTES, dtype=torch.uint8, device=dev)
    calib2 = torch.empty_like(calib)
    calib2.copy_(calib)
    torch.cuda.synchronize()
    del calib, calib2

    def attention():
        mbe.window_attention(c.q, c.k_pages, c.v_pages, c.page_table, c.prefix_lens, c.window_lens,
                             attn_case.block_size, out=out, max_prefix_len=max_p, max_window_len=max_w,
                             kv_split_tokens=args.kv_split_tokens, host_prefix_lens=hp, host_window_lens=hw)

    def edit():
        mbe.edit_select(logits, cur, edit_case.threshold, out=eo)

    for _ in range(args.warmup):
        attention()
        if edit_case is not None:
            edit()
    torch.cuda.synchronize()

    n = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n)]
    stream = torch.cuda.current_stream(dev)
    # Before every timed step a 512 MiB buffer is read (a float32 sum, reduced
    # in place), outside the events, so that no input of the step is served
    # from the 256 MB infinity cache.  It is only read: a written buffer would
    # leave the cache full of dirty lines whose write-back to HBM would then
    # land inside the timed step.
    flush = None
    if not args.no_flush:
        flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
        flush.fill_(1)          # 0x01010101: a small positive float
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for i in range(n):
        if flush is not None:
            flush.view(torch.float32).sum()
        ev[i][0].record(stream)
        attention()
        ev[i][1].record(stream)
        if edit_case is not None:
            edit()
        ev[i][2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    del flush
    d_attn = np.array([e[0].elapsed_time(e[1]) for e in ev]) / 1e3
    d_edit = np.array([e[1].elapsed_time(e[2]) for e in ev]) / 1e3
    t_attn = float(np.mean(d_attn))
    t_edit = float(np.mean(d_edit)) if edit_case is not None else 0.0
    t_step = float(np.mean([e[0].elapsed_time(e[2]) for e in ev])) / 1e3

    flops, attn_bytes = attention_work(attn_case)
    e_bytes = edit_bytes(R, V) if edit_case is not None else 0
    sol = flops / (PEAK_BF16_TFLOPS * 1e12) + e_bytes / (PEAK_HBM_GBS * 1e9)
    attn_tflops = flops / t_attn / 1e12
    # the attention roofline of this workload: min(MFMA peak, intensity x HBM peak)
    attn_roof = min(PEAK_BF16_TFLOPS, flops / attn_bytes * PEAK_HBM_GBS / 1e3)
    edit_gbs = e_bytes / t_edit / 1e9 if edit_case is not None else None

    # the same call with the other V page layout (same values), timed the same way
    other_v = c.v_pages.transpose(2, 3).contiguous()
    d_other = []
    flush = None if args.no_flush else torch.empty(512 << 20, dtype=torch.uint8, device=dev).fill_(1)
    for i in range(min(n, 20) + 3):
        if flush is not None:
            flush.view(torch.float32).sum()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        mbe.window_attention(c.q, c.k_pages, other_v, c.page_table, c.prefix_lens, c.window_lens,
                             attn_case.block_size, out=out, max_prefix_len=max_p, max_window_len=max_w,
                             kv_split_tokens=args.kv_split_tokens, host_prefix_lens=hp, host_window_lens=hw)
        e1.record(stream)
        torch.cuda.synchronize()
        if i >= 3:
            d_other.append(e0.elapsed_time(e1) / 1e3)
    del other_v, flush
    t_other = float(np.mean(d_other))
    kernel = attention_kernel_name(attn_case, 0, vt, args.kv_split_tokens)
    kernel_other = attention_kernel_name(attn_case, 0, not vt, args.kv_split_tokens)

    traffic = measured_traffic("window_attention", workload_tag(args), variant=kernel)
    res = {
        "metric": METRIC,
        "value": round(100.0 * sol / t_step, 3),
        "unit": "% of MI355X peak (speed-of-light step time / measured step time)",
        "n_gpus": 1,
        "steps": n,
        "warmup": args.warmup,
        "ms_per_step": round(t_step * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) Q/K/V, N(0,3) logits with planted peaks; shuffled 16-token pages)",
        "config": {
            "workload": args.workload,
            "batch": attn_case.batch,
            "prefix_lens": [int(attn_case.prefix_lens.min()), int(attn_case.prefix_lens.max())],
            "block_size": attn_case.block_size,
            "window_blocks": max_w // attn_case.block_size,
            "q_heads": attn_case.num_q_heads, "kv_heads": attn_case.num_kv_heads,
            "head_dim": attn_case.head_dim, "page_size": 16, "mask": "bidirectional window",
            "edit_rows": R if edit_case is not None else 0, "vocab": V if edit_case is not None else 0,
            "kv_split_tokens": args.kv_split_tokens,
            "v_page_layout": "token-major [16][D]" if vt else "token-minor [D][16]",
        },
        "attention": {"ms": round(t_attn * 1e3, 4), "ms_median": round(float(np.median(d_attn)) * 1e3, 4),
                      "ms_min": round(float(np.min(d_attn)) * 1e3, 4), "tflops": round(attn_tflops, 2),
                      "pct_mfma_peak": round(100 * attn_tflops / PEAK_BF16_TFLOPS, 2),
                      "gflop": round(flops / 1e9, 2), "algorithmic_mb": round(attn_bytes / 1e6, 1),
                      "flop_per_byte": round(flops / attn_bytes, 1),
                      "roofline_tflops": round(attn_roof, 1),
                      "pct_of_roofline": round(100 * attn_tflops / attn_roof, 2),
                      "kernel": kernel},
        "attention_other_v_layout": {"v_page_layout": "token-minor [D][16]" if vt else "token-major [16][D]",
                                     "kernel": kernel_other, "ms": round(t_other * 1e3, 4),
                                     "ms_median": round(float(np.median(d_other)) * 1e3, 4),
                                     "tflops": round(flops / t_other / 1e12, 2),
                                     "pct_mfma_peak": round(100 * flops / t_other / 1e12 / PEAK_BF16_TFLOPS, 2)},
        "cache": "cold: 512 MiB read before every step" if not args.no_flush else "warm (no flush)",
        "edit_select": ({"ms": round(t_edit * 1e3, 4), "ms_median": round(float(np.median(d_edit)) * 1e3, 4),
                         "ms_min": round(float(np.min(d_edit)) * 1e3, 4), "gbs": round(edit_gbs, 1),
                         "pct_hbm_peak": round(100 * edit_gbs / PEAK_HBM_GBS, 2),
                         "algorithmic_mb": round(e_bytes / 1e6, 1),
                         "traffic": measured_traffic("edit_select", workload_tag(args))}
                        if edit_case is not None else None),
        "roofline": attention_roofline(flops, attn_bytes, t_attn, kernel, traffic),
        "wall_s": round(wall, 3),
    }
    if args.power_sample > 0:
        idle = _amdsmi_sample()
        res["power_clock"] = {
            "idle": {"socket_power_w": idle[0], "gfx_clock_mhz_mean": round(float(np.mean(idle[1])), 1)} if idle else None,
            "attention": sample_power(attention, args.power_sample),
            "edit_select": sample_power(edit, args.power_sample) if edit_case is not None else None,
            "source": "amd-smi metric --power --clock --json, read by a host thread while the kernel ran back to back"}
    if edit_case is not None and not args.no_next:
        res["next_rows"] = bench_next_rows(mbe, attn_case, c, logits, cur, R, V, args.steps, edit_case)
    if not args.no_others:
        res["other_workloads"] = bench_other_workloads(mbe, args.workload, min(args.steps, 20))
    if not args.no_cpu_baseline and edit_case is not None:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(wl, attn_case, edit_case, flops, e_bytes,
                                           args.attn_sample, args.edit_sample)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
