#!/usr/bin/env python3
"""Throughput of one TreeFlash drafting step on one MI355X.

A step is the whole hot path for one batch: stage 1 (marginal LM head and
top-M), the AR approximator on every conditional row, the stage-2 LM head with
log-softmax and top-K2, and the best-first tree.  Inputs are synthetic
(seeded, drawn on the GPU) and resident in HBM before timing starts; several
independent weight copies rotate between steps so that no step finds its
weights in the 256 MB last-level cache.

Prints ONE JSON line: draft trees/s (value), rows/s, per-stage times, the
roofline of the dominant kernel (the stage-2 LM-head GEMM, timed alone with HIP
events recorded around its launch), and the CPU oracle timed on a bounded
sample on this host.

Offline helpers (no GPU): --summarize-trace, --summarize-pmc and
--summarize-mfma turn rocprofv3 output into the text summaries kept under
profiles/; the HBM traffic
summary is read back into roofline.traffic while the kernel sources are
unchanged since the counters were taken.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import re
import sqlite3
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2606_03819_amd import binding, synth  # noqa: E402

METRIC = "draft trees/sec (+ conditional rows/sec) at Qwen3-8B shape; HBM GB/s or MFMA % of peak"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
NOMINAL_GHZ = 2.4              # the clock the MFMA peak is rated at
XCDS = 8                       # accelerator dies (GRBM counters sum over them)
SIMDS = 1024                   # 256 CUs x 4 SIMDs
FP32_PEAK_TFLOPS = 157.3       # MI355X fp32 vector/MFMA
RIDGE = BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
PROFILES = os.path.join(ROOT, "profiles")
# sources that define the LM-head GEMM kernel; counters taken on another
# version of them say nothing about this one
KERNEL_SOURCES = ["lmhead.hip", "stream_gemm.hpp", "work.hpp", "plan.hpp", "rows.hpp", "common.hpp", "limits.hpp"]
COPY_BYTES = 1 << 30      # plain copy used to scale the traffic counters


def kernel_source_digest() -> str:
    hsh = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2606_03819_amd", "csrc", name), "rb") as f:
            hsh.update(name.encode() + b"\0" + f.read())
    return hsh.hexdigest()


def lm_kernel_pattern(rows: int, d: int) -> str:
    """Regex for the bf16 LM-head kernel instance the plan picks for `rows` rows
    (template arguments: weight tiles per wave, activation tiles, waves, ...):
    every tile shape goes to the LDS-DMA kernel when d is a multiple of its k
    step (64; beyond two row blocks in 256-row blocks), else to the
    register-staged kernel."""
    nt = 1 if rows <= 32 else (2 if rows <= 64 else 4)
    if rows <= 256 and d % 64 == 0:   # 32-row tiles, or the wave grid up to two row blocks
        return rf"lmhead_dma_kernel<\d+, {nt}, "
    if nt == 4 and rows > 128 and d % 64 == 0:    # 256-row blocks
        return r"lmhead_dma_kernel<\d+, 8, "
    return rf"lmhead_bf16_kernel<\d+, {nt}, "


def traffic_file(workload: str) -> str:
    return os.path.join(PROFILES, f"lmhead_stage2_{workload}_hbm_traffic.md")


def read_traffic(workload: str):
    """HBM bytes per launch of the stage-2 LM-head kernel from the committed counter summary,
    or None when there is none or the kernel sources changed since it was taken."""
    path = traffic_file(workload)
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("source_sha256") != kernel_source_digest() or rec.get("workload") != workload:
        return None
    return rec["traffic_bytes"]


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="qwen3-8b-shape", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--copies", type=int, default=4, help="independent weight copies rotated per step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="time only the headline workload (not the other four benchmark workloads)")
    ap.add_argument("--cpu-seconds", type=float, default=30.0, help="rough cap on the CPU baseline's work")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after timing, copy 1 GiB three times (torch.neg, read 1 GiB + write 1 GiB) "
                         "for counter calibration")
    ap.add_argument("--summarize-trace", metavar="DIR", help="print a kernel-trace summary of a rocprofv3 run")
    ap.add_argument("--summarize-mfma", metavar="DIR", help="print the MFMA use of the stage-2 LM-head kernel "
                    "from a rocprofv3 run with SQ_VALU_MFMA_BUSY_CYCLES and GRBM_GUI_ACTIVE")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print the HBM traffic summary from FETCH_SIZE and WRITE_SIZE rocprofv3 runs")
    ap.add_argument("--summarize-mops", metavar="DIR", help="print the bf16 MFMA work per kernel from a rocprofv3 run "
                    "with SQ_INSTS_VALU_MFMA_MOPS_BF16")
    ap.add_argument("--summarize-mlp-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print the HBM traffic summary of the AR approximator's kernels")
    ap.add_argument("--command", default="", help="command line recorded in a summary")
    ap.add_argument("--sweep", action="store_true",
                    help="drafting cost over budgets B = 16..512 (M = 8) and branchings M = 4..64 (B = 32) "
                         "at the workload's shape; prints one JSON line of its own")
    return ap.parse_args()


def make_copies(w, n):
    dev = torch.device("cuda", 0)
    copies = []
    for i in range(n):
        wi = w.replace(weight_seed=w.weight_seed + 1000 * i)
        device = synth.default_device_for(w)
        ws = synth.make_weights(wi, device)
        copies.append({k: v.to(dev) for k, v in ws.items()})
    states = synth.make_states(w, synth.default_device_for(w))
    return copies, {k: v.to(dev) for k, v in states.items()}


def host_cpu():
    """(usable host cores, CPU model name)."""
    cores = len(os.sched_getaffinity(0))
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return cores, model


def cpu_baseline(w, weights, states, budget_s, repeats=3):
    """The oracle, untuned, on one sequence's full step (one draft tree), with
    BLAS threads = every usable host core; the median of `repeats` runs (fewer
    when one run takes more than a third of `budget_s`)."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits
    import oracle

    cores, model = host_cpu()
    inputs = {k: synth.to_numpy64(v) for k, v in weights.items()}
    inputs["h"] = synth.to_numpy64(states["h"][:1])
    inputs["root"] = synth.to_numpy64(states["root"][:1])
    inputs["context"] = synth.to_numpy64(states["context"][:1])
    draft = oracle.draft_2prev if w.approximator == "2prev" else oracle.draft
    times = []
    with threadpool_limits(limits=cores):
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
        for _ in range(repeats):
            t0 = time.perf_counter()
            draft(inputs, w.gamma, w.k, w.B, w.inv_temperature, mirror_bf16=(w.dtype == "bf16"))
            times.append(time.perf_counter() - t0)
            if sum(times) > budget_s or times[0] > budget_s / 3:
                break
    dt = sorted(times)[len(times) // 2]
    return {"value": 1.0 / dt, "unit": "trees/s", "cores": int(threads), "kind": "oracle",
            "sample": f"one sequence's full drafting step (stage 1, {w.rows} conditional rows, tree) of "
                      f"{w.name}; median of {len(times)} run(s), {dt:.2f} s each in NumPy float64",
            "seconds": dt, "runs": len(times), "host_cores": cores, "cpu_model": model}


def _db(path):
    dbs = sorted(glob.glob(os.path.join(path, "**", "*.db"), recursive=True))
    if not dbs:
        raise SystemExit(f"no rocprofv3 database under {path}")
    return sqlite3.connect(dbs[0])


def summarize_trace(args):
    """Markdown table of per-kernel durations from a rocprofv3 --kernel-trace run."""
    cur = _db(args.summarize_trace).cursor()
    rows = cur.execute("select name, count(*), avg(duration), min(duration), max(duration), sum(duration) "
                       "from kernels where name like '%tf::%' group by name order by sum(duration) desc").fetchall()
    durs = {}
    for name, dur in cur.execute("select name, duration from kernels where name like '%tf::%'"):
        durs.setdefault(name, []).append(dur)
    med = {k: sorted(v)[len(v) // 2] for k, v in durs.items()}
    print(f"# Kernel trace: TreeFlash drafting step, {args.workload}\n")
    print(f"Command (repository root, `cd /tmp && export TMPDIR=/tmp` first):\n\n```\n{args.command}\n```\n")
    print("The library's kernels only (the PyTorch kernels that draw the synthetic inputs are left out); "
          "each bench step runs every kernel once, the merge twice (stage 1 and stage 2).\n")
    print("| kernel | calls | avg us | median us | min us | max us | total ms |\n|---|---|---|---|---|---|---|")
    for name, n, avg, mn, mx, tot in rows:
        short = name.split("(")[0].replace("void ", "")
        print(f"| `{short}` | {n} | {avg / 1e3:.1f} | {med[name] / 1e3:.1f} | {mn / 1e3:.1f} | {mx / 1e3:.1f} | "
              f"{tot / 1e6:.2f} |")


def summarize_pmc(args):
    """HBM traffic of the stage-2 LM-head kernel, scaled by a plain copy of known size."""
    w = synth.get_workload(args.workload)
    pattern = lm_kernel_pattern(w.rows * w.b, w.d)

    def per_kernel(path, counter):
        cur = _db(path).cursor()
        out = {}
        for name, v, n in cur.execute("select name, avg(counter_value), count(*) from pmc_events "
                                      "where counter_name = ? group by name", (counter,)):
            out[name] = (v, n)
        return out

    fetch, write = per_kernel(args.summarize_pmc[0], "FETCH_SIZE"), per_kernel(args.summarize_pmc[1], "WRITE_SIZE")

    def pick(d, pred):
        hits = [(k, v) for k, v in d.items() if pred(k)]
        if not hits:
            raise SystemExit("kernel not found in the counter runs")
        return max(hits, key=lambda kv: kv[1][0])

    lm_f = pick(fetch, lambda k: re.search(pattern, k) is not None)
    lm_w = pick(write, lambda k: re.search(pattern, k) is not None)
    cp_f = pick(fetch, lambda k: "neg" in k.lower())
    cp_w = pick(write, lambda k: "neg" in k.lower())
    kib = COPY_BYTES / 1024.0
    f_fac, w_fac = kib / cp_f[1][0], kib / cp_w[1][0]
    read_b = lm_f[1][0] * 1024.0 * f_fac
    write_b = lm_w[1][0] * 1024.0 * w_fac
    es = 2 if w.dtype == "bf16" else 4
    alg = w.V * w.d * es + w.rows * w.b * w.d * es
    rec = {"workload": w.name, "kernel": lm_f[0].split("(")[0], "dispatches": lm_f[1][1],
           "fetch_size_kib": lm_f[1][0], "write_size_kib": lm_w[1][0],
           "copy_kernel": cp_f[0].split("(")[0][:120], "copy_bytes": COPY_BYTES,
           "copy_fetch_size_kib": cp_f[1][0], "copy_write_size_kib": cp_w[1][0],
           "fetch_factor": f_fac, "write_factor": w_fac, "read_bytes": read_b, "write_bytes": write_b,
           "traffic_bytes": read_b + write_b, "algorithmic_bytes": alg,
           "traffic_over_algorithmic": (read_b + write_b) / alg, "source_sha256": kernel_source_digest()}
    print(f"# HBM traffic of the stage-2 LM-head kernel, {w.name}\n")
    print("Two rocprofv3 counter runs of the same bench command, one counter each; the 1 GiB copy "
          "(torch.neg over float32) that `--copy-calibration` adds gives the factor that turns each "
          "counter into bytes. "
          "`bench.py` reports `traffic_bytes` as `roofline.traffic` while the kernel sources hash to "
          "`source_sha256`.\n")
    print(f"Commands (repository root, `cd /tmp && export TMPDIR=/tmp` first):\n\n```\n{args.command}\n```\n")
    print(f"- LM-head kernel `{rec['kernel']}`: FETCH_SIZE {rec['fetch_size_kib']:.0f} KiB, "
          f"WRITE_SIZE {rec['write_size_kib']:.0f} KiB per dispatch ({rec['dispatches']} dispatches)")
    print(f"- copy of {COPY_BYTES} B: FETCH_SIZE {rec['copy_fetch_size_kib']:.0f} KiB, WRITE_SIZE "
          f"{rec['copy_write_size_kib']:.0f} KiB -> factors {f_fac:.3f} (read), {w_fac:.3f} (write)")
    print(f"- traffic {rec['traffic_bytes'] / 1e6:.1f} MB per launch = {rec['traffic_over_algorithmic']:.3f} x the "
          f"algorithmic {alg / 1e6:.1f} MB (lm_head + activation rows)\n")
    print("```json\n" + json.dumps(rec, indent=1) + "\n```")


def mlp_kernel_bytes(w):
    """(regex, label, algorithmic bytes) of the AR approximator's kernels on the
    one-row-block path: weights, inputs and outputs each counted once."""
    es = 2 if w.dtype == "bf16" else 4
    R, S, d, I = w.rows * w.b, w.gamma * w.b, w.d, w.I
    ew = d
    nproj = 1 if w.approximator == "silu" else 2
    gate = nproj * I * (d + ew) * es + (S * d + R * ew) * es + R * 2 * I * es
    down = d * I * es + R * 2 * I * es + S * d * es + R * d * es
    norm = S * d * es + R * ew * es + 2 * d * es + (S * d + R * ew) * es
    return [(r"mlp_dma_kernel<\d+, \d+, false,", "gate/up (or gate) projection: `mlp_dma_kernel<..., false, ...>`", gate),
            (r"mlp_dma_kernel<\d+, \d+, true,", "down projection: `mlp_dma_kernel<..., true, ...>`", down),
            (r"rmsnorm_rows", "gather + RMSNorm: `rmsnorm_rows_bf16_kernel`", norm)]


def summarize_mlp_pmc(args):
    """HBM traffic of the AR approximator's kernels, scaled like the LM head's."""
    w = synth.get_workload(args.workload)

    def per_kernel(path, counter):
        cur = _db(path).cursor()
        return {name: (v, n) for name, v, n in cur.execute(
            "select name, avg(counter_value), count(*) from pmc_events where counter_name = ? group by name",
            (counter,))}

    fetch = per_kernel(args.summarize_mlp_pmc[0], "FETCH_SIZE")
    write = per_kernel(args.summarize_mlp_pmc[1], "WRITE_SIZE")

    def pick(d, pat):
        hits = [(k, v) for k, v in d.items() if re.search(pat, k)]
        if not hits:
            raise SystemExit(f"kernel {pat} not found in the counter runs")
        return max(hits, key=lambda kv: kv[1][0])

    cp_f, cp_w = pick(fetch, "neg"), pick(write, "neg")
    kib = COPY_BYTES / 1024.0
    f_fac, w_fac = kib / cp_f[1][0], kib / cp_w[1][0]
    recs = []
    for pat, label, alg in mlp_kernel_bytes(w):
        kf, kw = pick(fetch, pat), pick(write, pat)
        rd, wr = kf[1][0] * 1024.0 * f_fac, kw[1][0] * 1024.0 * w_fac
        recs.append({"kernel": kf[0].split("(")[0], "what": label, "dispatches": kf[1][1],
                     "fetch_size_kib": kf[1][0], "write_size_kib": kw[1][0], "read_bytes": rd, "write_bytes": wr,
                     "traffic_bytes": rd + wr, "algorithmic_bytes": alg, "traffic_over_algorithmic": (rd + wr) / alg})
    print(f"# HBM traffic of the AR approximator's kernels, {w.name}\n")
    print("Two rocprofv3 counter runs of the same bench command, one counter each; the 1 GiB copy "
          "(torch.neg over float32) that `--copy-calibration` adds gives the factor that turns each counter "
          "into bytes.  Algorithmic bytes: weights, input rows and outputs, each once (the gate/up activation "
          "as bf16 hi/lo pairs).\n")
    print(f"Commands (repository root, `cd /tmp && export TMPDIR=/tmp` first):\n\n```\n{args.command}\n```\n")
    print(f"- copy of {COPY_BYTES} B: factors {f_fac:.3f} (read), {w_fac:.3f} (write)")
    for r in recs:
        print(f"- {r['what']}: FETCH_SIZE {r['fetch_size_kib']:.0f} KiB, WRITE_SIZE {r['write_size_kib']:.0f} KiB per "
              f"dispatch ({r['dispatches']} dispatches) -> {r['traffic_bytes'] / 1e6:.1f} MB = "
              f"{r['traffic_over_algorithmic']:.3f} x the algorithmic {r['algorithmic_bytes'] / 1e6:.1f} MB")
    print("\n```json\n" + json.dumps({"workload": w.name, "fetch_factor": f_fac, "write_factor": w_fac,
                                        "kernels": recs}, indent=1) + "\n```")


def summarize_mops(args):
    """bf16 MFMA work per dispatch of every library kernel (SQ_INSTS_VALU_MFMA_MOPS_BF16,
    512 FLOP per MOP, summed over the counter's instances of a dispatch)."""
    cur = _db(args.summarize_mops).cursor()
    per = {}
    for name, disp, v in cur.execute("select name, dispatch_id, sum(counter_value) from pmc_events "
                                     "where counter_name = 'SQ_INSTS_VALU_MFMA_MOPS_BF16' group by name, dispatch_id"):
        if "tf::" in name and v > 0:
            per.setdefault(name.split("(")[0], []).append(v * 512.0)
    print(f"# bf16 MFMA work per kernel, {args.workload}\n")
    print(f"Command (repository root, `cd /tmp && export TMPDIR=/tmp` first):\n\n```\n{args.command}\n```\n")
    print("| kernel | dispatches | GFLOP per dispatch (median) |\n|---|---|---|")
    for k, v in sorted(per.items(), key=lambda kv: -sorted(kv[1])[len(kv[1]) // 2]):
        print(f"| `{k}` | {len(v)} | {sorted(v)[len(v) // 2] / 1e9:.1f} |")


def summarize_mfma(args):
    """MFMA busy cycles and the clock of the stage-2 LM-head kernel (the longest
    dispatches of its instance), against the FLOP rate they imply."""
    w = synth.get_workload(args.workload)
    pattern = lm_kernel_pattern(w.rows * w.b, w.d)
    cur = _db(args.summarize_mfma).cursor()
    per = {}
    for name, c, disp, v, dur in cur.execute("select name, counter_name, dispatch_id, sum(counter_value), "
                                             "avg(duration) from pmc_events group by name, counter_name, "
                                             "dispatch_id"):
        if re.search(pattern, name):
            per.setdefault(disp, {"name": name.split("(")[0], "dur_ns": dur})[c] = v
    if not per:
        raise SystemExit("kernel not found in the counter run")
    longest = max(d["dur_ns"] for d in per.values())
    picks = [d for d in per.values() if d["dur_ns"] > 0.5 * longest]   # stage 2 (stage 1 has fewer rows)
    flops = 2.0 * w.rows * w.b * w.V * w.d
    rows_out = []
    for d in picks:
        t = d["dur_ns"] * 1e-9
        clock = d["GRBM_GUI_ACTIVE"] / XCDS / t
        busy = d["SQ_VALU_MFMA_BUSY_CYCLES"] / (clock * t * SIMDS)
        rows_out.append((d["dur_ns"] / 1e3, clock / 1e9, busy, flops / t / 1e12))
    n = len(rows_out)
    avg = [sum(r[i] for r in rows_out) / n for i in range(4)]
    print(f"# MFMA use of the stage-2 LM-head kernel, {w.name}\n")
    print(f"One rocprofv3 counter run of the bench command; `SQ_VALU_MFMA_BUSY_CYCLES` summed over the "
          f"{SIMDS} SIMDs, the clock from `GRBM_GUI_ACTIVE` (summed over {XCDS} XCDs) over the dispatch "
          f"duration.  {w.rows * w.b} rows x V = {w.V} x d = {w.d}: {flops / 1e12:.3f} TFLOP per launch.\n")
    print(f"Command (repository root, `cd /tmp && export TMPDIR=/tmp` first):\n\n```\n{args.command}\n```\n")
    print("| dispatch | us | clock GHz | MFMA busy | TFLOP/s | of 2.5 PF | of peak at this clock |")
    print("|---|---|---|---|---|---|---|")
    for i, (us, ghz, busy, tf) in enumerate(rows_out):
        print(f"| {i} | {us:.0f} | {ghz:.3f} | {busy:.3f} | {tf:.0f} | {tf / BF16_PEAK_TFLOPS:.3f} | "
              f"{tf / (BF16_PEAK_TFLOPS * ghz / NOMINAL_GHZ):.3f} |")
    print(f"\nKernel `{picks[0]['name']}`; mean over {n} dispatches: {avg[0]:.0f} us at {avg[1]:.3f} GHz, MFMA "
          f"busy {avg[2]:.3f} of SIMD cycles, {avg[3]:.0f} TFLOP/s = {avg[3] / BF16_PEAK_TFLOPS:.3f} of the "
          f"2.5 PF peak (rated at {NOMINAL_GHZ} GHz).  The busy fraction exceeds the FLOP fraction at the "
          f"measured clock by the padded rows ({-(-(w.rows * w.b) // 128) * 128} computed for {w.rows * w.b}).")


def make_drafter(w, weights):
    """The drafter of the workload's approximator (its buffers and workspace)."""
    cls = binding.Drafter2Prev if w.approximator == "2prev" else binding.Drafter
    return cls(weights, w.b, w.gamma, w.k, w.B, w.inv_temperature)


def approx_hidden(wt, h, root, context, topk_idx, workspace, hp, V):
    """Stage 2's first half: Eq. 1's SwiGLU (the plain SiLU MLP without an up
    projection), the w/ Linear layer when the weights hold one, or the w/
    2-prev SwiGLU when gate/up read three d-blocks."""
    d = h.shape[2]
    if "w_lin" in wt:
        binding.treeflash_arapprox_linear_hidden(h, root, topk_idx, wt["emb"], wt["norm_h_gain"],
                                                 wt["norm_e_gain"], wt["w_lin"], 1e-6, workspace, hp, V)
    elif wt["w_gate"].shape[1] == 3 * d:
        binding.treeflash_arapprox_2prev_hidden(h, context, root, topk_idx, wt["emb"], wt["norm_h_gain"],
                                                wt["norm_e_gain"], wt["w_gate"], wt["w_up"], wt["w_down"], 1e-6,
                                                workspace, hp, V)
    else:
        binding.treeflash_arapprox_hidden(h, root, topk_idx, wt["emb"], wt["norm_h_gain"], wt["norm_e_gain"],
                                          wt["w_gate"], wt.get("w_up"), wt["w_down"], 1e-6, workspace, hp, V)


def build_tree(w, dr):
    if w.approximator == "2prev":
        binding.treeflash_build_tree_2prev(dr.cond_idx, dr.cond_lp, dr.topk_idx, w.B, dr.tree)
    else:
        binding.treeflash_build_tree(dr.cond_idx, dr.cond_lp, dr.topk_idx, w.B, dr.tree)


def time_steps(w, copies, h, root, steps, warmup, context=None):
    """Mean GPU time per stage of the drafting step for workload w (events around each call)."""
    dev = torch.device("cuda", 0)
    dr = make_drafter(w, copies[0])
    hp = torch.empty((w.b, w.rows, w.d), dtype=w.torch_dtype, device=dev)

    def step(i, ev=None):
        wt = copies[i % len(copies)]
        if ev is not None:
            ev[0].record()
        binding.treeflash_marginal_topk(h, wt["lm_head"], w.k, w.inv_temperature, dr.workspace, dr.topk_idx,
                                        dr.topk_lp)
        if ev is not None:
            ev[1].record()
        approx_hidden(wt, h, root, context, dr.topk_idx, dr.workspace, hp, w.V)
        if ev is not None:
            ev[2].record()
        binding.treeflash_marginal_topk(hp, wt["lm_head"], dr.topk2, w.inv_temperature, dr.workspace,
                                        dr.cond_idx, dr.cond_lp, dr.cond_lse)
        if ev is not None:
            ev[3].record()
        build_tree(w, dr)
        if ev is not None:
            ev[4].record()

    for i in range(warmup):
        step(i)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
    torch.cuda.synchronize()
    for i in range(steps):
        step(i, evs[i])
    torch.cuda.synchronize()
    names = ["stage1_lmhead_topk", "arapprox_mlp", "stage2_lmhead_topk", "tree"]
    us = {n: 1000.0 * sum(e[j].elapsed_time(e[j + 1]) for e in evs) / steps for j, n in enumerate(names)}
    # whole steps with no event between the calls (each one idles the GPU briefly)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for i in range(steps):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    us["step"] = 1000.0 * e0.elapsed_time(e1) / steps
    return us


def sweep(args):
    """Drafting cost over budgets and branchings at the workload's shape (the paper's
    B and M sweeps, as a systems curve)."""
    base = synth.get_workload(args.workload)
    copies, st = make_copies(base, max(1, args.copies))
    h, root, context = st["h"], st["root"], st["context"]
    out = []
    points = [("B", B, base.replace(name=f"{base.name}-B{B}", B=B)) for B in (16, 32, 64, 128, 256, 512)]
    points += [("M", M, base.replace(name=f"{base.name}-M{M}", k=M)) for M in (4, 8, 16, 32, 64)]
    for axis, val, w in points:
        us = time_steps(w, copies, h, root, args.steps, args.warmup, context)
        out.append({"axis": axis, "value": val, "B": w.B, "M": w.k, "conditional_rows": w.rows * w.b,
                    "trees_per_s": w.b * 1e6 / us["step"], "stage_us": us})
    print(json.dumps({"metric": "drafting cost over draft budget B and branching M", "unit": "us",
                      "workload": base.name, "steps": args.steps, "warmup": args.warmup, "sweep": out}),
          flush=True)


def mlp_weight_bytes(w):
    """Bytes of the AR approximator's weights (read once per step)."""
    es = 2 if w.dtype == "bf16" else 4
    d, I = w.d, w.I
    kin = 3 * d if w.approximator == "2prev" else 2 * d
    if w.approximator == "linear":
        return 2 * d * d * es
    nin = 1 if w.approximator == "silu" else 2      # gate (and up) projections
    return (nin * I * kin + d * I) * es


def mlp_flops(w):
    """Algorithmic FLOPs of the AR approximator: the h~ half of the input
    projections once per drafter state (b * gamma), the rest per conditional row."""
    d, I = w.d, w.I
    states, rows = w.b * w.gamma, w.b * w.rows
    ew = 2 * d if w.approximator == "2prev" else d
    if w.approximator == "linear":
        return 2.0 * d * d * states + 2.0 * d * d * rows
    nin = 1 if w.approximator == "silu" else 2
    return 2.0 * nin * I * (d * states + ew * rows) + 2.0 * d * I * rows


def stage_roofline(w, stage_us):
    """The treeflash_arapprox_expand stage (gather + norms, the approximator,
    the stage-2 LM head with log-softmax and top-K2): algorithmic bytes and
    FLOPs against its measured time (the evented pass: AR approximator +
    stage-2 LM head and merge)."""
    es = 2 if w.dtype == "bf16" else 4
    rows = w.b * w.rows
    npre = 2 if w.approximator == "2prev" else 1
    nbytes = (mlp_weight_bytes(w) + rows * npre * w.d * es + w.b * w.gamma * w.d * es
              + w.V * w.d * es + rows * w.d * es)
    flops = mlp_flops(w) + 2.0 * rows * w.V * w.d
    t = (stage_us["arapprox_mlp"] + stage_us["stage2_lmhead_topk"]) * 1e-6
    peak_f = BF16_PEAK_TFLOPS if w.dtype == "bf16" else FP32_PEAK_TFLOPS
    t_ideal = max(nbytes / (HBM_PEAK_GBS * 1e9), flops / (peak_f * 1e12))
    return {"us": t * 1e6, "alg_bytes": nbytes, "alg_flops": flops,
            "hbm_frac": nbytes / t / 1e9 / HBM_PEAK_GBS, "mfma_frac": flops / t / 1e12 / peak_f,
            "frac": t_ideal / t, "bound": "hbm" if nbytes / (HBM_PEAK_GBS * 1e9) >= flops / (peak_f * 1e12) else "mfma"}


def lm_roofline(w, gemm):
    """Roofline of the dominant kernel, the stage-2 LM-head GEMM (the per-row
    merge is a separate kernel); algorithmic bytes per launch: lm_head [V, d]
    once plus the activation rows h' [rows, d]."""
    es = 2 if w.dtype == "bf16" else 4
    rows, V, d = w.b * w.rows, w.V, w.d
    t_lm = gemm["mean"] * 1e-6
    alg_bytes = V * d * es + rows * d * es
    alg_flops = 2.0 * rows * V * d
    if w.dtype == "bf16" and rows > RIDGE:
        roof = {"bound": "mfma", "achieved": alg_flops / t_lm / 1e12, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": alg_bytes / t_lm / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = read_traffic(w.name)
    roof["kernel"] = ("stage-2 LM head on h': " + lm_kernel_pattern(rows, d).split("<")[0]) if w.dtype == "bf16" \
        else "stage-2 LM head on h': lmhead_f32_kernel"
    roof["kernel_us"] = gemm
    roof["alg_bytes_per_launch"] = alg_bytes
    roof["alg_flops_per_launch"] = alg_flops
    roof["hbm_frac"] = alg_bytes / t_lm / 1e9 / HBM_PEAK_GBS
    roof["mfma_frac"] = alg_flops / t_lm / 1e12 / BF16_PEAK_TFLOPS
    return roof


EVENT_EVERY = 4   # timed steps per pair of events around the stage-2 LM-head kernel


def measure(w, copies, st, steps, warmup, copy_calibration=False):
    """Timed drafting steps of workload w (only the two events around the
    stage-2 LM-head kernel inside the timed region, on every EVENT_EVERY-th
    step), then an untimed pass with events between the calls for the
    per-stage split."""
    dev = torch.device("cuda", 0)
    d, V, R, b = w.d, w.V, w.rows, w.b
    dr = make_drafter(w, copies[0])
    hp = torch.empty((b, R, d), dtype=w.torch_dtype, device=dev)
    h, root, context = st["h"], st["root"], st["context"]

    def step(i, ev=None, stages=False):
        wt = copies[i % len(copies)]
        if stages:
            ev[0].record()
        binding.treeflash_marginal_topk(h, wt["lm_head"], w.k, w.inv_temperature, dr.workspace, dr.topk_idx,
                                        dr.topk_lp)
        if stages:
            ev[1].record()
        approx_hidden(wt, h, root, context, dr.topk_idx, dr.workspace, hp, V)
        if stages:
            ev[2].record()
        binding.treeflash_marginal_topk(hp, wt["lm_head"], dr.topk2, w.inv_temperature, dr.workspace,
                                        dr.cond_idx, dr.cond_lp, dr.cond_lse,
                                        events=None if ev is None else (ev[5].cuda_event, ev[6].cuda_event))
        if stages:
            ev[3].record()
        build_tree(w, dr)
        if stages:
            ev[4].record()

    def make_events():
        # events 0..4 bracket the four calls; 5, 6 bracket the stage-2 LM-head GEMM kernel
        # (recorded inside the library on this stream); recording once creates them
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(7)] for _ in range(steps)]
        for e in evs:
            for x in e:
                x.record()
        torch.cuda.synchronize()
        return evs

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    # timed steps: the two events around the stage-2 LM-head kernel, for its live
    # duration, on every EVENT_EVERY-th step only (an event on the stream leaves
    # a few microseconds of idle GPU: every step would carry ~6 us of it)
    every = EVENT_EVERY if steps >= 4 * EVENT_EVERY else 1
    evs = make_events()
    t0 = time.perf_counter()
    for i in range(steps):
        step(i, evs[i] if i % every == 0 else None)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gemm_us = sorted(1000.0 * e[5].elapsed_time(e[6]) for i, e in enumerate(evs) if i % every == 0)

    # per-stage split from a second, untimed pass with events between the calls
    sevs = make_events()
    for i in range(steps):
        step(i, sevs[i], stages=True)
    torch.cuda.synchronize()
    names = ["stage1_lmhead_topk", "arapprox_mlp", "stage2_lmhead_topk", "tree"]
    stage_us = {n: 1000.0 * sum(e[j].elapsed_time(e[j + 1]) for e in sevs) / steps for j, n in enumerate(names)}
    gemm = {"mean": sum(gemm_us) / len(gemm_us), "median": gemm_us[len(gemm_us) // 2],
            "p10": gemm_us[len(gemm_us) // 10], "p90": gemm_us[(9 * len(gemm_us)) // 10]}
    if copy_calibration:
        # an elementwise kernel that reads COPY_BYTES and writes COPY_BYTES (torch's
        # same-dtype copy_ goes to the runtime's blit kernel, shared with other copies)
        a = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
        c = torch.empty_like(a)
        for _ in range(3):
            torch.neg(a, out=c)
        torch.cuda.synchronize()
        del a, c
    return {"elapsed_s": elapsed, "stage_us": stage_us, "lm_kernel_us": gemm, "drafter": dr}


# The other workloads of the benchmark's five (the headline one is timed above).
OTHER_CONFIGS = ["tiny-f32", "qwen3-4b-shape", "qwen3-8b-shape-k16-b64", "qwen3-8b-shape-batch16"]


def other_configs(headline, args):
    """Throughput, the dominant kernel's roofline and the a2-a4 stage fraction of
    every other workload (fewer steps: the headline line is the one the metric
    is quoted on)."""
    out = {}
    steps, warmup = max(5, args.steps // 2), max(2, args.warmup // 2)
    for name in OTHER_CONFIGS:
        if name == headline:
            continue
        w = synth.get_workload(name)
        copies, st = make_copies(w, max(1, args.copies))
        m = measure(w, copies, st, steps, warmup)
        roof = lm_roofline(w, m["lm_kernel_us"])
        out[name] = {"trees_per_s": w.b * steps / m["elapsed_s"],
                     "rows_per_s": w.b * w.rows * steps / m["elapsed_s"],
                     "ms_per_step": 1000.0 * m["elapsed_s"] / steps, "steps": steps, "warmup": warmup,
                     "stage_us": m["stage_us"],
                     "stage2_lm_kernel": {k: roof[k] for k in ("bound", "achieved", "peak", "unit", "frac",
                                                               "hbm_frac", "mfma_frac", "kernel_us")},
                     "arapprox_expand_stage": stage_roofline(w, m["stage_us"])}
        del m, copies, st
        torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.summarize_trace:
        summarize_trace(args)
        return
    if args.summarize_mfma:
        summarize_mfma(args)
        return
    if args.summarize_pmc:
        summarize_pmc(args)
        return
    if args.summarize_mlp_pmc:
        summarize_mlp_pmc(args)
        return
    if args.summarize_mops:
        summarize_mops(args)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; multi-GPU sharding is a design note only",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(2)
    torch.cuda.set_device(0)
    binding.lib()
    if args.sweep:
        sweep(args)
        return
    w = synth.get_workload(args.workload)
    copies, st = make_copies(w, max(1, args.copies))
    dev = torch.device("cuda", 0)
    d, V, R, b = w.d, w.V, w.rows, w.b
    h, root, context = st["h"], st["root"], st["context"]
    m = measure(w, copies, st, args.steps, args.warmup, args.copy_calibration)
    dr = m.pop("drafter")
    elapsed = m["elapsed_s"]
    ms_per_step = 1000.0 * elapsed / args.steps
    trees_per_s = b * args.steps / elapsed
    rows = b * R
    stage_us = m["stage_us"]
    gemm = m["lm_kernel_us"]

    # verification hand-off on the last step's trees: tree-attention inputs and the
    # acceptance walk for a synthetic verifier that agrees with the drafter's best
    # child at every position (so tau is the depth of the greedy path + 1)
    tree_cpu = {f: dr.tree[f].cpu() for f in ("token", "parent")}
    target = torch.full((b, w.B + 1), -1, dtype=torch.int32)
    for s in range(b):
        seen = set()
        for j in range(w.B):
            p = int(tree_cpu["parent"][s, j])
            if p not in seen:
                seen.add(p)
                target[s, p + 1] = tree_cpu["token"][s, j]
    target = target.to(dev)
    vi = binding.treeflash_tree_attention_inputs(root, dr.tree)
    acc = binding.treeflash_accept(dr.tree, target, w.gamma)
    vevs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        vevs[i][0].record()
        binding.treeflash_tree_attention_inputs(root, dr.tree, vi)
        vevs[i][1].record()
        binding.treeflash_accept(dr.tree, target, w.gamma, acc)
        vevs[i][2].record()
    torch.cuda.synchronize()
    handoff = {"tree_attention_inputs_us": 1000.0 * sum(e[0].elapsed_time(e[1]) for e in vevs) / args.steps,
               "accept_us": 1000.0 * sum(e[1].elapsed_time(e[2]) for e in vevs) / args.steps,
               "tau_greedy_verifier": float(acc["accept_len"].float().mean().item()) + 1.0,
               "what": "verifier input (tokens, positions, ancestor mask) and the greedy acceptance walk; "
                       "synthetic verifier = the drafter's best child at every position"}

    # the marginal baseline (DDTree: stage 1 with K = min(B, V), marginal tree) on the
    # same workload and weight rotation, for the cost of AR-approximation
    md = binding.MarginalDrafter(copies[0]["lm_head"], b, w.gamma, w.B, w.inv_temperature)
    for i in range(args.warmup):
        md.step(h, copies[i % len(copies)]["lm_head"])
    mevs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for i in range(args.steps):
        mevs[i][0].record()
        md.step(h, copies[i % len(copies)]["lm_head"])
        mevs[i][1].record()
    torch.cuda.synchronize()
    m_elapsed = time.perf_counter() - t1
    ddtree = {"trees_per_s": b * args.steps / m_elapsed, "ms_per_step": 1000.0 * m_elapsed / args.steps,
              "gpu_us_per_step": 1000.0 * sum(e[0].elapsed_time(e[1]) for e in mevs) / args.steps,
              "K": md.K, "what": "stage 1 with K = min(B, V) entries per depth + marginal OPT-Tree"}
    del md

    roof = lm_roofline(w, gemm)
    es = 2 if w.dtype == "bf16" else 4
    step_bytes = 2 * V * d * es + mlp_weight_bytes(w)
    out = {
        "metric": METRIC, "value": trees_per_s, "unit": "trees/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "b": b, "d": d, "V": V, "gamma": w.gamma, "k": w.k, "B": w.B, "I": w.I,
                   "approximator": w.approximator, "inv_temperature": w.inv_temperature, "conditional_rows": rows, "gamma_k_b": w.gamma * w.k * b,
                   "weight_copies": len(copies)},
        "rows_per_s": rows * args.steps / elapsed,
        "stage_us": stage_us,
        "step_hbm_frac": step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "roofline": roof,
        "arapprox_expand_stage": stage_roofline(w, stage_us),
        "ddtree_baseline": ddtree,
        "verify_handoff": handoff,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, copies[0], st, args.cpu_seconds)
    del dr, copies, st
    if not args.no_configs:
        out["configs"] = other_configs(w.name, args)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
