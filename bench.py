"""Benchmark: one MoE layer, forward + backward, on one MI355X.

A step is the whole hot path on one batch: route, dispatch index build,
expert FFN forward (two grouped GEMMs), combine, expert FFN backward (four
grouped GEMMs + gate-gradient reduction), token-gradient combine and router
backward. Inputs and weights are resident in HBM before the timed region.

Prints one JSON line: tokens/s (whole job), per-kernel times from HIP events
recorded on the launch stream inside the timed region, the roofline of the
dominant kernel, saved and peak activation bytes per token next to a
materialised-permutation PyTorch baseline, and the CPU oracle timed on a
bounded token sample of the same workload.

python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload few_large_e8k2]

The default workload is the largest of the layer workloads that fits one GPU
(T=32768, d=4096, f=14336, E=8, k=2), with the h-on-load policy (no SwiGLU
intermediate in HBM); --h-buffered times the policy that passes h and g*h
between the GEMMs through transient buffers.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None,
                    help="layer workload (default: few_large_e8k2; mem_sweep_e64k8 for --sweep)")
    ap.add_argument("--act", choices=("swiglu", "silu", "relu"), default=None,
                    help="expert activation (default: the workload's own)")
    ap.add_argument("--h-buffered", dest="h_on_load", action="store_false",
                    help="buffer h (forward) and g*h (backward) between the GEMMs instead of "
                         "forming them on load (MOE_H_ON_LOAD, the default)")
    ap.add_argument("--h-on-load", dest="h_on_load", action="store_true",
                    help="form h and g*h on load, no SwiGLU intermediate in HBM (the default)")
    ap.set_defaults(h_on_load=True)
    ap.add_argument("--atomic-combine", dest="atomic_combine", action="store_true",
                    help="fold the combine into the epilogues of the second GEMM and the dX GEMM "
                         "(MOE_ATOMIC_COMBINE: packed-bf16 atomic adds into y and dx, no strips); "
                         "default: only where that is deterministic (k <= 2)")
    ap.add_argument("--strip-combine", dest="atomic_combine", action="store_false",
                    help="combine strip by strip with the ordered gather-reduce")
    ap.set_defaults(atomic_combine=None)
    ap.add_argument("--graph", action="store_true",
                    help="also time the step captured once in a HIP graph and replayed "
                         "(graph_replay in the JSON line; the main figures stay eager)")
    ap.add_argument("--recompute", action="store_true",
                    help="full-recompute checkpoint policy: save only the routing decision; the "
                         "dispatch and the expert FFN run over token chunks, and the backward "
                         "rebuilds each chunk's maps and first layer")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate CPU time budget of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-baseline-memory", action="store_true")
    ap.add_argument("--no-reference-rates", action="store_true",
                    help="skip the two measured ceilings (device copy, hipBLASLt dense GEMM)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a 1 GiB device copy (reference for HBM byte counters)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the per-kernel HBM traffic summary from two rocprofv3 --pmc "
                         "runs (FETCH_SIZE, WRITE_SIZE) of this script with --copy-calibration")
    ap.add_argument("--pmc-out", default=None)
    ap.add_argument("--summarize-stats", metavar="KERNEL_STATS_CSV",
                    help="write the short per-kernel timing summary of a rocprofv3 "
                         "--kernel-trace --stats run of this script")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("TCP_CSV", "SQ_CSV"),
                    help="write the per-kernel L1-to-L2 request and MFMA-busy summary from two "
                         "rocprofv3 --pmc runs of this script (TCP_TCC_READ_REQ_sum "
                         "TCP_TCC_READ_REQ_LATENCY_sum TCP_TCC_WRITE_REQ_sum "
                         "TCP_PENDING_STALL_CYCLES_sum, then SQ_VALU_MFMA_BUSY_CYCLES "
                         "SQ_BUSY_CYCLES GRBM_GUI_ACTIVE)")
    ap.add_argument("--summarize-lds", metavar="LDS_CSV",
                    help="write the per-kernel LDS bank-conflict summary from a rocprofv3 "
                         "--pmc run of this script (SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE "
                         "SQ_INSTS_LDS GRBM_GUI_ACTIVE)")
    ap.add_argument("--summarize-table1", metavar="JSON",
                    help="write profiles/table1_sweep.txt from the last line of a --table1 run")
    ap.add_argument("--summarize-sweep", metavar="JSON",
                    help="write the memory-sweep summary from the last line of a --sweep run")
    ap.add_argument("--profile-command", default="",
                    help="the rocprofv3 command(s) the summarised files came from")
    ap.add_argument("--summary-out", default=None)
    ap.add_argument("--sweep", action="store_true",
                    help="memory-capacity sweep: double T from the workload's T until out of "
                         "memory, for this path and for the materialised-permutation baseline")
    ap.add_argument("--sweep-max-doublings", type=int, default=9)
    ap.add_argument("--table1", action="store_true",
                    help="the seven shapes of the paper's Table 1 (SiLU and SwiGLU experts): "
                         "this path against a materialised PyTorch layer, time and memory")
    args = ap.parse_args()
    if args.workload is None:
        args.workload = "mem_sweep_e64k8" if args.sweep else "few_large_e8k2"
    return args


CSRC = os.path.join(ROOT, "paper_2601_05296_amd", "csrc")
COPY_BYTES = 1 << 30


def code_tokens(src: str) -> str:
    """C/C++ source without its comments, whitespace runs collapsed to one
    space (string and character literals kept as they are)."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c in "\"'":                                  # literal
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
            out.append(" ")
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def source_digest(csrc: str = CSRC) -> str:
    """sha256 over the code of the HIP sources (comments and layout left out):
    a traffic summary is valid only for that code."""
    import hashlib
    h = hashlib.sha256()
    for name in sorted(os.listdir(csrc)):
        if not name.endswith((".hip", ".hpp", ".cpp", ".h")):
            continue
        with open(os.path.join(csrc, name), encoding="utf-8") as fh:
            h.update(name.encode() + b"\0" + code_tokens(fh.read()).encode())
    return h.hexdigest()


def traffic_path(workload):
    return os.path.join(ROOT, "profiles", "hbm_traffic_%s.txt" % workload)


def kernel_short_name(full: str) -> str:
    """'void moe::(anonymous namespace)::g5_kernel(...)' -> 'g5_kernel'."""
    name = full.replace("(anonymous namespace)", "")
    return name.split("(")[0].split("::")[-1].split("<")[0].split()[-1]


def summarize_pmc(fetch_csv, write_csv, out, workload, cmd):
    """Average FETCH_SIZE / WRITE_SIZE (KiB per dispatch) per kernel, and the
    scale factors that make the copy kernel read and write exactly the bytes
    it moved."""
    import csv
    def load(path, counter):
        acc = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            acc.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return {k: float(np.mean(v)) for k, v in acc.items()}
    fetch, write = load(fetch_csv, "FETCH_SIZE"), load(write_csv, "WRITE_SIZE")
    copy = [k for k in fetch if "copy" in k.lower() or "elementwise" in k.lower()]
    copy = max(copy, key=lambda k: fetch[k])
    ff = COPY_BYTES / 1024.0 / fetch[copy]
    wf = COPY_BYTES / 1024.0 / write[copy]
    lines = ["# HBM traffic per dispatch (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE)",
             "# workload: %s" % workload,
             "# command: %s" % cmd,
             "# copy kernel (%d bytes read and written): %s" % (COPY_BYTES, kernel_short_name(copy)),
             "# scale factors: fetch %.4f, write %.4f (bytes = KiB * 1024 * factor)" % (ff, wf),
             "source_sha256 %s" % source_digest(),
             "fetch_factor %.6f" % ff, "write_factor %.6f" % wf,
             "# kernel fetch_KiB write_KiB"]
    for k in sorted(fetch, key=lambda k: -fetch[k]):
        short = kernel_short_name(k)
        if k == copy:
            short = "copy_calibration"
        lines.append("kernel %s %.1f %.1f" % (short, fetch[k], write.get(k, float("nan"))))
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("wrote", out)


def summarize_stats(stats_csv, out, workload, cmd, profile_cmd):
    """Per-kernel calls and durations from rocprofv3's kernel_stats.csv."""
    import csv
    from paper_2601_05296_amd import synth
    cfg = synth.CONFIGS[workload]
    rows = list(csv.DictReader(open(stats_csv)))
    lines = ["# rocprofv3 kernel statistics, workload %s (T=%d d=%d f=%d E=%d k=%d, %s)"
             % (workload, cfg.T, cfg.d, cfg.f, cfg.E, cfg.k, cfg.dtype),
             "# profile: %s" % profile_cmd,
             "# summary: python %s" % cmd,
             "# kernel calls avg_us total_ms pct min_us max_us"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        lines.append("%-22s %4d %10.1f %9.3f %6.2f %9.1f %9.1f" % (
            kernel_short_name(r["Name"])[:22], int(r["Calls"]), float(r["AverageNs"]) / 1e3,
            float(r["TotalDurationNs"]) / 1e6, float(r["Percentage"]),
            float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3))
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("wrote", out)


def summarize_table1(json_path, out, cmd, profile_cmd):
    """Text summary of a --table1 run (its last output line)."""
    rows = json.loads(open(json_path).read().strip().splitlines()[-1])["table1"]
    policy = (", this path with MOE_H_ON_LOAD (no h / g*h buffers)"
              if rows and rows[0].get("h_on_load") else "")
    lines = ["# Table 1 shapes (paper Section 6.1): this path vs a materialised PyTorch MoE layer"
             + policy,
             "# run: %s" % profile_cmd,
             "# summary: python %s" % cmd,
             "# one MI355X, bf16, f = 4d, T = batch x seq_len, plain top-k softmax gates; "
             "device-side seeded inputs",
             "# baseline: argsort + index_select routed-token buffer, one torch matmul (hipBLASLt) "
             "per expert, every",
             "#   intermediate kept by autograd (bench.materialised_step); saved bytes from "
             "saved-tensor hooks",
             "# bytes are per token; peak = max(forward peak, step peak less weight gradients), "
             "inputs and weights excluded",
             "# conf act T d f E k | ours_ms base_ms speedup | ours_saved base_saved ratio | "
             "ours_peak base_peak ratio | ours tokens/s"]
    for r in rows:
        lines.append("%s %s %d %d %d %d %d | %.3f %.3f %.2fx | %.0f %.0f %.2fx | %.0f %.0f %.2fx | %.0f" % (
            r["conf"], r["act"], r["T"], r["d"], r["f"], r["E"], r["k"], r["ours_ms"], r["base_ms"],
            r["speedup"], r["ours_saved_bytes_per_token"], r["base_saved_bytes_per_token"],
            r["saved_ratio"], r["ours_peak_bytes_per_token"], r["base_peak_bytes_per_token"],
            r["base_peak_bytes_per_token"] / r["ours_peak_bytes_per_token"], r["ours_tokens_per_s"]))
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("wrote", out)


def summarize_sweep(json_path, out, cmd, profile_cmd):
    """Text summary of a --sweep run (its last output line)."""
    from paper_2601_05296_amd import synth
    res = json.loads(open(json_path).read().strip().splitlines()[-1])["sweep"]
    c = synth.CONFIGS[res["workload"]]
    policy = ("full recompute over token chunks (only the routing decision saved)"
              if res.get("recompute") else
              "h and g*h formed on load (MOE_H_ON_LOAD)" if res.get("h_on_load") else
              "h and g*h buffered between the GEMMs")
    if res.get("atomic_combine"):
        policy += "; combine folded into the GEMM epilogues (MOE_ATOMIC_COMBINE)"
    lines = ["# Memory-capacity sweep, workload %s (d=%d f=%d E=%d k=%d, %s), one MI355X; "
             "this path: %s" % (c.name, c.d, c.f, c.E, c.k, c.dtype, policy),
             "# run: %s" % profile_cmd,
             "# summary: python %s" % cmd,
             "# ours: one forward + backward through the C ABI (moe_ffn_fwd_combine / "
             "moe_ffn_bwd_combine); peak =",
             "#       max(forward allocator peak, backward allocator peak less weight gradients), "
             "weights and inputs excluded",
             "# baseline: materialised-permutation PyTorch layer, forward only (saved tensors + "
             "forward temporaries;",
             "#           a lower bound on its training peak)",
             "# HBM: %d bytes" % res["hbm_bytes"],
             "# T  ours_peak_B/token  ours_saved_B/token  baseline_fwd_peak_B/token  "
             "baseline_saved_B/token"]
    def cell(r, key, oom):
        if key in r:
            return "%11.1f" % r[key]
        return "%11s" % ("OOM" if r.get(oom) else "-")
    for r in res["points"]:
        lines.append("%8d %s %s %s %s" % (
            r["T"], cell(r, "ours_peak_bytes_per_token", "ours_oom"),
            cell(r, "ours_saved_bytes_per_token", "ours_oom"),
            cell(r, "baseline_fwd_peak_bytes_per_token", "baseline_oom"),
            cell(r, "baseline_saved_bytes_per_token", "baseline_oom")))
    lines.append("# largest T that fits: ours %d, materialised baseline (forward alone) %d"
                 % (res["max_T_ours"], res["max_T_baseline_fwd"]))
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("wrote", out)


N_CU, N_XCD, SIMD_PER_CU = 256, 8, 4


def summarize_counters(tcp_csv, sq_csv, out, workload, cmd, profile_cmd):
    """Per-kernel means per launch of the L1-to-L2 request counters and of
    the MFMA busy cycles. GRBM_GUI_ACTIVE is summed over the XCDs, so one
    XCD's cycles are GUI/8; the mean number of read requests in flight per CU
    is the latency sum (request-cycles) over CU-cycles. The clock is one XCD's
    cycles over the dispatch's duration (meaningful for launches of a
    millisecond or more; short ones count the dispatch overhead's cycles)."""
    import csv
    acc, launches, dur = {}, {}, {}
    for path in (tcp_csv, sq_csv):
        seen = {}
        for r in csv.DictReader(open(path)):
            name = kernel_short_name(r["Kernel_Name"])
            a = acc.setdefault(name, {})
            a[r["Counter_Name"]] = a.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
            ids = seen.setdefault(name, set())
            if path == sq_csv and r["Dispatch_Id"] not in ids:
                dur[name] = dur.get(name, 0.0) + (int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
            ids.add(r["Dispatch_Id"])
        for name, ids in seen.items():
            launches[name] = max(launches.get(name, 0), len(ids))
    lines = ["# L1-to-L2 requests, MFMA busy time and clock per launch, workload %s" % workload,
             "# profile: %s" % profile_cmd,
             "# summary: python %s" % cmd,
             "# cycles = GRBM_GUI_ACTIVE / %d (one XCD); %d CUs, %d SIMDs per CU" % (N_XCD, N_CU, SIMD_PER_CU),
             "# rd_req: TCP_TCC_READ_REQ; lat: mean read latency in cycles; inflight: mean read "
             "requests in flight per CU; pend: share of CU-cycles the L1 stalls on pending "
             "requests; wr_req: TCP_TCC_WRITE_REQ; mfma: MFMA busy share of SIMD-cycles; "
             "us: mean duration; clk: cycles / duration (GHz)",
             "# kernel launches cycles rd_req lat inflight pend wr_req mfma us clk"]
    def per(a, key, n):
        return a.get(key, 0.0) / n
    order = sorted(acc, key=lambda k: -acc[k].get("GRBM_GUI_ACTIVE", 0.0))
    for name in order:
        a, n = acc[name], launches[name]
        cyc = per(a, "GRBM_GUI_ACTIVE", n) / N_XCD
        if cyc <= 0:
            continue
        rq = per(a, "TCP_TCC_READ_REQ_sum", n)
        lat_sum = per(a, "TCP_TCC_READ_REQ_LATENCY_sum", n)
        us = dur.get(name, 0.0) / n / 1e3
        lines.append("%-20s %4d %9.0f %10.3g %6.0f %8.1f %6.2f %10.3g %6.2f %9.1f %5.2f" % (
            name[:40], n, cyc, rq, lat_sum / rq if rq else float("nan"), lat_sum / (N_CU * cyc),
            per(a, "TCP_PENDING_STALL_CYCLES_sum", n) / (N_CU * cyc),
            per(a, "TCP_TCC_WRITE_REQ_sum", n),
            per(a, "SQ_VALU_MFMA_BUSY_CYCLES", n) / (N_CU * SIMD_PER_CU * cyc),
            us, cyc / (us * 1e3) if us > 0 else float("nan")))
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("wrote", out)


def summarize_lds(lds_csv, out, workload, cmd, profile_cmd):
    """Per-kernel means per launch of the LDS counters: cycles the LDS was
    busy with indexed accesses, the part of them lost to bank conflicts, and
    LDS instructions (summed over all CUs)."""
    import csv
    acc, ids = {}, {}
    for r in csv.DictReader(open(lds_csv)):
        name = kernel_short_name(r["Kernel_Name"])
        a = acc.setdefault(name, {})
        a[r["Counter_Name"]] = a.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        ids.setdefault(name, set()).add(r["Dispatch_Id"])
    lines = ["# LDS bank conflicts per launch, workload %s" % workload,
             "# profile: %s" % profile_cmd,
             "# summary: python %s" % cmd,
             "# active: SQ_LDS_IDX_ACTIVE; conflict: SQ_LDS_BANK_CONFLICT (cycles, all CUs); "
             "share: conflict / active; insts: SQ_INSTS_LDS",
             "# kernel launches active conflict share insts"]
    order = sorted(acc, key=lambda k: -acc[k].get("SQ_LDS_IDX_ACTIVE", 0.0) / len(ids[k]))
    for name in order:
        a, n = acc[name], len(ids[name])
        act = a.get("SQ_LDS_IDX_ACTIVE", 0.0) / n
        if act <= 0:
            continue
        bc = a.get("SQ_LDS_BANK_CONFLICT", 0.0) / n
        lines.append("%-20s %4d %10.3g %10.3g %6.3f %10.3g" % (
            name[:40], n, act, bc, bc / act, a.get("SQ_INSTS_LDS", 0.0) / n))
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("wrote", out)


def read_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed summary, or None if
    absent or taken on different sources."""
    p = traffic_path(workload)
    if not os.path.exists(p):
        return None
    vals, kern = {}, {}
    for line in open(p):
        parts = line.split()
        if not parts or parts[0].startswith("#"):
            continue
        if parts[0] == "kernel":
            kern[parts[1]] = (float(parts[2]), float(parts[3]))
        else:
            vals[parts[0]] = parts[1]
    if vals.get("source_sha256") != source_digest() or kernel not in kern:
        return None
    f_kib, w_kib = kern[kernel]
    return round((f_kib * float(vals["fetch_factor"]) + w_kib * float(vals["write_factor"])) * 1024.0)


def kernel_model(name, cfg, elem, recompute=False):
    """Algorithmic work of one kernel over one whole step (all its launches:
    the strips of the second GEMM, of the dX GEMM and of the combine, both
    combine passes, the recomputed first GEMM): (amount, unit, bound)."""
    T, d, f, E, k = cfg.T, cfg.d, cfg.f, cfg.E, cfg.k
    S = T * k
    g = 2.0 * S * d * f  # flops of one [S x d] x [d x f] product
    nb = 2 if cfg.act == "swiglu" else 1   # right operands of g1, g5, g6
    flops = {"g1_kernel": nb * g * (2 if recompute else 1), "g2_kernel": g, "g2h_kernel": g,
             "g3_kernel": g, "g3h_kernel": g,
             "g4_kernel": g, "g5_kernel": nb * g, "g6_kernel": nb * g}
    if name in flops:
        return flops[name], "TFLOP/s", "mfma"
    nparts = -(-f // 256) * 4   # gate-gradient partials per slot (G4: 256-column tiles, 4 waves across)
    nbuild = 2 if recompute else 1   # full recompute builds the maps again in the backward
    byts = {
        "route_bf16": T * d * elem + E * d * elem + T * E * 4 + T * k * 8,
        "tile_hist": nbuild * S * 4,
        "tile_scan": 0,
        "tile_rank": nbuild * (S * 4 + 3 * S * 4),
        "combine": 2 * (S * d * elem + T * d * elem + T * k * 8),   # forward and backward
        "dgate_reduce": S * nparts * 4 + S * 8,
        "slot_gates": S * 12,
        "fwd_slot_gates": S * 12,
        "zero_bf16": 2 * T * d * elem,   # y in the forward, dx in the backward
        "expert_ranks": E * 4 + E * 16,
        "rb_dlogits": T * E * 4 * 2 + T * k * 12,
        "rb_dx": T * E * 4 + E * d * elem + 2 * T * d * elem,
        "rb_dwg_partial": T * E * 4 + T * d * elem,
        "rb_dwg_reduce": 0,
    }
    return float(byts.get(name, 0)), "GB/s", "hbm"


def materialised_saved_bytes(x, w_gate, bias, w1, w3, w2, k, renorm, act="swiglu"):
    """Saved-for-backward bytes of a conventional MoE layer that materialises
    the permuted tokens and every expert intermediate (plain PyTorch autograd,
    forward only; weights are parameters and not counted)."""
    import torch
    # storages of the parameters and of the caller's input: not activations
    excluded = {t.untyped_storage().data_ptr() for t in (x, w_gate, w1, w3, w2) if t is not None}
    seen = {}

    def pack(t):
        if t.untyped_storage().data_ptr() not in excluded:
            seen[(t.data_ptr(), t.dtype, tuple(t.shape))] = t.numel() * t.element_size()
        return t

    T, d = x.shape
    E = w1.shape[0]
    xs = x.detach().requires_grad_(True)
    wg = w_gate.detach().requires_grad_(True)
    W1, W3, W2 = (None if w is None else w.detach().requires_grad_(True) for w in (w1, w3, w2))
    with torch.autograd.graph.saved_tensors_hooks(pack, lambda t: t):
        logits = (xs @ wg.t()).float()
        if bias is not None:
            logits = logits + bias
        p = torch.softmax(logits, dim=1)
        g, ids = torch.topk(p, k, dim=1)
        if renorm:
            g = g / g.sum(dim=1, keepdim=True)
        flat = ids.reshape(-1)
        order = torch.argsort(flat, stable=True)
        tok = order // k
        x_perm = xs.index_select(0, tok)               # routed-token buffer
        counts = torch.bincount(flat, minlength=E).tolist()
        outs = []
        o0 = 0
        for e in range(E):
            xe = x_perm[o0:o0 + counts[e]]
            a = xe @ W1[e]
            if act == "swiglu":
                h = torch.nn.functional.silu(a) * (xe @ W3[e])
            elif act == "relu":
                h = torch.relu(a)
            else:
                h = torch.nn.functional.silu(a)
            outs.append(h @ W2[e])
            o0 += counts[e]
        O = torch.cat(outs, 0)
        gw = g.reshape(-1)[order].to(O.dtype)
        y = torch.zeros_like(xs).index_add_(0, tok, O * gw[:, None])
    del y
    return sum(seen.values())


def materialised_step(x, w_gate, bias, w1, w3, w2, dy, k, renorm, act):
    """One forward + backward of a conventional MoE layer in plain PyTorch: the
    permuted tokens and every expert intermediate are materialised, one matmul
    per expert, autograd for the backward. Returns the gradients."""
    import torch
    xs = x.detach().requires_grad_(True)
    wg = w_gate.detach().requires_grad_(True)
    W1, W3, W2 = (None if w is None else w.detach().requires_grad_(True) for w in (w1, w3, w2))
    E = w1.shape[0]
    logits = (xs @ wg.t()).float()
    if bias is not None:
        logits = logits + bias
    p = torch.softmax(logits, dim=1)
    g, ids = torch.topk(p, k, dim=1)
    if renorm:
        g = g / g.sum(dim=1, keepdim=True)
    flat = ids.reshape(-1)
    order = torch.argsort(flat, stable=True)
    tok = order // k
    x_perm = xs.index_select(0, tok)
    counts = torch.bincount(flat, minlength=E).tolist()
    outs = []
    o0 = 0
    for e in range(E):
        xe = x_perm[o0:o0 + counts[e]]
        a = xe @ W1[e]
        if act == "swiglu":
            h = torch.nn.functional.silu(a) * (xe @ W3[e])
        elif act == "relu":
            h = torch.relu(a)
        else:
            h = torch.nn.functional.silu(a)
        outs.append(h @ W2[e])
        o0 += counts[e]
    O = torch.cat(outs, 0)
    gw = g.reshape(-1)[order].to(O.dtype)
    y = torch.zeros_like(xs).index_add_(0, tok, O * gw[:, None])
    y.backward(dy)
    return [t.grad for t in (xs, wg, W1, W3, W2) if t is not None]


def table1_sweep(args):
    """The seven shapes of the paper's Table 1 (Section 6.1), with the
    non-gated SiLU expert and with SwiGLU: time per fwd+bwd step, saved and
    peak activation bytes per token, for this path and for the materialised
    PyTorch layer (materialised_step). Inputs are drawn on the device from a
    seeded generator with the workloads' distributions."""
    import torch
    from paper_2601_05296_amd import layer, synth
    dev = torch.device("cuda:0")
    bf = torch.bfloat16
    hol = bool(args.h_on_load)   # this path with MOE_H_ON_LOAD
    rows = []
    for act in ("silu", "swiglu"):
        for name in synth.TABLE1:
            cfg = synth.CONFIGS["table1_" + name].with_(act=act)
            T, d, f, E, k = cfg.T, cfg.d, cfg.f, cfg.E, cfg.k
            gated = act == "swiglu"
            gen = torch.Generator(device=dev)
            gen.manual_seed(cfg.seed)
            rnd = lambda shape, std: (torch.randn(shape, generator=gen, device=dev) * std).to(bf)
            wg = rnd((E, d), 0.02)
            w1 = rnd((E, d, f), d ** -0.5)
            w3 = rnd((E, d, f), d ** -0.5) if gated else None
            w2 = rnd((E, f, d), f ** -0.5)
            x = rnd((T, d), 1.0)
            dy = rnd((T, d), 1.0)
            row = {"conf": name, "act": act, "T": T, "d": d, "f": f, "E": E, "k": k,
                   "h_on_load": hol}

            def timed(fn, steps, warm):
                for _ in range(warm):
                    fn()
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(steps):
                    fn()
                e1.record()
                torch.cuda.synchronize()
                return e0.elapsed_time(e1) / steps

            def ours():
                y, saved = layer.forward(x, wg, None, w1, w3, w2, k, False, act=act, h_on_load=hol)
                return layer.backward(saved, dy, x, wg, w1, w3, w2)

            def base():
                return materialised_step(x, wg, None, w1, w3, w2, dy, k, False, act)

            for which, fn in (("ours", ours), ("base", base)):
                torch.cuda.empty_cache()
                row[which + "_ms"] = round(timed(fn, args.steps, args.warmup), 4)
                torch.cuda.synchronize()
                # forward peak, then the peak of the whole step less the weight
                # gradients (which live only in the backward); the larger counts
                torch.cuda.reset_peak_memory_stats(dev)
                m0 = torch.cuda.memory_allocated(dev)
                if which == "ours":
                    y, saved = layer.forward(x, wg, None, w1, w3, w2, k, False, act=act, h_on_load=hol)
                    del y, saved
                else:
                    materialised_saved_bytes(x, wg, None, w1, w3, w2, k, False, act)
                torch.cuda.synchronize()
                fwd_peak = torch.cuda.max_memory_allocated(dev) - m0
                torch.cuda.reset_peak_memory_stats(dev)
                out = fn()
                torch.cuda.synchronize()
                peak = torch.cuda.max_memory_allocated(dev) - m0
                grads = sum(t.numel() * t.element_size()
                            for t in (out.values() if isinstance(out, dict) else out)
                            if t is not None and t.dim() == 3)  # weight gradients
                row[which + "_peak_bytes_per_token"] = round(max(fwd_peak, peak - grads) / T, 1)
                del out
            torch.cuda.empty_cache()
            y, saved = layer.forward(x, wg, None, w1, w3, w2, k, False, act=act, h_on_load=hol)
            row["ours_saved_bytes_per_token"] = round(saved.nbytes() / T, 1)
            del y, saved
            row["base_saved_bytes_per_token"] = round(
                materialised_saved_bytes(x, wg, None, w1, w3, w2, k, False, act) / T, 1)
            row["speedup"] = round(row["base_ms"] / row["ours_ms"], 3)
            row["saved_ratio"] = round(row["base_saved_bytes_per_token"] /
                                       row["ours_saved_bytes_per_token"], 3)
            row["ours_tokens_per_s"] = round(T / (row["ours_ms"] * 1e-3), 1)
            rows.append(row)
            print(json.dumps(row), flush=True)
            del x, dy, w1, w2, w3, wg
            torch.cuda.empty_cache()
    return rows


def memory_sweep(cfg, max_doublings, h_on_load=False, recompute=False, atomic_combine=None):
    """Peak activation bytes per token and the largest T that fits, for this
    path (one forward + backward) and for the materialised-permutation
    baseline (forward only: its saved tensors plus forward temporaries, a
    lower bound on its training peak). Inputs are drawn on the device from a
    seeded generator with the workload's distributions."""
    import torch
    from paper_2601_05296_amd import layer
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg.seed)
    d, f, E, k = cfg.d, cfg.f, cfg.E, cfg.k
    if atomic_combine is None:   # the layer's default
        atomic_combine = k <= 2
    bf = torch.bfloat16
    wg = (torch.randn((E, d), generator=gen, device=dev) * 0.02).to(bf)
    w1 = (torch.randn((E, d, f), generator=gen, device=dev) * d ** -0.5).to(bf)
    gated = cfg.act == "swiglu"
    w3 = (torch.randn((E, d, f), generator=gen, device=dev) * d ** -0.5).to(bf) if gated else None
    w2 = (torch.randn((E, f, d), generator=gen, device=dev) * f ** -0.5).to(bf)
    grad_bytes = 4 * ((3 if gated else 2) * E * d * f + E * d)
    rows = []
    ours_ok = base_ok = True
    for n in range(max_doublings + 1):
        T = cfg.T << n
        row = {"T": T}
        for which in ("ours", "baseline"):
            if (which == "ours" and not ours_ok) or (which == "baseline" and not base_ok):
                continue
            torch.cuda.empty_cache()
            try:
                x = torch.randn((T, d), generator=gen, device=dev).to(bf)
                dy = torch.randn((T, d), generator=gen, device=dev).to(bf) if which == "ours" else None
                torch.cuda.synchronize()
                torch.cuda.reset_peak_memory_stats(dev)
                base = torch.cuda.memory_allocated(dev)
                if which == "ours":
                    y, saved = layer.forward(x, wg, None, w1, w3, w2, k, cfg.renorm, act=cfg.act,
                                             h_on_load=h_on_load, recompute=recompute,
                                             atomic_combine=atomic_combine)
                    sb = saved.nbytes()
                    torch.cuda.synchronize()
                    fwd_peak = torch.cuda.max_memory_allocated(dev) - base
                    torch.cuda.reset_peak_memory_stats(dev)
                    g = layer.backward(saved, dy, x, wg, w1, w3, w2)
                    torch.cuda.synchronize()
                    peak = max(fwd_peak, torch.cuda.max_memory_allocated(dev) - base - grad_bytes)
                    del y, saved, g
                    row["ours_peak_bytes_per_token"] = round(peak / T, 1)
                    row["ours_saved_bytes_per_token"] = round(sb / T, 1)
                else:
                    sb = materialised_saved_bytes(x, wg, None, w1, w3, w2, k, cfg.renorm, cfg.act)
                    torch.cuda.synchronize()
                    peak = torch.cuda.max_memory_allocated(dev) - base
                    row["baseline_fwd_peak_bytes_per_token"] = round(peak / T, 1)
                    row["baseline_saved_bytes_per_token"] = round(sb / T, 1)
                del x, dy
            except torch.cuda.OutOfMemoryError:
                row[which + "_oom"] = True
                if which == "ours":
                    ours_ok = False
                else:
                    base_ok = False
            torch.cuda.empty_cache()
        rows.append(row)
        print(json.dumps(row), flush=True)
        if not ours_ok and not base_ok:
            break
    fits = lambda key: max([r["T"] for r in rows if key in r], default=0)
    return {"workload": cfg.name, "h_on_load": bool(h_on_load), "recompute": bool(recompute),
            "atomic_combine": bool(atomic_combine), "points": rows,
            "max_T_ours": fits("ours_peak_bytes_per_token"),
            "max_T_baseline_fwd": fits("baseline_fwd_peak_bytes_per_token"),
            "hbm_bytes": torch.cuda.get_device_properties(dev).total_memory}


def cpu_oracle_baseline(inp, cfg, budget_s):
    """Time the CPU oracle (fwd + bwd of the whole layer) on the first tokens
    of the same workload; the sample grows until about budget_s of work."""
    from oracle import oracle
    v = {n: (None if a is None else a.astype(np.float64)) for n, a in inp.vals.items()}

    def run(n):
        t0 = time.perf_counter()
        fw = oracle.layer_forward(v["x"][:n], v["w_gate"], v["bias"], v["w1"], v["w3"], v["w2"],
                                  cfg.k, cfg.renorm, act=cfg.act)
        oracle.layer_backward(fw, v["dy"][:n], v["x"][:n], v["w_gate"], v["w1"], v["w3"],
                              v["w2"], cfg.renorm)
        return time.perf_counter() - t0

    # two calibration runs fit time = a + b*n (a: the per-expert weight
    # gradient work, independent of n); the timed sample is sized for budget_s
    n0, n1 = 8, 32
    t0 = run(n0)
    t1 = run(n1)
    b = max((t1 - t0) / (n1 - n0), 1e-6)
    a = max(t0 - b * n0, 0.0)
    # the proportional estimate n1 * budget / t1 never overshoots (a >= 0); the
    # fit may, when the two runs differ by little more than noise: at most 2x
    n_prop = n1 * budget_s / max(t1, 1e-3)
    n = int(min(cfg.T, max(n1, min((budget_s - a) / b, 2.0 * n_prop))))
    t = run(n)
    cores = oracle.threads()
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": n / t, "unit": "tokens/s", "cores": cores, "kind": "oracle", "cpu": cpu,
            "sample": "first %d of %d tokens of %s, whole-layer fwd+bwd in fp64 "
                      "(%.1f s; calibration runs of %d and %d tokens, %.1f s, not counted)"
                      % (n, cfg.T, cfg.name, t, n0, n1, t0 + t1)}


def reference_rates(cfg, dev):
    """Two ceilings measured on this GPU beside the kernels, with events on the
    current stream, 5 timed calls after 2 untimed: a device-to-device copy of
    1 GiB (1 GiB read + 1 GiB written, the rate an HBM-bound gather-reduce can
    hope for), and hipBLASLt's dense bf16 GEMM (torch.matmul, contiguous
    operands) at one expert's even share of the first FFN product,
    [S/E x d] x [d x f], the rate a dense library GEMM of the same shape
    reaches. Neither is on the layer's path."""
    import torch

    def timed(fn, n=5):
        for _ in range(2):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n
    out = {}
    src = torch.empty(COPY_BYTES // 2, dtype=torch.bfloat16, device=dev)
    dst = torch.empty_like(src)
    ms = timed(lambda: dst.copy_(src))
    out["device_copy"] = {"bytes_read_plus_written": 2 * COPY_BYTES, "ms": round(ms, 4),
                          "GB_per_s": round(2 * COPY_BYTES / ms / 1e6, 1)}
    del src, dst
    m = max(256, (cfg.T * cfg.k // cfg.E) // 256 * 256)
    g = torch.Generator(device=dev).manual_seed(1)
    a = torch.randn((m, cfg.d), device=dev, generator=g).to(torch.bfloat16)
    b = torch.randn((cfg.d, cfg.f), device=dev, generator=g).to(torch.bfloat16)
    ms = timed(lambda: torch.matmul(a, b))
    out["hipblaslt_dense_bf16"] = {"M": m, "N": cfg.f, "K": cfg.d, "ms": round(ms, 4),
                                   "TFLOP_per_s": round(2.0 * m * cfg.d * cfg.f / ms / 1e9, 1)}
    del a, b
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1],
                      args.pmc_out or traffic_path(args.workload), args.workload,
                      " ".join(sys.argv))
        return
    if args.summarize_stats:
        summarize_stats(args.summarize_stats,
                        args.summary_out or os.path.join(ROOT, "profiles", "kernel_stats_%s.txt" % args.workload),
                        args.workload, " ".join(sys.argv), args.profile_command)
        return
    if args.summarize_table1:
        summarize_table1(args.summarize_table1,
                         args.summary_out or os.path.join(ROOT, "profiles", "table1_sweep.txt"),
                         " ".join(sys.argv), args.profile_command)
        return
    if args.summarize_sweep:
        summarize_sweep(args.summarize_sweep,
                        args.summary_out or os.path.join(ROOT, "profiles", "memory_sweep_mem_sweep_e64k8.txt"),
                        " ".join(sys.argv), args.profile_command)
        return
    if args.summarize_lds:
        summarize_lds(args.summarize_lds,
                      args.summary_out or os.path.join(ROOT, "profiles", "lds_bank_conflicts_%s.txt" % args.workload),
                      args.workload, " ".join(sys.argv), args.profile_command)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters[0], args.summarize_counters[1],
                           args.summary_out or os.path.join(ROOT, "profiles", "l2_requests_mfma_%s.txt" % args.workload),
                           args.workload, " ".join(sys.argv), args.profile_command)
        return
    if args.table1:
        print(json.dumps({"table1": table1_sweep(args)}), flush=True)
        return
    if args.sweep:
        from paper_2601_05296_amd import synth
        res = memory_sweep(synth.CONFIGS[args.workload], args.sweep_max_doublings,
                           h_on_load=args.h_on_load, recompute=args.recompute,
                           atomic_combine=args.atomic_combine)
        print(json.dumps({"sweep": res}), flush=True)
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the MoE layer here has no multi-GPU path "
              "(expert or data parallelism is not implemented); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2601_05296_amd import binding as B
    from paper_2601_05296_amd import layer, synth

    cfg = synth.CONFIGS[args.workload]
    if args.act:
        cfg = cfg.with_(act=args.act)
    assert cfg.dtype == "bf16", "the benchmark workloads are bf16"
    elem = 2
    dev = torch.device("cuda:0")
    inp = synth.make_inputs(cfg)

    def up(a):
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    x, wg, w1, w3, w2, dy = (up(inp.store[n]) for n in ("x", "w_gate", "w1", "w3", "w2", "dy"))
    bias = up(inp.store["bias"])
    T, d, f, E, k = cfg.T, cfg.d, cfg.f, cfg.E, cfg.k

    atomic = args.atomic_combine if args.atomic_combine is not None else k <= 2

    def step():
        y, saved = layer.forward(x, wg, bias, w1, w3, w2, k, cfg.renorm, act=cfg.act,
                                 recompute=args.recompute, h_on_load=args.h_on_load,
                                 atomic_combine=atomic)
        g = layer.backward(saved, dy, x, wg, w1, w3, w2)
        return y, saved, g

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # peak activation bytes of one step (weights, inputs and weight gradients
    # excluded): the forward's peak and the backward's, the larger one counts
    torch.cuda.reset_peak_memory_stats(dev)
    base = torch.cuda.memory_allocated(dev)
    y, saved = layer.forward(x, wg, bias, w1, w3, w2, k, cfg.renorm, act=cfg.act,
                             recompute=args.recompute, h_on_load=args.h_on_load,
                             atomic_combine=atomic)
    torch.cuda.synchronize()
    fwd_peak = torch.cuda.max_memory_allocated(dev) - base
    saved_bytes = saved.nbytes()   # before the backward (which may recompute A, B into it)
    torch.cuda.reset_peak_memory_stats(dev)
    g = layer.backward(saved, dy, x, wg, w1, w3, w2)
    torch.cuda.synchronize()
    grad_bytes = sum(g[n].numel() * 4 for n in ("dw1", "dw3", "dw2", "dw_gate") if g[n] is not None)
    bwd_peak = torch.cuda.max_memory_allocated(dev) - base - grad_bytes
    peak = max(fwd_peak, bwd_peak)
    formula = layer.saved_bytes_per_token(d, f, E, k, elem, T, cfg.act, args.recompute) * T
    assert abs(saved_bytes - formula) < 1, (saved_bytes, formula)
    del y, saved, g

    # records per step (one event per kernel launch and one per entry point),
    # counted on one untimed step with room to spare
    B.moe_probe_enable(4096)
    step()
    torch.cuda.synchronize()
    per_step_records = B.moe_probe_count() + 16
    assert B.moe_probe_dropped() == 0, "probe pool too small for one step"
    B.moe_probe_disable()

    # timed region: K whole steps, per-kernel events recorded on the stream
    B.moe_probe_enable(2 * per_step_records * args.steps + 64)
    bounds = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    bounds[0].record()
    for i in range(args.steps):
        step()
        bounds[i + 1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    step_ms = [bounds[i].elapsed_time(bounds[i + 1]) for i in range(args.steps)]
    dropped = B.moe_probe_dropped()
    recs = [B.moe_probe_get(i) for i in range(B.moe_probe_count())]
    B.moe_probe_disable()
    if dropped:
        raise RuntimeError("timing probe dropped %d records; per-kernel rates would be wrong"
                           % dropped)
    ms_step = (t1 - t0) * 1e3 / args.steps
    tokens_per_s = T * args.steps / (t1 - t0)

    kern = {}
    for name, ms in recs:
        kern.setdefault(name, []).append(ms)
    kernels = {}
    for name, lst in kern.items():
        avg = float(np.mean(lst))
        per_step_ms = float(np.sum(lst)) / args.steps
        if len(lst) % args.steps:
            raise RuntimeError("%s: %d launches over %d steps is not a whole number per step"
                               % (name, len(lst), args.steps))
        launches = len(lst) // args.steps
        amount, unit, bound = kernel_model(name, cfg, elem, args.recompute)
        # work of all the step's launches over their total time = the
        # per-launch work over the average launch
        rate = amount / (per_step_ms * 1e-3) / (1e12 if unit == "TFLOP/s" else 1e9) if amount else None
        peak_ = PEAK_BF16_TFLOPS if unit == "TFLOP/s" else PEAK_HBM_GBS
        kernels[name] = {"avg_ms": round(avg, 4), "launches_per_step": launches,
                         "ms_per_step": round(per_step_ms, 4),
                         "per_launch": amount / launches,
                         "bound": bound, "achieved": None if rate is None else round(rate, 1),
                         "unit": unit, "frac": None if rate is None else round(rate / peak_, 4)}
    dom = max(kernels, key=lambda n: kernels[n]["ms_per_step"])
    kd = kernels[dom]
    unit, bound = kd["unit"], kd["bound"]
    roofline = {"bound": bound, "achieved": kd["achieved"], "unit": unit,
                "peak": PEAK_BF16_TFLOPS if unit == "TFLOP/s" else PEAK_HBM_GBS,
                "frac": kd["frac"], "traffic": read_traffic(cfg.name, dom), "kernel": dom,
                "per_launch": kd["per_launch"], "avg_ms": kd["avg_ms"],
                "launches_per_step": kd["launches_per_step"]}
    gemm_ms = sum(kernels[n]["ms_per_step"] for n in kernels if n.startswith("g") and n[1].isdigit())
    # per-stage kernel time (ms per step); the router's two stages are the part
    # a sparse-to-sparse timing leaves out
    stage_of = {"route": ("route_",), "build": ("tile_",), "ffn_fwd": ("g1_", "g2_", "g2h_", "f32_g1", "f32_g2"),
                "combine": ("combine", "zero_", "fwd_slot_gates"), "ffn_bwd": ("g3_", "g3h_", "g4_", "g5_", "g6_", "dgate", "slot_gates", "expert_ranks", "f32_g3",
                                                      "f32_g4", "f32_g5", "f32_g6"),
                "route_bwd": ("rb_",)}
    stages = {st: round(sum(v["ms_per_step"] for n, v in kernels.items()
                            if any(n.startswith(p) for p in pre)), 4)
              for st, pre in stage_of.items()}
    router_ms = stages["route"] + stages["route_bwd"]
    gemm_flops = (18.0 if cfg.act == "swiglu" else 12.0) * T * k * d * f
    if args.recompute:   # the first layer runs again in the backward
        gemm_flops += (4.0 if cfg.act == "swiglu" else 2.0) * T * k * d * f
    out = {
        "metric": "MoE layer fwd+bwd tokens/sec + peak activation bytes/token, 1 MI355X",
        "value": round(tokens_per_s, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        # per-step device times from events between the steps (the mean above is
        # the host clock over the whole timed region)
        "ms_per_step_median": round(float(np.median(step_ms)), 4),
        "ms_per_step_min_max": [round(min(step_ms), 4), round(max(step_ms), 4)],
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": cfg.name, "T": T, "d": d, "f": f, "E": E, "k": k,
                   "renorm": cfg.renorm, "zipf_s": cfg.zipf_s, "act": cfg.act,
                   "checkpoint": "recompute" if args.recompute else "A,B",
                   "h_on_load": bool(args.h_on_load),
                   "combine": "atomic" if atomic else "strips",
                   "parallelism": "none"},
        "peak_activation_bytes_per_token": round(peak / T, 1),
        "peak_activation_bytes_per_token_fwd_bwd": [round(fwd_peak / T, 1), round(bwd_peak / T, 1)],
        "saved_activation_bytes_per_token": round(saved_bytes / T, 1),
        "roofline": roofline,
        "gemm": {"ms_per_step": round(gemm_ms, 4),
                 "tflops": round(gemm_flops / (gemm_ms * 1e-3) / 1e12, 1),
                 "frac": round(gemm_flops / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)},
        "stages_ms": stages,
        "dispatch_us": {"route_plus_build": round((stages["route"] + stages["build"]) * 1e3, 1),
                        "build": round(stages["build"] * 1e3, 1)},
        "sparse_to_sparse_tokens_per_s": round(T / ((ms_step - router_ms) * 1e-3), 1),
        "kernels": kernels,
    }
    # the same steps with the 256 MB MALL evicted before each one (a 1 GiB
    # scratch fill between steps, outside the events that time the step)
    scratch = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    fl = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        scratch.fill_(i & 0x7F)
        fl[i][0].record()
        step()
        fl[i][1].record()
    torch.cuda.synchronize()
    del scratch
    flushed = [a.elapsed_time(b) for a, b in fl]
    out["mall_flushed"] = {"steps": args.steps,
                           "ms_per_step_median": round(float(np.median(flushed)), 4),
                           "ms_per_step_min_max": [round(min(flushed), 4), round(max(flushed), 4)]}
    if args.graph:
        # the same step captured once in a HIP graph (every entry point is
        # capturable: no allocation, memset or synchronisation inside), then
        # replayed: the launch overhead the eager step pays is the difference
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        graph.replay()
        torch.cuda.synchronize()
        g0 = time.perf_counter()
        for _ in range(args.steps):
            graph.replay()
        torch.cuda.synchronize()
        g1 = time.perf_counter()
        del graph
        out["graph_replay"] = {"steps": args.steps,
                               "ms_per_step": round((g1 - g0) * 1e3 / args.steps, 4),
                               "tokens_per_s": round(T * args.steps / (g1 - g0), 1)}
    if not (args.recompute or args.no_baseline_memory):
        # the other operating point of the same layer: the other h policy
        # (bit-identical results; buffering h and g*h costs memory, forming
        # them on load costs vector work)
        other = not args.h_on_load
        def lean_step():
            y_, s_ = layer.forward(x, wg, bias, w1, w3, w2, k, cfg.renorm, act=cfg.act,
                                   h_on_load=other, atomic_combine=atomic)
            return y_, s_, layer.backward(s_, dy, x, wg, w1, w3, w2)
        lean_step()
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats(dev)
        b0 = torch.cuda.memory_allocated(dev)
        y_, s_ = layer.forward(x, wg, bias, w1, w3, w2, k, cfg.renorm, act=cfg.act, h_on_load=other,
                               atomic_combine=atomic)
        torch.cuda.synchronize()
        lf = torch.cuda.max_memory_allocated(dev) - b0
        torch.cuda.reset_peak_memory_stats(dev)
        g_ = layer.backward(s_, dy, x, wg, w1, w3, w2)
        torch.cuda.synchronize()
        lb = torch.cuda.max_memory_allocated(dev) - b0 - grad_bytes
        del y_, s_, g_
        n_lean = max(3, args.steps // 2)
        t2 = time.perf_counter()
        for _ in range(n_lean):
            lean_step()
        torch.cuda.synchronize()
        t3 = time.perf_counter()
        out["h_buffered_policy" if other is False else "h_on_load_policy"] = {
            "checkpoint": ("A,B; h and g*h formed on load (MOE_H_ON_LOAD)" if other else
                           "A,B; h and g*h passed through transient buffers"),
            "steps": n_lean, "ms_per_step": round((t3 - t2) * 1e3 / n_lean, 4),
            "tokens_per_s": round(T * n_lean / (t3 - t2), 1),
            "peak_activation_bytes_per_token": round(max(lf, lb) / T, 1),
            "peak_activation_bytes_per_token_fwd_bwd": [round(lf / T, 1), round(lb / T, 1)]}
    if not args.no_reference_rates:
        out["reference_rates"] = reference_rates(cfg, dev)
    if args.copy_calibration:
        src = torch.empty(COPY_BYTES // 2, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_baseline_memory:
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats(dev)
        base = torch.cuda.memory_allocated(dev)
        mb = materialised_saved_bytes(x, wg, bias, w1, w3, w2, k, cfg.renorm, cfg.act)
        torch.cuda.synchronize()
        out["materialised_baseline_saved_bytes_per_token"] = round(mb / T, 1)
        out["materialised_baseline_fwd_peak_bytes_per_token"] = round(
            (torch.cuda.max_memory_allocated(dev) - base) / T, 1)
        torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_oracle_baseline(inp, cfg, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
