"""Benchmark: layer-wise broadcast GNN inference on one MI355X.

Default workload (the largest configuration one GPU holds in core):
sage3-fanout-rmat-100m -- 3-layer GraphSAGE-mean, fanout-sampled (15, 10, 5)
by hash rank, on an RMAT(0.57, 0.19, 0.19) graph with 100,000,000 vertices
and 1,600,000,000 edges; N(0,1) bf16 features of width 128 with fp32
accumulation; layer widths 128 -> 256 -> 256 -> 172; 65,536-vertex source
chunks.  Inputs (edge list, features) are seeded synthetic data, generated on
the host and resident in HBM before any timed region.

One step = the whole hot path once: the CSR build from the edge list, then
per layer the in-edge lists (first layer) and the fanout sampler, layer init
(pending counts, the chunk index of the kept edges, weights), every chunk
push (MFMA transform, scatter-aggregate with arrival counters, self messages
and the fused finalise) and finalize, each layer's output feeding the next.
The CSR build and the layers are timed in two loops of K repetitions each
(the edge list is freed after the first loop: with it resident, the three
layers' buffers do not fit in HBM), and a step's time is their sum.

Output: one JSON line.  value = aggregated edges per second per layer (the
propagated edges of all layers / step time) in GTEPS.  roofline = the
scatter kernel's algorithmic HBM bytes over its HIP-event-timed launches,
against 8 TB/s.  gemm_roofline = the transform's flops over its
HIP-event-timed launches (a separate untimed pass), against
min(bf16 MFMA peak, arithmetic intensity x HBM bandwidth).  cpu_baseline =
the CPU oracle on a bounded sample: its in-lists and sampler over the whole
graph, and the layer maths for 65,536 seeded destinations plus the 256
largest in-degrees and up to 256 without in-edges per layer, each layer fed
the GPU's previous layer; the same sample checks the GPU's outputs.

--workload gcn2-rmat-1m (with --variant) runs the 1M-vertex in-memory
workloads instead (2-layer GCN / GIN / GAT, exact or sampled).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "aggregated edges/sec per layer (GTEPS) + % HBM/host-link roofline, 1 GPU"
HBM_PEAK_GBS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3
BF16_MFMA_PEAK_TFLOPS = 2500.0


# Model variants on the same graph and features: (family, fanouts per layer,
# description).  Sampled layers keep min(d_in(v), k) in-edges per destination.
VARIANTS = {
    "gcn": (1, (), "2-layer GCN 128->128->64 (symmetric norm, self loops), exact"),
    "gcn-sampled": (1, (10, 5), "2-layer GCN 128->128->64, fanouts (10, 5), norms of the sampled graph"),
    "gin": (2, (), "2-layer GIN 128->128->64 (linear apply, eps = 0), exact"),
    "gin-sampled": (2, (10, 5), "2-layer GIN 128->128->64, fanouts (10, 5)"),
    "gat": (3, (), "2-layer single-head GAT 128->128->64 (LeakyReLU 0.2), exact: transform, softmax statistics "
                   "and aggregation passes"),
    "gat-sampled": (3, (10, 5), "2-layer single-head GAT 128->128->64, fanouts (10, 5)"),
    "gin-mlp": (4, (), "2-layer GIN 128->128->64 with a two-layer perceptron apply (hidden = output width, "
                       "eps = 0), exact: W1 before aggregation, ReLU(+b1) at completion, W2 on each chunk's "
                       "completed rows"),
    "gin-mlp-sampled": (4, (10, 5), "2-layer GIN with perceptron apply, fanouts (10, 5)"),
}


# A segment's slots are its messages plus, for the segment from the
# destination's own chunk, the self message.  Segments of at most SHORT_LEN
# slots are short units; longer ones are cut into pieces of at most PIECE_LEN
# slots, and a segment cut into several is completed by the fix-up kernel.
# The library's work-unit counts are checked against the ones derived here.
PIECE_LEN = 512
SHORT_LEN = 16


def flush_model(src, dst, n: int, chunk: int) -> dict:
    """Flush structure of one exact layer, from the graph alone.

    A segment is the run of messages from one source chunk to one
    destination; a destination's segment from its own chunk also carries its
    self message, and a destination without one flushes its self message
    alone when its own chunk is pushed.  With chunks pushed in ascending
    order, v's first flush is in chunk min(first message chunk, own chunk)
    (no accumulator read) and its last in max(last message chunk, own
    chunk) (output row written instead of the accumulator)."""
    import numpy as np
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    key = (src // chunk) * n + dst
    seg, lens = np.unique(key, return_counts=True)
    ch, v = seg // n, seg % n
    cv = v // chunk
    minch = np.full(n, np.iinfo(np.int64).max, dtype=np.int64)
    maxch = np.full(n, -1, dtype=np.int64)
    np.minimum.at(minch, v, ch)
    np.maximum.at(maxch, v, ch)
    own_v = np.arange(n, dtype=np.int64) // chunk
    first = np.minimum(minch, own_v)
    last = np.maximum(maxch, own_v)
    fresh = ch == first[v]
    final = ch == last[v]
    slots = lens + (ch == cv)
    split = slots > PIECE_LEN
    pieces = np.where(slots > SHORT_LEN, (slots + PIECE_LEN - 1) // PIECE_LEN, 1)
    has_own = np.zeros(n, dtype=bool)
    has_own[v[ch == cv]] = True
    alone = ~has_own                      # vertices flushing their self message alone
    return {
        "messages": int(src.size), "segments": int(seg.size), "units": int(pieces.sum()),
        "short_units": int((slots <= SHORT_LEN).sum()), "split_segments": int(split.sum()),
        "active_src": int(np.unique(src).size), "own_segments": int(has_own.sum()),
        "sc_flush": int((~split).sum()), "sc_fresh": int((~split & fresh).sum()),
        "sc_final": int((~split & final).sum()), "split_pieces": int(pieces[split].sum()),
        "fx_fresh": int((split & fresh).sum()), "fx_final": int((split & final).sum()),
        "alone": int(alone.sum()), "alone_fresh": int((alone & (own_v == first)).sum()),
        "alone_final": int((alone & (own_v == last)).sum()),
    }


def kernel_bytes(fm: dict, n: int, d_o: int, out_bytes: int, sage: bool) -> dict:
    """Algorithmic HBM bytes of each per-layer kernel (all its launches).

    flush: counts read 8 + written 4; the accumulator row read (4 d_o) unless
    the flush is v's first; the accumulator row written (4 d_o), or the output
    row (out_bytes d_o) for v's last flush.
    scatter: 16 per work unit, 4 per message (source code), the chunk
    transform's rows once -- every vertex's self row, and for GraphSAGE also
    the aggregation half of each source's row (4 d_o each) -- one flag byte
    per vertex for the self pass, the flushes it owns (segments that are not
    split, and vertices flushing their self message alone), and a hub piece's
    partial row and count (4 d_o + 4) to the carry buffer.
    fix-up: 16 per hub segment, its pieces' carries read back, one flush."""
    def flushes(k, fresh, final):
        return 12.0 * k + 4.0 * d_o * (k - fresh) + out_bytes * d_o * final + 4.0 * d_o * (k - final)
    y_rows = n + (fm["active_src"] if sage else 0)
    sc = (16.0 * fm["units"] + 4.0 * fm["messages"] + 4.0 * d_o * y_rows + 1.0 * n
          + flushes(fm["sc_flush"], fm["sc_fresh"], fm["sc_final"])
          + flushes(fm["alone"], fm["alone_fresh"], fm["alone_final"])
          + (4.0 * d_o + 4.0) * fm["split_pieces"])
    fx = (16.0 * fm["split_segments"] + (4.0 * d_o + 4.0) * fm["split_pieces"]
          + flushes(fm["split_segments"], fm["fx_fresh"], fm["fx_final"]))
    return {"scatter": sc, "fixup": fx}


# ---------------------------------------------------------------- profiles --
PROFILE_DIR = os.path.join(ROOT, "profiles")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2607_17374_amd", "csrc", "layer.hip")
GIB_KIB = float(1 << 20)
WORKLOADS = ("sage3-fanout-rmat-100m", "gcn2-rmat-1m", "sage2-ooc-rmat-269m", "gcn2-skew-rmat-50m")
LINK_PEAK_GBS = 64.0      # PCIe Gen5 x16, per direction


def profile_path(workload: str) -> str:
    return os.path.join(PROFILE_DIR, f"k_scatter_{workload}.md")


def profile_commands(workload: str) -> list:
    """The commands whose output a workload's profile summary digests, run
    from the repository root (counter runs profile the scatter, the
    transform and the calibration copy only)."""
    tag = "c3" if workload == WORKLOADS[0] else "c2"
    base = "python3 bench.py" + ("" if workload == WORKLOADS[0] else f" --workload {workload}")
    timed = " --steps 3 --warmup 1" if workload == WORKLOADS[0] else " --steps 10 --warmup 2"
    once = " --steps 1 --warmup 0 --no-cpu-baseline --no-profile --copy-calibration"
    sel = '--kernel-include-regex "k_scatter|k_gemm_panel|k_transform_fixup|neg"'
    mfma = ("SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_VALU_MFMA_BUSY_CYCLES "
            "SQ_BUSY_CU_CYCLES GRBM_GUI_ACTIVE")
    return [
        f"rocprofv3 --kernel-trace --stats --output-format csv -d gpurun_out/prof_{tag} -o {tag} -- "
        f"{base}{timed} --no-cpu-baseline",
        f"rocprofv3 --pmc FETCH_SIZE {sel} --output-format csv -d gpurun_out/pmc_fetch_{tag} -o p -- {base}{once}",
        f"rocprofv3 --pmc WRITE_SIZE {sel} --output-format csv -d gpurun_out/pmc_write_{tag} -o p -- {base}{once}",
        f"rocprofv3 --pmc {mfma} {sel} --output-format csv -d gpurun_out/pmc_mfma_{tag} -o p -- {base}{once}",
        f"python3 bench.py --summarize-profile {workload} gpurun_out/prof_{tag} gpurun_out/pmc_fetch_{tag} "
        f"gpurun_out/pmc_write_{tag} gpurun_out/pmc_mfma_{tag}",
    ]


# the scatter kernels and their launch dispatch: the part of KERNEL_SOURCE
# between these two section lines, plus the device helpers they include
SCATTER_BEGIN = "// ---------------------------------------------------------- scatter kernels --"
SCATTER_END = "// ------------------------------------------------------------- chunk index --"
DEVICE_HELPERS = os.path.join(ROOT, "paper_2607_17374_amd", "csrc", "device.hpp")


def source_digest() -> str:
    """sha256 of the code that decides what k_scatter does: its kernels and
    launch dispatch (the whole source file if the section lines are gone)
    and the device helpers header."""
    import hashlib
    text = open(KERNEL_SOURCE).read()
    a, b = text.find(SCATTER_BEGIN), text.find(SCATTER_END)
    region = text[a:b] if 0 <= a < b else text
    h = hashlib.sha256(region.encode())
    h.update(open(DEVICE_HELPERS, "rb").read())
    return h.hexdigest()


def profiled_traffic(workload: str):
    """HBM bytes per k_scatter launch from the workload's committed counter
    summary, or None when there is none or the kernel source changed since
    it was taken."""
    try:
        text = open(profile_path(workload)).read()
    except OSError:
        return None
    vals = dict(line.strip().split(": ", 1) for line in text.splitlines()
                if line.startswith("    ") and ": " in line and not line.strip().startswith(("rocprofv3", "python3")))
    if vals.get("source_sha256") != source_digest():
        return None
    try:
        return float(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _short_name(name: str) -> str:
    import re
    name = name.replace("(anonymous namespace)::", "")
    return re.sub(r"\(.*", "", name).replace("void ", "").strip()


def _counter_means(d: str, counter: str) -> dict:
    """kernel short name -> (dispatches, mean counter value per dispatch)."""
    import csv
    import glob
    acc = {}
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            k = _short_name(r["Kernel_Name"])
            n, t = acc.get(k, (0, 0.0))
            acc[k] = (n + 1, t + float(r["Counter_Value"]))
    return {k: (n, t / n) for k, (n, t) in acc.items()}


def _pick(d: dict, pred):
    """(dispatches, dispatch-weighted mean) over the kernels whose name passes pred."""
    ks = [k for k in d if pred(k)]
    n = sum(d[k][0] for k in ks)
    return n, (sum(d[k][0] * d[k][1] for k in ks) / n if n else float("nan"))


WORKLOAD_TITLE = {
    WORKLOADS[0]: "sage3-fanout-rmat-100m (3-layer GraphSAGE-mean 128->256->256->172, fanouts (15, 10, 5), "
                  "RMAT 100M vertices / 1.6B edges, bf16 features, 65,536-vertex chunks)",
    WORKLOADS[1]: "gcn2-rmat-1m (2-layer GCN 128->128->64, RMAT 1M vertices / 20M edges, fp32, "
                  "65,536-vertex chunks)",
}


OOC_PROFILE_SCALE = 16


def copy_profile_command() -> str:
    return ("rocprofv3 --memory-copy-trace --kernel-trace --stats --output-format csv -d gpurun_out/prof_c4 -o c4 -- "
            f"python3 bench.py --workload {WORKLOADS[2]} --scale {OOC_PROFILE_SCALE} --steps 2 --warmup 1 "
            "--no-cpu-baseline")


def summarize_copies(trace_dir: str) -> str:
    """Host-link summary of the out-of-core bench from a memory-copy trace:
    each layer's chunk copies run on that layer's own copy stream, so the
    streams in order of their first copy alternate layer 1, layer 2 (one
    pair per pass); each streams the layer's whole input once."""
    import csv
    import glob
    from fixtures import workloads as WL
    base = WL.SAGE_OOC_RMAT_269M
    n = base.n // OOC_PROFILE_SCALE
    tr = glob.glob(os.path.join(trace_dir, "**", "*memory_copy_trace.csv"), recursive=True)
    ks = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not tr or not ks:
        raise SystemExit(f"no memory-copy trace or kernel stats under {trace_dir}")
    rows = [r for r in csv.DictReader(open(tr[0])) if r["Direction"] == "MEMORY_COPY_HOST_TO_DEVICE"]
    by = {}
    for r in rows:
        by.setdefault(r["Stream_Id"], []).append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    copy_streams = sorted((v for k, v in by.items() if k != "0"), key=lambda v: min(a for a, _ in v))
    out = [f"# Host link on {WORKLOADS[2]} at 1/{OOC_PROFILE_SCALE} ({n:,} vertices, {base.e // OOC_PROFILE_SCALE:,} "
           "edges, 131,072-vertex chunks)", "",
           "Command, from the repository root on one MI355X:", "", "    " + copy_profile_command(),
           f"    python3 bench.py --summarize-copies gpurun_out/prof_c4", "",
           "Layer 1's chunks are filled by the library's loader (the seeded generator on host threads) and copied "
           "on layer 1's copy stream; layer 2 streams layer 1's output back from pinned host memory on its own "
           "copy stream.  Each stream carries its layer's whole input once (n x d_in x 4 bytes).  Engine rate = "
           "bytes / summed copy durations; effective rate = bytes / (first copy start to last copy end).  "
           "Nominal link: 64 GB/s per direction (PCIe Gen5 x16).", "",
           "| pass | layer | copies | GB | summed copy ms | engine GB/s | span ms | effective GB/s | of 64 GB/s |",
           "|---|---|---|---|---|---|---|---|---|"]
    for k, v in enumerate(copy_streams):
        layer = k % 2 + 1
        d_in = base.dims[layer - 1]
        gb = n * d_in * 4 / 1e9
        busy = sum(b - a for a, b in v) / 1e6
        span = (max(b for _, b in v) - min(a for a, _ in v)) / 1e6
        out.append(f"| {k // 2 + 1}{' (warm-up)' if k < 2 else ''} | {layer} | {len(v)} | {gb:.2f} | {busy:.1f} | "
                   f"{gb / busy * 1e3:.1f} | {span:.1f} | {gb / span * 1e3:.1f} | {gb / span * 1e3 / 64:.3f} |")
    cal = sorted(by.get("0", []), key=lambda t: t[1] - t[0], reverse=True)[:3]
    if cal:
        ms = sum(b - a for a, b in cal) / len(cal) / 1e6
        out += ["", f"Plain pinned copy of 4 GiB on the default stream (the bench's link calibration), mean of "
                    f"{len(cal)}: {ms:.1f} ms = {(4 << 30) / ms / 1e6:.1f} GB/s."]
    krow = list(csv.DictReader(open(ks[0])))
    out += ["", "## Kernel time (same run)", "", "| kernel | calls | total ms | average us |", "|---|---|---|---|"]
    for r in krow[:12]:
        out.append(f"| {_short_name(r['Name'])} | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.1f} | "
                   f"{float(r['AverageNs']) / 1e3:.1f} |")
    return "\n".join(out)


def c5_profile_command() -> str:
    return ("rocprofv3 --kernel-trace --stats --output-format csv -d gpurun_out/prof_c5 -o c5 -- "
            f"python3 bench.py --workload {WORKLOADS[3]} --steps 1 --warmup 1")


def summarize_reorder(trace_dir: str) -> str:
    """Kernel-time summary of the reordered skewed GCN bench: every
    kernel, and the Alg. 1 kernels (k_ta_*) and the degree/BFS kernels
    grouped."""
    import csv
    import glob
    ks = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not ks:
        raise SystemExit(f"no kernel stats under {trace_dir}")
    rows = list(csv.DictReader(open(ks[0])))
    out = [f"# Reordering kernels (Alg. 1, degree/BFS, RCMK) on {WORKLOADS[3]} (50M vertices, 1B edges, "
           "random IDs)", "",
           "Command, from the repository root on one MI355X:", "", "    " + c5_profile_command(),
           "    python3 bench.py --summarize-reorder gpurun_out/prof_c5", "",
           "The run makes two steps (one warm-up) of: CSR build, degree/BFS order, Alg. 1 from it (5 updates), "
           "relabel, both GCN layers; then each ordering once on its own (degree/BFS and RCMK, Alg. 1 from each "
           "with 5 updates), with the layers in each.  Alg. 1 therefore runs 4 times (20 updates), the degree/BFS "
           "order 3 times and RCMK once.", ""]
    ta = ("k_sum_short", "k_sum_piece", "k_sum_combine", "k_rank_short", "k_rank_piece", "k_rank_combine",
          "k_sum_terms", "k_ta_")
    groups = {"Alg. 1 kernels (sums, ranks, positions; its position sort is counted with the radix sorts)":
              lambda k: any(x in k for x in ta),
              "radix sorts (CSR builds, relabelling, Alg. 1's position sort, indexes)": lambda k: "k_radix" in k}
    out += ["| group | calls | total ms |", "|---|---|---|"]
    for g, pred in groups.items():
        sel = [r for r in rows if pred(r["Name"])]
        out.append(f"| {g} | {sum(int(r['Calls']) for r in sel)} | "
                   f"{sum(float(r['TotalDurationNs']) for r in sel) / 1e6:.1f} |")
    out += ["", "| kernel | calls | total ms | average us | % |", "|---|---|---|---|---|"]
    for r in rows[:40]:
        out.append(f"| {_short_name(r['Name'])} | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.2f} | "
                   f"{float(r['AverageNs']) / 1e3:.1f} | {float(r['Percentage']):.1f} |")
    return "\n".join(out)


def summarize_profile(workload: str, trace_dir: str, fetch_dir: str, write_dir: str, mfma_dir: str = None) -> str:
    import csv
    import glob
    stats = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not stats:
        raise SystemExit(f"no kernel_stats.csv under {trace_dir}")
    rows = list(csv.DictReader(open(stats[0])))
    out = [f"# k_scatter on {WORKLOAD_TITLE[workload]}", "",
           "Commands, from the repository root on one MI355X (counter runs one at a time):", ""]
    out += ["    " + c for c in profile_commands(workload)]
    out += ["", "## Kernel time (--kernel-trace --stats, every pass of the run)", "",
            "| kernel | calls | total ms | average us | % |", "|---|---|---|---|---|"]
    for r in rows[:20]:
        out.append(f"| {_short_name(r['Name'])} | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.3f} | "
                   f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['Percentage']):.1f} |")
    sc = [r for r in rows if "k_scatter<" in r["Name"]]
    calls = sum(int(r["Calls"]) for r in sc)
    tot_ns = sum(float(r["TotalDurationNs"]) for r in sc)
    fetch = _counter_means(fetch_dir, "FETCH_SIZE")
    write = _counter_means(write_dir, "WRITE_SIZE")
    _, f_cal = _pick(fetch, lambda k: "neg_kernel" in k)
    _, w_cal = _pick(write, lambda k: "neg_kernel" in k)
    nf, f_sc = _pick(fetch, lambda k: "k_scatter<" in k)
    nw, w_sc = _pick(write, lambda k: "k_scatter<" in k)
    ff, fw = GIB_KIB / f_cal, GIB_KIB / w_cal
    traffic = (f_sc * ff + w_sc * fw) * 1024.0
    out += ["", "## HBM traffic (--pmc, one counter per run)", "",
            f"Calibration: torch neg over 1 GiB (1,048,576 KiB read and written) reads FETCH_SIZE "
            f"{f_cal:.0f} KiB and WRITE_SIZE {w_cal:.0f} KiB per dispatch, so the factors are "
            f"{ff:.3f} (fetch) and {fw:.3f} (write).", "",
            f"k_scatter, mean over {nf} / {nw} dispatches (all layers): FETCH_SIZE {f_sc:.0f} KiB, "
            f"WRITE_SIZE {w_sc:.0f} KiB per dispatch; scaled: {traffic / 1e6:.1f} MB per launch."]
    gemm_pred = lambda k: "k_gemm_panel" in k or "k_transform_fixup" in k
    ng, f_g = _pick(fetch, gemm_pred)
    _, w_g = _pick(write, gemm_pred)
    if ng:
        out += ["", f"Transform (k_gemm_panel / k_transform_fixup), mean over {ng} dispatches: FETCH_SIZE "
                    f"{f_g:.0f} KiB, WRITE_SIZE {w_g:.0f} KiB per dispatch; scaled: "
                    f"{(f_g * ff + w_g * fw) * 1024.0 / 1e6:.1f} MB per launch."]
    if mfma_dir:
        gt = [r for r in rows if gemm_pred(r["Name"])]
        g_calls = sum(int(r["Calls"]) for r in gt)
        g_us = sum(float(r["TotalDurationNs"]) for r in gt) / max(g_calls, 1) / 1e3
        mops = {c: _pick(_counter_means(mfma_dir, c), gemm_pred) for c in
                ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_VALU_MFMA_MOPS_F32", "SQ_VALU_MFMA_BUSY_CYCLES",
                 "SQ_BUSY_CU_CYCLES", "GRBM_GUI_ACTIVE")}
        flops = 512.0 * sum(v[1] for k, v in mops.items() if "MOPS" in k and v[0])
        busy, cu_busy = mops["SQ_VALU_MFMA_BUSY_CYCLES"][1], mops["SQ_BUSY_CU_CYCLES"][1]
        out += ["", "## Matrix cores in the transform (--pmc)", "",
                f"Mean per dispatch over {mops['SQ_INSTS_VALU_MFMA_MOPS_BF16'][0]} dispatches:",
                "", "| counter | mean per dispatch |", "|---|---|"]
        out += [f"| {k} | {v[1]:.4g} |" for k, v in mops.items()]
        out += ["", f"MFMA work from the counters: 512 x MOPS = {flops / 1e9:.3f} GFLOP per dispatch; over the "
                    f"traced mean duration {g_us:.2f} us that is {flops / (g_us * 1e-6) / 1e12:.1f} TFLOP/s.  "
                    f"Matrix-core busy cycles over CU busy cycles: {busy / cu_busy:.3f}."]
    out += ["", "Machine-readable (bench.py reports traffic only while the kernel source digest matches):", "",
            "    kernel: k_scatter",
            f"    launches: {calls}",
            f"    avg_launch_us: {tot_ns / max(calls, 1) / 1e3:.2f}",
            f"    fetch_factor: {ff:.4f}",
            f"    write_factor: {fw:.4f}",
            f"    traffic_bytes_per_launch: {traffic:.0f}",
            f"    source_sha256: {source_digest()}"]
    return "\n".join(out)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default 3, or 10 for gcn2-rmat-1m)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps (default 1, or 2 for gcn2-rmat-1m)")
    ap.add_argument("--workload", choices=WORKLOADS, default=WORKLOADS[0])
    ap.add_argument("--scale", type=int, default=1,
                    help="divide vertices and edges by this: trial runs of sage3-fanout-rmat-100m (not a result); "
                         "sage2-ooc-rmat-269m needs 16 or more (its pinned host memory)")
    ap.add_argument("--chunk", type=int, default=0,
                    help="sage3-fanout-rmat-100m only: source chunk size (default: the workload's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--loader-threads", type=int, default=2,
                    help="sage2-ooc-rmat-269m: loader threads (each fill spreads a chunk over the host cores)")
    ap.add_argument("--no-profile", action="store_true", help="time without per-kernel events")
    ap.add_argument("--full-profile", action="store_true",
                    help="events around every kernel (adds the transform's MFMA roofline; more events in the stream)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 1 GiB device copy, the reference kernel for HBM byte counters")
    ap.add_argument("--variant", choices=sorted(VARIANTS), default="gcn",
                    help="gcn2-rmat-1m only: model family on the same graph (default: the exact GCN workload)")
    ap.add_argument("--summarize-profile", nargs="+", metavar="ARG",
                    help="WORKLOAD TRACE_DIR FETCH_DIR WRITE_DIR [MFMA_DIR]: print the profile summary of a "
                         "kernel-trace run and FETCH_SIZE / WRITE_SIZE (and matrix-core counter) runs")
    ap.add_argument("--summarize-copies", metavar="TRACE_DIR",
                    help="print the host-link summary of a memory-copy trace of the out-of-core bench")
    ap.add_argument("--summarize-reorder", metavar="TRACE_DIR",
                    help="print the kernel summary of a trace of the reordered skewed GCN bench")
    args = ap.parse_args()
    if args.summarize_reorder:
        print(summarize_reorder(args.summarize_reorder))
        return
    if args.summarize_copies:
        print(summarize_copies(args.summarize_copies))
        return
    if args.summarize_profile:
        if len(args.summarize_profile) not in (4, 5) or args.summarize_profile[0] not in WORKLOADS[:2]:
            raise SystemExit("--summarize-profile WORKLOAD TRACE_DIR FETCH_DIR WRITE_DIR [MFMA_DIR]")
        print(summarize_profile(*args.summarize_profile))
        return
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the path has no multi-GPU mode)", file=sys.stderr)
        sys.exit(2)
    if args.workload == "gcn2-rmat-1m":
        args.steps = 10 if args.steps is None else args.steps
        args.warmup = 2 if args.warmup is None else args.warmup
        return bench_rmat_1m(args)
    if args.workload == "gcn2-skew-rmat-50m":
        args.steps = 3 if args.steps is None else args.steps
        args.warmup = 1 if args.warmup is None else args.warmup
        return bench_c5(args)
    if args.workload == "sage2-ooc-rmat-269m":
        args.steps = 2 if args.steps is None else args.steps
        args.warmup = 1 if args.warmup is None else args.warmup
        if args.scale < 16:
            raise SystemExit("sage2-ooc-rmat-269m: --scale 16 or more (pinned host memory: at 1/16 both layers' "
                             "outputs and the store for evicted rows already take 43 GB)")
        return bench_ooc(args)
    args.steps = 3 if args.steps is None else args.steps
    args.warmup = 1 if args.warmup is None else args.warmup
    return bench_sage3_100m(args)


def bench_rmat_1m(args):
    import numpy as np
    import torch
    import fixtures as F
    from fixtures import workloads as WL
    import paper_2607_17374_amd as T
    from tests import harness as H

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    import dataclasses
    agg, fanouts, desc = VARIANTS[args.variant]
    w = dataclasses.replace(WL.GCN_RMAT_1M, agg=agg, fanouts=fanouts)
    sampled = bool(fanouts)
    src, dst = WL.graph(w)
    X = torch.from_numpy(WL.input_features(w)).to(dev)
    src_d = torch.from_numpy(src).to(dev)
    dst_d = torch.from_numpy(dst).to(dev)
    specs = H.layer_specs(w)
    outs = [torch.empty((w.n, s["d_out"]), dtype=torch.float32, device=dev) for s in specs]
    # HIP events around the scatter launches only (2), or every kernel (1)
    profile = 0 if args.no_profile else (1 if args.full_profile else 2)
    if args.copy_calibration:
        # a plain streaming kernel of known size for the byte counters:
        # neg reads 1 GiB and writes 1 GiB
        a = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        c = torch.empty_like(a)
        for _ in range(3):
            torch.neg(a, out=c)
        del a, c
    torch.cuda.synchronize()
    fm = flush_model(src, dst, w.n, w.chunk)
    setup = torch.cuda.Stream()

    def step(prof):
        t0 = time.perf_counter()
        row_off, col_dst = T.build_csr(w.n, src_d, dst_d)
        t_csr = time.perf_counter() - t0
        tp = time.perf_counter()
        plan = T.Plan(w.n, row_off, col_dst, w.chunk)
        t_plan = time.perf_counter() - tp
        h = X
        per = []

        def make(li):
            # a later layer is set up on a stream of its own, beside the
            # previous layer's queued chunks
            t = time.perf_counter()
            L = T.Layer(w.n, row_off, col_dst, out=outs[li], chunk=w.chunk, profile=prof, plan=plan,
                        setup_stream=setup if li > 0 else None, **specs[li])
            return L, time.perf_counter() - t

        L, t_init = make(0)
        for li in range(len(specs)):
            tl = time.perf_counter()
            L.push_all(h)
            # the next layer's set-up runs beside this layer's queued chunks
            nxt = make(li + 1) if li + 1 < len(specs) else None
            st = L.finalize()
            L.destroy()
            # push through finalize; the first layer also counts its set-up
            # (the chunk index), later layers' set-up falls inside the layer
            # before them
            st["wall_ms"] = (time.perf_counter() - tl + (t_init if li == 0 else 0.0)) * 1e3
            per.append(st)
            h = outs[li]
            if nxt:
                L, t_init = nxt
        plan.destroy()
        return t_csr * 1e3, t_plan * 1e3, per

    for _ in range(args.warmup):
        step(profile)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    # per-kernel events in the first timed step only: each event pair costs
    # about 6 us of the step
    runs = [step(profile if i == 0 else 0) for i in range(args.steps)]
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_step = elapsed * 1e3 / args.steps

    # per-layer figures, averaged over the timed steps
    nl = len(specs)
    layers = []
    tot = {"scatter": [0.0, 0.0, 0], "fixup": [0.0, 0.0, 0]}  # bytes, ms, launches
    gemm_flops = gemm_ms = 0.0
    model_ok = True
    for li in range(nl):
        sts = [r[2][li] for r in runs]
        d_o, d_in = specs[li]["d_out"], specs[li]["d_in"]
        ncols = d_o  # GCN and GIN transform width (GIN's perceptron: W1, then W2 at graduation)
        wall = float(np.mean([s["wall_ms"] for s in sts]))
        st = sts[-1]
        kb = kernel_bytes(fm, w.n, d_o, 4, sage=False)
        checks = (st["short_units"] == fm["short_units"], st["wave_units"] == fm["units"] - fm["short_units"],
                  st["split_segments"] == fm["split_segments"], st["pairs"] == fm["segments"] + fm["alone"],
                  st["messages"] == fm["messages"])
        if sampled:
            checks = ()      # the flush model describes exact layers only
        if not all(checks):
            model_ok = False
            print(f"warning: layer {li + 1} work counts differ from the flush model: {checks}", file=sys.stderr)
        prof = sts[:1] if profile else []  # the step with events
        timed = ("gemm", "scatter", "fixup")
        ms = {k: float(np.mean([s[f"ms_{k}"] for s in (prof if k in timed else sts)])) if (prof or k not in timed)
              else 0.0 for k in ("gemm", "scatter", "fixup", "init", "index")}
        # GAT aggregates in its own passes; GIN's perceptron writes a completed
        # row into its accumulator row instead of the output, the same bytes
        if prof and not sampled and agg != WL.GAT_ATT:
            for k in tot:
                tot[k][0] += kb[k] * len(prof)
                tot[k][1] += sum(s[f"ms_{k}"] for s in prof)
                tot[k][2] += sum(s[f"launches_{k}"] for s in prof)
        if prof:
            gemm_flops += 2.0 * w.n * d_in * ncols * len(prof)
            gemm_ms += sum(s["ms_gemm"] for s in prof)
        layers.append({
            "layer": li + 1, "d_in": d_in, "d_out": d_o, "edges": st["messages"], "pairs": st["pairs"],
            "wall_ms": round(wall, 3), "gteps": round(st["messages"] / (wall * 1e-3) / 1e9, 3),
            "vertices_per_s": round(w.n / (wall * 1e-3), 1),
            **{f"{k}_ms": round(v, 3) for k, v in ms.items()},
            "short_units": st["short_units"], "wave_units": st["wave_units"],
            "split_segments": st["split_segments"],
            **({} if sampled else {f"{k}_algorithmic_gb": round(kb[k] / 1e9, 4) for k in kb}),
            **({} if sampled else {f"{k}_gbs": (round(kb[k] / (ms[k] * 1e-3) / 1e9, 1) if ms[k] > 0 else None)
                                   for k in kb}),
        })
    csr_ms = float(np.mean([r[0] for r in runs]))
    plan_ms = float(np.mean([r[1] for r in runs]))
    total_edges = sum(l["edges"] for l in layers)
    value = total_edges / (ms_step * 1e-3) / 1e9

    roofline = None
    if profile and tot["scatter"][1] > 0:
        byt, ms_, nlaunch = tot["scatter"]
        achieved = byt / (ms_ * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": profiled_traffic("gcn2-rmat-1m"), "kernel": "k_scatter",
                    "avg_launch_us": round(ms_ * 1e3 / nlaunch, 2), "bytes_per_launch": round(byt / nlaunch, 0),
                    "model_check": model_ok}
    gemm = None
    if profile and gemm_ms > 0:
        tf = gemm_flops / (gemm_ms * 1e-3) / 1e12
        gemm = {"bound": "mfma", "achieved": round(tf, 2), "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tf / FP32_MFMA_PEAK_TFLOPS, 4), "kernel": "k_gemm_panel"}

    cpu = None
    if not args.no_cpu_baseline:
        import oracle as O
        t0 = time.perf_counter()
        g, zs = H.oracle_model(w, src, dst)
        t_or = time.perf_counter() - t0
        cpu = {"value": round(total_edges / t_or / 1e9, 5), "unit": "GTEPS", "cores": O.threads(),
               "kind": "oracle", "seconds": round(t_or, 2),
               "sample": "the full workload once: oracle CSR and in-lists, then both layers for all "
                         f"1,000,000 destinations in fp64 (value = both layers' {total_edges / 1e6:.1f}M "
                         "propagated edges / wall time)"}

    line = {
        "metric": METRIC, "value": round(value, 4), "unit": "GTEPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{'gcn2-rmat-1m' if args.variant == 'gcn' else 'rmat-1m-' + args.variant}: "
                               f"{desc}; "
                               "RMAT(0.57,0.19,0.19) 1,000,000 vertices / 20,000,000 edges; N(0,1) fp32 features; "
                               "65,536-vertex source chunks; step = CSR build + chunk index"
                               f"{' (sampled: per-layer in-edge lists and masks)' if sampled else ''} + both layers",
                   "n": w.n, "e": w.e, "chunk": w.chunk, "csr_ms": round(csr_ms, 3),
                   "plan_ms": round(plan_ms, 3)},
        "per_layer": layers,
        "roofline": roofline,
        "gemm_roofline": gemm,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def sampled_scatter_bytes(st: dict, n: int, d_o: int, out_bytes: int, sage: bool) -> float:
    """Algorithmic HBM bytes of one layer's scatter launches, from the
    library's statistics.  Per work unit 16 (its descriptor); per message 4
    (the source's row code); the chunk transform's rows once -- every
    vertex's self row and, for GraphSAGE, each source's aggregation row
    (4 d_o each); one flag byte per vertex (self pass); per flush 12 (counts
    read and written); the accumulator row read on every flush but a
    vertex's first and written on every flush but its last (a vertex's first
    and last flush are one each of its P flushes), and its output row once.
    In-core GraphSAGE layers take the self messages of the A vertices
    without a segment from their own chunk in the transform (A =
    self_in_transform, of which self_fresh found nothing accumulated and
    self_last completed the vertex, counted in a profiled run): the scatter
    then reads no self row for them and only updates their counts (12), and
    the transform_self_bytes of those flushes leave its total.
    Exact when no segment is split into pieces, which holds for fanouts up to
    15 (a segment then holds at most 15 messages and the self message)."""
    if st["split_segments"]:
        raise ValueError("the byte model holds for layers without split segments")
    P = st["pairs"]
    A = st.get("self_in_transform", 0)
    if A and min(st["self_fresh"], st["self_last"]) < 0:
        raise ValueError("the self-message counts are taken in profiled runs only")
    units = st["short_units"] + st["wave_units"]
    y_rows = n * (2 if sage else 1) - A
    return (16.0 * units + 4.0 * st["messages"] + 4.0 * d_o * y_rows + 1.0 * n + 12.0 * P
            + 8.0 * d_o * (P - n) + out_bytes * d_o * n - transform_self_bytes(st, d_o, out_bytes, counts=False))


def transform_self_bytes(st: dict, d_o: int, out_bytes: int, counts: bool = True) -> float:
    """Accumulator and output bytes of the self messages an in-core
    GraphSAGE layer's transform takes (none otherwise): each reads the row
    (4 d_o) unless it found nothing accumulated, and writes it (4 d_o) or,
    as the vertex's last arrival, the output row (out_bytes d_o); with
    counts, also each such vertex's flag byte and counts (9) that the
    transform reads."""
    A = st.get("self_in_transform", 0)
    if not A:
        return 0.0
    fresh, last = st["self_fresh"], st["self_last"]
    return (4.0 * d_o * (A - fresh) + 4.0 * d_o * (A - last) + out_bytes * d_o * last
            + (9.0 * A if counts else 0.0))


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def destination_sample(seed: int, deg_in, count: int = 65536):
    """count seeded uniform destinations, the 256 largest in-degrees (ties by
    lower ID) and up to 256 vertices without in-edges, sorted."""
    import numpy as np
    n = deg_in.size
    rng = np.random.default_rng(seed)
    uni = rng.choice(n, min(count, n), replace=False)
    cand = np.argpartition(-deg_in.astype(np.int64), 256)[:512] if n > 512 else np.arange(n)
    top = cand[np.lexsort((cand, -deg_in[cand].astype(np.int64)))][:256]
    zero = np.flatnonzero(deg_in == 0)[:256]
    return np.unique(np.concatenate([uni, top, zero]).astype(np.int64))


def bench_sage3_100m(args):
    import numpy as np
    import torch
    import fixtures as F
    from fixtures import workloads as WL
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import torch_dtype
    from tests import harness as H

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    t_start = time.perf_counter()

    def say(msg):
        print(f"[bench {time.perf_counter() - t_start:7.1f}s] {msg}", file=sys.stderr, flush=True)

    w = WL.SAGE_FANOUT_RMAT_100M
    if args.scale > 1:
        w = w.scaled(n=w.n // args.scale, e=w.e // args.scale)
    if args.chunk > 0:
        import dataclasses
        w = dataclasses.replace(w, chunk=args.chunk)
    specs = H.layer_specs(w)
    nl = len(specs)
    src, dst = WL.graph(w)
    say(f"{w.name}: edge list {src.size} edges")
    xh = WL.input_features(w)
    say("features")
    X = torch.from_numpy(xh.view(np.int16)).to(dev).view(torch_dtype(w.feat_dtype))
    src_d = torch.from_numpy(src).to(dev)
    dst_d = torch.from_numpy(dst).to(dev)
    # output buffers: layer 1 and layer 3 share one (layer 1's output is dead
    # once layer 2 has run), layer 2 has its own
    nbytes = [w.n * s["d_out"] * (4 if s["out_dtype"] == F.F32 else 2) for s in specs]
    buf_a = torch.empty(max(nbytes[0], nbytes[2]), dtype=torch.uint8, device=dev)
    buf_b = torch.empty(nbytes[1], dtype=torch.uint8, device=dev)

    if args.copy_calibration:
        # a plain streaming kernel of known size for the byte counters:
        # neg reads 1 GiB and writes 1 GiB
        ca = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        cb = torch.empty_like(ca)
        for _ in range(3):
            torch.neg(ca, out=cb)
        del ca, cb
        torch.cuda.synchronize()

    def out_view(li):
        buf = buf_b if li == 1 else buf_a
        dt = torch_dtype(specs[li]["out_dtype"])
        return buf[:nbytes[li]].view(dt).view(w.n, specs[li]["d_out"])

    # ---- a1: the CSR build, K timed builds while the edge list is resident
    for _ in range(args.warmup):
        row_off, col_dst = T.build_csr(w.n, src_d, dst_d)
        del row_off, col_dst
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        row_off, col_dst = T.build_csr(w.n, src_d, dst_d)
    torch.cuda.synchronize()
    csr_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    say(f"CSR build {csr_ms:.1f} ms")
    del src_d, dst_d
    torch.cuda.empty_cache()

    # ---- a3-a11: sampler and the three layers, K timed passes.  Each layer
    # is set up after the previous one is gone: setting it up beside the
    # previous layer's chunks (desc.setup_stream) holds two layers' indexes
    # and temporaries at once, which at this size runs the device out of
    # memory, so that the memory cache frees and re-allocates blocks of GBs
    # (about 150 ms each; measured 1.43 s a step against 0.84 s)
    def layers_pass(profile, hook=None):
        per = []
        plan = T.Plan(w.n, row_off, col_dst, w.chunk)
        h = X
        for li in range(nl):
            out = out_view(li)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            L = T.Layer(w.n, row_off, col_dst, out=out, chunk=w.chunk, profile=profile, plan=plan, **specs[li])
            L.push_all(h)
            st = L.finalize()
            torch.cuda.synchronize()
            st["wall_ms"] = (time.perf_counter() - t0) * 1e3
            if hook:
                hook(li, L, out)
            L.destroy()
            per.append(st)
            h = out
        plan.destroy()
        return per

    profile = 0 if args.no_profile else 2
    for _ in range(args.warmup):
        layers_pass(profile)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    # events around the scatter launches in the first timed pass only: each
    # event pair costs about 6 us of the step
    runs = [layers_pass(profile if i == 0 else 0) for i in range(args.steps)]
    torch.cuda.synchronize()
    layers_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    ms_step = csr_ms + layers_ms
    say(f"layers {layers_ms:.1f} ms per pass")

    layers = []
    sc_bytes = sc_ms = 0.0
    sc_launches = 0
    for li in range(nl):
        sts = [r[li] for r in runs]
        st = sts[-1]
        d_o, d_in = specs[li]["d_out"], specs[li]["d_in"]
        ob = 4 if specs[li]["out_dtype"] == F.F32 else 2
        wall = float(np.mean([x["wall_ms"] for x in sts]))
        prof = sts[:1] if profile else []  # the pass with events (and the self-message counts)
        kb = sampled_scatter_bytes(prof[0], w.n, d_o, ob, sage=True) if prof else None
        ms_sc = float(np.mean([x["ms_scatter"] for x in prof])) if prof else 0.0
        if prof:
            sc_bytes += kb * len(prof)
            sc_ms += sum(x["ms_scatter"] for x in prof)
            sc_launches += sum(x["launches_scatter"] for x in prof)
        layers.append({
            "layer": li + 1, "d_in": d_in, "d_out": d_o, "fanout": specs[li]["fanout"], "edges": st["messages"],
            "pairs": st["pairs"], "wall_ms": round(wall, 3), "gteps": round(st["messages"] / (wall * 1e-3) / 1e9, 4),
            "vertices_per_s": round(w.n / (wall * 1e-3), 1),
            "init_ms": round(float(np.mean([x["ms_init"] for x in sts])), 3),
            "sample_and_index_ms": round(float(np.mean([x["ms_index"] for x in sts])), 3),
            "scatter_ms": round(ms_sc, 3), "scatter_algorithmic_gb": round(kb / 1e9, 3) if kb else None,
            "scatter_gbs": round(kb / (ms_sc * 1e-3) / 1e9, 1) if ms_sc > 0 and kb else None,
            "self_in_transform": st["self_in_transform"],
            "short_units": st["short_units"], "wave_units": st["wave_units"],
        })
    total_edges = sum(l["edges"] for l in layers)
    value = total_edges / (ms_step * 1e-3) / 1e9
    roofline = None
    if profile and sc_ms > 0:
        achieved = sc_bytes / (sc_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": None if args.scale > 1 or args.chunk > 0 else profiled_traffic(w.name),
                    "kernel": "k_scatter",
                    "avg_launch_us": round(sc_ms * 1e3 / sc_launches, 2),
                    "bytes_per_launch": round(sc_bytes / sc_launches, 0)}

    # ---- untimed pass with events around every kernel (transform figures),
    # copying out the rows the oracle sample reads
    cpu = check = None
    gemm = None
    need_rows = {}
    got_rows = {}
    ids = keeps = g = None
    t_or = {}
    if not args.no_cpu_baseline:
        import oracle as O
        t0 = time.perf_counter()
        g = O.EdgeGraph(w.n, src, dst)
        t_or["in_lists"] = time.perf_counter() - t0
        say(f"oracle in-lists {t_or['in_lists']:.1f} s")
        ids, keeps, kept_in_sample = [], [], []
        for li in range(1, nl + 1):
            t0 = time.perf_counter()
            _, keep_in, m = O.sample(g, w.seed, li, w.fanout(li))
            t_or[f"sample_{li}"] = time.perf_counter() - t0
            keeps.append(keep_in)
            ids.append(destination_sample(w.seed * 1000 + li, g.deg_in))
            kept_in_sample.append(int(m[ids[-1]].sum()))
            # rows of layer li's input the oracle reads: the destinations and their kept in-neighbours
            need_rows[li] = np.unique(np.concatenate([ids[-1], H.in_neighbours(g, ids[-1], keep_in)]))
            say(f"oracle sampler layer {li}: {t_or[f'sample_{li}']:.1f} s, {len(need_rows[li])} input rows needed")

    def hook(li, L, out):
        if need_rows:
            if li + 1 < nl:
                got_rows[("in", li + 2)] = out.index_select(0, torch.from_numpy(need_rows[li + 2]).to(dev)).cpu()
            got_rows[("out", li + 1)] = out.index_select(0, torch.from_numpy(ids[li]).to(dev)).cpu()

    per = layers_pass(1, hook) if (need_rows or not args.no_profile) else []
    gf = gb = gms = 0.0
    for li, st in enumerate(per):
        d_in, d_o = specs[li]["d_in"], specs[li]["d_out"]
        gf += 2.0 * w.n * d_in * 2 * d_o
        # bf16 rows in, fp32 transform rows out (the self half only for the
        # vertices whose self message is a segment slot), and the self
        # messages the transform takes
        A = st["self_in_transform"]
        ob = 4 if specs[li]["out_dtype"] == F.F32 else 2
        gb += w.n * d_in * 2.0 + (2 * w.n - A) * d_o * 4.0 + transform_self_bytes(st, d_o, ob)
        gms += st["ms_gemm"]
        layers[li]["gemm_ms"] = round(st["ms_gemm"], 3)
    if gms > 0:
        tf = gf / (gms * 1e-3) / 1e12
        ai = gf / gb
        cap = min(BF16_MFMA_PEAK_TFLOPS, ai * HBM_PEAK_GBS / 1e3)
        gemm = {"bound": "mfma" if cap >= BF16_MFMA_PEAK_TFLOPS else "hbm", "achieved": round(tf, 2),
                "peak": round(cap, 1), "unit": "TFLOP/s", "frac": round(tf / cap, 4),
                "mfma_peak": BF16_MFMA_PEAK_TFLOPS, "ai_flop_per_byte": round(ai, 1),
                "achieved_gbs": round(gb / (gms * 1e-3) / 1e9, 1), "kernel": "k_gemm_panel (bf16)",
                "note": "untimed pass with events around every kernel"}

    if need_rows:
        import oracle as O
        zs_cmp = []
        t_layer = {}
        for li in range(1, nl + 1):
            p = WL.layer_params(w, li)
            in_dt, out_dt = w.layer_dtypes(li)
            if li == 1:
                Hin = xh
            else:
                rows = got_rows[("in", li)]
                Hin = np.zeros((w.n, rows.shape[1]), np.uint16 if in_dt != F.F32 else np.float32)
                Hin[need_rows[li]] = rows.view(torch.int16).numpy().view(np.uint16) if in_dt != F.F32 else rows.numpy()
            t0 = time.perf_counter()
            z = O.layer(w.agg, g, Hin, in_dt, p.W, p.b, li < nl, keep_in=keeps[li - 1], dst_ids=ids[li - 1])
            t_layer[li] = time.perf_counter() - t0
            y = H.to_numpy_f64(got_rows[("out", li)], out_dt)
            r = H.compare(y, z, H.RTOL[w.feat_dtype])
            zs_cmp.append({"layer": li, "destinations": int(len(ids[li - 1])), "mismatches": r["n_bad"],
                           "max_abs": r["max_abs"], "mean_rel": r["mean_rel"]})
            say(f"oracle layer {li}: {t_layer[li]:.2f} s, mismatches {r['n_bad']} of {len(ids[li - 1])}")
            del Hin
        check = zs_cmp
        t_sample_work = t_or["in_lists"] + sum(t_or[f"sample_{li}"] for li in range(1, nl + 1))
        t_layers_sample = sum(t_layer.values())
        t_extrap = t_sample_work + sum(t_layer[li] * w.n / len(ids[li - 1]) for li in range(1, nl + 1))
        cpu = {"value": round(total_edges / t_extrap / 1e9, 6), "unit": "GTEPS", "cores": O.threads(),
               "kind": "oracle", "cpu_model": _cpu_model(), "seconds": round(t_sample_work + t_layers_sample, 2),
               "extrapolated_full_step_s": round(t_extrap, 1),
               "sample": "in-lists and the fanout sampler of all three layers over the whole graph "
                         f"({t_sample_work:.1f} s), then the layer maths for 65,536 seeded destinations, the 256 "
                         "largest in-degrees and up to 256 without in-edges per layer, each fed the GPU's previous "
                         f"layer ({t_layers_sample:.2f} s); value = all layers' {total_edges / 1e6:.0f}M propagated "
                         "edges / the full step extrapolated linearly from the sampled destinations (extrapolated)"}

    line = {
        "metric": METRIC, "value": round(value, 4), "unit": "GTEPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{w.name}: 3-layer GraphSAGE-mean 128->256->256->172, fanouts (15, 10, 5) by "
                               "hash rank; RMAT(0.57,0.19,0.19) "
                               f"{w.n:,} vertices / {w.e:,} edges; N(0,1) bf16 features, fp32 accumulation; "
                               f"{w.chunk:,}-vertex source chunks; step = CSR build + per layer sampler, chunk "
                               "index and chunk pushes",
                   "n": w.n, "e": w.e, "chunk": w.chunk, "csr_ms": round(csr_ms, 3),
                   "layers_ms": round(layers_ms, 3), **({"scale": f"1/{args.scale}"} if args.scale > 1 else {})},
        "per_layer": layers,
        "roofline": roofline,
        "gemm_roofline": gemm,
        "cpu_baseline": cpu,
        "oracle_check": check,
    }
    print(json.dumps(line), flush=True)


def bench_c5(args):
    """gcn2-skew-rmat-50m: 2-layer GCN 256 -> 256 -> 64 (fp16 storage, fp32
    accumulation) on a skewed RMAT(0.65, 0.15, 0.15) graph with 50M vertices
    and 1B edges in random vertex IDs, reordered before the layers.  One
    step = CSR build + degree/BFS order + Alg. 1 (5 updates of the
    topology-aware order from it) + relabelling the graph and permuting the
    features + both layers in the new IDs.  Beside the step: each ordering
    (random IDs, degree/BFS, RCMK, Alg. 1 from either) timed on its own with
    the layers' time in that order, its total edge span C(pi) and
    dispersion J(pi)."""
    import numpy as np
    import torch
    from fixtures import workloads as WL
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import torch_dtype
    from tests import harness as H

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    t_start = time.perf_counter()

    def say(msg):
        print(f"[bench {time.perf_counter() - t_start:7.1f}s] {msg}", file=sys.stderr, flush=True)

    w = WL.GCN_SKEW_RMAT_50M
    if args.scale > 1:
        w = w.scaled(w.n // args.scale, w.e // args.scale)
    specs = H.layer_specs(w)
    src, dst = WL.graph(w)
    say(f"{w.name}: edge list {src.size} edges (random IDs)")
    xh = WL.input_features(w)
    X = torch.from_numpy(xh.view(np.int16)).to(dev).view(torch_dtype(w.feat_dtype))
    del xh
    src_d = torch.from_numpy(src).to(dev)
    dst_d = torch.from_numpy(dst).to(dev)
    del src, dst
    outs = [T.alloc_device((w.n, sp["d_out"]), torch_dtype(sp["out_dtype"]), dev) for sp in specs]

    def sync_ms(t0):
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3

    def layers(row_off, col_dst, x):
        t0 = time.perf_counter()
        plan = T.Plan(w.n, row_off, col_dst, w.chunk)
        h = x
        for li, sp in enumerate(specs):
            L = T.Layer(w.n, row_off, col_dst, out=outs[li], chunk=w.chunk, plan=plan, **sp)
            L.push_all(h)
            L.finalize()
            L.destroy()
            h = outs[li]
        plan.destroy()
        return sync_ms(t0)

    def step():
        t = {}
        t0 = time.perf_counter()
        row_off, col_dst = T.build_csr(w.n, src_d, dst_d)
        t["csr_ms"] = sync_ms(t0)
        t0 = time.perf_counter()
        pi0 = T.reorder(w.n, row_off, col_dst)
        t["bfs_ms"] = sync_ms(t0)
        t0 = time.perf_counter()
        ta = T.reorder_ta(w.n, row_off, col_dst, pi0, 5)
        t["alg1_ms"] = sync_ms(t0)
        t0 = time.perf_counter()
        r2, c2 = T.relabel_graph(w.n, row_off, col_dst, ta.pi)
        x2 = T.permute_rows(X, ta.pi)
        t["relabel_ms"] = sync_ms(t0)
        del row_off, col_dst
        t["layers_ms"] = layers(r2, c2, x2)
        return t, ta

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    runs = [step() for _ in range(args.steps)]
    ms_step = sync_ms(t0) / args.steps
    phases = {k: round(float(np.mean([r[0][k] for r in runs])), 2) for k in runs[0][0]}
    ta = runs[-1][1]
    say(f"step {ms_step:.1f} ms: {phases}")

    # each ordering on its own: its time, the layers' time in it, C(pi), J(pi)
    row_off, col_dst = T.build_csr(w.n, src_d, dst_d)
    orders = []
    ident = torch.arange(w.n, dtype=torch.int32, device=dev)
    base = T.reorder_ta(w.n, row_off, col_dst, ident, 1)   # index 0: C and J of the identity
    orders.append({"order": "random IDs", "order_ms": 0.0, "span": int(base.spans[0]), "J": float(base.disp[0]),
                   "layers_ms": round(layers(row_off, col_dst, X), 1)})
    for label, fn in (("degree/BFS", T.reorder), ("RCMK", T.reorder_rcm)):
        t0 = time.perf_counter()
        pi = fn(w.n, row_off, col_dst)
        o_ms = sync_ms(t0)
        t0 = time.perf_counter()
        got = T.reorder_ta(w.n, row_off, col_dst, pi, 5)
        ta_ms = sync_ms(t0)
        for name, perm, ms, sp, dj in ((label, pi, o_ms, int(got.spans[0]), float(got.disp[0])),
                                       (f"Alg. 1 from {label} (5 updates)", got.pi, o_ms + ta_ms,
                                        int(got.spans[got.done]), float(got.disp[got.done]))):
            r2, c2 = T.relabel_graph(w.n, row_off, col_dst, perm)
            x2 = T.permute_rows(X, perm)
            orders.append({"order": name, "order_ms": round(ms, 1), "span": sp, "J": dj,
                           "layers_ms": round(layers(r2, c2, x2), 1)})
            if name.startswith("Alg. 1"):
                orders[-1]["alg1_ms"] = round(ta_ms, 1)
                orders[-1]["updates"] = int(got.done)
                orders[-1]["spans_per_update"] = [int(x) for x in got.spans[:got.done + 1]]
                orders[-1]["J_per_update"] = [float(x) for x in got.disp[:got.done + 1]]
            del r2, c2, x2
            torch.cuda.empty_cache()
        say(f"{label}: {orders[-2]} / {orders[-1]['order']} {orders[-1]['order_ms']} ms")
    edges = 2 * w.e
    line = {
        "metric": METRIC, "value": round(edges / (ms_step * 1e-3) / 1e9, 4), "unit": "GTEPS", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f16", "data": "synthetic",
        "config": {"workload": f"{w.name}: 2-layer GCN 256->256->64, fp16 storage, fp32 accumulation; skewed "
                               f"RMAT(0.65,0.15,0.15) {w.n:,} vertices / {w.e:,} edges in random IDs; "
                               f"{w.chunk:,}-vertex chunks; step = CSR build + degree/BFS order + Alg. 1 "
                               "(5 updates) + relabel + both layers",
                   "n": w.n, "e": w.e, "chunk": w.chunk, "phases_ms": phases,
                   **({"scale": f"1/{args.scale}"} if args.scale > 1 else {})},
        "alg1": {"updates": int(ta.done), "spans": [int(x) for x in ta.spans[:ta.done + 1]],
                 "J": [float(x) for x in ta.disp[:ta.done + 1]], "ms": phases["alg1_ms"]},
        "orders": orders,
        "roofline": None,
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


def pinned_copy_gbs(dev, gib: int = 4) -> float:
    """Plain pinned host-to-device copy rate (GB/s), the measured link ceiling."""
    import torch
    from paper_2607_17374_amd.api import alloc_pinned
    h = alloc_pinned((gib << 30,), torch.uint8)
    d = torch.empty(gib << 30, dtype=torch.uint8, device=dev)
    d.copy_(h, non_blocking=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(3):
        d.copy_(h, non_blocking=True)
    torch.cuda.synchronize()
    rate = 3 * (gib << 30) / (time.perf_counter() - t0) / 1e9
    del h, d
    torch.cuda.empty_cache()
    return rate


def bench_ooc(args):
    """sage2-ooc-rmat-269m at 1/scale: 2-layer GraphSAGE-mean 512 -> 256 ->
    128 (fp32, U[-1, 1) features) on RMAT with 1% resident hubs, the
    accumulators under the HBM budget scaled with the graph (eviction to
    pinned host memory), 131,072-vertex chunks.  Layer 1's input is never
    resident anywhere: the library's loader fills each chunk with the seeded
    generator on host threads into a ring of pinned buffers while earlier
    chunks copy and compute.  Layer 1 writes its output to pinned host
    memory, which layer 2 streams back in (and writes its own there).  One
    step = CSR build + both layers; roofline = the host link: the bytes
    layer 1 moves over it per second of its streaming, against 64 GB/s."""
    import dataclasses
    import numpy as np
    import torch
    import fixtures as F
    from fixtures import workloads as WL
    import paper_2607_17374_amd as T
    from tests import harness as H

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    t_start = time.perf_counter()

    def say(msg):
        print(f"[bench {time.perf_counter() - t_start:7.1f}s] {msg}", file=sys.stderr, flush=True)

    base = WL.SAGE_OOC_RMAT_269M
    w = base.scaled(base.n // args.scale, base.e // args.scale, name=f"{base.name}-div{args.scale}")
    w = dataclasses.replace(w, hbm_budget=base.hbm_budget // args.scale)
    specs = H.layer_specs(w)
    link = pinned_copy_gbs(dev)
    say(f"pinned host-to-device copy {link:.1f} GB/s")
    src, dst = WL.graph(w)
    say(f"{w.name}: edge list {src.size} edges")
    src_d = torch.from_numpy(src).to(dev)
    dst_d = torch.from_numpy(dst).to(dev)
    for _ in range(args.warmup):
        row_off, col_dst = T.build_csr(w.n, src_d, dst_d)
        del row_off, col_dst
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        row_off, col_dst = T.build_csr(w.n, src_d, dst_d)
    torch.cuda.synchronize()
    csr_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    del src_d, dst_d
    torch.cuda.empty_cache()
    say(f"CSR build {csr_ms:.1f} ms")
    outs = [T.api.alloc_pinned((w.n, sp["d_out"]), torch.float32) for sp in specs]
    say("pinned outputs")
    fill_fn, fill_ctx = F.feature_fill(w.seed, w.feat_dist, w.dims[0], F.F32)

    def one_pass():
        per = []
        plan = T.Plan(w.n, row_off, col_dst, w.chunk)
        for li, sp in enumerate(specs):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            L = T.Layer(w.n, row_off, col_dst, out=outs[li], chunk=w.chunk, plan=plan, hbm_budget=w.hbm_budget,
                        hub_fraction=w.hub_fraction, **sp)
            t1 = time.perf_counter()
            if li == 0:
                ls = L.stream(fill_fn, fill_ctx, threads=args.loader_threads)
            else:
                ls = None
                L.push_all(outs[li - 1])
            t2 = time.perf_counter()
            st = L.finalize()
            torch.cuda.synchronize()
            t3 = time.perf_counter()
            L.destroy()
            st.update(init_s=t1 - t0, push_s=t2 - t1, layer_s=t3 - t0, stream_s=t3 - t1, loader=ls)
            per.append(st)
        plan.destroy()
        return per

    for _ in range(args.warmup):
        one_pass()
    t0 = time.perf_counter()
    runs = [one_pass() for _ in range(args.steps)]
    torch.cuda.synchronize()
    layers_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    ms_step = csr_ms + layers_ms
    say(f"layers {layers_ms:.1f} ms per pass")
    layers = []
    for li in range(len(specs)):
        sts = [r[li] for r in runs]
        st = sts[-1]
        mean = lambda k: float(np.mean([x[k] for x in sts]))
        d = {"layer": li + 1, "d_in": specs[li]["d_in"], "d_out": specs[li]["d_out"], "edges": st["messages"],
             "wall_ms": round(mean("layer_s") * 1e3, 1), "init_ms": round(mean("init_s") * 1e3, 1),
             "gteps": round(st["messages"] / mean("layer_s") / 1e9, 4),
             "h2d_gb": round(st["h2d_bytes"] / 1e9, 2), "d2h_gb": round(st["d2h_bytes"] / 1e9, 2),
             "h2d_gbs": round(st["h2d_bytes"] / mean("stream_s") / 1e9, 2),
             "d2h_gbs": round(st["d2h_bytes"] / mean("stream_s") / 1e9, 2),
             "evictions": st["evictions"], "reloads": st["reloads"], "hub_message_share": st["hub_message_share"],
             "device_gb": round(st["device_bytes"] / 1e9, 2), "input": "loader" if li == 0 else "pinned host"}
        if st["loader"]:
            lw = float(np.mean([x["loader"]["wall_seconds"] for x in sts]))
            d["loader"] = {k: round(float(np.mean([x["loader"][k] for x in sts])), 3)
                           for k in ("fill_seconds", "wait_seconds", "push_seconds", "wall_seconds")}
            d["generator_gbs"] = round(st["loader"]["bytes"] / (d["loader"]["fill_seconds"] / args.loader_threads)
                                       / 1e9, 2)
            d["loader_gbs"] = round(st["loader"]["bytes"] / lw / 1e9, 2)
        layers.append(d)
    total_edges = sum(l["edges"] for l in layers)
    value = total_edges / (ms_step * 1e-3) / 1e9
    l1 = runs[-1][0]
    stream_s = float(np.mean([r[0]["stream_s"] for r in runs]))
    achieved = l1["h2d_bytes"] / stream_s / 1e9
    waited = layers[0]["loader"]["wait_seconds"]
    roofline = {"bound": "host-link", "achieved": round(achieved, 2), "peak": LINK_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / LINK_PEAK_GBS, 4), "traffic": None, "kernel": "host-to-device chunk copies",
                "measured_pinned_copy_gbs": round(link, 2), "frac_of_measured": round(achieved / link, 4),
                "d2h_gbs": layers[0]["d2h_gbs"],
                "note": "layer 1: every chunk generated on host threads and copied while earlier chunks compute; "
                        f"the pushing thread waited {waited:.2f} s of {stream_s:.2f} s for the generator"}

    check = cpu = None
    if not args.no_cpu_baseline:
        import oracle as O
        t0 = time.perf_counter()
        g = O.EdgeGraph(w.n, src, dst)
        t_lists = time.perf_counter() - t0
        del src, dst
        ids = [destination_sample(w.seed * 1000 + li, g.deg_in) for li in range(1, w.layers + 1)]
        need1 = np.unique(np.concatenate([ids[0], ids[1], H.in_neighbours(g, ids[1])]))
        need0 = np.unique(np.concatenate([need1, H.in_neighbours(g, need1)]))
        X = np.zeros((w.n, w.dims[0]), np.float32)      # only the rows the oracle reads are touched
        X[need0] = F.features_rows(w.seed, w.feat_dist, need0, w.dims[0])
        say(f"oracle in-lists {t_lists:.1f} s; {need0.size} input rows")
        t0 = time.perf_counter()
        zs = H.oracle_sampled_layers(w, g, X, ids)
        t_or = time.perf_counter() - t0
        check = []
        for li, z in enumerate(zs, start=1):
            y = outs[li - 1].numpy()[ids[li - 1]].astype(np.float64)
            r = H.compare(y, z, H.RTOL[F.F32])
            check.append({"layer": li, "destinations": int(len(ids[li - 1])), "mismatches": r["n_bad"],
                          "max_abs": r["max_abs"], "mean_rel": r["mean_rel"]})
            say(f"oracle layer {li}: mismatches {r['n_bad']} of {len(ids[li - 1])}")
        rows = need0.size + need1.size
        t_extrap = t_lists + t_or * (w.n * w.layers) / rows
        cpu = {"value": round(total_edges / t_extrap / 1e9, 6), "unit": "GTEPS", "cores": O.threads(),
               "kind": "oracle", "cpu_model": _cpu_model(), "seconds": round(t_lists + t_or, 2),
               "extrapolated_full_step_s": round(t_extrap, 1),
               "sample": f"in-lists over the whole graph ({t_lists:.1f} s), then both layers at {rows} rows (the "
                         "65,536 seeded destinations, the 256 largest in-degrees and up to 256 without in-edges per "
                         f"layer, and the layer-1 rows layer 2 reads) ({t_or:.2f} s); value = both layers' "
                         f"{total_edges / 1e6:.0f}M edges / the step extrapolated linearly in rows (extrapolated)"}

    line = {
        "metric": METRIC, "value": round(value, 4), "unit": "GTEPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{w.name}: 2-layer GraphSAGE-mean 512->256->128, fp32, U[-1,1) features; "
                               f"RMAT(0.57,0.19,0.19) {w.n:,} vertices / {w.e:,} edges; {w.chunk:,}-vertex chunks; "
                               f"HBM budget {w.hbm_budget / 1e9:.0f} GB with 1% resident hubs; layer-1 chunks "
                               "generated on host threads by the library's loader, outputs in pinned host memory; "
                               "step = CSR build + both layers",
                   "n": w.n, "e": w.e, "chunk": w.chunk, "scale": f"1/{args.scale}", "csr_ms": round(csr_ms, 3),
                   "layers_ms": round(layers_ms, 3), "loader_threads": args.loader_threads},
        "per_layer": layers,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "oracle_check": check,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
