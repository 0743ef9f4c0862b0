"""Benchmark: layer-wise broadcast GNN inference on one MI355X.

Workload: 2-layer GCN (symmetric normalisation with self loops), exact,
RMAT(0.57, 0.19, 0.19) graph with 1,000,000 vertices and 20,000,000 edges,
N(0,1) fp32 features of width 128, layer widths 128 -> 128 -> 64, sources
streamed in 65,536-vertex chunks.  Inputs (edge list, features) are seeded
synthetic data resident in HBM before the timed region.

One step = the whole hot path once: CSR build from the edge list, the
chunk index (a plan shared by both exact layers), then for each layer init
(pending counts, weights), all chunk pushes (MFMA transform, scatter with
fused finalise, fix-up) and finalize.

Output: one JSON line.  value = aggregated edges per second per layer
(sum over layers of the propagated edges / step time) in GTEPS.  roofline =
the scatter kernel's algorithmic HBM bytes over its HIP-event-timed
duration, against 8 TB/s.  cpu_baseline = the CPU oracle timed on this
host over the same workload.
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


def scatter_algorithmic_bytes(st: dict, d_o: int, ncols: int, out_bytes: int) -> float:
    """Bytes the scatter step must move for one layer (all its launches).

    the work-unit table (16 bytes per unit) and each item's source code (4);
    the chunk transform Y read once (4 * ncols per vertex); pending/expected
    counts 8 read + 4 written per (destination, chunk) pair; accumulator
    rows: every pair but a vertex's first reads its row and every pair but
    its last writes it (4 * d_o each); one output row per vertex.  Hub
    segments completed by the fix-up pass are taken out (their accumulator
    traffic is the fix-up kernel's)."""
    n, items, pairs = st["n"], st["messages"] + st["self_terms"], st["pairs"]
    units, splits = st["short_units"] + st["wave_units"], st["split_segments"]
    return (16.0 * units + 4.0 * items + 4.0 * n * ncols + 12.0 * pairs + 8.0 * d_o * (pairs - n)
            + out_bytes * d_o * n - 8.0 * d_o * splits)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="time without per-kernel events")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 1 GiB device copy, the reference kernel for HBM byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the path has no multi-GPU mode; see DESIGN.md for how it would shard)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import fixtures as F
    from fixtures import workloads as WL
    import paper_2607_17374_amd as T
    from tests import harness as H

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    w = WL.GCN_RMAT_1M
    src, dst = WL.graph(w)
    X = torch.from_numpy(WL.input_features(w)).to(dev)
    src_d = torch.from_numpy(src).to(dev)
    dst_d = torch.from_numpy(dst).to(dev)
    specs = H.layer_specs(w)
    outs = [torch.empty((w.n, s["d_out"]), dtype=torch.float32, device=dev) for s in specs]
    profile = not args.no_profile
    if args.copy_calibration:
        a = torch.ones(1 << 28, dtype=torch.float32, device=dev)     # 1 GiB
        c = torch.empty_like(a)
        for _ in range(3):
            c.copy_(a)
        del a, c
    torch.cuda.synchronize()

    def step():
        t0 = time.perf_counter()
        row_off, col_dst = T.build_csr(w.n, src_d, dst_d)
        t_csr = time.perf_counter() - t0
        tp = time.perf_counter()
        plan = T.Plan(w.n, row_off, col_dst, w.chunk)
        t_plan = time.perf_counter() - tp
        h = X
        per = []
        for spec, out in zip(specs, outs):
            tl = time.perf_counter()
            L = T.Layer(w.n, row_off, col_dst, out=out, chunk=w.chunk, profile=profile, plan=plan, **spec)
            L.push_all(h)
            st = L.finalize()
            L.destroy()
            st["wall_ms"] = (time.perf_counter() - tl) * 1e3
            per.append(st)
            h = out
        plan.destroy()
        return t_csr * 1e3, t_plan * 1e3, per

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    runs = [step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_step = elapsed * 1e3 / args.steps

    # per-layer figures, averaged over the timed steps
    nl = len(specs)
    layers = []
    tot_bytes = tot_ms = tot_launch = 0.0
    gemm_flops = gemm_ms = 0.0
    for li in range(nl):
        sts = [r[2][li] for r in runs]
        d_o, d_in = specs[li]["d_out"], specs[li]["d_in"]
        ncols = d_o  # GCN transform width
        wall = float(np.mean([s["wall_ms"] for s in sts]))
        st = sts[-1]
        b = scatter_algorithmic_bytes(st, d_o, ncols, 4)
        sc_ms = float(np.mean([s["ms_scatter"] for s in sts]))
        launches = st["launches_scatter"]
        if profile:
            tot_bytes += b * len(sts)
            tot_ms += sum(s["ms_scatter"] for s in sts)
            tot_launch += launches * len(sts)
            gemm_flops += 2.0 * w.n * d_in * ncols * len(sts)
            gemm_ms += sum(s["ms_gemm"] for s in sts)
        layers.append({
            "layer": li + 1, "d_in": d_in, "d_out": d_o, "edges": st["messages"], "pairs": st["pairs"],
            "wall_ms": round(wall, 3), "gteps": round(st["messages"] / (wall * 1e-3) / 1e9, 3),
            "vertices_per_s": round(w.n / (wall * 1e-3), 1), "init_ms": round(float(np.mean([s["ms_init"] for s in sts])), 3),
            "gemm_ms": round(float(np.mean([s["ms_gemm"] for s in sts])), 3), "scatter_ms": round(sc_ms, 3),
            "fixup_ms": round(float(np.mean([s["ms_fixup"] for s in sts])), 3),
            "scatter_launches": launches, "short_units": st["short_units"], "wave_units": st["wave_units"],
            "split_segments": st["split_segments"],
            "scatter_algorithmic_gb": round(b / 1e9, 4),
            "scatter_gbs": round(b / (sc_ms * 1e-3) / 1e9, 1) if sc_ms > 0 else None,
        })
    csr_ms = float(np.mean([r[0] for r in runs]))
    plan_ms = float(np.mean([r[1] for r in runs]))
    total_edges = sum(l["edges"] for l in layers)
    value = total_edges / (ms_step * 1e-3) / 1e9

    roofline = None
    if profile and tot_ms > 0:
        achieved = tot_bytes / (tot_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "k_scatter",
                    "avg_launch_us": round(tot_ms * 1e3 / tot_launch, 2),
                    "bytes_per_launch": round(tot_bytes / tot_launch, 0)}
    gemm = None
    if profile and gemm_ms > 0:
        tf = gemm_flops / (gemm_ms * 1e-3) / 1e12
        gemm = {"bound": "mfma", "achieved": round(tf, 2), "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tf / FP32_MFMA_PEAK_TFLOPS, 4), "kernel": "k_gemm_f32"}

    cpu = None
    if not args.no_cpu_baseline:
        import oracle as O
        t0 = time.perf_counter()
        g, zs = H.oracle_model(w, src, dst)
        t_or = time.perf_counter() - t0
        cpu = {"value": round(total_edges / t_or / 1e9, 5), "unit": "GTEPS", "cores": O.threads(),
               "kind": "oracle", "seconds": round(t_or, 2),
               "sample": "the full workload once: oracle CSR and in-lists, then both layers for all "
                         "1,000,000 destinations in fp64 (value = both layers' 40M propagated edges / wall time)"}

    line = {
        "metric": METRIC, "value": round(value, 4), "unit": "GTEPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "gcn2-rmat-1m: 2-layer GCN 128->128->64 (symmetric norm, self loops), exact; "
                               "RMAT(0.57,0.19,0.19) 1,000,000 vertices / 20,000,000 edges; N(0,1) fp32 features; "
                               "65,536-vertex source chunks; step = CSR build + chunk index + both layers",
                   "n": w.n, "e": w.e, "chunk": w.chunk, "csr_ms": round(csr_ms, 3),
                   "plan_ms": round(plan_ms, 3)},
        "per_layer": layers,
        "roofline": roofline,
        "gemm_roofline": gemm,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
