"""Full-size parity runs of the large workloads on one GPU, against the oracle.

    python tests/fullsize.py gcn2-skew-rmat-50m          # 50M vertices, 1B edges
    python tests/fullsize.py sage3-fanout-rmat-100m      # 100M vertices, 1.6B edges
    python tests/fullsize.py sage2-ooc-rmat-269m --scale 8   # out of core, at 1/8
    python tests/fullsize.py <workload> --scale 64       # the same recipe at 1/64

Not collected by pytest (a run takes minutes and most of the GPU's memory);
every step prints a line when it ends, and a JSON summary goes to
gpurun_out/fullsize_<workload>.json.

Checks, all against the oracle (which never reads anything the GPU made):
  - CSR: the GPU's CSR has the canonical shape (rows strictly ascending, no
    self loop, offsets from 0 to e) and the same edge-set digest as the
    generated edge list, so it is the canonical CSR of that list;
  - fanout masks (sampled layers): the digest and count of the CSR edges the
    GPU keeps equal those of the in-edges the oracle's sampler keeps;
  - degree/BFS order (reordered workloads): bit for bit against the oracle;
  - embeddings: per layer, 65,536 seeded destinations plus the 256 largest
    in-degrees and up to 256 zero in-degree vertices, against the oracle
    chain (each layer evaluated on the vertices the next layer reads, fed the
    oracle's own previous layer), with the tolerance of the test suite;
  - reordered workloads: the reordered run, un-permuted, against the run in
    the original IDs, every element.

The out-of-core workload streams every chunk from pinned host memory
(generated before the timed layers, so the host link and not the generator
is measured), writes its outputs to pinned host memory and keeps its
accumulators under the HBM budget (scaled with the graph) with 1% resident
hubs; it reports the host-link bytes and rates beside a plain pinned copy.
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

T0 = time.time()


def say(msg: str) -> None:
    print(f"[{time.time() - T0:7.1f}s] {msg}", flush=True)


def destination_sample(seed: int, deg_in: np.ndarray, count: int = 65536) -> np.ndarray:
    """count seeded uniform destinations, the 256 largest in-degrees (ties by
    lower ID) and up to 256 vertices without in-edges."""
    n = deg_in.size
    rng = np.random.default_rng(seed)
    uni = rng.choice(n, min(count, n), replace=False)
    cand = np.argpartition(-deg_in.astype(np.int64), 256)[:512] if n > 512 else np.arange(n)
    top = cand[np.lexsort((cand, -deg_in[cand].astype(np.int64)))][:256]
    zero = np.flatnonzero(deg_in == 0)[:256]
    return np.unique(np.concatenate([uni, top, zero]).astype(np.int64))


def rows_to_host(t, ids: np.ndarray, dtype_code: int) -> np.ndarray:
    import torch
    from tests import harness as H
    sel = t.index_select(0, torch.from_numpy(ids).to(t.device))
    return H.to_numpy_f64(sel, dtype_code)


def check_csr(n: int, row_off, col_dst, digest_list: tuple) -> dict:
    import oracle as O
    ro = row_off.cpu().numpy()
    cd = col_dst.cpu().numpy()
    shape = O.csr_check(n, ro, cd)
    dg = O.digest_csr(n, ro, cd)
    ok = shape == 0 and dg == digest_list
    say(f"CSR: shape rule {shape}, digest {'equal' if dg == digest_list else 'DIFFERENT'} ({dg[0]} edges)")
    return {"csr_shape_rule": shape, "csr_digest_equal": dg == digest_list, "ok": ok, "_host": (ro, cd)}


def embeddings(w, g, X, runs: dict, ids: list, keeps: list) -> dict:
    """Oracle chain on the samples vs the GPU rows of each run, already on the host."""
    from tests import harness as H
    zs = H.oracle_sampled_layers(w, g, X, ids, keeps)
    out = {}
    for name, outs_host in runs.items():
        res = []
        for li, (y, z) in enumerate(zip(outs_host, zs), start=1):
            r = H.compare(y, z, H.RTOL[w.feat_dtype])
            r.pop("worst", None)
            r["layer"], r["destinations"] = li, int(len(ids[li - 1]))
            say(f"{name} layer {li}: {r['destinations']} destinations, mismatches {r['n_bad']}, "
                f"max abs {r['max_abs']:.3e}, mean rel {r['mean_rel']:.3e}")
            res.append(r)
        out[name] = res
    return out


def run_model(w, row_off, col_dst, X, plan_chunk, ids, mask_check=None, keep_input=True):
    """All layers through the C ABI; returns (sampled output rows per layer on
    the host, per-layer stats and wall times, last output tensor).  With
    keep_input False the caller holds no other reference to X and its memory
    is given back after the first layer."""
    import torch
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import torch_dtype
    from tests import harness as H
    plan = T.Plan(w.n, row_off, col_dst, plan_chunk)
    dev = X.device
    h = X
    host, stats = [], []
    for li, spec in enumerate(H.layer_specs(w), start=1):
        out = T.alloc_device((w.n, spec["d_out"]), torch_dtype(spec["out_dtype"]), dev)
        torch.cuda.synchronize()
        t0 = time.time()
        L = T.Layer(w.n, row_off, col_dst, out=out, chunk=w.chunk, plan=plan, **spec)
        t_init = time.time() - t0
        if mask_check is not None:
            mask_check(li, L)
        t1 = time.time()
        L.push_all(h)
        st = L.finalize()
        torch.cuda.synchronize()
        t_run = time.time() - t1
        L.destroy()
        st.update(layer=li, init_s=round(t_init, 3), push_finalize_s=round(t_run, 3),
                  gteps=round(st["messages"] / (t_init + t_run) / 1e9, 3))
        say(f"layer {li}: {st['messages']} messages, {st['pairs']} pairs, init {t_init:.2f} s, "
            f"chunks {t_run:.2f} s, completed {st['completed']}/{w.n}")
        assert st["pending_left"] == 0
        stats.append(st)
        host.append(rows_to_host(out, ids[li - 1], spec["out_dtype"]))
        del h
        if not keep_input:
            X = None
        h = out
        torch.cuda.empty_cache()
    plan.destroy()
    return host, stats, h


def residency_run(w, g, pi_host, row_off, col_dst, X, slot_list) -> dict:
    """Residency of one ordering: the oracle's chunk-level profile A[k] of
    the order, then the second layer of w (on input X) in core and under
    budgets that leave about each of `slot_list` pool rows with 1% hubs.
    Outputs must equal the in-core run bit for bit; reports evictions,
    reloads and host-link bytes."""
    import torch
    import oracle as O
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import torch_dtype
    from tests import harness as H
    A = O.active_profile(g, pi_host, w.chunk)
    res = {"peak_active": int(A.max()), "mean_active": float(A.mean()), "budgeted": []}
    say(f"  residency: peak A {res['peak_active']}, mean A {res['mean_active']:.0f}")
    spec = H.layer_specs(w)[1]

    def run(budget):
        out = T.alloc_device((w.n, spec["d_out"]), torch_dtype(spec["out_dtype"]), X.device)
        torch.cuda.synchronize()
        t0 = time.time()
        L = T.Layer(w.n, row_off, col_dst, out=out, chunk=w.chunk, hbm_budget=budget,
                    hub_fraction=0.01 if budget else 0.0, **spec)
        L.push_all(X)
        st = L.finalize()
        L.destroy()
        torch.cuda.synchronize()
        return out, st, time.time() - t0

    ref, st0, t_ref = run(0)
    res["t_in_core"] = t_ref
    for slots in slot_list:
        budget = H.pool_budget(st0, w.n, spec["d_out"], spec["d_in"], w.chunk, slots)
        try:
            out, st, t = run(budget)
        except T.TaurusError as ex:
            if ex.status != -6:
                raise
            res["budgeted"].append({"slots_asked": slots, "refused": str(ex)})
            say(f"  residency: about {slots} pool rows refused: {ex}")
            continue
        r = dict(slots_asked=slots, pool_rows=st["pool_rows"], equal_to_in_core=bool(torch.equal(ref, out)),
                 evictions=st["evictions"], reloads=st["reloads"], d2h_bytes=st["d2h_bytes"],
                 h2d_bytes=st["h2d_bytes"], device_bytes=st["device_bytes"], seconds=t)
        res["budgeted"].append(r)
        say(f"  residency: {r['pool_rows']} pool rows: {r['evictions']} evictions, {r['reloads']} reloads, "
            f"{r['d2h_bytes'] / 1e9:.2f} GB out, {t:.2f} s (in core {t_ref:.2f} s), "
            f"equal to in core: {r['equal_to_in_core']}")
        del out
    del ref
    torch.cuda.empty_cache()
    return res


def run_c5(w) -> dict:
    import torch
    import oracle as O
    import paper_2607_17374_amd as T
    from tests import harness as H
    from fixtures import workloads as WL
    from paper_2607_17374_amd.api import torch_dtype
    res = {"workload": w.name, "n": w.n, "e": w.e}
    src, dst = WL.graph(w)
    say(f"edge list: {src.size} edges (random IDs)")
    g = O.EdgeGraph(w.n, src, dst, out_lists=True)
    dig = O.digest_edges(src, dst)
    say("oracle in-lists and edge digest")
    s = torch.from_numpy(src).cuda()
    d = torch.from_numpy(dst).cuda()
    row_off, col_dst = T.build_csr(w.n, s, d)
    torch.cuda.synchronize()
    del s, d
    torch.cuda.empty_cache()
    say("GPU CSR")
    c = check_csr(w.n, row_off, col_dst, dig)
    del c["_host"]
    res["csr"] = c
    del src, dst
    ident = np.arange(w.n, dtype=np.int32)
    res["span_random_ids"] = O.total_span(g, ident)
    orders = {}
    for label, gpu_fn, oracle_fn in (("degree/BFS order", T.reorder, O.reorder_bfs),
                                     ("RCMK order", T.reorder_rcm, O.reorder_rcm)):
        t0 = time.time()
        pi = gpu_fn(w.n, row_off, col_dst)
        torch.cuda.synchronize()
        t_gpu = time.time() - t0
        say(f"GPU {label} in {t_gpu:.2f} s")
        want = oracle_fn(g)
        ok = bool(np.array_equal(pi.cpu().numpy(), want))
        span = O.total_span(g, want)
        res[label] = {"bit_exact": ok, "span": span, "gpu_s": t_gpu}
        say(f"{label} bit-exact vs oracle: {ok}; total span {res['span_random_ids']} -> {span}")
        orders[label] = pi
        # Alg. 1 from this bootstrap
        ta_label = f"topology-aware order from {label.split()[0]}"
        t0 = time.time()
        got = T.reorder_ta(w.n, row_off, col_dst, pi, 5)
        torch.cuda.synchronize()
        t_gpu = time.time() - t0
        done = got.done
        say(f"GPU {ta_label} in {t_gpu:.2f} s: spans {got.spans[:done + 1].tolist()} "
            f"J {got.disp[:done + 1].tolist()}")
        want_ta = O.reorder_ta(g, want, 5)
        try:
            differ = H.check_ta(g, got, want_ta, ta_label)
            ok = True
        except AssertionError as ex:
            differ, ok = -1, False
            say(f"{ta_label} check failed: {ex}")
        res[ta_label] = {"matches_oracle": ok, "ranks_differing_near_ties": differ,
                         "spans": got.spans[:done + 1].tolist(), "disp": got.disp[:done + 1].tolist(),
                         "gpu_s": t_gpu}
        say(f"{ta_label} vs oracle: {ok} ({differ} ranks differ at near ties)")
        orders[ta_label] = got.pi
        del want, want_ta
    ids = [destination_sample(w.seed * 1000 + li, g.deg_in) for li in range(1, w.layers + 1)]
    xh = WL.input_features(w)
    say("features")
    X = torch.from_numpy(xh.view(np.int16)).cuda().view(torch_dtype(w.feat_dtype))
    host_a, stats_a, last_a = run_model(w, row_off, col_dst, X, w.chunk, ids)
    res["random_ids"] = {"stats": stats_a}
    slots = [w.n * 7 // 25, w.n * 6 // 25, w.n // 5]      # 28%, 24% and 20% of the rows
    res["random_ids"]["residency"] = residency_run(w, g, ident, row_off, col_dst, X, slots)
    last_a_host = last_a.cpu()
    del last_a
    torch.cuda.empty_cache()
    # reordered runs: relabel the graph, permute the features, run, un-permute
    runs = {"random IDs": host_a}
    for label, perm in orders.items():
        r2, c2 = T.relabel_graph(w.n, row_off, col_dst, perm)
        X2 = T.permute_rows(X, perm)
        torch.cuda.empty_cache()
        say(f"{label}: relabelled graph and features")
        ph = perm.cpu().numpy()
        ids_new = [ph[i].astype(np.int64) for i in ids]   # the same vertices under their new IDs
        host_b, stats_b, last_b = run_model(w, r2, c2, X2, w.chunk, ids_new)
        res[label]["stats"] = stats_b
        res[label]["residency"] = residency_run(w, g, ph, r2, c2, X2, slots)
        del r2, c2, X2
        back = T.permute_rows(last_b, perm, inverse=True).cpu()
        del last_b
        a64, b64 = last_a_host.double(), back.double()
        rms = float(a64.pow(2).mean().sqrt())
        bound = 1e-2 * (a64.abs() + rms)
        res[label]["vs_random_ids_last_layer"] = {"max_abs": float((a64 - b64).abs().max()),
                                                  "n_bad": int(((a64 - b64).abs() > bound).sum())}
        say(f"{label} vs random IDs, last layer, every element: {res[label]['vs_random_ids_last_layer']}")
        del a64, b64, back
        runs[label] = host_b
        torch.cuda.empty_cache()
    del row_off, col_dst, X, last_a_host
    res["embeddings"] = embeddings(w, g, xh, runs, ids, [None] * w.layers)
    return res


def run_c3(w) -> dict:
    import torch
    import oracle as O
    import paper_2607_17374_amd as T
    from fixtures import workloads as WL
    from paper_2607_17374_amd.api import torch_dtype
    res = {"workload": w.name, "n": w.n, "e": w.e}
    src, dst = WL.graph(w)
    say(f"edge list: {src.size} edges")
    g = O.EdgeGraph(w.n, src, dst)
    dig = O.digest_edges(src, dst)
    say("oracle in-lists and edge digest")
    s = torch.from_numpy(src).cuda()
    d = torch.from_numpy(dst).cuda()
    row_off, col_dst = T.build_csr(w.n, s, d)
    torch.cuda.synchronize()
    del s, d, src, dst
    torch.cuda.empty_cache()
    say("GPU CSR")
    c = check_csr(w.n, row_off, col_dst, dig)
    ro_h, cd_h = c.pop("_host")
    res["csr"] = c
    keeps = []
    masks = []

    def mask_check(li, L):
        words, kept = L.sampled_edges()
        _, keep_in, m = O.sample(g, w.seed, li, w.fanout(li))
        got = O.digest_csr(w.n, ro_h, cd_h, words)
        want = O.digest_in_lists(g, keep_in)
        ok = got == want and kept == int(m.sum())
        say(f"layer {li} fanout {w.fanout(li)}: kept {kept} edges, mask digest {'equal' if got == want else 'DIFFERENT'}")
        masks.append({"layer": li, "kept": int(kept), "digest_equal": got == want, "count_equal": kept == int(m.sum())})
        keeps.append(keep_in)

    ids = [destination_sample(w.seed * 1000 + li, g.deg_in) for li in range(1, w.layers + 1)]
    xh = WL.input_features(w)
    say("features")
    host, stats, last = run_model(w, row_off, col_dst,
                                  torch.from_numpy(xh.view(np.int16)).cuda().view(torch_dtype(w.feat_dtype)),
                                  w.chunk, ids, mask_check=mask_check, keep_input=False)
    res["masks"] = masks
    res["stats"] = stats
    del last
    torch.cuda.empty_cache()
    del ro_h, cd_h
    res["embeddings"] = embeddings(w, g, xh, {"GPU": host}, ids, keeps)
    return res


def link_peak_gbs(gib: int = 4) -> float:
    """Host-to-device rate of one large copy from pinned memory (the link as
    the copy engines see it)."""
    import torch
    src = torch.empty(gib << 28, dtype=torch.float32).pin_memory()
    dst = torch.empty_like(src, device="cuda")
    dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    t = time.time()
    for _ in range(3):
        dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    gbs = 3 * src.numel() * 4 / (time.time() - t) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return gbs


def run_c4(w) -> dict:
    import torch
    import oracle as O
    import paper_2607_17374_amd as T
    import fixtures as F
    from fixtures import workloads as WL
    from tests import harness as H
    res = {"workload": w.name, "n": w.n, "e": w.e, "hbm_budget": w.hbm_budget, "hub_fraction": w.hub_fraction}
    res["link_peak_h2d_gbs"] = round(link_peak_gbs(), 2)
    say(f"pinned host-to-device copy: {res['link_peak_h2d_gbs']} GB/s")
    src, dst = WL.graph(w)
    say(f"edge list: {src.size} edges")
    g = O.EdgeGraph(w.n, src, dst)
    dig = O.digest_edges(src, dst)
    say("oracle in-lists and edge digest")
    s = torch.from_numpy(src).cuda()
    d = torch.from_numpy(dst).cuda()
    row_off, col_dst = T.build_csr(w.n, s, d)
    torch.cuda.synchronize()
    del s, d, src, dst
    torch.cuda.empty_cache()
    c = check_csr(w.n, row_off, col_dst, dig)
    del c["_host"]
    res["csr"] = c
    # layer-1 input in pinned host memory, in pieces of whole chunks of at
    # most 8 GiB each (pinned allocations are capped on this host)
    row_bytes = w.dims[0] * 4
    step = max(w.chunk, ((8 << 30) // row_bytes) // w.chunk * w.chunk)
    pieces = []
    for v0 in range(0, w.n, step):
        v1 = min(w.n, v0 + step)
        piece = torch.from_numpy(F.features(w.seed, w.feat_dist, v0, v1, w.dims[0], F.F32)).pin_memory()
        pieces.append((v0, v1, piece))
        say(f"features rows {v1}/{w.n} (pinned)")

    def push_layer1(L):
        for v0, v1, piece in pieces:
            for b in range(v0, v1, w.chunk):
                L.push_chunk(b, min(b + w.chunk, v1), piece[b - v0:min(b + w.chunk, v1) - v0])


    ids = [destination_sample(w.seed * 1000 + li, g.deg_in) for li in range(1, w.layers + 1)]
    h = None
    host, stats = [], []
    plan = T.Plan(w.n, row_off, col_dst, w.chunk)
    for li, spec in enumerate(H.layer_specs(w), start=1):
        out = torch.empty((w.n, spec["d_out"]), dtype=torch.float32).pin_memory()
        torch.cuda.synchronize()
        t0 = time.time()
        L = T.Layer(w.n, row_off, col_dst, out=out, chunk=w.chunk, plan=plan, hbm_budget=w.hbm_budget,
                    hub_fraction=w.hub_fraction, **spec)
        t_init = time.time() - t0
        t1 = time.time()
        if h is None:
            push_layer1(L)
        else:
            L.push_all(h)
        st = L.finalize()
        t_run = time.time() - t1
        L.destroy()
        link = st["h2d_bytes"] + st["d2h_bytes"]
        st.update(layer=li, init_s=round(t_init, 3), push_finalize_s=round(t_run, 3),
                  h2d_gbs=round(st["h2d_bytes"] / t_run / 1e9, 2), link_gbs=round(link / t_run / 1e9, 2),
                  gteps=round(st["messages"] / (t_init + t_run) / 1e9, 3))
        say(f"layer {li}: {st['messages']} messages, init {t_init:.2f} s, chunks {t_run:.2f} s; "
            f"h2d {st['h2d_bytes'] / 1e9:.1f} GB ({st['h2d_gbs']} GB/s), d2h {st['d2h_bytes'] / 1e9:.1f} GB, "
            f"evictions {st['evictions']}, reloads {st['reloads']}, hub messages {st['hub_message_share']:.3f}, "
            f"device bytes {st['device_bytes'] / 1e9:.1f} GB, completed {st['completed']}/{w.n}")
        assert st["pending_left"] == 0
        stats.append(st)
        host.append(out.numpy()[ids[li - 1]].astype(np.float64))
        del h
        h = out
        torch.cuda.empty_cache()
    plan.destroy()
    del h, out
    res["stats"] = stats
    # the oracle gets the layer-1 input as one host array (built from the pieces)
    X = np.concatenate([piece.numpy() for _, _, piece in pieces])
    pieces.clear()
    res["embeddings"] = embeddings(w, g, X, {"GPU": host}, ids, [None] * w.layers)
    return res


def main():
    from fixtures import workloads as WL
    import argparse
    ap = argparse.ArgumentParser()
    ap.add_argument("workload", nargs="?", default="gcn2-skew-rmat-50m")
    ap.add_argument("--scale", type=int, default=1, help="run the recipe at 1/scale of the vertices and edges")
    ap.add_argument("--chunk", type=int, default=0, help="override the chunk size (out of core: after scaling)")
    ap.add_argument("--budget-frac", type=float, default=1.0, help="out of core: multiply the HBM budget")
    ap.add_argument("--tag", default="", help="suffix of the summary file name")
    args = ap.parse_args()
    w = {x.name: x for x in WL.ALL}[args.workload]
    if args.scale > 1:
        import dataclasses
        w = w.scaled(w.n // args.scale, w.e // args.scale, name=f"{w.name}-div{args.scale}")
        if w.out_of_core:
            # budget and chunk scale with the graph: the same number of chunks,
            # so each chunk holds the full-size share of the edges
            w = dataclasses.replace(w, hbm_budget=w.hbm_budget // args.scale,
                                    chunk=max(1024, w.chunk // args.scale))
    if args.chunk or args.budget_frac != 1.0 or args.tag:
        import dataclasses
        w = dataclasses.replace(w, chunk=args.chunk or w.chunk, hbm_budget=int(w.hbm_budget * args.budget_frac),
                                name=w.name + (f"-{args.tag}" if args.tag else ""))
    import torch
    assert torch.cuda.is_available(), "needs a GPU"
    import oracle as O
    say(f"{w.name}: n={w.n} e={w.e}; oracle threads {O.threads()}")
    res = run_c5(w) if w.reorder else (run_c4(w) if w.out_of_core else run_c3(w))
    res["seconds"] = round(time.time() - T0, 1)
    os.makedirs(os.path.join(ROOT, "gpurun_out"), exist_ok=True)
    path = os.path.join(ROOT, "gpurun_out", f"fullsize_{w.name}.json")
    with open(path, "w") as f:
        json.dump(res, f, indent=1, default=lambda o: o.item() if hasattr(o, "item") else str(o))
    say(f"summary in {path}")


if __name__ == "__main__":
    main()
