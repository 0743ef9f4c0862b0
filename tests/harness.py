"""Shared test/measurement helpers: run a workload on the GPU through the C
ABI, run the oracle on the CPU, and compare the two.

The GPU side and the oracle side only meet here, in the comparison; their
inputs come from ``fixtures`` (the seeded generator both may use)."""
from __future__ import annotations

import numpy as np

import fixtures as F
from fixtures import workloads as WL

# tolerance of the embedding comparison: fp32 paths 1e-4, 16-bit storage 1e-2
RTOL = {F.F32: 1e-4, F.BF16: 1e-2, F.F16: 1e-2}


def compare(y: np.ndarray, o: np.ndarray, rtol: float) -> dict:
    """Element-wise |y - o| <= rtol * (|o| + RMS(o)); RMS over the whole
    layer output of the oracle guards ReLU zeros and cancellation.  Also the
    paper's summary statistics: mean per-vertex max abs error and mean
    relative error."""
    y = np.asarray(y, np.float64)
    o = np.asarray(o, np.float64)
    assert y.shape == o.shape, (y.shape, o.shape)
    if o.size == 0:
        return dict(n_bad=0, max_abs=0.0, mean_vertex_max_abs=0.0, mean_rel=0.0, rms=0.0, worst=None)
    rms = float(np.sqrt(np.mean(o * o)))
    err = np.abs(y - o)
    bound = rtol * (np.abs(o) + rms)
    bad = err > bound
    rel = err / (np.abs(o) + rms + 1e-300)
    worst = np.unravel_index(int(np.argmax(err - bound)), err.shape)
    return dict(n_bad=int(bad.sum()), max_abs=float(err.max()), mean_vertex_max_abs=float(err.max(axis=1).mean()),
                mean_rel=float(rel.mean()), max_rel=float(rel.max()), rms=rms,
                worst=(tuple(int(i) for i in worst), float(y[worst]), float(o[worst])))


def layer_specs(w: WL.Workload, fanouts=None):
    """Per-layer keyword arguments of paper_2607_17374_amd.Layer for workload w."""
    specs = []
    for li in range(1, w.layers + 1):
        p = WL.layer_params(w, li)
        in_dt, out_dt = w.layer_dtypes(li)
        specs.append(dict(agg=w.agg, d_in=p.d_in, d_out=p.d_out, weight_cat=p.weight_cat(), bias=p.b,
                          in_dtype=in_dt, out_dtype=out_dt, relu=li < w.layers,
                          fanout=(fanouts[li - 1] if fanouts else w.fanout(li)), layer=li, seed=w.seed,
                          attn=p.attn))
    return specs


def oracle_layer(w: WL.Workload, p, g, H, h_dtype, relu, keep_in=None, dst_ids=None):
    """The oracle layer of w's family with layer parameters p."""
    import oracle as O
    if w.agg == WL.GAT_ATT:
        return O.gat_layer(g, H, h_dtype, p.W, p.attn, p.b, relu, keep_in=keep_in, dst_ids=dst_ids)
    return O.layer(w.agg, g, H, h_dtype, p.W, p.b, relu, keep_in=keep_in, dst_ids=dst_ids)


def oracle_model(w: WL.Workload, src=None, dst=None):
    """Full oracle run of workload w -> (oracle graph, [fp64 outputs per layer])."""
    import oracle as O
    if src is None:
        src, dst = WL.graph(w)
    g = O.Graph(w.n, src, dst)
    X = WL.input_features(w)
    H, h_dtype = X, w.feat_dtype
    zs = []
    for li in range(1, w.layers + 1):
        p = WL.layer_params(w, li)
        keep = None
        if w.fanout(li) > 0:
            _, keep, _ = O.sample(g, w.seed, li, w.fanout(li))
        z = oracle_layer(w, p, g, H, h_dtype, li < w.layers, keep_in=keep)
        zs.append(z)
        _, out_dt = w.layer_dtypes(li)
        H = O.round_store(z, out_dt)
        h_dtype = out_dt
    return g, zs


def gpu_graph(w: WL.Workload, src=None, dst=None, device="cuda"):
    import torch
    import paper_2607_17374_amd as T
    if src is None:
        src, dst = WL.graph(w)
    s = torch.from_numpy(np.ascontiguousarray(src)).to(device)
    d = torch.from_numpy(np.ascontiguousarray(dst)).to(device)
    row_off, col_dst = T.build_csr(w.n, s, d)
    return row_off, col_dst


def gpu_model(w: WL.Workload, row_off, col_dst, X=None, chunk=None, order=None, profile=False, stream=None,
              use_plan=True):
    """Run every layer of w through the C ABI; returns ([outputs], [stats]).
    The layers share one plan (exact chunk index, in-edge lists for sampling)
    unless use_plan is False."""
    import torch
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import torch_dtype
    if X is None:
        xh = WL.input_features(w)
        X = torch.from_numpy(xh.view(np.int16) if xh.dtype == np.uint16 else xh).cuda()
        if w.feat_dtype != F.F32:
            X = X.view(torch_dtype(w.feat_dtype))
    chunk = chunk or w.chunk
    h = X
    outs, stats = [], []
    specs = layer_specs(w)
    plan = T.Plan(w.n, row_off, col_dst, chunk, stream=stream) if use_plan else None
    for spec in specs:
        out = T.alloc_device((w.n, spec["d_out"]), torch_dtype(spec["out_dtype"]), X.device)
        L = T.Layer(w.n, row_off, col_dst, out=out, chunk=chunk, profile=profile, stream=stream,
                    plan=plan, **spec)
        L.push_all(h, order=order)
        stats.append(L.finalize())
        L.destroy()
        outs.append(out)
        h = out
    if plan is not None:
        plan.destroy()
    return outs, stats


def pool_budget(stats_incore: dict, n: int, d_out: int, d_in: int, chunk: int, slots: int) -> int:
    """An hbm_budget that leaves about `slots` accumulator rows, from the
    statistics of the same layer run in core (mirrors the library's planning:
    everything but the dense rows, about 42 bytes of residency arrays per
    vertex, two staging buffers, then the pool, each with 1/8 rounding
    room)."""
    row = d_out * 4
    dense = n * row
    other = stats_incore["device_bytes"] - dense
    staging = 2 * min(chunk, n) * d_in * 4 * 9 // 8
    return int(other + 42 * n * 9 // 8 + 4096 + staging + slots * (row + 4) * 9 // 8 + (1 << 20))


def to_numpy_f64(t, dtype_code: int) -> np.ndarray:
    import torch
    return t.detach().to(torch.float64).cpu().numpy() if dtype_code != F.F32 else t.detach().cpu().numpy().astype(np.float64)


def in_neighbours(g, vs: np.ndarray, keep_in: np.ndarray | None = None) -> np.ndarray:
    """Sources of the in-edges of the vertices vs (kept ones only when a
    sampled layer's keep_in mask over the in-lists is given), as a sorted
    unique array."""
    vs = np.asarray(vs, np.int64)
    lo, hi = g.in_off[vs], g.in_off[vs + 1]
    cnt = hi - lo
    if cnt.sum() == 0:
        return np.zeros(0, np.int64)
    pos = np.repeat(lo - np.concatenate([[0], np.cumsum(cnt)[:-1]]), cnt) + np.arange(cnt.sum())
    if keep_in is not None:
        pos = pos[keep_in[pos] != 0]
    return np.unique(g.in_src[pos].astype(np.int64))


def oracle_sampled_layers(w: WL.Workload, g, X: np.ndarray, ids: list, keeps: list | None = None) -> list:
    """Oracle outputs (fp64) of every layer of w at the destination sample
    ids[l - 1], each layer fed the oracle's own previous layer, which is
    evaluated only on the vertices the later layers read (the samples, the
    destinations' own rows and their propagated in-neighbours).  X: the
    layer-1 input in storage dtype; keeps[l - 1]: the oracle sampler's keep_in
    for sampled layers, else None."""
    import oracle as O
    L = w.layers
    keeps = keeps or [None] * L
    need = [None] * L
    need[L - 1] = np.unique(np.asarray(ids[L - 1], np.int64))
    for li in range(L - 1, 0, -1):          # layer li's outputs read by layer li + 1
        nxt = need[li]
        need[li - 1] = np.unique(np.concatenate([np.asarray(ids[li - 1], np.int64), nxt,
                                                 in_neighbours(g, nxt, keeps[li])]))
    H, h_dtype = X, w.feat_dtype
    out = []
    for li in range(1, L + 1):
        p = WL.layer_params(w, li)
        z = oracle_layer(w, p, g, H, h_dtype, li < L, keep_in=keeps[li - 1], dst_ids=need[li - 1])
        pos = np.searchsorted(need[li - 1], np.asarray(ids[li - 1], np.int64))
        out.append(z[pos])
        if li < L:
            _, out_dt = w.layer_dtypes(li)
            rows = O.round_store(z, out_dt)
            H = np.zeros((w.n, rows.shape[1]), rows.dtype)
            H[need[li - 1]] = rows
            h_dtype = out_dt
    return out
