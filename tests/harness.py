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
        extra = {}
        if w.agg == WL.GIN_MLP:   # the perceptron's second layer, row-major [d_hidden][d_out]
            extra = dict(d_hidden=p.d_out, weight2=np.ascontiguousarray(p.W2.T, np.float32), bias2=p.b2)
        specs.append(dict(agg=w.agg, d_in=p.d_in, d_out=p.d_out, weight_cat=p.weight_cat(), bias=p.b,
                          in_dtype=in_dt, out_dtype=out_dt, relu=li < w.layers,
                          fanout=(fanouts[li - 1] if fanouts else w.fanout(li)), layer=li, seed=w.seed,
                          attn=p.attn, **extra))
    return specs


def oracle_layer(w: WL.Workload, p, g, H, h_dtype, relu, keep_in=None, dst_ids=None):
    """The oracle layer of w's family with layer parameters p."""
    import oracle as O
    if w.agg == WL.GAT_ATT:
        return O.gat_layer(g, H, h_dtype, p.W, p.attn, p.b, relu, keep_in=keep_in, dst_ids=dst_ids)
    if w.agg == WL.GIN_MLP:
        return O.gin_mlp_layer(g, H, h_dtype, p.W, p.b, p.W2, p.b2, relu, keep_in=keep_in, dst_ids=dst_ids)
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


# ---- Alg. 1 (Sec. 3.8): GPU positions and orders against the oracle ------

U64 = 2.0 ** -53   # unit roundoff of fp64


def _gamma(k):
    k = np.asarray(k, np.float64)
    return k * U64 / (1.0 - k * U64)


def ta_position_bound(g, updates: int) -> np.ndarray:
    """Relative error bound rho(w) of the fp64 positions after ``updates``
    updates of Alg. 1, valid for any summation order (the standard bound
    gamma(k) = k u / (1 - k u) on a sum of k non-negative terms, errors of
    non-negative inputs composed multiplicatively).  Per update:
      centre of v, a sum of d(v) positions then two divisions:
        1 + rho_q(v) = (1 + max_{N(v)} rho_r)(1 + gamma(d(v)))(1 + u)^2;
      position of w, a sum over S(w) = {w} + out(w) of those terms divided by
      a sum of the 1/d(v) (each rounded once):
        1 + rho_r(w) = (1 + max_{S(w)} rho_q)(1 + gamma(|S(w)|))(1 + u)
                       / (1 - ((1 + u)(1 + gamma(|S(w)|)) - 1)).
    Both the GPU and the oracle are within rho(w) r_exact(w), so they differ
    by at most 2 rho(w) r_exact(w)."""
    n = g.n
    din = np.diff(g.in_off).astype(np.int64)
    dout = np.diff(g.row_off).astype(np.int64)
    d = din + 1
    s = dout + 1
    rho = np.zeros(n)

    def list_max(own, off, idx, lens):
        # max of own[v] and x[idx[k]] over v's list (lists are contiguous)
        out = own.copy()
        if idx.size:
            nz = lens > 0
            seg = np.maximum.reduceat(own[idx], off[:-1][nz])
            out[nz] = np.maximum(out[nz], seg)
        return out

    for _ in range(updates):
        m = list_max(rho, g.in_off, g.in_src, din)
        rq = (1 + m) * (1 + _gamma(d)) * (1 + U64) ** 2 - 1
        mq = list_max(rq, g.row_off, g.col_dst, dout)
        den = (1 + U64) * (1 + _gamma(s)) - 1
        rho = (1 + mq) * (1 + _gamma(s)) * (1 + U64) / (1 - den) - 1
    return rho


def check_ta(g, gpu, ora, tag=""):
    """Alg. 1 on the GPU (api.TaOrder) against the oracle (oracle.TaResult),
    both after the same number of updates requested:
    - the same number of updates made;
    - positions within the rounding bound of ta_position_bound;
    - the GPU order ranks its own positions, ties by ID (bit-exact);
    - the GPU order sorts the oracle's positions except between positions
      closer than their two bounds (near ties may fall either way), and each
      vertex it ranks differently from the oracle sits at such a near tie;
    - C(pi) of the GPU's order equals the oracle's span of that order, J(pi)
      the oracle's dispersion of it within fp64 rounding; the bootstrap's
      C and J equal the oracle's.
    Returns the number of vertices whose rank differs from the oracle's."""
    import oracle as O
    n = g.n
    assert gpu.done == ora.done, (tag, gpu.done, ora.done)
    pos = gpu.positions.cpu().numpy()
    pi = gpu.pi.cpu().numpy()
    rho = ta_position_bound(g, ora.done)
    tol = 2 * rho / (1 - rho) * np.abs(ora.positions) + 1e-300
    err = np.abs(pos - ora.positions)
    assert np.all(err <= tol), (tag, float((err / tol).max()), int(np.argmax(err / tol)))
    order = np.argsort(pi, kind="stable")
    assert np.array_equal(np.sort(pi), np.arange(n)), tag
    assert np.array_equal(order, np.lexsort((np.arange(n), pos))), tag
    ro = ora.positions[order]
    slack = tol[order][:-1] + tol[order][1:]
    gaps = ro[1:] - ro[:-1]
    assert np.all(gaps >= -slack), (tag, float(gaps.min()))
    t = ora.done
    assert gpu.spans[t] == O.total_span(g, pi), tag
    assert gpu.disp[t] == pytest_approx(O.dispersion(g, pi.astype(np.float64)), 1e-9), tag
    assert gpu.spans[0] == ora.spans[0] and gpu.disp[0] == pytest_approx(ora.disp[0], 1e-9), tag
    wrong = np.nonzero(pi != ora.pi)[0]
    if wrong.size:
        at_rank = np.empty(n, np.int64)
        at_rank[ora.pi] = np.arange(n)
        other = at_rank[pi[wrong]]
        assert np.all(np.abs(ora.positions[wrong] - ora.positions[other]) <= tol[wrong] + tol[other]), tag
    return int(wrong.size)


def check_ta_updates(g, run_gpu, pi0, iterations, tag=""):
    """check_ta after every update: run_gpu(t) runs t updates on the GPU.
    Each prefix must repeat the full run's C and J (the GPU run is
    deterministic), and every update's order is checked against the oracle's
    run of that many updates.  Returns the full run and the ranks differing
    (near ties) after each update."""
    import oracle as O
    full = run_gpu(iterations)
    diffs = []
    for t in range(1, full.done + 1):
        got = full if t == full.done else run_gpu(t)
        assert got.done == t, (tag, t, got.done)
        assert np.array_equal(got.spans[:t + 1], full.spans[:t + 1]), (tag, t)
        assert np.array_equal(got.disp[:t + 1], full.disp[:t + 1]), (tag, t)
        diffs.append(check_ta(g, got, O.reorder_ta(g, pi0, t), f"{tag} after {t}"))
    assert full.done == O.reorder_ta(g, pi0, iterations).done, tag
    return full, diffs


def pytest_approx(x, rel):
    import pytest
    return pytest.approx(x, rel=rel, abs=0)
