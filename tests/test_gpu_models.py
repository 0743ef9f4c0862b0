"""GIN layers (sum and perceptron apply; exact and sampled), sampled GCN and
GAT layers on the GPU vs the oracle (needs an MI355X)."""
import dataclasses
import sys

import numpy as np
import pytest

import fixtures as F
from fixtures import workloads as WL
from tests import harness as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _note(msg):
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def _graph(rng, n):
    """Simple digraph with in-degrees 0, small, medium and one vertex fed by
    nearly every other vertex."""
    pairs = set()
    for v in range(n):
        r = rng.random()
        d = 0 if r < 0.2 else int(rng.integers(1, 16)) if r < 0.7 else int(rng.integers(16, 200))
        for u in rng.choice(n, size=min(d, n - 1), replace=False):
            if u != v:
                pairs.add((int(u), v))
    hub = int(rng.integers(0, n))
    for u in range(n):
        if u != hub and rng.random() < 0.9:
            pairs.add((u, hub))
    a = np.array(sorted(pairs), dtype=np.int32)
    return a[:, 0].copy(), a[:, 1].copy()


@pytest.mark.parametrize("agg,k", [(WL.GIN_SUM, 0), (WL.GIN_SUM, 5), (WL.GIN_SUM, 15),
                                   (WL.GCN_SYM, 1), (WL.GCN_SYM, 5), (WL.GCN_SYM, 15)])
def test_layer_matches_oracle(torch_cuda, agg, k):
    """One fp32 layer (d 48 -> 40, bias, ReLU) over 3,000 vertices in three
    chunks, every row against the oracle (the sampled GCN normalised by the
    sampled graph's degrees)."""
    import oracle as O
    import paper_2607_17374_amd as T
    torch = torch_cuda
    rng = np.random.default_rng(300 + 10 * agg + k)
    n, d_in, d_out, seed, layer = 3000, 48, 40, 77, 2
    src, dst = _graph(rng, n)
    _note(f"agg {agg} fanout {k}: n={n} e={src.size}")
    g = O.Graph(n, src, dst)
    X = rng.standard_normal((n, d_in)).astype(np.float32)
    W = (rng.standard_normal((d_out, d_in)) * 0.2).astype(np.float32)
    b = rng.standard_normal(d_out).astype(np.float32)
    row_off, col_dst = T.build_csr(n, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda())
    out = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    L = T.Layer(n, row_off, col_dst, agg=agg, d_in=d_in, d_out=d_out, weight_cat=np.ascontiguousarray(W.T), bias=b,
                out=out, relu=True, fanout=k, layer=layer, seed=seed, chunk=1024)
    L.push_all(torch.from_numpy(X).cuda())
    st = L.finalize()
    if k:
        words, kept = L.sampled_edges()
    L.destroy()
    keep = None
    if k:
        want, keep, m = O.sample(g, seed, layer, k)
        assert np.array_equal(words, want) and kept == int(m.sum()) == st["messages"]
    z = O.layer(agg, g, X, O.F32, W.astype(np.float64), b.astype(np.float64), True, keep_in=keep)
    r = H.compare(out.cpu().numpy(), z, H.RTOL[F.F32])
    assert r["n_bad"] == 0, r


@pytest.mark.parametrize("agg,dtype", [(WL.GIN_SUM, F.F32), (WL.GIN_SUM, F.BF16), (WL.GCN_SYM, F.BF16)])
def test_sampled_model_on_rmat(torch_cuda, agg, dtype):
    """A 2-layer model with fanouts (10, 5) on the RMAT recipe of the
    in-memory workload at 1/16 of its vertices and edges, in 8,192-vertex
    chunks, every row of each layer against the oracle fed its own previous
    layer."""
    import oracle as O
    torch = torch_cuda
    w = dataclasses.replace(WL.GCN_RMAT_1M, agg=agg, feat_dtype=dtype, fanouts=(10, 5)).scaled(
        n=1_000_000 // 16, e=20_000_000 // 16, chunk=8192, name=f"rmat-1m-div16-agg{agg}-{dtype}")
    _note(f"{w.name}")
    src, dst = WL.graph(w)
    g, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, stats = H.gpu_model(w, row_off, col_dst)
    for li, (o, z, st) in enumerate(zip(outs, zs, stats), start=1):
        _, keep, m = O.sample(g, w.seed, li, w.fanout(li))
        assert st["messages"] == int(m.sum())
        _, out_dt = w.layer_dtypes(li)
        r = H.compare(H.to_numpy_f64(o, out_dt), z, H.RTOL[dtype])
        _note(f"  layer {li}: {r['n_bad']} bad, max abs {r['max_abs']:.2e}")
        assert r["n_bad"] == 0, (li, r)


def test_gin_closed_form_and_unknown_family(torch_cuda):
    """GIN with unit features and weights counts each vertex's in-degree
    plus one; an unknown family (5) is refused."""
    import paper_2607_17374_amd as T
    torch = torch_cuda
    n = 100
    src = np.arange(1, n, dtype=np.int32)
    dst = np.zeros(n - 1, dtype=np.int32)
    row_off, col_dst = T.build_csr(n, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda())
    out = torch.empty((n, 4), dtype=torch.float32, device="cuda")
    with pytest.raises(T.TaurusError) as ex:
        T.Layer(n, row_off, col_dst, agg=5, d_in=8, d_out=4, weight_cat=np.zeros((8, 4), np.float32), bias=None,
                out=out, chunk=64)
    assert ex.value.status == -1
    L = T.Layer(n, row_off, col_dst, agg=WL.GIN_SUM, d_in=8, d_out=4, weight_cat=np.ones((8, 4), np.float32),
                bias=None, out=out, chunk=64)
    L.push_all(torch.ones((n, 8), dtype=torch.float32, device="cuda"))
    L.finalize()
    L.destroy()
    # vertex 0 sums 99 sources and itself: 100 * 8 per output; the others 8
    got = out.cpu().numpy()
    assert np.all(got[0] == 800.0) and np.all(got[1:] == 8.0)


@pytest.mark.parametrize("k", [0, 5])
def test_gat_layer_matches_oracle(torch_cuda, k):
    """One single-head GAT layer (d 48 -> 40, bias, ReLU), exact and with
    fanout 5, over 3,000 vertices in three chunks; the hub's segments are cut
    into pieces, so the piece statistics and the fix-up run.  Every row
    against the oracle."""
    import oracle as O
    import paper_2607_17374_amd as T
    torch = torch_cuda
    rng = np.random.default_rng(400 + k)
    n, d_in, d_out, seed, layer = 3000, 48, 40, 31, 1
    src, dst = _graph(rng, n)
    _note(f"gat fanout {k}: n={n} e={src.size}")
    g = O.Graph(n, src, dst)
    X = rng.standard_normal((n, d_in)).astype(np.float32)
    W = (rng.standard_normal((d_out, d_in)) * 0.2).astype(np.float32)
    attn = rng.standard_normal((2, d_out)).astype(np.float32)
    b = rng.standard_normal(d_out).astype(np.float32)
    row_off, col_dst = T.build_csr(n, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda())
    out = torch.empty((n, d_out), dtype=torch.float32, device="cuda")
    L = T.Layer(n, row_off, col_dst, agg=WL.GAT_ATT, d_in=d_in, d_out=d_out, weight_cat=np.ascontiguousarray(W.T),
                bias=b, out=out, relu=True, fanout=k, layer=layer, seed=seed, chunk=1024, attn=attn)
    L.push_all(torch.from_numpy(X).cuda())
    st = L.finalize()
    L.destroy()
    assert st["completed"] == n and (k or st["split_segments"] > 0)   # exact: the hub's segments are split
    keep = O.sample(g, seed, layer, k)[1] if k else None
    z = O.gat_layer(g, X, O.F32, W.astype(np.float64), attn.astype(np.float64), b.astype(np.float64), True,
                    keep_in=keep)
    r = H.compare(out.cpu().numpy(), z, H.RTOL[F.F32])
    assert r["n_bad"] == 0, r


@pytest.mark.parametrize("dtype,fanouts", [(F.F32, ()), (F.BF16, ()), (F.F32, (10, 5))])
def test_gat_model_on_rmat(torch_cuda, dtype, fanouts):
    """A 2-layer GAT on the RMAT recipe of the in-memory workload at 1/16,
    8,192-vertex chunks, every row of each layer against the oracle fed its
    own previous layer."""
    torch = torch_cuda
    w = dataclasses.replace(WL.GCN_RMAT_1M, agg=WL.GAT_ATT, feat_dtype=dtype, fanouts=fanouts).scaled(
        n=1_000_000 // 16, e=20_000_000 // 16, chunk=8192, name=f"gat-rmat-1m-div16-{dtype}-{len(fanouts)}")
    _note(w.name)
    src, dst = WL.graph(w)
    g, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, stats = H.gpu_model(w, row_off, col_dst)
    for li, (o, z) in enumerate(zip(outs, zs), start=1):
        _, out_dt = w.layer_dtypes(li)
        r = H.compare(H.to_numpy_f64(o, out_dt), z, H.RTOL[dtype])
        _note(f"  layer {li}: {r['n_bad']} bad, max abs {r['max_abs']:.2e}")
        assert r["n_bad"] == 0, (li, r)


def test_gat_argument_errors(torch_cuda):
    import paper_2607_17374_amd as T
    torch = torch_cuda
    n = 100
    src = np.arange(1, n, dtype=np.int32)
    dst = np.zeros(n - 1, dtype=np.int32)
    row_off, col_dst = T.build_csr(n, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda())
    out = torch.empty((n, 4), dtype=torch.float32, device="cuda")
    base = dict(agg=WL.GAT_ATT, d_in=8, d_out=4, weight_cat=np.zeros((8, 4), np.float32), bias=None, out=out,
                chunk=64)
    for bad in (dict(), dict(attn=np.zeros((2, 4), np.float32), hbm_budget=1 << 30)):
        with pytest.raises(T.TaurusError) as ex:
            T.Layer(n, row_off, col_dst, **dict(base, **bad))
        assert ex.value.status == -1, bad


@pytest.mark.parametrize("k,dtype,out_dtype,d_hidden,d_out", [
    (0, F.F32, F.F32, 72, 40), (5, F.F32, F.F32, 136, 200), (0, F.BF16, F.BF16, 64, 48),
    (15, F.F32, F.BF16, 32, 40), (1, F.F16, F.F32, 256, 132)])
def test_gin_mlp_layer_matches_oracle(torch_cuda, k, dtype, out_dtype, d_hidden, d_out):
    """GIN with a two-layer perceptron apply (d_in 48 -> d_hidden -> d_out,
    both biases, ReLU after each layer), exact and sampled, over 3,000
    vertices in three chunks (the last ragged): every row against the
    oracle.  Widths above 128 put the second layer's columns in several
    workgroup panels."""
    import oracle as O
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import torch_dtype
    torch = torch_cuda
    rng = np.random.default_rng(500 + 7 * k + d_hidden)
    n, d_in, seed, layer = 3000, 48, 91, 2
    src, dst = _graph(rng, n)
    _note(f"gin-mlp fanout {k} dtype {dtype}->{out_dtype} d {d_in}->{d_hidden}->{d_out}: n={n} e={src.size}")
    g = O.Graph(n, src, dst)
    X = rng.standard_normal((n, d_in)).astype(np.float32)
    W1 = (rng.standard_normal((d_hidden, d_in)) * 0.2).astype(np.float32)
    b1 = rng.standard_normal(d_hidden).astype(np.float32)
    W2 = (rng.standard_normal((d_out, d_hidden)) * (1.0 / np.sqrt(d_hidden))).astype(np.float32)
    b2 = rng.standard_normal(d_out).astype(np.float32)
    if dtype != F.F32:   # 16-bit storage of the inputs and the first layer's weights
        Xh = F.round16(X, dtype)
        W1 = F.bits_to_float(F.round16(W1, dtype), dtype).reshape(W1.shape)
        x = torch.from_numpy(Xh.view(np.int16)).cuda().view(torch_dtype(dtype))
        H_in = Xh
    else:
        x = torch.from_numpy(X).cuda()
        H_in = X
    row_off, col_dst = T.build_csr(n, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda())
    out = torch.empty((n, d_out), dtype=torch_dtype(out_dtype), device="cuda")
    L = T.Layer(n, row_off, col_dst, agg=WL.GIN_MLP, d_in=d_in, d_out=d_out, weight_cat=np.ascontiguousarray(W1.T),
                bias=b1, out=out, in_dtype=dtype, out_dtype=out_dtype, relu=True, fanout=k, layer=layer,
                seed=seed, chunk=1024, d_hidden=d_hidden, weight2=np.ascontiguousarray(W2.T), bias2=b2)
    L.push_all(x)
    st = L.finalize()
    L.destroy()
    assert st["completed"] == n and st["pending_left"] == 0
    keep = O.sample(g, seed, layer, k)[1] if k else None
    z = O.gin_mlp_layer(g, H_in, dtype, W1.astype(np.float64), b1.astype(np.float64), W2.astype(np.float64),
                        b2.astype(np.float64), True, keep_in=keep)
    tol = H.RTOL[F.F32] if dtype == F.F32 and out_dtype == F.F32 else H.RTOL[F.BF16]
    r = H.compare(H.to_numpy_f64(out, out_dtype), z, tol)
    assert r["n_bad"] == 0, r


@pytest.mark.parametrize("dtype,fanouts", [(F.F32, ()), (F.BF16, (10, 5))])
def test_gin_mlp_model_on_rmat(torch_cuda, dtype, fanouts):
    """A 2-layer GIN with perceptron apply on the RMAT recipe of the
    in-memory workload at 1/16, 8,192-vertex chunks: every row of each layer
    against the oracle fed its own previous layer."""
    torch = torch_cuda
    w = dataclasses.replace(WL.GCN_RMAT_1M, agg=WL.GIN_MLP, feat_dtype=dtype, fanouts=fanouts).scaled(
        n=1_000_000 // 16, e=20_000_000 // 16, chunk=8192, name=f"gin-mlp-rmat-1m-div16-{dtype}-{len(fanouts)}")
    _note(w.name)
    src, dst = WL.graph(w)
    g, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, stats = H.gpu_model(w, row_off, col_dst)
    for li, (o, z) in enumerate(zip(outs, zs), start=1):
        _, out_dt = w.layer_dtypes(li)
        r = H.compare(H.to_numpy_f64(o, out_dt), z, H.RTOL[dtype])
        _note(f"  layer {li}: {r['n_bad']} bad, max abs {r['max_abs']:.2e}")
        assert r["n_bad"] == 0, (li, r)


def test_gin_mlp_argument_errors(torch_cuda):
    """A perceptron layer needs a hidden width (positive, a multiple of 4,
    at most 1024), its second layer's weights and no budget; arrays of the
    wrong size are refused by the binding before the library reads them."""
    import paper_2607_17374_amd as T
    torch = torch_cuda
    n = 100
    src = np.arange(1, n, dtype=np.int32)
    dst = np.zeros(n - 1, dtype=np.int32)
    row_off, col_dst = T.build_csr(n, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda())
    out = torch.empty((n, 4), dtype=torch.float32, device="cuda")

    def base(dh):
        return dict(agg=WL.GIN_MLP, d_in=8, d_out=4, weight_cat=np.zeros((8, dh), np.float32), bias=None,
                    out=out, chunk=64, d_hidden=dh, weight2=np.zeros((dh, 4), np.float32))
    for dh, bad in ((8, dict(weight2=None)), (8, dict(hbm_budget=1 << 30)), (6, {}), (1028, {}), (0, {})):
        with pytest.raises(T.TaurusError) as ex:
            T.Layer(n, row_off, col_dst, **dict(base(dh), **bad))
        assert ex.value.status == -1, (dh, bad)
    with pytest.raises(ValueError):
        T.Layer(n, row_off, col_dst, **dict(base(8), weight2=np.zeros((4, 4), np.float32)))
