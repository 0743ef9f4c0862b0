"""Fanout sampler and 16-bit layer inputs on the GPU vs the oracle (needs an MI355X)."""
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


def _degree_mix_graph(rng, n):
    """Simple digraph whose in-degrees span 0, <= 15, (15, 64], (64, 1000] and
    one vertex fed by nearly every other vertex (a hub far above 64)."""
    pairs = set()
    for v in range(n):
        r = rng.random()
        d = 0 if r < 0.2 else int(rng.integers(1, 16)) if r < 0.7 else int(rng.integers(16, 65)) if r < 0.95 \
            else int(rng.integers(65, 1000))
        for u in rng.choice(n, size=min(d, n - 1), replace=False):
            if u != v:
                pairs.add((int(u), v))
    hub = int(rng.integers(0, n))
    for u in range(n):
        if u != hub and rng.random() < 0.9:
            pairs.add((u, hub))
    a = np.array(sorted(pairs), dtype=np.int32)
    return a[:, 0].copy(), a[:, 1].copy()


def _device_edges(torch, src, dst):
    return torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda()


def _gpu_mask(torch, n, row_off, col_dst, k, layer, seed, plan=None, chunk=1024):
    """Mask of a sampled GraphSAGE layer, read right after init."""
    import paper_2607_17374_amd as T
    out = torch.empty((n, 4), dtype=torch.float32, device="cuda")
    L = T.Layer(n, row_off, col_dst, agg=WL.SAGE_MEAN, d_in=8, d_out=4, weight_cat=np.zeros((8, 8), np.float32),
                bias=None, out=out, fanout=k, layer=layer, seed=seed, chunk=chunk, plan=plan)
    words, kept = L.sampled_edges()
    L.destroy()
    return words, kept


@pytest.mark.parametrize("k", [1, 5, 15, 64, 65, 300, 512])
def test_sampler_mask_bit_exact(torch_cuda, k):
    import oracle as O
    import paper_2607_17374_amd as T
    rng = np.random.default_rng(100 + k)
    n = 3000
    src, dst = _degree_mix_graph(rng, n)
    _note(f"sampler mask k={k} n={n} e={src.size}")
    g = O.Graph(n, src, dst)
    row_off, col_dst = T.build_csr(n, *_device_edges(torch_cuda, src, dst))
    plan = T.Plan(n, row_off, col_dst, 1024)
    d_in = np.bincount(dst, minlength=n)
    for layer in (1, 2, 3):
        for seed in (7, 2**63 + 11):
            words, kept = _gpu_mask(torch_cuda, n, row_off, col_dst, k, layer, seed, plan=plan)
            want, keep_in, m = O.sample(g, seed, layer, k)
            assert np.array_equal(words, want), (k, layer, seed)
            assert kept == int(np.minimum(d_in, k).sum()) == int(m.sum())
    plan.destroy()


def test_sampler_without_plan_and_other_chunk(torch_cuda):
    import paper_2607_17374_amd as T
    rng = np.random.default_rng(5)
    n = 2000
    src, dst = _degree_mix_graph(rng, n)
    _note("sampler mask: plan / no plan / chunk size give the same mask")
    row_off, col_dst = T.build_csr(n, *_device_edges(torch_cuda, src, dst))
    a, _ = _gpu_mask(torch_cuda, n, row_off, col_dst, 10, 2, 99, plan=None, chunk=1024)
    plan = T.Plan(n, row_off, col_dst, 333)
    b, _ = _gpu_mask(torch_cuda, n, row_off, col_dst, 10, 2, 99, plan=plan, chunk=333)
    plan.destroy()
    assert np.array_equal(a, b)


def test_fanout_above_max_degree_equals_exact(torch_cuda):
    """k >= max in-degree keeps every edge, so the sampled layer is the exact one."""
    import paper_2607_17374_amd as T
    torch = torch_cuda
    w = WL.SAGE_RMAT_4K
    src, dst = WL.graph(w)
    keep = np.bincount(dst, minlength=w.n)[dst] <= 64   # drop the in-edges of vertices above 64
    src, dst = np.ascontiguousarray(src[keep]), np.ascontiguousarray(dst[keep])
    _note(f"fanout 64 >= max in-degree on {src.size} edges")
    row_off, col_dst = T.build_csr(w.n, *_device_edges(torch, src, dst))
    X = torch.from_numpy(WL.input_features(w)).cuda()
    spec = H.layer_specs(w)[0]
    outs = []
    for fanout in (0, 64):
        out = torch.empty((w.n, spec["d_out"]), dtype=torch.float32, device="cuda")
        s = dict(spec, fanout=fanout)
        L = T.Layer(w.n, row_off, col_dst, out=out, chunk=w.chunk, **s)
        words, kept = L.sampled_edges()
        assert kept == src.size
        L.push_all(X)
        L.finalize()
        L.destroy()
        outs.append(out.cpu().numpy())
    assert np.array_equal(outs[0], outs[1])


def _destination_sample(rng, g, count):
    d_in = np.diff(g.in_off)
    ids = set(rng.choice(g.n, size=min(count, g.n), replace=False).tolist())
    ids.update(np.argsort(-d_in, kind="stable")[:64].tolist())
    ids.update(np.flatnonzero(d_in == 0)[:64].tolist())
    return np.array(sorted(ids), dtype=np.int64)


def test_sampled_bf16_model_c3_shape(torch_cuda):
    """3-layer GraphSAGE-mean with fanouts (15, 10, 5), bf16 storage, widths
    128 -> 256 -> 256 -> 172 on an RMAT graph of the same recipe at 1/800 of
    the vertices.  Per layer: the mask bit-exact against the oracle's
    sampler, and a seeded destination sample (plus the top in-degrees and
    zero in-degree vertices) against the oracle, each layer fed the oracle's
    own previous layer."""
    import oracle as O
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import torch_dtype
    torch = torch_cuda
    w = WL.SAGE_FANOUT_RMAT_100M.scaled(n=1 << 17, e=16 << 17, chunk=16384)
    _note(f"{w.name}: n={w.n} e={w.e}")
    src, dst = WL.graph(w)
    g = O.Graph(w.n, src, dst)
    row_off, col_dst = T.build_csr(w.n, *_device_edges(torch, src, dst))
    xh = WL.input_features(w)
    X = torch.from_numpy(xh.view(np.int16)).cuda().view(torch_dtype(w.feat_dtype))
    plan = T.Plan(w.n, row_off, col_dst, w.chunk)
    rng = np.random.default_rng(31)
    h = X
    outs, all_ids, keeps = [], [], []
    for li, spec in enumerate(H.layer_specs(w), start=1):
        _note(f"  layer {li} fanout {spec['fanout']}")
        out = torch.empty((w.n, spec["d_out"]), dtype=torch_dtype(spec["out_dtype"]), device="cuda")
        L = T.Layer(w.n, row_off, col_dst, out=out, chunk=w.chunk, plan=plan, **spec)
        words, kept = L.sampled_edges()
        want, keep_in, m = O.sample(g, w.seed, li, spec["fanout"])
        assert np.array_equal(words, want), li
        L.push_all(h)
        st = L.finalize()
        L.destroy()
        assert st["messages"] == kept == int(m.sum())
        all_ids.append(_destination_sample(rng, g, 2048))
        keeps.append(keep_in)
        outs.append(out)
        h = out
    plan.destroy()
    zs = H.oracle_sampled_layers(w, g, xh, all_ids, keeps)
    for li, (out, ids, z, spec) in enumerate(zip(outs, all_ids, zs, H.layer_specs(w)), start=1):
        y = H.to_numpy_f64(out, spec["out_dtype"])[ids]
        r = H.compare(y, z, H.RTOL[w.feat_dtype])
        assert r["n_bad"] == 0, (li, r)


@pytest.mark.parametrize("base,dtype", [(WL.SAGE_RMAT_4K, F.BF16), (WL.SAGE_RMAT_4K, F.F16),
                                        (WL.GCN_RMAT_1M, F.F16), (WL.GCN_RMAT_1M, F.BF16)])
def test_16bit_inputs_exact_model(torch_cuda, base, dtype):
    """Exact models with 16-bit storage: the transform runs on the bf16/fp16
    matrix cores; every vertex of every layer against the oracle."""
    w = dataclasses.replace(base, feat_dtype=dtype, name=f"{base.name}-{dtype}")
    if w.n > 100_000:
        w = w.scaled(n=1 << 15, e=1 << 19, chunk=4096)
    _note(f"{w.name}: n={w.n} e={w.e}")
    src, dst = WL.graph(w)
    _, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, _ = H.gpu_model(w, row_off, col_dst)
    for li, (o, z) in enumerate(zip(outs, zs), start=1):
        _, out_dt = w.layer_dtypes(li)
        r = H.compare(H.to_numpy_f64(o, out_dt), z, H.RTOL[dtype])
        assert r["n_bad"] == 0, (li, r)


def test_sampling_error_paths(torch_cuda):
    import paper_2607_17374_amd as T
    torch = torch_cuda
    w = WL.SAGE_RMAT_4K
    _note("sampling and 16-bit argument errors")
    row_off, col_dst = H.gpu_graph(w)
    spec = H.layer_specs(w)[0]
    out = torch.empty((w.n, spec["d_out"]), dtype=torch.float32, device="cuda")
    for bad in (dict(fanout=513), dict(fanout=-1), dict(fanout=5, agg=7, weight_cat=np.zeros((64, 64), np.float32)),
                dict(fanout=5, layer=0), dict(in_dtype=F.BF16, d_in=60, weight_cat=np.zeros((60, 128), np.float32))):
        with pytest.raises(T.TaurusError) as ex:
            T.Layer(w.n, row_off, col_dst, out=out, chunk=1024, **dict(spec, **bad))
        assert ex.value.status == -1, bad
