"""GPU path vs the oracle, through the C ABI (needs an MI355X)."""
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


def _random_simple_graph(rng, n, e):
    u = rng.integers(0, n, size=e * 2, dtype=np.int64)
    v = rng.integers(0, n, size=e * 2, dtype=np.int64)
    keep = u != v
    key = np.unique(u[keep] * n + v[keep])
    rng.shuffle(key)
    key = key[:e]
    return (key // n).astype(np.int32), (key % n).astype(np.int32)


# ------------------------------------------------------------------ CSR ----

# the last case is sparse: runs of hundreds of empty rows between edges, the
# row offsets of long runs filled by the build's second pass
@pytest.mark.parametrize("n,e,seed", [(1, 0, 0), (5, 0, 1), (37, 200, 2), (1000, 20000, 3), (70000, 400000, 4),
                                      (1 << 20, 30000, 6)])
def test_csr_random_bit_exact(torch_cuda, n, e, seed):
    import oracle as O
    _note(f"csr random n={n} e={e} seed={seed}")
    rng = np.random.default_rng(seed)
    src, dst = _random_simple_graph(rng, n, e) if e else (np.zeros(0, np.int32), np.zeros(0, np.int32))
    w = WL.SAGE_RMAT_4K.scaled(n, len(src))
    row_off, col_dst = H.gpu_graph(w, src, dst)
    g = O.Graph(n, src, dst)
    assert np.array_equal(row_off.cpu().numpy(), g.row_off)
    assert np.array_equal(col_dst.cpu().numpy(), g.col_dst)


@pytest.mark.parametrize("w", [WL.SAGE_RMAT_4K, WL.GCN_RMAT_1M], ids=lambda w: w.name)
def test_csr_workload_bit_exact(torch_cuda, w):
    import oracle as O
    _note(f"csr workload {w.name}")
    src, dst = WL.graph(w)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    g = O.Graph(w.n, src, dst)
    assert np.array_equal(row_off.cpu().numpy(), g.row_off)
    assert np.array_equal(col_dst.cpu().numpy(), g.col_dst)


@pytest.mark.parametrize("bad", ["self_loop", "repeat", "range"])
def test_csr_rejects_non_simple(torch_cuda, bad):
    import paper_2607_17374_amd as T
    torch = torch_cuda
    _note(f"csr rejects {bad}")
    src = np.array([0, 1, 2, 3], np.int32)
    dst = np.array([1, 2, 3, 0], np.int32)
    if bad == "self_loop":
        dst[2] = 2
    elif bad == "repeat":
        src[3], dst[3] = 0, 1
    else:
        dst[1] = 9
    with pytest.raises(T.TaurusError) as ex:
        T.build_csr(5, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda())
    assert ex.value.status == -1


# -------------------------------------------------------------- layers -----

def _check_model(w, outs, zs, label):
    for li, (out, z) in enumerate(zip(outs, zs), start=1):
        _, out_dt = w.layer_dtypes(li)
        y = H.to_numpy_f64(out, out_dt)
        r = H.compare(y, z, H.RTOL[out_dt if out_dt != F.F32 else w.feat_dtype])
        assert r["n_bad"] == 0, f"{label} layer {li}: {r}"


def test_sage_small_workload_full(torch_cuda):
    w = WL.SAGE_RMAT_4K
    _note(f"layers {w.name} full")
    src, dst = WL.graph(w)
    _, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, stats = H.gpu_model(w, row_off, col_dst)
    _check_model(w, outs, zs, w.name)
    for st in stats:
        assert st["pending_left"] == 0 and st["completed"] == w.n
        assert st["messages"] == w.e and st["self_terms"] == w.n
        assert st["chunks_pushed"] == st["chunks"] == 4


@pytest.mark.parametrize("chunk", [1, 7, 1000, 4096, 10000])
@pytest.mark.parametrize("use_plan", [True, False])
def test_chunk_size_invariance(torch_cuda, chunk, use_plan):
    w = WL.SAGE_RMAT_4K
    _note(f"chunk invariance chunk={chunk} plan={use_plan}")
    src, dst = WL.graph(w)
    _, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, _ = H.gpu_model(w, row_off, col_dst, chunk=chunk, use_plan=use_plan)
    _check_model(w, outs, zs, f"chunk {chunk}")


def test_plan_mismatch_rejected(torch_cuda):
    import paper_2607_17374_amd as T
    torch = torch_cuda
    _note("plan mismatch")
    w = WL.SAGE_RMAT_4K
    row_off, col_dst = H.gpu_graph(w)
    plan = T.Plan(w.n, row_off, col_dst, 512)
    spec = H.layer_specs(w)[0]
    out = torch.empty((w.n, spec["d_out"]), dtype=torch.float32, device="cuda")
    with pytest.raises(T.TaurusError) as ex:
        T.Layer(w.n, row_off, col_dst, out=out, chunk=1024, plan=plan, **spec)
    assert ex.value.status == -1
    # a layer keeps the shared index alive after the plan is destroyed
    L = T.Layer(w.n, row_off, col_dst, out=out, chunk=512, plan=plan, **spec)
    plan.destroy()
    L.push_all(torch.from_numpy(WL.input_features(w)).cuda())
    assert L.finalize()["pending_left"] == 0
    L.destroy()


def test_chunk_order_invariance(torch_cuda):
    w = WL.SAGE_RMAT_4K
    _note("reverse and shuffled chunk order")
    src, dst = WL.graph(w)
    _, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, _ = H.gpu_model(w, row_off, col_dst, order=[3, 2, 1, 0])
    _check_model(w, outs, zs, "reverse")
    outs, _ = H.gpu_model(w, row_off, col_dst, order=[2, 0, 3, 1])
    _check_model(w, outs, zs, "shuffled")


def _expected_self_counts(src, dst, n, chunk, order):
    """Vertices without an in-edge from their own chunk (their self message
    is taken by the transform), and of those the ones whose self message
    comes before / after every other message when chunks are pushed in
    `order`: counted from the edge list."""
    pos = np.empty(len(order), np.int64)
    pos[np.asarray(order)] = np.arange(len(order))
    own_pos = pos[np.arange(n) // chunk]
    msg_pos = pos[src.astype(np.int64) // chunk]
    own_seg = np.zeros(n, bool)
    own_seg[dst[msg_pos == own_pos[dst]]] = True
    first = np.full(n, len(order), np.int64)
    last = np.full(n, -1, np.int64)
    np.minimum.at(first, dst, msg_pos)
    np.maximum.at(last, dst, msg_pos)
    alone = ~own_seg
    return (int(alone.sum()), int((alone & (first > own_pos)).sum()), int((alone & (last < own_pos)).sum()))


@pytest.mark.parametrize("order", ["ascending", "shuffled"])
def test_sage_self_messages_in_transform(torch_cuda, order):
    """In-core GraphSAGE: the transform takes the self messages of vertices
    with no in-edge from their own chunk; outputs match the oracle and the
    layer's counts of those messages (all, into an empty row, completing the
    vertex) match the edge list."""
    w = WL.SAGE_RMAT_4K
    chunk = 256
    nch = w.n // chunk
    seq = list(range(nch)) if order == "ascending" else [int(c) for c in np.random.default_rng(5).permutation(nch)]
    _note(f"self messages in the transform, chunk {chunk}, order {order}")
    src, dst = WL.graph(w)
    _, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, stats = H.gpu_model(w, row_off, col_dst, chunk=chunk, order=seq, profile=True)
    _check_model(w, outs, zs, f"chunk {chunk} {order}")
    want = _expected_self_counts(src, dst, w.n, chunk, seq)
    assert want[0] > 0 and want[1] > 0 and want[2] > 0, want
    for st in stats:
        assert (st["self_in_transform"], st["self_fresh"], st["self_last"]) == want
    # without profiling the counts are not taken
    _, stats = H.gpu_model(w, row_off, col_dst, chunk=chunk, order=seq)
    assert all((st["self_in_transform"], st["self_fresh"], st["self_last"]) == (want[0], -1, -1) for st in stats)


def test_gcn_scaled_workload(torch_cuda):
    w = WL.GCN_RMAT_1M.scaled(30000, 400000, chunk=4096)
    _note(f"layers {w.name}")
    src, dst = WL.graph(w)
    _, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, stats = H.gpu_model(w, row_off, col_dst)
    _check_model(w, outs, zs, w.name)
    assert all(st["split_segments"] > 0 for st in stats)   # hubs straddle tiles


@pytest.mark.parametrize("which", ["gcn-scaled", "sage-4k"])
def test_lean_index_build_same_lists(torch_cuda, which):
    """The memory-lean chunk-index build (work lists one at a time, used for
    large graphs) gives the same work lists as the single-scan build: the
    outputs are bit-identical and match the oracle."""
    import os
    w = WL.GCN_RMAT_1M.scaled(30000, 400000, chunk=4096) if which == "gcn-scaled" else WL.SAGE_RMAT_4K
    _note(f"lean index {w.name}")
    src, dst = WL.graph(w)
    _, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    got = {}
    try:
        for lean in ("0", "1"):
            os.environ["TAURUS_INDEX_LEAN"] = lean
            outs, stats = H.gpu_model(w, row_off, col_dst)
            got[lean] = ([o.cpu() for o in outs], stats)
    finally:
        os.environ.pop("TAURUS_INDEX_LEAN", None)
    for a, b in zip(got["0"][0], got["1"][0]):
        assert torch_cuda.equal(a, b)
    for sa, sb in zip(got["0"][1], got["1"][1]):
        for k in ("short_units", "wave_units", "split_segments", "pairs", "messages"):
            assert sa[k] == sb[k], k
    _check_model(w, got["1"][0], zs, f"{w.name} lean")


def test_gcn_full_size_bench_configuration(torch_cuda):
    """The benchmark workload (1M vertices, 20M edges, 64K chunks), every output row."""
    w = WL.GCN_RMAT_1M
    _note(f"layers {w.name} full size")
    src, dst = WL.graph(w)
    _, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, stats = H.gpu_model(w, row_off, col_dst, profile=True)
    _check_model(w, outs, zs, w.name)
    assert stats[0]["launches_scatter"] == 16


@pytest.mark.parametrize("d_out", [16, 32, 172, 256, 512, 1024])
@pytest.mark.parametrize("agg", [WL.SAGE_MEAN, WL.GCN_SYM])
def test_row_shapes(torch_cuda, d_out, agg):
    """Every row-group layout (4..64 lanes, 1..4 float4 per lane, masked lanes)."""
    import oracle as O
    _note(f"row shape d_out={d_out} agg={agg}")
    w = WL.Workload("shape", 3000, 40000, WL.RMAT_STD, F.UNIFORM, F.F32, agg, (64, d_out), chunk=512, seed=9)
    src, dst = WL.graph(w)
    _, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, _ = H.gpu_model(w, row_off, col_dst)
    _check_model(w, outs, zs, f"d_out {d_out}")


@pytest.mark.parametrize("out_dtype", [F.BF16, F.F16])
def test_16bit_outputs(torch_cuda, out_dtype):
    """Hidden outputs stored in 16 bits are the RNE rounding of the fp32 result."""
    import oracle as O
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import torch_dtype
    torch = torch_cuda
    _note(f"16-bit outputs {out_dtype}")
    w = WL.SAGE_RMAT_4K
    src, dst = WL.graph(w)
    g, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    spec = H.layer_specs(w)[0]
    spec["out_dtype"] = out_dtype
    X = torch.from_numpy(WL.input_features(w)).cuda()
    out = torch.empty((w.n, spec["d_out"]), dtype=torch_dtype(out_dtype), device="cuda")
    L = T.Layer(w.n, row_off, col_dst, out=out, chunk=w.chunk, **spec)
    L.push_all(X)
    L.finalize()
    L.destroy()
    y = out.to(torch.float64).cpu().numpy()
    r = H.compare(y, zs[0], 1e-2)
    assert r["n_bad"] == 0, r


def test_star_hub_spans_many_tiles(torch_cuda):
    """One destination with 20000 in-neighbours in one chunk: its segment
    spans ~20 scatter tiles and is completed by the fix-up pass."""
    _note("star hub")
    n = 30000
    src = np.arange(1, 20001, dtype=np.int32)
    dst = np.zeros(20000, np.int32)
    rng = np.random.default_rng(5)
    s2, d2 = _random_simple_graph(rng, n, 50000)
    key = np.unique(np.concatenate([src.astype(np.int64) * n + dst, s2.astype(np.int64) * n + d2]))
    src, dst = (key // n).astype(np.int32), (key % n).astype(np.int32)
    for agg in (WL.SAGE_MEAN, WL.GCN_SYM):
        w = WL.Workload("star", n, len(src), WL.RMAT_STD, F.NORMAL, F.F32, agg, (32, 64), chunk=32768, seed=3)
        _, zs = H.oracle_model(w, src, dst)
        row_off, col_dst = H.gpu_graph(w, src, dst)
        outs, stats = H.gpu_model(w, row_off, col_dst)
        _check_model(w, outs, zs, f"star agg={agg}")
        assert stats[0]["split_segments"] >= 1


def test_edgeless_and_isolated(torch_cuda):
    _note("edgeless graph")
    w = WL.Workload("empty", 100, 0, WL.RMAT_STD, F.UNIFORM, F.F32, WL.SAGE_MEAN, (8, 8), chunk=16, seed=1)
    src = np.zeros(0, np.int32)
    dst = np.zeros(0, np.int32)
    _, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, _ = H.gpu_model(w, row_off, col_dst)
    _check_model(w, outs, zs, "edgeless")


@pytest.mark.parametrize("fanouts", [(), (3, 2)], ids=["exact", "sampled"])
def test_sparse_graph_models(torch_cuda, fanouts):
    """A graph far sparser than a tile of 4,096 edges is rows (1M vertices,
    30K edges): the item kernels find rows by searching row_off between a
    tile's first and last rows, and the CSR and in-edge offsets fill long
    runs of empty rows in their second pass.  Both GraphSAGE layers, exact
    and sampled, equal the oracle."""
    import dataclasses
    _note(f"sparse graph fanouts={fanouts}")
    rng = np.random.default_rng(11)
    n, e = 1 << 20, 30000
    src, dst = _random_simple_graph(rng, n, e)
    w = dataclasses.replace(WL.SAGE_RMAT_4K.scaled(n, len(src), chunk=65536), fanouts=fanouts,
                            name=f"sparse-{len(fanouts)}")
    _, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    outs, stats = H.gpu_model(w, row_off, col_dst)
    _check_model(w, outs, zs, w.name)
    for st in stats:
        assert st["pending_left"] == 0 and st["completed"] == w.n


# --------------------------------------------------------- error paths -----

def test_error_paths(torch_cuda):
    import paper_2607_17374_amd as T
    torch = torch_cuda
    _note("error paths")
    w = WL.SAGE_RMAT_4K
    row_off, col_dst = H.gpu_graph(w)
    spec = H.layer_specs(w)[0]
    X = torch.from_numpy(WL.input_features(w)).cuda()
    out = torch.empty((w.n, spec["d_out"]), dtype=torch.float32, device="cuda")
    L = T.Layer(w.n, row_off, col_dst, out=out, chunk=1024, **spec)
    with pytest.raises(T.TaurusError) as ex:
        L.push_chunk(10, 1034, X[10:1034])                     # not a whole chunk
    assert ex.value.status == -1
    L.push_chunk(0, 1024, X[0:1024])
    with pytest.raises(T.TaurusError) as ex:
        L.push_chunk(0, 1024, X[0:1024])                       # pushed twice
    assert ex.value.status == -4
    L.push_chunk(1024, 2048, X[1024:2048])
    with pytest.raises(T.TaurusError) as ex:
        L.finalize()                                           # chunks 2, 3 missing
    assert ex.value.status == -5
    L.push_chunk(2048, 3072, X[2048:3072])
    L.push_chunk(3072, 4096, X[3072:4096])
    st = L.finalize()
    assert st["pending_left"] == 0
    words, kept = L.sampled_edges()
    assert kept == w.e and np.all(words[:-1] == np.uint64(2**64 - 1))
    L.destroy()
    # budget too small for the layer's structures
    with pytest.raises(T.TaurusError) as ex:
        T.Layer(w.n, row_off, col_dst, out=out, chunk=1024, hbm_budget=4096, **spec)
    assert ex.value.status == -6
