"""Vertex orderings (degree/BFS, RCMK, the topology-aware Alg. 1),
relabelling and row permutation on the GPU vs the oracle (needs an MI355X)."""
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


def _simple(n, u, v):
    keep = u != v
    pairs = np.unique(np.stack([u[keep], v[keep]], axis=1).astype(np.int64), axis=0)
    return pairs[:, 0].astype(np.int32), pairs[:, 1].astype(np.int32)


def _cases():
    rng = np.random.default_rng(42)
    out = []
    n = 3000   # sparse random digraph: many components, isolated vertices
    out.append(("sparse-random", n, *_simple(n, rng.integers(0, n, 2500), rng.integers(0, n, 2500))))
    n = 2000   # denser, a few hubs
    u = np.concatenate([rng.integers(0, n, 20000), rng.integers(0, n, 3000)])
    v = np.concatenate([rng.integers(0, n, 20000), rng.integers(0, 5, 3000)])
    out.append(("dense-hubs", n, *_simple(n, u, v)))
    n = 1500   # one long path (deep search) plus a reversed path
    u = np.concatenate([np.arange(0, 999), np.arange(1001, 1499)])
    v = np.concatenate([np.arange(1, 1000), np.arange(1000, 1498)])
    out.append(("paths", n, *_simple(n, u, v)))
    n = 700    # star into 0, star out of 1
    u = np.concatenate([np.arange(2, 700), np.full(300, 1)])
    v = np.concatenate([np.zeros(698, np.int64), np.arange(400, 700)])
    out.append(("stars", n, *_simple(n, u, v)))
    out.append(("edgeless", 500, np.zeros(0, np.int32), np.zeros(0, np.int32)))
    n = 2500   # half the edges reciprocated: pairs that symmetrise to one neighbour
    u, v = rng.integers(0, n, 6000), rng.integers(0, n, 6000)
    back = rng.random(6000) < 0.5
    out.append(("reciprocal", n, *_simple(n, np.concatenate([u, v[back]]), np.concatenate([v, u[back]]))))
    return out


NCASES = 6


@pytest.mark.parametrize("case", range(NCASES))
def test_reorder_bit_exact(torch_cuda, case):
    import oracle as O
    import paper_2607_17374_amd as T
    name, n, src, dst = _cases()[case]
    _note(f"reorder {name}: n={n} e={src.size}")
    g = O.Graph(n, src, dst)
    s = torch_cuda.from_numpy(src).cuda()
    d = torch_cuda.from_numpy(dst).cuda()
    row_off, col_dst = T.build_csr(n, s, d)
    pi = T.reorder(n, row_off, col_dst).cpu().numpy()
    want = O.reorder_bfs(g)
    assert np.array_equal(pi, want)
    # relabelled CSR equals the oracle's CSR of the renamed edge list
    r2, c2 = T.relabel_graph(n, row_off, col_dst, torch_cuda.from_numpy(pi).cuda())
    g2 = O.Graph(n, want[src], want[dst])
    assert np.array_equal(r2.cpu().numpy(), g2.row_off)
    assert np.array_equal(c2.cpu().numpy(), g2.col_dst)


def test_reorder_skewed_rmat_random_ids(torch_cuda):
    """C5's recipe (skewed RMAT, random IDs) at 1/400 of the vertices."""
    import oracle as O
    import paper_2607_17374_amd as T
    w = WL.GCN_SKEW_RMAT_50M.scaled(n=1 << 17, e=1 << 21, chunk=8192)
    src, dst = WL.graph(w)
    _note(f"reorder {w.name}")
    g = O.Graph(w.n, src, dst)
    row_off, col_dst = T.build_csr(w.n, torch_cuda.from_numpy(src).cuda(), torch_cuda.from_numpy(dst).cuda())
    pi = T.reorder(w.n, row_off, col_dst).cpu().numpy()
    assert np.array_equal(pi, O.reorder_bfs(g))
    ident = np.arange(w.n, dtype=np.int32)
    assert O.total_span(g, pi) < O.total_span(g, ident)


def test_permute_rows_round_trip(torch_cuda):
    import paper_2607_17374_amd as T
    torch = torch_cuda
    rng = np.random.default_rng(3)
    n = 5000
    perm = rng.permutation(n).astype(np.int32)
    p = torch.from_numpy(perm).cuda()
    for width, dt in ((256, torch.float16), (3, torch.float32), (128, torch.float32)):
        _note(f"permute rows width {width} {dt}")
        x = torch.randn(n, width, device="cuda").to(dt)
        y = T.permute_rows(x, p)
        xn, yn = x.cpu().numpy(), y.cpu().numpy()
        assert np.array_equal(yn[perm], xn)
        back = T.permute_rows(y, p, inverse=True)
        assert torch.equal(back, x)


def test_reordered_fp16_gcn_matches_original_ids(torch_cuda):
    """C5 shape: GCN fp16 256 -> 256 -> 64 over a skewed RMAT graph with
    random IDs, run again after the degree/BFS reordering; the reordered run,
    un-permuted, matches the oracle in the original IDs."""
    import oracle as O
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import torch_dtype
    torch = torch_cuda
    w = WL.GCN_SKEW_RMAT_50M.scaled(n=1 << 15, e=1 << 19, chunk=4096)
    src, dst = WL.graph(w)
    _note(f"{w.name}: oracle")
    g, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    xh = WL.input_features(w)
    X = torch.from_numpy(xh.view(np.int16)).cuda().view(torch_dtype(w.feat_dtype))
    _note("reorder, relabel, permute features")
    pi = T.reorder(w.n, row_off, col_dst)
    r2, c2 = T.relabel_graph(w.n, row_off, col_dst, pi)
    X2 = T.permute_rows(X, pi)
    outs, _ = H.gpu_model(w, r2, c2, X=X2)
    for li, (o, z) in enumerate(zip(outs, zs), start=1):
        back = T.permute_rows(o, pi, inverse=True)
        _, out_dt = w.layer_dtypes(li)
        r = H.compare(H.to_numpy_f64(back, out_dt), z, H.RTOL[w.feat_dtype])
        assert r["n_bad"] == 0, (li, r)
    assert O.total_span(g, pi.cpu().numpy()) < O.total_span(g, np.arange(w.n, dtype=np.int32))


def test_reorder_error_paths(torch_cuda):
    import paper_2607_17374_amd as T
    torch = torch_cuda
    _note("reorder / relabel / permute errors")
    n = 100
    src = np.arange(1, n, dtype=np.int32)
    dst = np.zeros(n - 1, dtype=np.int32)
    row_off, col_dst = T.build_csr(n, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda())
    bad = torch.zeros(n, dtype=torch.int32, device="cuda")        # not a permutation
    with pytest.raises(T.TaurusError) as ex:
        T.relabel_graph(n, row_off, col_dst, bad)
    assert ex.value.status == -1
    with pytest.raises(T.TaurusError) as ex:
        T.permute_rows(torch.zeros(n, 4, device="cuda"), bad)
    assert ex.value.status == -1
    broken = col_dst.clone()
    broken[0] = n + 5                                               # destination out of range
    with pytest.raises(T.TaurusError) as ex:
        T.reorder(n, row_off, broken)
    assert ex.value.status == -1


@pytest.mark.parametrize("case", range(NCASES))
def test_reorder_rcm_bit_exact(torch_cuda, case):
    """RCMK order of the symmetrised graph: bit for bit against the oracle."""
    import oracle as O
    import paper_2607_17374_amd as T
    name, n, src, dst = _cases()[case]
    _note(f"reorder_rcm {name}: n={n} e={src.size}")
    g = O.Graph(n, src, dst)
    row_off, col_dst = T.build_csr(n, torch_cuda.from_numpy(src).cuda(), torch_cuda.from_numpy(dst).cuda())
    pi = T.reorder_rcm(n, row_off, col_dst)
    assert np.array_equal(pi.cpu().numpy(), O.reorder_rcm(g))
    if src.size:
        broken = col_dst.clone()
        broken[0] = n + 5
        with pytest.raises(T.TaurusError) as ex:
            T.reorder_rcm(n, row_off, broken)
        assert ex.value.status == -1


@pytest.mark.parametrize("case", range(NCASES))
@pytest.mark.parametrize("boot", ["identity", "bfs", "rcm"])
def test_reorder_ta_matches_oracle(torch_cuda, case, boot):
    """Alg. 1 (topology-aware order) against the oracle: the same number of
    updates, positions within the fp64 rounding bound, an order that ranks
    the oracle's positions (near ties aside), and C(pi), J(pi) of each
    update's order."""
    import oracle as O
    import paper_2607_17374_amd as T
    name, n, src, dst = _cases()[case]
    _note(f"reorder_ta {name} from {boot}: n={n} e={src.size}")
    g = O.Graph(n, src, dst)
    row_off, col_dst = T.build_csr(n, torch_cuda.from_numpy(src).cuda(), torch_cuda.from_numpy(dst).cuda())
    p0 = {"identity": lambda: None, "bfs": lambda: O.reorder_bfs(g), "rcm": lambda: O.reorder_rcm(g)}[boot]()
    p0d = None if p0 is None else torch_cuda.from_numpy(p0).cuda()
    got, diffs = H.check_ta_updates(g, lambda t: T.reorder_ta(n, row_off, col_dst, p0d, t), p0, 6,
                                    f"{name}/{boot}")
    _note(f"  updates {got.done}, spans {got.spans[:got.done + 1].tolist()}, ranks differing (near ties) {diffs}")


def test_reorder_ta_worked_example(torch_cuda):
    """The two-update example worked by hand (tests/golden): positions carried
    across updates reverse vertices 0 and 1 in the second update."""
    import paper_2607_17374_amd as T
    from tests.test_oracle_pins import _golden_alg1
    from tests.conftest import ROOT
    import os
    n, edges, fr, it = _golden_alg1(os.path.join(ROOT, "tests", "golden"))
    e = np.array(edges, np.int32)
    row_off, col_dst = T.build_csr(n, torch_cuda.from_numpy(e[:, 0].copy()).cuda(),
                                   torch_cuda.from_numpy(e[:, 1].copy()).cuda())
    _note("reorder_ta worked example")
    got = T.reorder_ta(n, row_off, col_dst, None, 2)
    assert got.done == 2 and got.pi.cpu().numpy().tolist() == it("pi2")
    assert np.allclose(got.positions.cpu().numpy(), fr("r2"), rtol=1e-15, atol=0)
    assert got.spans.tolist() == it("spans")
    assert np.allclose(got.disp, fr("disp"), rtol=1e-15, atol=0)


def test_reorder_ta_hub_pieces(torch_cuda):
    """Lists long enough to be cut into pieces on the GPU (a hub receiving
    from and sending to 9,000 vertices, beside a sparse random graph)."""
    import oracle as O
    import paper_2607_17374_amd as T
    rng = np.random.default_rng(7)
    n = 20000
    u = np.concatenate([rng.integers(1, n, 30000), np.arange(1, 9001), np.zeros(9000, np.int64)])
    v = np.concatenate([rng.integers(1, n, 30000), np.zeros(9000, np.int64), np.arange(10001, 19001)])
    src, dst = _simple(n, u, v)
    _note(f"reorder_ta hub pieces: n={n} e={src.size}")
    g = O.Graph(n, src, dst)
    row_off, col_dst = T.build_csr(n, torch_cuda.from_numpy(src).cuda(), torch_cuda.from_numpy(dst).cuda())
    boot = rng.permutation(n).astype(np.int32)
    bd = torch_cuda.from_numpy(boot).cuda()
    got, diffs = H.check_ta_updates(g, lambda t: T.reorder_ta(n, row_off, col_dst, bd, t), boot, 5, "hub pieces")
    _note(f"  spans {got.spans[:got.done + 1].tolist()}, ranks differing (near ties) {diffs}")


def test_reorder_ta_skewed_rmat_model(torch_cuda):
    """C5's recipe (skewed RMAT, random IDs, fp16 GCN) at 1/400 of the
    vertices: the RCMK order bit-exact with the oracle, Alg. 1 from it and
    from the degree/BFS order against the oracle, each lowering the total
    span; the model on the Alg. 1 relabelled graph, un-permuted, matches the
    oracle in the original IDs."""
    import oracle as O
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import torch_dtype
    torch = torch_cuda
    w = WL.GCN_SKEW_RMAT_50M.scaled(n=1 << 17, e=1 << 21, chunk=8192)
    src, dst = WL.graph(w)
    _note(f"reorder_ta {w.name}")
    g, zs = H.oracle_model(w, src, dst)
    row_off, col_dst = H.gpu_graph(w, src, dst)
    rcm = T.reorder_rcm(w.n, row_off, col_dst)
    assert np.array_equal(rcm.cpu().numpy(), O.reorder_rcm(g))
    for bname, boot in (("rcm", rcm), ("bfs", T.reorder(w.n, row_off, col_dst))):
        got, diffs = H.check_ta_updates(g, lambda t: T.reorder_ta(w.n, row_off, col_dst, boot, t),
                                        boot.cpu().numpy(), 5, bname)
        _note(f"  from {bname}: spans {got.spans[:got.done + 1].tolist()}, J {got.disp[:got.done + 1].tolist()}, "
              f"ranks differing (near ties) {diffs}")
        assert got.spans[got.done] < got.spans[0] and got.disp[got.done] < got.disp[0]
    pi = got.pi
    r2, c2 = T.relabel_graph(w.n, row_off, col_dst, pi)
    xh = WL.input_features(w)
    X2 = T.permute_rows(torch.from_numpy(xh.view(np.int16)).cuda().view(torch_dtype(w.feat_dtype)), pi)
    outs, _ = H.gpu_model(w, r2, c2, X=X2)
    for li, (o, z) in enumerate(zip(outs, zs), start=1):
        back = T.permute_rows(o, pi, inverse=True)
        _, out_dt = w.layer_dtypes(li)
        r = H.compare(H.to_numpy_f64(back, out_dt), z, H.RTOL[w.feat_dtype])
        assert r["n_bad"] == 0, (li, r)


def test_reorder_ta_error_paths(torch_cuda):
    import paper_2607_17374_amd as T
    torch = torch_cuda
    _note("reorder_ta errors")
    n = 100
    src = np.arange(1, n, dtype=np.int32)
    dst = np.zeros(n - 1, dtype=np.int32)
    row_off, col_dst = T.build_csr(n, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda())
    for bad in (torch.zeros(n, dtype=torch.int32, device="cuda"),            # repeated ranks
                torch.arange(1, n + 1, dtype=torch.int32, device="cuda")):   # a rank out of range
        with pytest.raises(T.TaurusError) as ex:
            T.reorder_ta(n, row_off, col_dst, bad, 3)
        assert ex.value.status == -1
    with pytest.raises(T.TaurusError) as ex:
        T.reorder_ta(n, row_off, col_dst, None, 0)
    assert ex.value.status == -1
