"""The library's chunk loader (taurus_stream_layer): host threads fill a
ring of pinned chunk buffers while the calling thread pushes them (needs an
MI355X)."""
import ctypes
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


# the out-of-core recipe (GraphSAGE-mean 512 -> 256, fp32, U[-1, 1)) small
W = dataclasses.replace(WL.SAGE_OOC_RMAT_269M, random_ids=True).scaled(n=1 << 15, e=1 << 19, chunk=1024)


@pytest.mark.parametrize("threads,ring,budget", [(3, 0, False), (1, 2, False), (4, 5, True)])
def test_loader_matches_device_pushes_and_oracle(torch_cuda, threads, ring, budget):
    """Layer 1 of the out-of-core recipe at 32K vertices fed by the loader
    (the seeded feature generator as its fill, on `threads` threads over a
    ring of `ring` pinned chunks; optionally under a budget that evicts)
    equals the run fed from device memory bit for bit, and 1,024 sampled
    destinations match the oracle."""
    import oracle as O
    import paper_2607_17374_amd as T
    torch = torch_cuda
    _note(f"loader threads {threads} ring {ring} budget {budget}")
    src, dst = WL.graph(W)
    row_off, col_dst = H.gpu_graph(W, src, dst)
    spec = H.layer_specs(W)[0]
    xh = WL.input_features(W)
    ref = torch.empty((W.n, spec["d_out"]), dtype=torch.float32, device="cuda")
    L = T.Layer(W.n, row_off, col_dst, out=ref, chunk=W.chunk, **spec)
    L.push_all(torch.from_numpy(xh).cuda())
    st0 = L.finalize()
    L.destroy()
    extra = {}
    if budget:  # a pool of a quarter of the rows beyond the hubs and one chunk's destinations
        from tests.test_gpu_resident import _max_chunk_destinations
        need = _max_chunk_destinations(src, dst, W.n, W.chunk)
        hubs = int(np.ceil(0.01 * W.n))
        slots = hubs + need + (W.n - hubs - need) // 4
        extra = dict(hbm_budget=H.pool_budget(st0, W.n, spec["d_out"], spec["d_in"], W.chunk, slots),
                     hub_fraction=0.01)
    out = torch.empty_like(ref)
    L = T.Layer(W.n, row_off, col_dst, out=out, chunk=W.chunk, **spec, **extra)
    fn, ctx = F.feature_fill(W.seed, W.feat_dist, W.dims[0], F.F32, threads=2)
    ls = L.stream(fn, ctx, threads=threads, ring=ring)
    st = L.finalize()
    L.destroy()
    nch = (W.n + W.chunk - 1) // W.chunk
    assert ls["chunks"] == nch and ls["bytes"] == W.n * W.dims[0] * 4, ls
    assert st["chunks_pushed"] == nch and st["pending_left"] == 0
    assert st["h2d_bytes"] >= W.n * W.dims[0] * 4
    if budget:
        assert st["evictions"] > 0, st
    assert torch.equal(out, ref)
    g = O.Graph(W.n, src, dst)
    ids = np.random.default_rng(5).choice(W.n, 1024, replace=False)
    p = WL.layer_params(W, 1)
    z = O.layer(W.agg, g, xh, F.F32, p.W, p.b, spec["relu"], dst_ids=ids)
    r = H.compare(out.cpu().numpy()[ids], z, H.RTOL[F.F32])
    assert r["n_bad"] == 0, r


def test_loader_python_fill_and_failure(torch_cuda):
    """A fill written in Python (a ctypes callback) gives the same output; a
    fill that returns nonzero stops the layer with TAURUS_E_INVALID naming
    the chunk, and the handle is poisoned afterwards."""
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd import _native as N
    torch = torch_cuda
    w = WL.SAGE_RMAT_4K
    row_off, col_dst = H.gpu_graph(w)
    spec = H.layer_specs(w)[0]
    xh = WL.input_features(w)
    ref = torch.empty((w.n, spec["d_out"]), dtype=torch.float32, device="cuda")
    L = T.Layer(w.n, row_off, col_dst, out=ref, chunk=w.chunk, **spec)
    L.push_all(torch.from_numpy(xh).cuda())
    L.finalize()
    L.destroy()
    row_bytes = w.dims[0] * 4
    calls = []

    def fill(ctx, b, e, dst):
        calls.append(b)
        ctypes.memmove(dst, xh[b:e].ctypes.data, (e - b) * row_bytes)
        return 0

    cb = N.FILL_FN(fill)
    out = torch.empty_like(ref)
    L = T.Layer(w.n, row_off, col_dst, out=out, chunk=w.chunk, **spec)
    L.stream(cb, None, threads=2, ring=3)
    L.finalize()
    L.destroy()
    assert torch.equal(out, ref) and sorted(calls) == list(range(0, w.n, w.chunk))

    def bad(ctx, b, e, dst):
        return 7 if b == 2 * w.chunk else fill(ctx, b, e, dst)

    cb_bad = N.FILL_FN(bad)
    L = T.Layer(w.n, row_off, col_dst, out=torch.empty_like(ref), chunk=w.chunk, **spec)
    with pytest.raises(T.TaurusError) as ex:
        L.stream(cb_bad, None, threads=1, ring=2)
    assert ex.value.status == -1 and "chunk 2" in str(ex.value), str(ex.value)
    with pytest.raises(T.TaurusError) as ex:
        L.push_chunk(3 * w.chunk, 4 * w.chunk, torch.from_numpy(xh[3 * w.chunk:4 * w.chunk]).cuda())
    assert ex.value.status == -4   # TAURUS_E_STATE: poisoned
    L.destroy()


def test_loader_argument_errors(torch_cuda):
    import paper_2607_17374_amd as T
    torch = torch_cuda
    w = WL.SAGE_RMAT_4K
    row_off, col_dst = H.gpu_graph(w)
    spec = H.layer_specs(w)[0]
    fn, ctx = F.feature_fill(w.seed, w.feat_dist, w.dims[0], F.F32)
    out = torch.empty((w.n, spec["d_out"]), dtype=torch.float32, device="cuda")
    L = T.Layer(w.n, row_off, col_dst, out=out, chunk=w.chunk, **spec)
    for threads, ring in ((0, 0), (65, 0), (4, 4), (2, 257)):
        with pytest.raises(T.TaurusError) as ex:
            L.stream(fn, ctx, threads=threads, ring=ring)
        assert ex.value.status == -1, (threads, ring)
    with pytest.raises(T.TaurusError) as ex:
        L.stream(0, ctx)
    assert ex.value.status == -1
    # after a chunk was pushed the loader is refused (it pushes every chunk)
    L.push_chunk(0, w.chunk, torch.from_numpy(WL.input_features(w)[:w.chunk]).cuda())
    with pytest.raises(T.TaurusError) as ex:
        L.stream(fn, ctx)
    assert ex.value.status == -4
    L.destroy()
