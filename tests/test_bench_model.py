"""The benchmark's algorithmic byte models (bench.py) against a flush-by-flush
count on small graphs: chunks pushed in ascending order, every segment
(one destination, one source chunk) and every self message enumerated."""
import numpy as np
import pytest

import bench


def _graph(seed, n, e):
    rng = np.random.default_rng(seed)
    u = rng.integers(0, n, size=3 * e)
    v = rng.integers(0, n, size=3 * e)
    keep = u != v
    key = np.unique(u[keep] * n + v[keep])[:e]
    # every vertex is a source (the sampled-layer model counts n aggregation rows)
    ring = np.arange(n) * n + (np.arange(n) + 1) % n
    key = np.unique(np.concatenate([key, ring]))
    return key // n, key % n


def _enumerate(src, dst, n, chunk, d_o, ob, sage, self_in_transform):
    """Bytes of the scatter and of the self messages a transform takes,
    flush by flush, following the documented per-item costs."""
    ins = [[] for _ in range(n)]
    for u, v in zip(src.tolist(), dst.tolist()):
        ins[v].append(u)
    # each vertex's flushes in push order: (chunk, messages, carries self)
    flushes = {v: [] for v in range(n)}
    for v in range(n):
        chunks = sorted({u // chunk for u in ins[v]} | {v // chunk})
        for c in chunks:
            m = sum(1 for u in ins[v] if u // chunk == c)
            flushes[v].append((c, m, c == v // chunk))
    scatter = transform = 0.0
    units = 0
    a = fresh = last = 0
    active = len(set(src.tolist()))
    scatter += 4.0 * d_o * active if sage else 0.0      # aggregation rows of Y
    scatter += 1.0 * n                                   # flag bytes
    for v in range(n):
        fl = flushes[v]
        for i, (c, m, own) in enumerate(fl):
            first, final = i == 0, i == len(fl) - 1
            rmw = (0.0 if first else 4.0 * d_o) + (ob * d_o if final else 4.0 * d_o)
            if own and m == 0 and sage and self_in_transform:
                # alone: the transform adds the self row, the scatter counts it
                a += 1
                fresh += first
                last += final
                transform += 9.0 + rmw
                scatter += 12.0
                continue
            if m > 0:
                units += 1
                scatter += 16.0 + 4.0 * m
            if own:
                scatter += 4.0 * d_o                     # the self row of Y (GCN: the vertex's one row)
            scatter += 12.0 + rmw
    pairs = sum(len(f) for f in flushes.values())
    st = {"split_segments": 0, "pairs": pairs, "short_units": units, "wave_units": 0, "messages": int(src.size),
          "self_in_transform": a, "self_fresh": fresh, "self_last": last}
    return scatter, transform, st


@pytest.mark.parametrize("seed,n,e,chunk", [(1, 300, 1500, 37), (2, 512, 700, 64), (3, 200, 3000, 20)])
@pytest.mark.parametrize("ob", [2, 4])
def test_sampled_scatter_bytes_flush_by_flush(seed, n, e, chunk, ob):
    src, dst = _graph(seed, n, e)
    d_o = 172
    for in_transform in (False, True):
        sc, tr, st = _enumerate(src, dst, n, chunk, d_o, ob, True, in_transform)
        assert (st["self_in_transform"] > 0) == in_transform
        assert bench.sampled_scatter_bytes(st, n, d_o, ob, sage=True) == pytest.approx(sc, rel=0, abs=1e-6)
        assert bench.transform_self_bytes(st, d_o, ob) == pytest.approx(tr, rel=0, abs=1e-6)


@pytest.mark.parametrize("seed,n,e,chunk", [(4, 300, 1500, 37), (5, 256, 4000, 50)])
def test_kernel_bytes_flush_by_flush(seed, n, e, chunk):
    src, dst = _graph(seed, n, e)
    d_o = 64
    sc, _, st = _enumerate(src, dst, n, chunk, d_o, 4, False, False)
    fm = bench.flush_model(src, dst, n, chunk)
    assert fm["split_segments"] == 0 and fm["units"] == st["short_units"]
    kb = bench.kernel_bytes(fm, n, d_o, 4, sage=False)
    assert kb["scatter"] == pytest.approx(sc, rel=0, abs=1e-6)
    assert kb["fixup"] == 0


def test_self_counts_needed_for_transform_layers():
    st = {"split_segments": 0, "pairs": 10, "short_units": 5, "wave_units": 0, "messages": 5,
          "self_in_transform": 3, "self_fresh": -1, "self_last": -1}
    with pytest.raises(ValueError):
        bench.sampled_scatter_bytes(st, 5, 8, 2, sage=True)
