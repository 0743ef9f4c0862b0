"""The large workloads' recipes at the largest scales that keep a GPU test
to about a minute, each checked against the oracle end to end with the
full-size runner's steps (tests/fullsize.py): the sampled 3-layer
GraphSAGE workload at 1/4 of its vertices and edges, the reordered skewed
GCN workload at 1/8, and the out-of-core workload at 1/64 streamed exactly
as at full size (needs an MI355X)."""
import dataclasses
import sys

import numpy as np
import pytest

from fixtures import workloads as WL

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


def _embeddings_clean(res):
    for run, layers in res["embeddings"].items():
        for r in layers:
            assert r["n_bad"] == 0, (run, r)
            assert r["destinations"] > 60000, (run, r)


def test_sampled_graphsage_quarter_scale(torch_cuda):
    """sage3-fanout-rmat-100m at 1/4 (25M vertices, 400M edges, bf16,
    fanouts 15/10/5, 65,536-vertex chunks): the GPU CSR is the canonical CSR
    of the edge list, every layer's kept-edge set equals the oracle
    sampler's (digest and count), and about 66K sampled destinations per
    layer match the oracle chain."""
    from tests import fullsize as FS
    base = WL.SAGE_FANOUT_RMAT_100M
    w = base.scaled(base.n // 4, base.e // 4, name=f"{base.name}-div4")
    _note(f"{w.name}: n={w.n} e={w.e}")
    res = FS.run_c3(w)
    assert res["csr"]["ok"], res["csr"]
    assert len(res["masks"]) == 3
    for m in res["masks"]:
        assert m["digest_equal"] and m["count_equal"], m
    for st in res["stats"]:
        assert st["completed"] == w.n and st["pending_left"] == 0
    _embeddings_clean(res)


def test_reordered_skewed_gcn_eighth_scale(torch_cuda):
    """gcn2-skew-rmat-50m at 1/8 (6.25M vertices, 125M edges, fp16, random
    IDs): degree/BFS and RCMK orders bit for bit against the oracle, Alg. 1
    from each (5 updates) against the oracle's positions and spans, the
    relabelled runs un-permuted against the run in the original IDs, and
    every run's sampled destinations against the oracle."""
    from tests import fullsize as FS
    base = WL.GCN_SKEW_RMAT_50M
    w = base.scaled(base.n // 8, base.e // 8, name=f"{base.name}-div8")
    _note(f"{w.name}: n={w.n} e={w.e}")
    res = FS.run_c5(w)
    assert res["csr"]["ok"], res["csr"]
    for label in ("degree/BFS order", "RCMK order"):
        assert res[label]["bit_exact"], label
        assert res[label]["span"] < res["span_random_ids"], label
        assert res[label]["vs_random_ids_last_layer"]["n_bad"] == 0, label
        ta = res[f"topology-aware order from {label.split()[0]}"]
        assert ta["matches_oracle"], ta
        assert ta["vs_random_ids_last_layer"]["n_bad"] == 0
    _embeddings_clean(res)


def test_out_of_core_streaming_sixty_fourth_scale(torch_cuda):
    """sage2-ooc-rmat-269m at 1/64 (4.2M vertices, 62.5M edges, fp32 512 ->
    256 -> 128) streamed as at full size: every chunk from pinned host
    memory, outputs into pinned host memory, accumulators under 3/4 of the
    scaled HBM budget with 1% resident hubs (rows evicted to the host and
    reloaded), chunks of 2,048 vertices; about 66K sampled destinations per
    layer against the oracle chain."""
    from tests import fullsize as FS
    base = WL.SAGE_OOC_RMAT_269M
    w = base.scaled(base.n // 64, base.e // 64, name=f"{base.name}-div64")
    # 3/4 of the budget scaled with the graph: the scaled budget itself
    # leaves room for every live row at this scale (about 1.66M at the
    # peak), 3/4 leaves about 1.0M slots, still above the 42K hubs plus one
    # chunk's 621K destinations
    w = dataclasses.replace(w, hbm_budget=base.hbm_budget // 64 * 3 // 4, chunk=max(1024, base.chunk // 64))
    _note(f"{w.name}: n={w.n} e={w.e} budget={w.hbm_budget} chunk={w.chunk}")
    res = FS.run_c4(w)
    assert res["csr"]["ok"], res["csr"]
    evicted = 0
    for li, st in enumerate(res["stats"], start=1):
        assert st["completed"] == w.n and st["pending_left"] == 0
        assert st["h2d_bytes"] >= w.n * w.dims[li - 1] * 4          # every chunk crossed the host link
        assert st["device_bytes"] <= w.hbm_budget + (1 << 20), st
        assert 0.0 < st["hub_message_share"] < 1.0
        evicted += st["evictions"]
    assert evicted > 0
    _embeddings_clean(res)
