"""A layer's set-up on a stream of its own (desc.setup_stream): the next
layer's sampler and chunk index run beside the previous layer's queued
chunks, and its dense accumulators are taken at its first push.  The
outputs equal those of the plain layer-after-layer run bit for bit (needs
an MI355X)."""
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


CASES = {
    # the sampled 3-layer GraphSAGE recipe (bf16, fanouts 15/10/5) small
    "sage3-sampled": WL.SAGE_FANOUT_RMAT_100M.scaled(n=1 << 16, e=1 << 20, chunk=4096),
    # the exact 2-layer GCN recipe (fp32), chunk index shared through the plan
    "gcn2-exact": WL.GCN_RMAT_1M.scaled(n=1 << 16, e=1 << 20, chunk=4096),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_overlapped_setup_matches_plain_run(torch_cuda, name):
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import torch_dtype
    torch = torch_cuda
    w = CASES[name]
    _note(f"{name}: n={w.n} e={w.e} chunk={w.chunk}")
    row_off, col_dst = H.gpu_graph(w)
    ref, _ = H.gpu_model(w, row_off, col_dst)
    xh = WL.input_features(w)
    X = torch.from_numpy(xh.view(np.int16) if xh.dtype == np.uint16 else xh).cuda()
    if w.feat_dtype != F.F32:
        X = X.view(torch_dtype(w.feat_dtype))
    specs = H.layer_specs(w)
    outs = [T.alloc_device((w.n, sp["d_out"]), torch_dtype(sp["out_dtype"]), X.device) for sp in specs]
    setup = torch.cuda.Stream()
    plan = T.Plan(w.n, row_off, col_dst, w.chunk)
    L = T.Layer(w.n, row_off, col_dst, out=outs[0], chunk=w.chunk, plan=plan, **specs[0])
    h = X
    for li in range(len(specs)):
        L.push_all(h)
        nxt = None
        if li + 1 < len(specs):  # set up while this layer's chunks are still queued
            nxt = T.Layer(w.n, row_off, col_dst, out=outs[li + 1], chunk=w.chunk, plan=plan,
                          setup_stream=setup, **specs[li + 1])
        st = L.finalize()
        assert st["completed"] == w.n and st["pending_left"] == 0, st
        L.destroy()
        h = outs[li]
        L = nxt
    torch.cuda.synchronize()
    plan.destroy()
    for li, (a, b) in enumerate(zip(ref, outs)):
        assert torch.equal(a, b), f"layer {li + 1} differs"


def test_setup_stream_layer_alone(torch_cuda):
    """One layer set up on another stream and pushed at once: its pushes wait
    for the set-up (the stream's wait is enqueued by the init) and the output
    equals the plain layer's."""
    import paper_2607_17374_amd as T
    torch = torch_cuda
    w = WL.SAGE_RMAT_4K
    row_off, col_dst = H.gpu_graph(w)
    spec = H.layer_specs(w)[0]
    X = torch.from_numpy(WL.input_features(w)).cuda()
    ref = torch.empty((w.n, spec["d_out"]), dtype=torch.float32, device="cuda")
    L = T.Layer(w.n, row_off, col_dst, out=ref, chunk=w.chunk, **spec)
    L.push_all(X)
    L.finalize()
    L.destroy()
    out = torch.empty_like(ref)
    L = T.Layer(w.n, row_off, col_dst, out=out, chunk=w.chunk, setup_stream=torch.cuda.Stream(), **spec)
    L.push_all(X)
    st = L.finalize()
    L.destroy()
    assert st["pending_left"] == 0 and torch.equal(out, ref)
