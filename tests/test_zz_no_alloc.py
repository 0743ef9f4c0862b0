"""taurus_build_csr_noalloc (temporaries in the library's fixed per-GPU
scratch array, no allocation) against taurus_build_csr and the oracle, bit
for bit, over calls in a row with shrinking inputs (needs an MI355X)."""
import sys

import numpy as np
import pytest

from fixtures import workloads as WL

pytestmark = pytest.mark.gpu


def _note(msg):
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _random_simple(rng, n, m):
    u = rng.integers(0, n, m)
    v = rng.integers(0, n, m)
    keep = u != v
    pairs = np.unique(np.stack([u[keep], v[keep]], axis=1), axis=0)
    perm = rng.permutation(pairs.shape[0])
    return pairs[perm, 0].astype(np.int32), pairs[perm, 1].astype(np.int32)


def test_noalloc_csr_matches_allocating_build(torch_cuda):
    import oracle as O
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import build_csr_noalloc, NOALLOC_MAX_EDGES
    torch = torch_cuda
    rng = np.random.default_rng(21)
    w = WL.SAGE_RMAT_4K
    cases = [("near the limit", 300_000, *_random_simple(rng, 300_000, NOALLOC_MAX_EDGES - 1000)),
             (w.name, w.n, *WL.graph(w)),
             ("small", 5000, *_random_simple(rng, 5000, 20_000)),
             ("edgeless", 17, np.zeros(0, np.int32), np.zeros(0, np.int32))]
    for name, n, src, dst in cases:
        _note(f"build_csr_noalloc {name}: n={n} e={src.size}")
        s = torch.from_numpy(src).cuda()
        d = torch.from_numpy(dst).cuda()
        ro_ref, cd_ref = T.build_csr(n, s, d)
        # outputs pre-filled with junk: every entry must be written
        ro = torch.full((n + 1,), -7, dtype=torch.int64, device="cuda")
        cd = torch.full((src.size,), -7, dtype=torch.int32, device="cuda")
        build_csr_noalloc(n, s, d, ro, cd)
        torch.cuda.synchronize()
        assert torch.equal(ro, ro_ref) and torch.equal(cd, cd_ref), name
        g = O.Graph(n, src, dst)
        assert np.array_equal(ro.cpu().numpy(), g.row_off) and np.array_equal(cd.cpu().numpy(), g.col_dst), name


def test_noalloc_csr_errors(torch_cuda):
    import paper_2607_17374_amd as T
    from paper_2607_17374_amd.api import build_csr_noalloc, NOALLOC_MAX_EDGES
    torch = torch_cuda
    _note("build_csr_noalloc errors")
    n = 100
    # a repeated pair and a self loop are reported, as by the allocating build
    for src, dst in (([1, 2, 1], [2, 3, 2]), ([4, 5], [4, 6])):
        s = torch.tensor(src, dtype=torch.int32, device="cuda")
        d = torch.tensor(dst, dtype=torch.int32, device="cuda")
        ro = torch.empty(n + 1, dtype=torch.int64, device="cuda")
        cd = torch.empty(len(src), dtype=torch.int32, device="cuda")
        with pytest.raises(T.TaurusError) as ex:
            build_csr_noalloc(n, s, d, ro, cd)
        assert ex.value.status == -1
    # above the limit: refused before any work
    e = NOALLOC_MAX_EDGES + 1
    big = torch.zeros(e, dtype=torch.int32, device="cuda")
    ro = torch.empty(n + 1, dtype=torch.int64, device="cuda")
    with pytest.raises(T.TaurusError) as ex:
        build_csr_noalloc(n, big, big, ro, big)
    assert ex.value.status == -1
    # a valid call afterwards still works
    s = torch.tensor([0, 1, 2], dtype=torch.int32, device="cuda")
    d = torch.tensor([1, 2, 0], dtype=torch.int32, device="cuda")
    ro = torch.empty(4, dtype=torch.int64, device="cuda")
    cd = torch.empty(3, dtype=torch.int32, device="cuda")
    build_csr_noalloc(3, s, d, ro, cd)
    assert ro.tolist() == [0, 1, 2, 3] and cd.tolist() == [1, 2, 0]
