"""Pins for the CPU oracle: each check below is something other than the
oracle itself -- a published value, a dense matrix product (numpy), a closed
form, brute force on a tiny input, or a hand-worked example -- chosen so that
a plausible slip in the oracle (a dropped term, a swapped degree, a wrong
index, a transposed weight) fails at least one of them."""
import numpy as np
import pytest

import oracle as O
import fixtures as F

G = 0x9e3779b97f4a7c15


def random_digraph(rng, n, p, isolated=0):
    """Simple random digraph with ``isolated`` vertices that have no edges at all."""
    A = rng.random((n, n)) < p
    np.fill_diagonal(A, False)
    if isolated:
        iso = rng.choice(n, isolated, replace=False)
        A[iso, :] = False
        A[:, iso] = False
    u, v = np.nonzero(A)
    perm = rng.permutation(u.size)          # edge list order must not matter
    return A, u[perm].astype(np.int32), v[perm].astype(np.int32)


# --------------------------------------------------------------- hashing --

def test_oracle_hash_matches_published_splitmix64(golden_dir):
    refs = [int(l, 16) for l in open(f"{golden_dir}/splitmix64_state0.txt")
            if l.strip() and not l.startswith("#")]
    for k, ref in enumerate(refs):
        assert O.hash_u64(0, (k * G) % 2**64) == ref


def test_oracle_hash_multi_argument_chain(golden_dir):
    """H(s, t, x) chains one mix per argument: H(0, 0, G) = mix64(mix64(G) + 2G);
    with H(0, 0) pinned above, check H(0,0,x) against H(H(0,0) , x) form."""
    h0 = O.hash_u64(0, 0)
    for x in (0, 1, 12345):
        assert O.hash_u64(0, 0, x) == O.hash_u64(h0, x)


# ------------------------------------------------------------------- CSR --

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_csr_brute_force(seed):
    rng = np.random.default_rng(seed)
    A, u, v = random_digraph(rng, 60, 0.08, isolated=5)
    g = O.Graph(60, u, v)
    pairs = sorted(zip(u.tolist(), v.tolist()))
    assert g.col_dst.tolist() == [b for _, b in pairs]
    for x in range(60):
        assert g.row_off[x + 1] - g.row_off[x] == sum(1 for a, _ in pairs if a == x)
    assert g.row_off[0] == 0 and g.row_off[-1] == u.size
    assert (np.diff(g.row_off) >= 0).all()
    assert np.array_equal(g.deg_out, A.sum(1)) and np.array_equal(g.deg_in, A.sum(0))
    # in-lists: ascending sources, and in_pos points back to the same edge
    for x in range(60):
        srcs = g.in_src[g.in_off[x]:g.in_off[x + 1]]
        assert srcs.tolist() == sorted(np.nonzero(A[:, x])[0].tolist())
        for k in range(g.in_off[x], g.in_off[x + 1]):
            p = g.in_pos[k]
            assert g.col_dst[p] == x and g.row_off[g.in_src[k]] <= p < g.row_off[g.in_src[k] + 1]


def test_csr_rejects_non_simple():
    with pytest.raises(ValueError):
        O.Graph(4, np.array([0, 1], np.int32), np.array([0, 2], np.int32))   # self loop
    with pytest.raises(ValueError):
        O.Graph(4, np.array([0, 0], np.int32), np.array([2, 2], np.int32))   # repeated pair
    with pytest.raises(ValueError):
        O.Graph(4, np.array([0], np.int32), np.array([4], np.int32))         # out of range


def test_csr_empty_graph():
    g = O.Graph(5, np.zeros(0, np.int32), np.zeros(0, np.int32))
    assert (g.row_off == 0).all() and g.e == 0


# --------------------------------------------------------------- sampler --

def test_sampler_brute_force_and_invariants():
    rng = np.random.default_rng(3)
    A, u, v = random_digraph(rng, 80, 0.15, isolated=4)
    g = O.Graph(80, u, v)
    seed, layer = 17, 2
    prev = None
    for k in (1, 2, 3, 5, 8):
        words, keep_in, m = O.sample(g, seed, layer, k)
        bits = O.mask_bits(words, g.e)
        assert np.array_equal(m, np.minimum(g.deg_in, k))
        assert bits.sum() == m.sum() and keep_in.sum() == m.sum()
        # brute force: enumerate each v's in-edges, rank by (hash, u), keep k smallest
        for x in range(80):
            srcs = g.in_src[g.in_off[x]:g.in_off[x + 1]].tolist()
            ranked = sorted(srcs, key=lambda s: (O.hash_u64(seed, 4, layer, x, s), s))
            want = set(ranked[:k])
            got = {s for j, s in enumerate(srcs) if keep_in[g.in_off[x] + j]}
            assert got == want
            # the CSR-order mask holds the same set
            for s in srcs:
                row = g.col_dst[g.row_off[s]:g.row_off[s + 1]]
                p = g.row_off[s] + int(np.searchsorted(row, x))
                assert bits[p] == (s in want)
        # nesting: the set for k is inside the set for k+1 ...
        if prev is not None:
            assert not (prev & ~bits).any()
        prev = bits


def test_sampler_large_fanout_keeps_everything():
    rng = np.random.default_rng(4)
    _, u, v = random_digraph(rng, 50, 0.2)
    g = O.Graph(50, u, v)
    words, keep_in, m = O.sample(g, 5, 1, int(g.deg_in.max()))
    assert O.mask_bits(words, g.e).all() and keep_in.all()
    assert np.array_equal(m, g.deg_in)
    words0, _, m0 = O.sample(g, 5, 1, 0)
    assert O.mask_bits(words0, g.e).all() and np.array_equal(m0, g.deg_in)


def test_sampler_layers_differ():
    rng = np.random.default_rng(5)
    _, u, v = random_digraph(rng, 120, 0.3)
    g = O.Graph(120, u, v)
    w1, _, _ = O.sample(g, 9, 1, 3)
    w2, _, _ = O.sample(g, 9, 2, 3)
    assert not np.array_equal(w1, w2)


# -------------------------------------------------------- layer maths ------

def dense_sage(A_keep, H, W_agg, W_self, b, relu):
    """GraphSAGE-mean as dense matrix products: D_M^-1 A_M^T H W_agg^T + H W_self^T + b."""
    m = A_keep.sum(0).astype(np.float64)
    inv = np.where(m > 0, 1.0 / np.maximum(m, 1), 0.0)
    agg = inv[:, None] * (A_keep.T.astype(np.float64) @ H)
    z = agg @ W_agg.T + H @ W_self.T + b
    return np.maximum(z, 0) if relu else z


def dense_gcn(A, H, W, b, relu):
    """Symmetric-normalised GCN with self loops as dense products:
    D_in^-1/2 (A+I)^T D_out^-1/2 H W^T + b, D from the row/column sums of A+I."""
    Ah = A.astype(np.float64) + np.eye(A.shape[0])
    dout = Ah.sum(1)
    din = Ah.sum(0)
    P = np.diag(din ** -0.5) @ Ah.T @ np.diag(dout ** -0.5)
    z = P @ H @ W.T + b
    return np.maximum(z, 0) if relu else z


@pytest.mark.parametrize("seed,relu", [(0, True), (1, False), (2, True)])
def test_sage_matches_dense(seed, relu):
    rng = np.random.default_rng(seed)
    n, d_in, d_out = 96, 12, 7
    A, u, v = random_digraph(rng, n, 0.06, isolated=6)
    g = O.Graph(n, u, v)
    H = rng.standard_normal((n, d_in))
    W = rng.standard_normal((d_out, 2 * d_in))
    b = rng.standard_normal(d_out)
    H32 = H.astype(np.float32)
    got = O.layer(O.SAGE_MEAN, g, H32, O.F32, W, b, relu)
    ref = dense_sage(A, H32.astype(np.float64), W[:, :d_in], W[:, d_in:], b, relu)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed,relu", [(0, True), (1, False)])
def test_gcn_matches_dense(seed, relu):
    rng = np.random.default_rng(seed + 10)
    n, d_in, d_out = 90, 9, 11
    A, u, v = random_digraph(rng, n, 0.07, isolated=5)
    g = O.Graph(n, u, v)
    H32 = rng.standard_normal((n, d_in)).astype(np.float32)
    W = rng.standard_normal((d_out, d_in))
    b = rng.standard_normal(d_out)
    got = O.layer(O.GCN_SYM, g, H32, O.F32, W, b, relu)
    ref = dense_gcn(A, H32.astype(np.float64), W, b, relu)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_sampled_sage_matches_dense_on_kept_edges():
    rng = np.random.default_rng(7)
    n, d_in, d_out = 100, 8, 5
    A, u, v = random_digraph(rng, n, 0.12, isolated=3)
    g = O.Graph(n, u, v)
    H32 = rng.standard_normal((n, d_in)).astype(np.float32)
    W = rng.standard_normal((d_out, 2 * d_in))
    b = rng.standard_normal(d_out)
    words, keep_in, _ = O.sample(g, 21, 1, 4)
    bits = O.mask_bits(words, g.e)
    A_keep = np.zeros_like(A)
    src_csr = np.repeat(np.arange(n), np.diff(g.row_off))
    A_keep[src_csr[bits], g.col_dst[bits]] = True
    got = O.layer(O.SAGE_MEAN, g, H32, O.F32, W, b, True, keep_in=keep_in)
    ref = dense_sage(A_keep, H32.astype(np.float64), W[:, :d_in], W[:, d_in:], b, True)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_sampled_gcn_matches_dense_on_kept_edges():
    """A sampled GCN layer is the GCN of the sampled graph: the kept edges
    plus one self loop per vertex, normalised by that graph's degrees."""
    rng = np.random.default_rng(17)
    n, d_in, d_out = 100, 8, 5
    A, u, v = random_digraph(rng, n, 0.12, isolated=3)
    g = O.Graph(n, u, v)
    H32 = rng.standard_normal((n, d_in)).astype(np.float32)
    W = rng.standard_normal((d_out, d_in))
    b = rng.standard_normal(d_out)
    for k in (1, 4):
        words, keep_in, _ = O.sample(g, 23, 2, k)
        bits = O.mask_bits(words, g.e)
        A_keep = np.zeros_like(A)
        src_csr = np.repeat(np.arange(n), np.diff(g.row_off))
        A_keep[src_csr[bits], g.col_dst[bits]] = True
        got = O.layer(O.GCN_SYM, g, H32, O.F32, W, b, True, keep_in=keep_in)
        ref = dense_gcn(A_keep, H32.astype(np.float64), W, b, True)
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def dense_gin(A, H, W, b, relu):
    """GIN with eps = 0 and a linear apply function: (A + I)^T H W^T + b."""
    z = (A.astype(np.float64) + np.eye(A.shape[0])).T @ H @ W.T + b
    return np.maximum(z, 0) if relu else z


@pytest.mark.parametrize("sampled", [False, True])
def test_gin_matches_dense(sampled):
    rng = np.random.default_rng(27)
    n, d_in, d_out = 90, 7, 6
    A, u, v = random_digraph(rng, n, 0.08, isolated=4)
    g = O.Graph(n, u, v)
    H32 = rng.standard_normal((n, d_in)).astype(np.float32)
    W = rng.standard_normal((d_out, d_in))
    b = rng.standard_normal(d_out)
    keep_in, A_used = None, A
    if sampled:
        words, keep_in, _ = O.sample(g, 5, 1, 3)
        bits = O.mask_bits(words, g.e)
        A_used = np.zeros_like(A)
        A_used[np.repeat(np.arange(n), np.diff(g.row_off))[bits], g.col_dst[bits]] = True
    got = O.layer(O.GIN_SUM, g, H32, O.F32, W, b, False, keep_in=keep_in)
    np.testing.assert_allclose(got, dense_gin(A_used, H32.astype(np.float64), W, b, False), rtol=1e-12, atol=1e-12)
    # closed form: constant features c and identity weights give c (d_in(v) + 1)
    ones = np.full((n, d_in), 0.5, np.float32)
    z = O.layer(O.GIN_SUM, g, ones, O.F32, np.eye(d_in), None, False)
    np.testing.assert_allclose(z, 0.5 * (np.diff(g.in_off)[:, None] + 1) * np.ones((1, d_in)), rtol=0, atol=0)


@pytest.mark.parametrize("sampled", [False, True])
def test_gin_mlp_matches_dense(sampled):
    """GIN with a two-layer perceptron apply function: ReLU(((A^T + I) H) W1^T
    + b1) W2^T + b2 as dense matrix products (numpy), exact and sampled;
    identity second layer and zero bias reduce it to ReLU of the linear GIN."""
    rng = np.random.default_rng(28)
    n, d_in, d_h, d_out = 80, 6, 9, 5
    A, u, v = random_digraph(rng, n, 0.09, isolated=3)
    g = O.Graph(n, u, v)
    H32 = rng.standard_normal((n, d_in)).astype(np.float32)
    W1, b1 = rng.standard_normal((d_h, d_in)), rng.standard_normal(d_h)
    W2, b2 = rng.standard_normal((d_out, d_h)), rng.standard_normal(d_out)
    keep_in, A_used = None, A
    if sampled:
        words, keep_in, _ = O.sample(g, 6, 2, 3)
        bits = O.mask_bits(words, g.e)
        A_used = np.zeros_like(A)
        A_used[np.repeat(np.arange(n), np.diff(g.row_off))[bits], g.col_dst[bits]] = True
    agg = (A_used.astype(np.float64) + np.eye(n)).T @ H32.astype(np.float64)
    for relu in (False, True):
        want = np.maximum(agg @ W1.T + b1, 0) @ W2.T + b2
        if relu:
            want = np.maximum(want, 0)
        got = O.gin_mlp_layer(g, H32, O.F32, W1, b1, W2, b2, relu, keep_in=keep_in)
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
    # W2 = I, no biases: ReLU of the linear GIN with W1
    z = O.gin_mlp_layer(g, H32, O.F32, W1, None, np.eye(d_h), None, False, keep_in=keep_in)
    lin = O.layer(O.GIN_SUM, g, H32, O.F32, W1, None, True, keep_in=keep_in)
    np.testing.assert_allclose(z, lin, rtol=1e-13, atol=1e-13)
    # subset of destinations equals rows of the full result
    ids = np.array([0, 5, 17, n - 1], np.int64)
    sub = O.gin_mlp_layer(g, H32, O.F32, W1, b1, W2, b2, True, keep_in=keep_in, dst_ids=ids)
    np.testing.assert_array_equal(sub, O.gin_mlp_layer(g, H32, O.F32, W1, b1, W2, b2, True, keep_in=keep_in)[ids])


def test_subset_of_destinations_equals_rows_of_full():
    rng = np.random.default_rng(8)
    n = 70
    A, u, v = random_digraph(rng, n, 0.1)
    g = O.Graph(n, u, v)
    H32 = rng.standard_normal((n, 6)).astype(np.float32)
    W = rng.standard_normal((4, 12))
    full = O.layer(O.SAGE_MEAN, g, H32, O.F32, W, None, True)
    ids = np.array([5, 0, 69, 5, 33], np.int64)
    part = O.layer(O.SAGE_MEAN, g, H32, O.F32, W, None, True, dst_ids=ids)
    assert np.array_equal(full[ids], part)


def test_closed_form_sage_constant_features():
    """Constant input c*1: every vertex with m >= 1 gets ReLU((W_agg + W_self) c1 + b),
    vertices with no in-neighbour get ReLU(W_self c1 + b)."""
    rng = np.random.default_rng(9)
    n, d = 64, 5
    A, u, v = random_digraph(rng, n, 0.05, isolated=4)
    g = O.Graph(n, u, v)
    c = 0.75
    H = np.full((n, d), c, np.float32)
    W = rng.standard_normal((3, 2 * d))
    b = rng.standard_normal(3)
    out = O.layer(O.SAGE_MEAN, g, H, O.F32, W, b, True)
    with_nb = np.maximum((W[:, :d] + W[:, d:]) @ np.full(d, c) + b, 0)
    without = np.maximum(W[:, d:] @ np.full(d, c) + b, 0)
    for x in range(n):
        np.testing.assert_allclose(out[x], with_nb if g.deg_in[x] > 0 else without, rtol=1e-13, atol=1e-13)


def test_closed_form_sage_identity_is_neighbour_average():
    """W_agg = I, W_self = 0, b = 0, no activation: the layer is plain averaging
    of the in-neighbours' features."""
    rng = np.random.default_rng(10)
    n, d = 50, 4
    A, u, v = random_digraph(rng, n, 0.1, isolated=2)
    g = O.Graph(n, u, v)
    H = rng.standard_normal((n, d)).astype(np.float32)
    W = np.concatenate([np.eye(d), np.zeros((d, d))], axis=1)
    out = O.layer(O.SAGE_MEAN, g, H, O.F32, W, None, False)
    for x in range(n):
        nb = [a for a, bb in zip(u.tolist(), v.tolist()) if bb == x]
        want = np.mean(H[nb].astype(np.float64), axis=0) if nb else np.zeros(d)
        np.testing.assert_allclose(out[x], want, rtol=1e-13, atol=1e-13)


def test_closed_form_gcn_degrees_only():
    """Constant c, W = I, b = 0, no activation:
    out(v) = c * d^_in(v)^-1/2 * sum_{u in N-(v) + {v}} d^_out(u)^-1/2."""
    rng = np.random.default_rng(11)
    n, d = 40, 3
    A, u, v = random_digraph(rng, n, 0.1, isolated=3)
    g = O.Graph(n, u, v)
    c = -1.25
    H = np.full((n, d), c, np.float32)
    out = O.layer(O.GCN_SYM, g, H, O.F32, np.eye(d), None, False)
    dout = A.sum(1) + 1.0
    din = A.sum(0) + 1.0
    for x in range(n):
        srcs = list(np.nonzero(A[:, x])[0]) + [x]
        want = c * din[x] ** -0.5 * sum(dout[s] ** -0.5 for s in srcs)
        np.testing.assert_allclose(out[x], np.full(d, want), rtol=1e-13)


@pytest.mark.parametrize("kind", ["cycle", "complete"])
def test_closed_form_gcn_regular_symmetric_graph_preserves_constants(kind):
    n, d, c = 12, 4, 0.3
    if kind == "cycle":
        u = np.concatenate([np.arange(n), (np.arange(n) + 1) % n])
        v = np.concatenate([(np.arange(n) + 1) % n, np.arange(n)])
    else:
        uu, vv = np.nonzero(~np.eye(n, dtype=bool))
        u, v = uu, vv
    g = O.Graph(n, u.astype(np.int32), v.astype(np.int32))
    out = O.layer(O.GCN_SYM, g, np.full((n, d), c, np.float32), O.F32, np.eye(d), None, False)
    np.testing.assert_allclose(out, float(np.float32(c)), rtol=1e-13)


def test_gcn_symmetric_equals_kipf_form():
    """On a symmetric graph the directed reading reduces to D^-1/2 (A+I) D^-1/2."""
    rng = np.random.default_rng(12)
    n = 30
    A = rng.random((n, n)) < 0.15
    A = A | A.T
    np.fill_diagonal(A, False)
    u, v = np.nonzero(A)
    g = O.Graph(n, u.astype(np.int32), v.astype(np.int32))
    H = rng.standard_normal((n, 5)).astype(np.float32)
    W = rng.standard_normal((5, 5))
    Ah = A + np.eye(n)
    Dm = np.diag(Ah.sum(1) ** -0.5)
    ref = Dm @ Ah @ Dm @ H.astype(np.float64) @ W.T
    got = O.layer(O.GCN_SYM, g, H, O.F32, W, None, False)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_layer_16bit_inputs_widen_exactly():
    rng = np.random.default_rng(13)
    n, d = 30, 4
    A, u, v = random_digraph(rng, n, 0.2)
    g = O.Graph(n, u, v)
    x32 = rng.standard_normal((n, d)).astype(np.float32)
    W = rng.standard_normal((3, 2 * d))
    for code in (F.BF16, F.F16):
        bits = F.round16(x32, code)
        wide = F.bits_to_float(bits, code).reshape(n, d)
        assert np.array_equal(O.widen(bits, code), wide.astype(np.float64))
        got = O.layer(O.SAGE_MEAN, g, bits, code, W, None, False)
        ref = O.layer(O.SAGE_MEAN, g, wide, O.F32, W, None, False)
        assert np.array_equal(got, ref)


def test_round_store_matches_library_conversions():
    import torch
    rng = np.random.default_rng(14)
    x = np.concatenate([rng.standard_normal(2000) * 10.0 ** rng.integers(-9, 5, 2000),
                        [0.0, -0.0, 65519.99, 65520.0, 1e6, 2**-24, 2**-25, 1 + 2**-11]])
    f32 = O.round_store(x, O.F32)
    assert np.array_equal(f32, x.astype(np.float32))
    assert np.array_equal(O.round_store(x, O.F16), x.astype(np.float32).astype(np.float16).view(np.uint16))
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(O.round_store(x, O.BF16), ref)


# --------------------------------------------------------------- reorder --

def _g(n, edges):
    e = np.array(edges, np.int32).reshape(-1, 2)
    return O.Graph(n, e[:, 0].copy(), e[:, 1].copy())


def test_reorder_star():
    # leaves 1..5 send to hub 0: hub first, then its sources by (d_in desc, id)
    g = _g(6, [(i, 0) for i in range(1, 6)])
    pi = O.reorder_bfs(g)
    assert pi.tolist() == [0, 1, 2, 3, 4, 5]
    # same star with the hub named 5
    g = _g(6, [(i, 5) for i in range(0, 5)])
    assert O.reorder_bfs(g).tolist() == [1, 2, 3, 4, 5, 0]


def test_reorder_edgeless_is_identity():
    g = O.Graph(7, np.zeros(0, np.int32), np.zeros(0, np.int32))
    assert O.reorder_bfs(g).tolist() == list(range(7))


def test_reorder_path_and_two_components():
    # path 0 -> 1 -> 2 -> 3: in-degrees 0,1,1,1; root order 1, 2, 3, 0.
    # BFS over in-edges from 1 visits 0; root 2 adds only itself (its
    # in-neighbour 1 is seen), and so does root 3.
    g = _g(4, [(0, 1), (1, 2), (2, 3)])
    order = [1, 0, 2, 3]                       # visit order worked by hand
    pi = O.reorder_bfs(g)
    assert [int(np.nonzero(pi == i)[0][0]) for i in range(4)] == order
    # two components: {4 <- 5, 4 <- 6, 6 <- 7} and {0 <- 1, 0 <- 2, 0 <- 3}
    g = _g(8, [(5, 4), (6, 4), (7, 6), (1, 0), (2, 0), (3, 0)])
    # d_in: 0:3, 4:2, 6:1, others 0.  Roots: 0 (3), then 4 (2), then 6 (seen), ...
    # BFS(0): 0, 1, 2, 3.  BFS(4): 4, then in-nbrs {5 (d 0), 6 (d 1)} -> 6, 5; then 7 from 6.
    order = [0, 1, 2, 3, 4, 6, 5, 7]
    pi = O.reorder_bfs(g)
    assert [int(np.nonzero(pi == i)[0][0]) for i in range(8)] == order


def test_reorder_tree_levels():
    # a binary in-tree: 1,2 -> 0; 3,4 -> 1; 5,6 -> 2; extra 6 -> 4 gives 4 d_in 1
    g = _g(7, [(1, 0), (2, 0), (3, 1), (4, 1), (5, 2), (6, 2), (6, 4)])
    # d_in: 0:2, 1:2, 2:2, 4:1.  Root 0.  Children of 0: {1, 2} tie on d_in 2 -> 1, 2.
    # children of 1: {3 (0), 4 (1)} -> 4, 3; children of 2: {5, 6} (6 not yet seen) -> 5, 6
    # children of 4: {6} already seen.
    order = [0, 1, 2, 4, 3, 5, 6]
    pi = O.reorder_bfs(g)
    assert [int(np.nonzero(pi == i)[0][0]) for i in range(7)] == order


def search_order_is_valid(n, order, nbrs, key):
    """Properties that characterise a breadth-first visit order whose roots
    and children are ranked by ``key``: a bijection; each vertex is either a
    root (the first unvisited vertex in key order at its time) or appears
    after the earliest-placed vertex that lists it in ``nbrs`` (its
    discoverer); children of one discoverer are contiguous in key order and
    blocks of children follow their discoverers' order."""
    order = [int(x) for x in order]
    assert sorted(order) == list(range(n))
    pos = np.empty(n, np.int64)
    pos[order] = np.arange(n)
    disc = np.full(n, -1)
    # discoverer of w: the earliest vertex (by position) before w that lists w
    for x in order:
        for w in nbrs(x):
            if pos[w] > pos[x] and disc[w] < 0:
                disc[w] = x
    roots = [x for x in order if disc[x] < 0]
    # roots appear in root order among themselves
    assert roots == sorted(roots, key=key)
    # a root is the first unvisited vertex in global root order when it starts
    rank = sorted(range(n), key=key)
    for r in roots:
        assert all(pos[x] < pos[r] for x in rank[:rank.index(r)])
    # non-roots in visit order: discoverer positions never decrease (blocks of
    # children are contiguous and follow their parents' order), and each
    # block is sorted by key
    last = -1
    for i, x in enumerate(order):
        if disc[x] < 0:
            continue
        assert pos[disc[x]] < pos[x]
        assert pos[disc[x]] >= last
        if pos[disc[x]] == last:
            assert key(order[i - 1]) < key(x)
        last = pos[disc[x]]
    return True


def bfs_order_is_valid(g, pi):
    """The degree/BFS order: search over in-neighbours, key (d_in desc, id asc)."""
    order = np.empty(g.n, np.int64)
    order[np.asarray(pi, np.int64)] = np.arange(g.n)
    return search_order_is_valid(g.n, order, lambda x: g.in_src[g.in_off[x]:g.in_off[x + 1]],
                                 lambda x: (-int(g.deg_in[x]), int(x)))


def symmetric_neighbours(g):
    S = [set() for _ in range(g.n)]
    for u in range(g.n):
        for v in g.col_dst[g.row_off[u]:g.row_off[u + 1]]:
            S[u].add(int(v))
            S[int(v)].add(u)
    return S


def rcm_order_is_valid(g, pi):
    """RCMK: the reversed order is a Cuthill-McKee search of the symmetrised
    graph, key (symmetric degree asc, id asc)."""
    S = symmetric_neighbours(g)
    order = np.empty(g.n, np.int64)
    order[g.n - 1 - np.asarray(pi, np.int64)] = np.arange(g.n)
    return search_order_is_valid(g.n, order, lambda x: sorted(S[x]), lambda x: (len(S[x]), int(x)))


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_reorder_random_graphs_are_valid_bfs_orders(seed):
    rng = np.random.default_rng(seed + 40)
    _, u, v = random_digraph(rng, 70, 0.03, isolated=5)
    g = O.Graph(70, u, v)
    assert bfs_order_is_valid(g, O.reorder_bfs(g))


def test_total_span_hand_example():
    # every neighbourhood holds the self message: N(3) = {0,1,2,3} at ranks
    # 0..3 -> span 3; N(0) = {0,2} -> 2; N(1) = {1}, N(2) = {2} -> 0
    g = _g(4, [(0, 3), (1, 3), (2, 3), (2, 0)])
    assert O.total_span(g, np.arange(4, dtype=np.int32)) == 3 + 2
    # ranks 3,0,1,2: N(3) spans 0..3 -> 3; N(0) at ranks {3, 1} -> 2
    assert O.total_span(g, np.array([3, 0, 1, 2], np.int32)) == 3 + 2
    # ranks 1,2,0,3 put vertex 2 next to vertex 0: N(3) -> 3; N(0) at ranks {1, 0} -> 1
    assert O.total_span(g, np.array([1, 2, 0, 3], np.int32)) == 3 + 1
    # no edges: every span is 0
    assert O.total_span(_g(3, []), np.array([2, 0, 1], np.int32)) == 0


def test_span_equals_sum_of_active_counts():
    """C(pi) = sum_t A(t) with A(t) = #{v : a(v) <= t < c(v)} (Sec. 3.8)."""
    rng = np.random.default_rng(50)
    _, u, v = random_digraph(rng, 40, 0.1)
    g = O.Graph(40, u, v)
    pi = rng.permutation(40).astype(np.int32)
    total = 0
    for t in range(40):
        for x in range(40):
            nb = np.concatenate([[x], g.in_src[g.in_off[x]:g.in_off[x + 1]]])
            if pi[nb].min() <= t < pi[nb].max():
                total += 1
    assert O.total_span(g, pi) == total
    # the residency profile at chunk size 1 sums to the same total (M = C(pi)),
    # and at other chunk sizes counts the partial states held after each chunk
    assert O.active_profile(g, pi, 1).sum() == total
    for chunk in (3, 7, 40):
        A = O.active_profile(g, pi, chunk)
        for k in range(A.size):
            held = 0
            for x in range(40):
                nb = np.concatenate([[x], g.in_src[g.in_off[x]:g.in_off[x + 1]]])
                held += int(pi[nb].min() // chunk <= k < pi[nb].max() // chunk)
            assert A[k] == held
    # and the bandwidth bound C(pi) <= 2 |V| B, B = max edge length under pi
    B = int(np.abs(pi[u].astype(np.int64) - pi[v]).max())
    assert total <= 2 * 40 * B


# ---- large-graph helpers: in-lists from the edge list, set digests, CSR shape

def _edge_list(rng, n, p):
    _, u, v = random_digraph(rng, n, p, isolated=3)
    perm = rng.permutation(u.size)           # any edge order
    return u[perm].astype(np.int32), v[perm].astype(np.int32)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_edge_graph_in_lists_equal_graph(seed):
    rng = np.random.default_rng(seed + 70)
    u, v = _edge_list(rng, 60, 0.08)
    g = O.Graph(60, u, v)
    eg = O.EdgeGraph(60, u, v)
    assert np.array_equal(eg.in_off, g.in_off) and np.array_equal(eg.in_src, g.in_src)
    assert np.array_equal(eg.deg_out, g.deg_out) and np.array_equal(eg.deg_in, g.deg_in)
    eo = O.EdgeGraph(60, u, v, out_lists=True)
    assert np.array_equal(eo.row_off, g.row_off) and np.array_equal(eo.col_dst, g.col_dst)
    assert np.array_equal(O.reorder_ta(eo, None, 3)[0], O.reorder_ta(g, None, 3)[0])
    # the fanout sampler sees the same lists: same kept entries and counts
    for k in (1, 3):
        _, keep_g, m_g = O.sample(g, 11, 2, k)
        words, keep_e, m_e = O.sample(eg, 11, 2, k)
        assert words is None and np.array_equal(keep_g, keep_e) and np.array_equal(m_g, m_e)


def test_set_digests_agree_and_separate():
    rng = np.random.default_rng(80)
    u, v = _edge_list(rng, 50, 0.1)
    g = O.Graph(50, u, v)
    d = O.digest_edges(u, v)
    assert d[0] == u.size
    assert O.digest_csr(50, g.row_off, g.col_dst) == d == O.digest_in_lists(g)
    # one destination moved: a different set, a different digest
    col = g.col_dst.copy()
    i = int(np.flatnonzero(np.diff(g.row_off) > 0)[0])
    col[g.row_off[i]] = (col[g.row_off[i]] + 1) % 50
    assert O.digest_csr(50, g.row_off, col) != d
    # the kept edges of a sampled layer: mask over the CSR == keep_in over the in-lists
    words, keep_in, m = O.sample(g, 5, 1, 2)
    dm = O.digest_csr(50, g.row_off, g.col_dst, words)
    assert dm == O.digest_in_lists(g, keep_in) and dm[0] == int(m.sum())


def test_csr_check_rules():
    rng = np.random.default_rng(90)
    u, v = _edge_list(rng, 40, 0.1)
    g = O.Graph(40, u, v)
    assert O.csr_check(40, g.row_off, g.col_dst) == 0
    row = int(np.flatnonzero(np.diff(g.row_off) >= 2)[0])
    a = g.row_off[row]
    col = g.col_dst.copy(); col[a], col[a + 1] = col[a + 1], col[a]
    assert O.csr_check(40, g.row_off, col) == 3                # out of order
    col = g.col_dst.copy(); col[a] = row
    assert O.csr_check(40, g.row_off, col) in (3, 4)           # self loop (may also break the order)
    col = g.col_dst.copy(); col[a] = 40
    assert O.csr_check(40, g.row_off, col) in (2, 3)           # out of range
    ro = g.row_off.copy(); ro[-1] += 1
    assert O.csr_check(40, ro, g.col_dst) == 1                 # offsets


@pytest.mark.parametrize("which", ["sage-sampled", "gcn"])
def test_oracle_chain_on_samples_equals_full_oracle(which):
    """The sampled-destination chain (each layer on the vertices the next one
    reads, fed the oracle's own previous layer) equals the full oracle."""
    from fixtures import workloads as WL
    from tests import harness as H
    if which == "gcn":
        w = WL.GCN_RMAT_1M.scaled(n=3000, e=40000, chunk=1024)
    else:
        w = WL.SAGE_FANOUT_RMAT_100M.scaled(n=3000, e=40000, chunk=1024)
    src, dst = WL.graph(w)
    g, zs = H.oracle_model(w, src, dst)
    rng = np.random.default_rng(3)
    ids = [np.sort(rng.choice(w.n, 200, replace=False)) for _ in range(w.layers)]
    keeps = [O.sample(g, w.seed, li, w.fanout(li))[1] if w.fanout(li) else None for li in range(1, w.layers + 1)]
    out = H.oracle_sampled_layers(w, g, WL.input_features(w), ids, keeps)
    for li in range(w.layers):
        assert np.array_equal(out[li], zs[li][ids[li]]), li


# ---- topology-aware reordering (Sec. 3.8, Alg. 1)

def _dispersion(g, r, mu):
    """The objective of Sec. 3.8: J = sum_v 1/d(v) sum_{u in N(v)} (r(u) - mu(v))^2,
    N(v) = v's in-neighbours and v itself (the self message), d(v) = |N(v)|."""
    J = 0.0
    for v in range(g.n):
        nb = np.concatenate([[v], g.in_src[g.in_off[v]:g.in_off[v + 1]]])
        J += np.sum((r[nb] - mu[v]) ** 2) / nb.size
    return J


@pytest.mark.parametrize("seed", [0, 1])
def test_ta_updates_are_the_minimisers(seed):
    """mu* minimises J for fixed r, and r* minimises J for fixed mu: no
    perturbation of either lowers J (J is convex in each block)."""
    rng = np.random.default_rng(seed + 100)
    _, u, v = random_digraph(rng, 30, 0.12, isolated=2)
    g = O.Graph(30, u, v)
    r = rng.permutation(30).astype(np.float64) + rng.random(30)
    mu, r2 = O.ta_step(g, r)
    j_mu = _dispersion(g, r, mu)
    j_r = _dispersion(g, r2, mu)
    for _ in range(20):
        d = rng.normal(scale=0.3, size=30)
        assert _dispersion(g, r, mu + d) >= j_mu - 1e-9
        assert _dispersion(g, r2 + d, mu) >= j_r - 1e-9
    # one coordinate at a time (the minimiser is unique per coordinate)
    for k in range(30):
        e = np.zeros(30); e[k] = 1e-3
        assert _dispersion(g, r, mu + e) > j_mu and _dispersion(g, r, mu - e) > j_mu
        assert _dispersion(g, r2 + e, mu) > j_r and _dispersion(g, r2 - e, mu) > j_r


def test_ta_dispersion_never_increases():
    rng = np.random.default_rng(110)
    _, u, v = random_digraph(rng, 40, 0.08)
    g = O.Graph(40, u, v)
    r = rng.permutation(40).astype(np.float64)
    mu, _ = O.ta_step(g, r)
    prev = _dispersion(g, r, mu)
    for _ in range(6):
        _, r = O.ta_step(g, r)
        j_after_r = _dispersion(g, r, mu)
        mu, _ = O.ta_step(g, r)
        j_after_mu = _dispersion(g, r, mu)
        assert j_after_r <= prev + 1e-9 and j_after_mu <= j_after_r + 1e-9
        prev = j_after_mu


def test_ta_special_cases():
    # a directed path keeps its order: r = (1/6, 1, 2, 5/2) after one update
    g = _g(4, [(0, 1), (1, 2), (2, 3)])
    mu, r = O.ta_step(g, np.arange(4, dtype=np.float64))
    assert np.allclose(mu, [0, 0.5, 1.5, 2.5]) and np.allclose(r, [1 / 6, 1, 2, 2.5])
    res = O.reorder_ta(g, None, 5)
    # each of 1, 2, 3 spans itself and its predecessor; the order is unchanged
    # by the first update, so the loop stops there
    assert np.array_equal(res.pi, np.arange(4)) and res.done == 1 and res.spans[0] == res.spans[1] == 3
    assert np.allclose(res.positions, [1 / 6, 1, 2, 2.5])
    # no edges: every vertex is its own neighbourhood, so nothing moves
    g = _g(5, [])
    boot = np.array([3, 0, 4, 1, 2], np.int32)
    res = O.reorder_ta(g, boot, 5)
    assert np.array_equal(res.pi, boot) and res.done == 1 and res.spans[0] == 0 and res.disp[0] == 0
    assert np.array_equal(res.positions, boot.astype(np.float64))
    # a reciprocal pair 0 <-> 1 from ranks (2, 0): both centres and both
    # positions are (2 + 0) / 2 = 1, which the isolated vertex 2 (rank 1)
    # keeps too; the three-way tie is broken by ID, and the next update
    # leaves it there
    g = _g(3, [(0, 1), (1, 0)])
    res = O.reorder_ta(g, np.array([2, 0, 1], np.int32), 5)
    assert np.array_equal(res.positions, [1.0, 1.0, 1.0])
    assert res.pi.tolist() == [0, 1, 2] and res.done == 2
    # N(0) = N(1) = {0, 1}: ranks {2, 0} span 2 each (variance 1), then
    # ranks {0, 1} span 1 each (variance 1/4)
    assert res.spans[:3].tolist() == [4, 2, 2] and res.disp[:3].tolist() == [2.0, 0.5, 0.5]


def _golden_alg1(golden_dir):
    from fractions import Fraction
    vals = {}
    for line in open(f"{golden_dir}/alg1_worked_example.txt"):
        if line.startswith("#") or not line.strip():
            continue
        key, *rest = line.split()
        vals[key] = rest
    n = int(vals["n"][0])
    edges = [tuple(int(x) for x in e.split(",")) for e in vals["edges"]]
    fr = lambda k: [float(Fraction(x)) for x in vals[k]]
    it = lambda k: [int(x) for x in vals[k]]
    return n, edges, fr, it


def test_ta_worked_example(golden_dir):
    """Alg. 1 on the hand-worked graph of tests/golden: the positions are
    carried across updates, so the second update reverses vertices 0 and 1
    (restarting from the ranks would leave the order unchanged)."""
    n, edges, fr, it = _golden_alg1(golden_dir)
    g = _g(n, edges)
    one = O.reorder_ta(g, None, 1)
    assert one.done == 1 and one.pi.tolist() == it("pi1")
    assert np.allclose(one.positions, fr("r1"), rtol=1e-15, atol=0)
    two = O.reorder_ta(g, None, 2)
    assert two.done == 2 and two.pi.tolist() == it("pi2")
    assert np.allclose(two.positions, fr("r2"), rtol=1e-15, atol=0)
    assert two.spans.tolist() == it("spans")
    assert np.allclose(two.disp, fr("disp"), rtol=1e-15, atol=0)


def _dense_alg1(n, u, v, pi0, updates):
    """Alg. 1 as dense linear algebra: with Nm[v, w] = 1 when w is in N(v)
    (v's in-neighbours and v), d = Nm 1, one update is the linear map
    r -> (Nm^T D^-1 D^-1 Nm r) / (Nm^T D^-1 1), so the positions after t
    updates are that map applied t times to the bootstrap ranks."""
    Nm = np.eye(n)
    Nm[v, u] = 1.0
    d = Nm.sum(axis=1)
    B = (Nm.T @ np.diag(1.0 / d**2) @ Nm) / (Nm.T @ (1.0 / d))[:, None]
    r = pi0.astype(np.float64)
    out = []
    for _ in range(updates):
        r = B @ r
        out.append(r.copy())
    return out


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_ta_positions_follow_dense_operator(seed):
    """Positions after t updates equal the dense map applied t times to the
    bootstrap (the printed loop carries r); the order ranks them, ties by ID;
    spans and J are those of each update's order."""
    rng = np.random.default_rng(seed + 140)
    n = 50
    _, u, v = random_digraph(rng, n, 0.06, isolated=3)
    g = O.Graph(n, u, v)
    boot = rng.permutation(n).astype(np.int32)
    rs = _dense_alg1(n, u, v, boot, 4)
    for t in range(1, 5):
        res = O.reorder_ta(g, boot, t)
        if res.done < t:
            break
        want = rs[t - 1]
        assert np.allclose(res.positions, want, rtol=1e-12, atol=1e-12 * n)
        # the order sorts the positions (ties within rounding may go either way)
        order = np.argsort(res.pi)
        gaps = np.diff(want[order])
        assert np.all(gaps > -1e-9 * n), gaps.min()
        assert res.spans[t] == O.total_span(g, res.pi)
        ranks = res.pi.astype(np.float64)
        assert res.disp[t] == pytest.approx(O.dispersion(g, ranks), rel=1e-12)


def test_ta_stops_when_the_order_converges():
    """The loop ends at the first update that leaves pi unchanged, and not
    before: every earlier update changed the order."""
    rng = np.random.default_rng(150)
    stops = []
    for trial in range(6):
        n = 12
        _, u, v = random_digraph(rng, n, 0.15)
        g = O.Graph(n, u, v)
        boot = rng.permutation(n).astype(np.int32)
        full = O.reorder_ta(g, boot, 40)
        prev = boot
        for t in range(1, full.done + 1):
            cur = O.reorder_ta(g, boot, t)
            assert cur.done == t
            changed = not np.array_equal(cur.pi, prev)
            if t < full.done:
                assert changed, t
            elif full.done < 40:
                assert not changed
            prev = cur.pi
        stops.append(full.done)
        if full.done < 40:
            assert np.array_equal(prev, full.pi)
            again = O.reorder_ta(g, boot, full.done + 3)
            assert again.done == full.done and np.array_equal(again.pi, full.pi)
    # the cases include loops that converge after more than one update
    assert any(1 < d < 40 for d in stops), stops


@pytest.mark.parametrize("seed", [0, 1])
def test_dispersion_is_neighbourhood_variance(seed):
    """J = sum_v 1/d(v) sum_{u in N(v)} (x(u) - mu(v))^2 with mu the mean over
    N(v) is the sum of each neighbourhood's population variance (numpy var)."""
    rng = np.random.default_rng(seed + 160)
    n = 40
    _, u, v = random_digraph(rng, n, 0.1, isolated=2)
    g = O.Graph(n, u, v)
    for x in (rng.permutation(n).astype(np.float64), rng.normal(size=n) * 7):
        want = 0.0
        for w in range(n):
            nb = np.concatenate([[w], u[v == w]])
            want += np.var(x[nb])
        assert O.dispersion(g, x) == pytest.approx(want, rel=1e-12)


def test_ta_order_is_a_permutation_with_consistent_spans():
    rng = np.random.default_rng(120)
    _, u, v = random_digraph(rng, 60, 0.05, isolated=4)
    g = O.Graph(60, u, v)
    boot = rng.permutation(60).astype(np.int32)
    res = O.reorder_ta(g, boot, 4)
    assert np.array_equal(np.sort(res.pi), np.arange(60))
    assert res.spans[0] == O.total_span(g, boot) and res.spans[res.done] == O.total_span(g, res.pi)
    assert res.disp[0] == pytest.approx(O.dispersion(g, boot.astype(np.float64)), rel=1e-12)
    # the order is the ranks of the returned positions, ties by ID
    order = np.lexsort((np.arange(60), res.positions))
    assert np.array_equal(res.pi[order], np.arange(60))


def test_ta_lowers_span_on_skewed_rmat():
    """The trend the paper reports for Alg. 1 (Sec. 3.8, convergence study):
    C(pi) falls from both an uninformed (original / random-ID) bootstrap and
    a locality bootstrap.  Here on the skewed RMAT recipe with random IDs at
    1/400 of its size, from the identity and from the degree/BFS order."""
    from fixtures import workloads as WL
    w = WL.GCN_SKEW_RMAT_50M.scaled(n=125_000, e=2_500_000, chunk=512)
    src, dst = WL.graph(w)
    g = O.Graph(w.n, src, dst)
    for boot in (None, O.reorder_bfs(g)):
        res = O.reorder_ta(g, boot, 5)
        assert res.done == 5
        assert res.spans[1] < res.spans[0] and res.spans[5] < 0.75 * res.spans[0], res.spans
        assert res.spans[5] == O.total_span(g, res.pi)
        # J of the order falls with the span (Sec. 3.8 reports the two track)
        assert res.disp[5] < res.disp[0], res.disp


# ---- RCMK bootstrap (Sec. 3.8 bootstraps Alg. 1 with it)

def test_rcm_matches_scipy():
    """scipy's reverse_cuthill_mckee follows the same textbook rules (minimum
    degree root, children by ascending degree with ties in ID order,
    reversed); on connected graphs with a single minimum-degree vertex its
    order is fully determined, so the two must agree exactly."""
    import scipy.sparse as sp
    from scipy.sparse.csgraph import connected_components, reverse_cuthill_mckee
    rng = np.random.default_rng(140)
    checked = 0
    while checked < 40:
        n = int(rng.integers(5, 120))
        A, u, v = random_digraph(rng, n, float(rng.uniform(0.02, 0.2)))
        S = sp.csr_matrix((A | A.T).astype(np.int32))
        deg = np.diff(S.indptr)
        if u.size == 0 or connected_components(S)[0] != 1 or (deg == deg.min()).sum() != 1:
            continue
        perm = reverse_cuthill_mckee(S, symmetric_mode=True)
        want = np.empty(n, np.int32)
        want[perm] = np.arange(n)
        assert np.array_equal(O.reorder_rcm(O.Graph(n, u, v)), want)
        checked += 1


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_rcm_random_graphs_are_valid(seed):
    rng = np.random.default_rng(seed + 150)
    _, u, v = random_digraph(rng, 60, 0.03, isolated=6)       # several components
    g = O.Graph(60, u, v)
    assert rcm_order_is_valid(g, O.reorder_rcm(g))


def test_rcm_bandwidth_on_shuffled_path_and_grid():
    rng = np.random.default_rng(160)
    # a path with shuffled labels and random edge directions: bandwidth 1
    n = 50
    lab = rng.permutation(n)
    e = [(lab[i], lab[i + 1]) if rng.random() < 0.5 else (lab[i + 1], lab[i]) for i in range(n - 1)]
    g = _g(n, e)
    pi = O.reorder_rcm(g)
    assert np.abs(pi[g.col_dst] - np.repeat(pi[:n], np.diff(g.row_off))).max() == 1
    # a k x k grid with shuffled labels: Cuthill-McKee levels are anti-diagonals,
    # so no edge is longer than 2k - 1 (random labels give about k^2)
    k = 12
    lab = rng.permutation(k * k)
    e = []
    for i in range(k):
        for j in range(k):
            if j + 1 < k:
                e.append((lab[i * k + j], lab[i * k + j + 1]))
            if i + 1 < k:
                e.append((lab[(i + 1) * k + j], lab[i * k + j]))
    g = _g(k * k, e)
    pi = O.reorder_rcm(g)
    src = np.repeat(np.arange(k * k), np.diff(g.row_off))
    assert np.abs(pi[g.col_dst] - pi[src]).max() <= 2 * k - 1
    assert rcm_order_is_valid(g, pi)


def test_rcm_special_cases():
    # no edges: every vertex is a root, in ID order, then reversed
    assert O.reorder_rcm(_g(4, [])).tolist() == [3, 2, 1, 0]
    # a star (hub 0 sends to 1..4): the leaves have degree 1; root 1, then
    # the hub, then leaves 2, 3, 4; reversed
    g = _g(5, [(0, i) for i in range(1, 5)])
    assert O.reorder_rcm(g).tolist() == [3, 4, 2, 1, 0]
    # a reciprocal pair counts once in the symmetric degree: all four degrees
    # are 1, so the search starts at 0 (counted twice, 0 and 1 would have
    # degree 2 and the search would start at 2, giving [1, 0, 3, 2])
    g = _g(4, [(0, 1), (1, 0), (2, 3)])
    assert O.reorder_rcm(g).tolist() == [3, 2, 1, 0]


# ---- residency under a budget: eviction policies (Sec. 3.5.3 and the eviction study)

# Chunks of one source each and a pool of 3 rows: before chunk 3 the pool
# holds vertices 4 and 5 and chunk 3 needs rows for 3 and 6, so one of 4, 5
# goes.  Case 1: 4 took its row first (chunk 0) and was last touched at
# chunk 2 with 3 messages pending; 5 took its row at chunk 1, was last
# touched there and has 1 pending.  Case 2: 4 last touched at chunk 0 with 3
# pending; 5 admitted at chunk 1, touched at chunk 2, 2 pending.  The victim
# is reloaded exactly once, when its next message comes.
RES_CASES = {
    "case1": ([(0, 4), (2, 4), (5, 4), (6, 4), (1, 5), (6, 5), (3, 6)], {"pending": 5, "fifo": 4, "lru": 5}),
    "case2": ([(0, 4), (5, 4), (6, 4), (1, 5), (2, 5), (6, 5), (3, 6)], {"pending": 5, "fifo": 4, "lru": 4}),
}


@pytest.mark.parametrize("case", sorted(RES_CASES))
def test_residency_hand_cases(case):
    edges, victims = RES_CASES[case]
    g = _g(7, edges)
    for policy, victim in victims.items():
        ev, rl, per = O.residency_sim(g, 1, 3, 0, policy)
        want = np.zeros(7, np.int32)
        want[victim] = 1
        assert (ev, rl) == (1, 1) and np.array_equal(per, want), (policy, per)
    # random: the smaller of H(seed, 7, 3, v) >> 50 over v = 4, 5, ties by ID
    for seed in range(6):
        keys = {v: O.hash_u64(seed, 7, 3, v) >> 50 for v in (4, 5)}
        victim = min((4, 5), key=lambda v: (keys[v], v))
        _, _, per = O.residency_sim(g, 1, 3, 0, "random", seed=seed)
        assert per[victim] == 1 and per.sum() == 1
    # a pool too small for one chunk's destinations is refused
    with pytest.raises(RuntimeError):
        O.residency_sim(g, 1, 1, 0)


def test_residency_fifo_readmission():
    # pool of 2 rows, one source per chunk: 3 takes a row at chunk 0, is
    # evicted at chunk 1 for 6, and comes back at chunk 3 (its own self
    # message).  At chunk 4 vertex 4 needs a row: FIFO evicts 6 (admitted at
    # chunk 1), not 3 (admitted again at chunk 3).  6 comes back at chunk 6.
    g = _g(7, [(0, 3), (1, 6), (5, 3)])
    ev, rl, per = O.residency_sim(g, 1, 2, 0, "fifo")
    assert (ev, rl) == (2, 2) and per.tolist() == [0, 0, 0, 1, 0, 0, 1]


def big_pending_graph():
    """Three destinations whose pending counts are all far above 16,383 when
    one of them must go.  One source per chunk, a pool of 4 rows, no hubs.
      chunk 0: vertex 0 sends to A = 1, B = 2, C = 3 (rows: 0, A, B, C);
               0 has no in-edge, completes and frees its row;
      chunks 1-3: the self messages of A, B and C (no new rows);
      chunk 4: vertex 4 sends to 5: rows for 4 and 5, one free, so one of
               A, B, C is evicted, the fewest pending;
      chunk 5: 5 completes; chunks 6..: vertices 6.. send to A (20,000 of
               them), B (the first 17,000) and C (the first 18,000).
    Before chunk 4, pending = in-degree + 1 (self) - 1 (vertex 0) - 1 (own
    chunk): A 20,000, B 17,000, C 18,000, so B is the victim; it is reloaded
    at chunk 6 (two rows free then), and nothing else moves."""
    src = [0, 0, 0, 4]
    dst = [1, 2, 3, 5]
    for j in range(20000):
        w = 6 + j
        src.append(w); dst.append(1)
        if j < 17000:
            src.append(w); dst.append(2)
        if j < 18000:
            src.append(w); dst.append(3)
    return _g(6 + 20000, list(zip(src, dst)))


def test_residency_fewest_pending_is_exact_above_16383():
    """Sec. 3.5.3 ranks candidates by their exact pending count, however
    large (a capped count would tie A, B and C and take the lowest ID, A)."""
    g = big_pending_graph()
    ev, rl, per = O.residency_sim(g, 1, 4, 0, "pending")
    want = np.zeros(g.n, np.int32)
    want[2] = 1
    assert (ev, rl) == (1, 1) and np.array_equal(per, want), np.nonzero(per)


@pytest.mark.parametrize("seed", [0, 1])
def test_residency_invariants(seed):
    """Every eviction is followed by a reload (the victim is still pending);
    hubs never move; with a row for every vertex nothing is evicted."""
    rng = np.random.default_rng(seed + 170)
    _, u, v = random_digraph(rng, 300, 0.02, isolated=10)
    g = O.Graph(300, u, v)
    H = 6
    m = np.diff(g.in_off)
    hubs = np.lexsort((np.arange(300), -m))[:H]
    for policy in O.EVICTION:
        assert O.residency_sim(g, 16, 300, H, policy)[0] == 0
        for S in (150, 100):
            try:
                ev, rl, per = O.residency_sim(g, 16, S, H, policy, seed=3)
            except RuntimeError:
                continue
            assert ev == rl == per.sum() and (per[hubs] == 0).all()


def test_fewest_pending_reloads_least():
    """The eviction study's finding: evicting the states with the fewest
    pending messages causes fewer reloads than random, FIFO or LRU choices.
    Checked on the C4 recipe (RMAT, random IDs) at 1/2000 of its size with 1%
    hubs and a pool of 35% of the rows."""
    import dataclasses
    from fixtures import workloads as WL
    w = dataclasses.replace(WL.SAGE_OOC_RMAT_269M, random_ids=True).scaled(n=1 << 17, e=1 << 21, chunk=1024)
    src, dst = WL.graph(w)
    g = O.Graph(w.n, src, dst)
    H, S = int(np.ceil(0.01 * w.n)), int(0.35 * w.n)
    reloads = {p: O.residency_sim(g, w.chunk, S, H, p, seed=4)[1] for p in O.EVICTION}
    assert reloads["pending"] > 0
    assert all(reloads["pending"] < reloads[p] for p in ("random", "fifo", "lru")), reloads


# ---- GATConv (Sec. 3.9): single head, self message in every neighbourhood

def dense_gat(A, H, W, attn, b, relu, slope=0.2):
    """Dense GAT: scores on (A + I), column softmax, attention-weighted rows."""
    Hp = H @ W.T
    s, t = Hp @ attn[0], Hp @ attn[1]
    M = A.astype(bool) | np.eye(A.shape[0], dtype=bool)      # M[u, v]: u sends to v
    E = s[:, None] + t[None, :]
    E = np.where(E > 0, E, slope * E)
    E = np.where(M, E, -np.inf)
    P = np.exp(E - E.max(axis=0, keepdims=True))
    P /= P.sum(axis=0, keepdims=True)                       # P[u, v] = alpha_uv
    z = P.T @ Hp + b
    return np.maximum(z, 0) if relu else z


@pytest.mark.parametrize("sampled,relu", [(False, True), (False, False), (True, True)])
def test_gat_matches_dense(sampled, relu):
    rng = np.random.default_rng(210 + 2 * sampled + relu)
    n, d_in, d_out = 80, 7, 6
    A, u, v = random_digraph(rng, n, 0.09, isolated=4)
    g = O.Graph(n, u, v)
    H32 = rng.standard_normal((n, d_in)).astype(np.float32)
    W = rng.standard_normal((d_out, d_in))
    attn = rng.standard_normal((2, d_out))
    b = rng.standard_normal(d_out)
    keep_in, A_used = None, A
    if sampled:
        words, keep_in, _ = O.sample(g, 9, 1, 3)
        bits = O.mask_bits(words, g.e)
        A_used = np.zeros_like(A)
        A_used[np.repeat(np.arange(n), np.diff(g.row_off))[bits], g.col_dst[bits]] = True
    got = O.gat_layer(g, H32, O.F32, W, attn, b, relu, keep_in=keep_in)
    np.testing.assert_allclose(got, dense_gat(A_used, H32.astype(np.float64), W, attn, b, relu),
                               rtol=1e-11, atol=1e-11)


def test_gat_special_cases():
    rng = np.random.default_rng(220)
    n, d_in, d_out = 50, 5, 4
    A, u, v = random_digraph(rng, n, 0.1, isolated=3)
    g = O.Graph(n, u, v)
    H = rng.standard_normal((n, d_in)).astype(np.float32)
    W = rng.standard_normal((d_out, d_in))
    Hp = H.astype(np.float64) @ W.T
    M = (A | np.eye(n, dtype=bool)).astype(np.float64)
    mean = (M.T @ Hp) / M.sum(axis=0)[:, None]
    # zero attention, or attention on the destination only: every score of a
    # neighbourhood is equal, so GAT is the mean over N(v) and v
    for attn in (np.zeros((2, d_out)), np.stack([np.zeros(d_out), rng.standard_normal(d_out)])):
        np.testing.assert_allclose(O.gat_layer(g, H, O.F32, W, attn, None, False), mean, rtol=1e-12, atol=1e-12)
    # a vertex without in-edges attends only to itself
    iso = np.flatnonzero(np.diff(g.in_off) == 0)
    z = O.gat_layer(g, H, O.F32, W, rng.standard_normal((2, d_out)), None, False, dst_ids=iso)
    np.testing.assert_allclose(z, Hp[iso], rtol=1e-12, atol=1e-12)
