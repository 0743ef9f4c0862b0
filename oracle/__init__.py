"""ORACLE -- test infrastructure only.

numpy front end of ``oracle.c``: a plain, slow, destination-centric CPU
reference for layer-wise GNN inference (Taurus, arXiv 2607.17374), in fp64.
Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the GPU library
in ``paper_2607_17374_amd``; the only common code is the seeded input
generator in ``fixtures``.

Every function is pinned by the CPU tests in ``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import NamedTuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "oracle.c")

F32, BF16, F16 = 0, 1, 2
SAGE_MEAN, GCN_SYM, GIN_SUM, GAT_ATT, GIN_MLP = 0, 1, 2, 3, 4


def build(force: bool = True) -> str:
    if force or not os.path.exists(_SO):
        tmp = _SO + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _SO)
    return _SO


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        _lib = load(_SO)
    return _lib


def load(path: str):
    """Open a compiled oracle library and declare its entry points."""
    L = ctypes.CDLL(path)
    i64, u64, i32, vp = ctypes.c_int64, ctypes.c_uint64, ctypes.c_int, ctypes.c_void_p
    L.or_build_csr.restype = i32
    L.or_build_csr.argtypes = [i64, i64, vp, vp, vp, vp]
    L.or_build_in_lists.restype = i32
    L.or_build_in_lists.argtypes = [i64, vp, vp, vp, vp, vp]
    L.or_hash.restype = u64
    L.or_hash.argtypes = [u64, u64, i32, vp]
    L.or_sample.restype = None
    L.or_sample.argtypes = [i64, vp, vp, vp, vp, u64, i64, i64, vp, vp, vp]
    L.or_round_store.restype = None
    L.or_round_store.argtypes = [i64, vp, i32, vp]
    L.or_widen.restype = None
    L.or_widen.argtypes = [i64, vp, i32, vp]
    L.or_layer.restype = i32
    L.or_layer.argtypes = [i32, i64, vp, vp, vp, vp, vp, i32, i64, vp, vp, i64, i32, i64, vp, vp]
    L.or_gat_layer.restype = i32
    L.or_gat_layer.argtypes = [i64, vp, vp, vp, vp, i32, i64, vp, vp, vp, i64, i32, ctypes.c_double, i64, vp, vp]
    L.or_reorder_bfs.restype = i32
    L.or_reorder_bfs.argtypes = [i64, vp, vp, vp]
    L.or_reorder_rcm.restype = i32
    L.or_reorder_rcm.argtypes = [i64, vp, vp, vp, vp, vp]
    L.or_total_span.restype = i64
    L.or_active_profile.restype = None
    L.or_residency_sim.restype = i32
    L.or_residency_sim.argtypes = [i64, vp, vp, vp, i64, i64, i64, i32, u64, vp, vp, vp]
    L.or_active_profile.argtypes = [i64, vp, vp, vp, i64, vp]
    L.or_total_span.argtypes = [i64, vp, vp, vp]
    L.or_threads.restype = i32
    L.or_threads.argtypes = []
    L.or_in_lists_from_edges.restype = i32
    L.or_in_lists_from_edges.argtypes = [i64, i64, vp, vp, vp, vp, vp]
    L.or_digest_edges.restype = None
    L.or_digest_edges.argtypes = [i64, vp, vp, vp]
    L.or_digest_csr.restype = None
    L.or_digest_csr.argtypes = [i64, vp, vp, vp, vp]
    L.or_digest_in_lists.restype = None
    L.or_digest_in_lists.argtypes = [i64, vp, vp, vp, vp]
    L.or_csr_check.restype = i32
    L.or_csr_check.argtypes = [i64, i64, vp, vp]
    L.or_ta_step.restype = None
    L.or_ta_step.argtypes = [i64, vp, vp, vp, vp, vp, vp, vp]
    L.or_reorder_ta.restype = i32
    L.or_reorder_ta.argtypes = [i64, vp, vp, vp, vp, vp, i32, vp, vp, vp, vp, vp]
    L.or_gin_mlp_layer.restype = i32
    L.or_gin_mlp_layer.argtypes = [i64, vp, vp, vp, vp, i32, i64, vp, vp, i64, vp, vp, i64, i32, i64, vp, vp]
    L.or_dispersion.restype = ctypes.c_double
    L.or_dispersion.argtypes = [i64, vp, vp, vp]
    return L


def threads() -> int:
    return int(lib().or_threads())


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class Graph:
    """CSR by source plus in-neighbour lists, built by the oracle."""

    def __init__(self, n: int, src: np.ndarray, dst: np.ndarray, check_simple: bool = True):
        src = np.ascontiguousarray(src, np.int32)
        dst = np.ascontiguousarray(dst, np.int32)
        e = src.size
        self.n, self.e = n, e
        self.row_off = np.empty(n + 1, np.int64)
        self.col_dst = np.empty(e, np.int32)
        rc = lib().or_build_csr(n, e, _p(src), _p(dst), _p(self.row_off), _p(self.col_dst))
        if rc == -2 or rc == -3 or (rc == -1 and check_simple):
            raise ValueError(f"or_build_csr: {rc}")
        self.simple = rc == 0
        self.in_off = np.empty(n + 1, np.int64)
        self.in_src = np.empty(e, np.int32)
        self.in_pos = np.empty(e, np.int64)
        rc = lib().or_build_in_lists(n, _p(self.row_off), _p(self.col_dst), _p(self.in_off),
                                     _p(self.in_src), _p(self.in_pos))
        if rc:
            raise MemoryError("or_build_in_lists")
        self.deg_out = np.diff(self.row_off).astype(np.int32)
        self.deg_in = np.diff(self.in_off).astype(np.int32)


class EdgeGraph:
    """In-neighbour lists and out-degrees built straight from the edge list
    (no CSR and no sort of the pairs), for graphs too large for ``Graph``.
    Usable by ``layer``, ``sample`` (keep_in and m only) and
    ``reorder_bfs``; with out_lists also the CSR (the out-lists, built the
    same way from the reversed pairs), which ``reorder_ta`` needs."""

    def __init__(self, n: int, src: np.ndarray, dst: np.ndarray, out_lists: bool = False):
        src = np.ascontiguousarray(src, np.int32)
        dst = np.ascontiguousarray(dst, np.int32)
        self.n, self.e = n, src.size
        self.in_off = np.empty(n + 1, np.int64)
        self.in_src = np.empty(self.e, np.int32)
        self.deg_out = np.empty(n, np.int32)
        if lib().or_in_lists_from_edges(n, self.e, _p(src), _p(dst), _p(self.in_off), _p(self.in_src),
                                        _p(self.deg_out)):
            raise MemoryError("or_in_lists_from_edges")
        self.deg_in = np.diff(self.in_off).astype(np.int32)
        self.row_off = None
        self.col_dst = None
        self.in_pos = None
        if out_lists:
            self.row_off = np.empty(n + 1, np.int64)
            self.col_dst = np.empty(self.e, np.int32)
            scratch = np.empty(n, np.int32)
            if lib().or_in_lists_from_edges(n, self.e, _p(dst), _p(src), _p(self.row_off), _p(self.col_dst),
                                            _p(scratch)):
                raise MemoryError("or_in_lists_from_edges")


def digest_edges(src: np.ndarray, dst: np.ndarray) -> tuple:
    """(count, sum, xor) set digest of the pairs (src[i], dst[i])."""
    src = np.ascontiguousarray(src, np.int32)
    dst = np.ascontiguousarray(dst, np.int32)
    out = np.zeros(3, np.uint64)
    lib().or_digest_edges(src.size, _p(src), _p(dst), _p(out))
    return tuple(int(x) for x in out)


def digest_csr(n: int, row_off: np.ndarray, col_dst: np.ndarray, mask_words: np.ndarray | None = None) -> tuple:
    """Set digest of a CSR's edges (only those whose mask bit is set, if given)."""
    row_off = np.ascontiguousarray(row_off, np.int64)
    col_dst = np.ascontiguousarray(col_dst, np.int32)
    mw = None if mask_words is None else np.ascontiguousarray(mask_words, np.uint64)
    out = np.zeros(3, np.uint64)
    lib().or_digest_csr(n, _p(row_off), _p(col_dst), _p(mw), _p(out))
    return tuple(int(x) for x in out)


def digest_in_lists(g, keep_in: np.ndarray | None = None) -> tuple:
    """Set digest of the (u, v) pairs of g's in-lists (kept entries only, if given)."""
    kin = None if keep_in is None else np.ascontiguousarray(keep_in, np.uint8)
    out = np.zeros(3, np.uint64)
    lib().or_digest_in_lists(g.n, _p(g.in_off), _p(g.in_src), _p(kin), _p(out))
    return tuple(int(x) for x in out)


def csr_check(n: int, row_off: np.ndarray, col_dst: np.ndarray) -> int:
    """0 if the CSR has the canonical shape (see or_csr_check), else the rule it breaks."""
    row_off = np.ascontiguousarray(row_off, np.int64)
    col_dst = np.ascontiguousarray(col_dst, np.int32)
    return int(lib().or_csr_check(n, col_dst.size, _p(row_off), _p(col_dst)))


def hash_u64(seed: int, tag: int, *args: int) -> int:
    a = np.array(args, dtype=np.uint64) if args else np.zeros(1, np.uint64)
    return int(lib().or_hash(seed & (2**64 - 1), tag, len(args), _p(a)))


def sample(g, seed: int, layer: int, k: int):
    """Fanout mask of one layer -> (mask_words uint64[ceil(e/64)], keep_in uint8[e], m int32[n]).
    For an EdgeGraph (no CSR positions) mask_words is None."""
    words = np.zeros((g.e + 63) // 64, np.uint64) if g.in_pos is not None else None
    keep_in = np.zeros(g.e, np.uint8)
    m = np.zeros(g.n, np.int32)
    lib().or_sample(g.n, _p(g.row_off), _p(g.in_off), _p(g.in_src), _p(g.in_pos),
                    seed & (2**64 - 1), layer, k, _p(words), _p(keep_in), _p(m))
    return words, keep_in, m


def layer(agg: int, g: Graph, H: np.ndarray, h_dtype: int, W: np.ndarray, b: np.ndarray | None,
          relu: bool, keep_in: np.ndarray | None = None, dst_ids: np.ndarray | None = None) -> np.ndarray:
    """One layer in fp64 for ``dst_ids`` (all vertices if None).

    ``W`` in the paper's orientation (rows = d_out; SAGE cols = 2 d_in =
    [W_agg | W_self]); ``H`` is the layer input in its storage dtype (16-bit
    types as uint16 bit patterns)."""
    H = np.ascontiguousarray(H)
    d_in = H.shape[1]
    W = np.ascontiguousarray(W, np.float64)
    d_out = W.shape[0]
    cols = 2 * d_in if agg == SAGE_MEAN else d_in
    assert W.shape[1] == cols, (W.shape, cols)
    bb = None if b is None else np.ascontiguousarray(b, np.float64)
    ids = None if dst_ids is None else np.ascontiguousarray(dst_ids, np.int64)
    count = g.n if ids is None else ids.size
    out = np.empty((count, d_out), np.float64)
    kin = None if keep_in is None else np.ascontiguousarray(keep_in, np.uint8)
    deg_out = g.deg_out
    if kin is not None:
        # a sampled layer propagates over the kept edges: their out-degrees
        deg_out = np.bincount(g.in_src[kin != 0], minlength=g.n).astype(np.int32)
    rc = lib().or_layer(agg, g.n, _p(g.in_off), _p(g.in_src), _p(kin), _p(deg_out),
                        _p(H), h_dtype, d_in, _p(W), _p(bb), d_out, int(relu),
                        count, _p(ids), _p(out))
    if rc:
        raise RuntimeError(f"or_layer: {rc}")
    return out


def gin_mlp_layer(g, H: np.ndarray, h_dtype: int, W1: np.ndarray, b1: np.ndarray | None, W2: np.ndarray,
                  b2: np.ndarray | None, relu: bool, keep_in: np.ndarray | None = None,
                  dst_ids: np.ndarray | None = None) -> np.ndarray:
    """GIN layer with a two-layer perceptron apply function (eps = 0) in fp64
    for ``dst_ids`` (all if None): W1 [d_h][d_in], W2 [d_out][d_h]."""
    H = np.ascontiguousarray(H)
    d_in = H.shape[1]
    W1 = np.ascontiguousarray(W1, np.float64)
    W2 = np.ascontiguousarray(W2, np.float64)
    d_h, d_out = W1.shape[0], W2.shape[0]
    assert W1.shape[1] == d_in and W2.shape[1] == d_h
    c1 = None if b1 is None else np.ascontiguousarray(b1, np.float64)
    c2 = None if b2 is None else np.ascontiguousarray(b2, np.float64)
    ids = None if dst_ids is None else np.ascontiguousarray(dst_ids, np.int64)
    count = g.n if ids is None else ids.size
    out = np.empty((count, d_out), np.float64)
    kin = None if keep_in is None else np.ascontiguousarray(keep_in, np.uint8)
    rc = lib().or_gin_mlp_layer(g.n, _p(g.in_off), _p(g.in_src), _p(kin), _p(H), h_dtype, d_in, _p(W1), _p(c1),
                                d_h, _p(W2), _p(c2), d_out, int(relu), count, _p(ids), _p(out))
    if rc:
        raise RuntimeError(f"or_gin_mlp_layer: {rc}")
    return out


GAT_SLOPE = 0.2   # LeakyReLU negative slope of the attention scores


def gat_layer(g: Graph, H: np.ndarray, h_dtype: int, W: np.ndarray, attn: np.ndarray, b: np.ndarray | None,
              relu: bool, keep_in: np.ndarray | None = None, dst_ids: np.ndarray | None = None,
              slope: float = GAT_SLOPE) -> np.ndarray:
    """Single-head GAT layer in fp64 for ``dst_ids`` (all if None).  W [d_out][d_in];
    attn [2][d_out] (row 0 source, row 1 destination)."""
    H = np.ascontiguousarray(H)
    d_in = H.shape[1]
    W = np.ascontiguousarray(W, np.float64)
    d_out = W.shape[0]
    assert W.shape[1] == d_in and np.shape(attn) == (2, d_out)
    a = np.ascontiguousarray(attn, np.float64)
    bb = None if b is None else np.ascontiguousarray(b, np.float64)
    ids = None if dst_ids is None else np.ascontiguousarray(dst_ids, np.int64)
    count = g.n if ids is None else ids.size
    out = np.empty((count, d_out), np.float64)
    kin = None if keep_in is None else np.ascontiguousarray(keep_in, np.uint8)
    rc = lib().or_gat_layer(g.n, _p(g.in_off), _p(g.in_src), _p(kin), _p(H), h_dtype, d_in, _p(W), _p(a), _p(bb),
                            d_out, int(relu), float(slope), count, _p(ids), _p(out))
    if rc:
        raise MemoryError("or_gat_layer")
    return out


def round_store(x: np.ndarray, dtype: int) -> np.ndarray:
    """fp64 -> fp32 -> (bf16 | fp16), round to nearest even; 16-bit as uint16 bits."""
    x = np.ascontiguousarray(x, np.float64)
    out = np.empty(x.shape, np.float32 if dtype == F32 else np.uint16)
    lib().or_round_store(x.size, _p(x), dtype, _p(out))
    return out


def widen(x: np.ndarray, dtype: int) -> np.ndarray:
    x = np.ascontiguousarray(x)
    out = np.empty(x.shape, np.float64)
    lib().or_widen(x.size, _p(x), dtype, _p(out))
    return out


def reorder_bfs(g: Graph) -> np.ndarray:
    out = np.empty(g.n, np.int32)
    if lib().or_reorder_bfs(g.n, _p(g.in_off), _p(g.in_src), _p(out)):
        raise MemoryError("or_reorder_bfs")
    return out


def reorder_rcm(g: Graph) -> np.ndarray:
    """RCMK order of the symmetrised graph (Sec. 3.8's bootstrap) -> new_of_old int32[n]."""
    out = np.empty(g.n, np.int32)
    if lib().or_reorder_rcm(g.n, _p(g.row_off), _p(g.col_dst), _p(g.in_off), _p(g.in_src), _p(out)):
        raise MemoryError("or_reorder_rcm")
    return out


def ta_step(g: Graph, r: np.ndarray):
    """One update of Alg. 1 (Sec. 3.8): positions r -> (centres mu, new positions r)."""
    r = np.ascontiguousarray(r, np.float64)
    mu = np.empty(g.n, np.float64)
    r2 = np.empty(g.n, np.float64)
    lib().or_ta_step(g.n, _p(g.row_off), _p(g.col_dst), _p(g.in_off), _p(g.in_src), _p(r), _p(mu), _p(r2))
    return mu, r2


class TaResult(NamedTuple):
    """Result of Alg. 1: the order, the real positions it ranks, and per update
    (index 0 = the bootstrap) the total span C(pi) and the dispersion J(pi)."""
    pi: np.ndarray          # int32[n], new ID of each vertex
    positions: np.ndarray   # float64[n], r after the last update made
    spans: np.ndarray       # int64[iterations + 1]; 0 past the last update made
    disp: np.ndarray        # float64[iterations + 1]; 0 past the last update made
    done: int               # updates made


def reorder_ta(g: Graph, pi0: np.ndarray | None = None, iterations: int = 5) -> TaResult:
    """Alg. 1 (Sec. 3.8) from bootstrap pi0 (identity if None): r = pi0 once,
    then per update mu*, r*, pi = ArgSort(r) (ties by ID), carrying r forward,
    until pi stops changing or after ``iterations`` updates."""
    pi = np.empty(g.n, np.int32)
    pos = np.empty(g.n, np.float64)
    spans = np.zeros(iterations + 1, np.int64)
    disp = np.zeros(iterations + 1, np.float64)
    done = ctypes.c_int(0)
    p0 = None if pi0 is None else np.ascontiguousarray(pi0, np.int32)
    if lib().or_reorder_ta(g.n, _p(g.row_off), _p(g.col_dst), _p(g.in_off), _p(g.in_src), _p(p0), iterations,
                           _p(pi), _p(pos), _p(spans), _p(disp), ctypes.byref(done)):
        raise MemoryError("or_reorder_ta")
    return TaResult(pi, pos, spans, disp, done.value)


def dispersion(g: Graph, x: np.ndarray) -> float:
    """J of Sec. 3.8 for positions x (float64[n], or the ranks of an order) at
    the centres mu*(x), the self message in every neighbourhood."""
    x = np.ascontiguousarray(x, np.float64)
    return float(lib().or_dispersion(g.n, _p(g.in_off), _p(g.in_src), _p(x)))


def total_span(g: Graph, pi: np.ndarray) -> int:
    """C(pi) of Sec. 3.8 with the self message in every neighbourhood."""
    pi = np.ascontiguousarray(pi, np.int32)
    return int(lib().or_total_span(g.n, _p(g.in_off), _p(g.in_src), _p(pi)))


def active_profile(g: Graph, pi: np.ndarray, chunk: int) -> np.ndarray:
    """A[k] of Sec. 3.8 at chunk granularity: destinations holding a partial
    state after chunk k of the order pi (self message included)."""
    pi = np.ascontiguousarray(pi, np.int32)
    A = np.empty((g.n + chunk - 1) // chunk, np.int64)
    lib().or_active_profile(g.n, _p(g.in_off), _p(g.in_src), _p(pi), chunk, _p(A))
    return A


EVICTION = {"pending": 0, "random": 1, "fifo": 2, "lru": 3}


def residency_sim(g: Graph, chunk: int, slots: int, hubs: int, policy: str = "pending", seed: int = 0,
                  keep: np.ndarray | None = None):
    """Slot-level simulation of a budgeted layer's residency (Sec. 3.5) ->
    (evictions, reloads, reloads per vertex int32[n]).  keep: bool per CSR
    edge (propagated edges of a sampled layer), None = every edge.  Raises
    RuntimeError when the pool cannot free enough rows."""
    ev, rl = ctypes.c_int64(0), ctypes.c_int64(0)
    per = np.zeros(g.n, np.int32)
    kp = None if keep is None else np.ascontiguousarray(keep, np.uint8)
    rc = lib().or_residency_sim(g.n, _p(g.row_off), _p(g.col_dst), _p(kp), chunk, slots, hubs, EVICTION[policy],
                                seed & (2**64 - 1), ctypes.byref(ev), ctypes.byref(rl), _p(per))
    if rc == -3:
        raise MemoryError("or_residency_sim")
    if rc:
        raise RuntimeError("residency: the pool cannot free enough rows")
    return ev.value, rl.value, per


def mask_bits(words: np.ndarray, e: int) -> np.ndarray:
    """Unpack a little-endian bit mask (bit i of word i//64) into a bool array of length e."""
    b = np.unpackbits(np.ascontiguousarray(words, np.uint64).view(np.uint8), bitorder="little")
    return b[:e].astype(bool)


def run_model(w, g: Graph, X: np.ndarray, params):
    """Full-graph layer-wise inference through every layer of workload ``w``.

    Returns the list of per-layer outputs in storage dtype (hidden layers in
    the workload's feature dtype, last layer fp32), and the fp64 outputs of
    the last layer.  Sampled layers draw their fanout masks with the oracle's
    own sampler."""
    H, h_dtype = X, w.feat_dtype
    outs = []
    z = None
    for li in range(1, w.layers + 1):
        p = params[li - 1]
        keep = None
        if w.fanout(li) > 0:
            _, keep, _ = sample(g, w.seed, li, w.fanout(li))
        relu = li < w.layers
        if w.agg == GAT_ATT:
            z = gat_layer(g, H, h_dtype, p.W, p.attn, p.b, relu, keep_in=keep)
        else:
            z = layer(w.agg, g, H, h_dtype, p.W, p.b, relu, keep_in=keep)
        _, out_dtype = w.layer_dtypes(li)
        H = round_store(z, out_dtype)
        h_dtype = out_dtype
        outs.append(H)
    return outs, z
