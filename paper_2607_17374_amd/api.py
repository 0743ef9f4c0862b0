"""Torch-facing wrapper of the C ABI.

Torch provides device memory and streams; each function below only turns
tensors into pointers and calls the library.  Names follow the C ABI:
``build_csr`` = taurus_build_csr, ``Layer`` = taurus_layer_init / push_chunk /
finalize / sampled_edges / destroy.
"""
from __future__ import annotations

import ctypes
from typing import NamedTuple, Optional, Sequence

import numpy as np
import torch

from . import _native as N

_TORCH_DTYPE = {N.F32: torch.float32, N.BF16: torch.bfloat16, N.F16: torch.float16}


def torch_dtype(code: int):
    return _TORCH_DTYPE[code]


def _stream_ptr(stream: Optional[torch.cuda.Stream]) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _dev_ptr(t: torch.Tensor, dtype: torch.dtype, what: str) -> int:
    if not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{what} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return t.data_ptr()


def _buf_ptr(t: torch.Tensor, dtype: torch.dtype, what: str):
    """(pointer, on_host) of a device tensor or of a pinned host tensor."""
    if t.dtype != dtype:
        raise ValueError(f"{what} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if t.is_cuda:
        return t.data_ptr(), 0
    if not t.is_pinned():
        raise ValueError(f"{what} on the host must be pinned memory")
    return t.data_ptr(), 1


def hash_u64(seed: int, tag: int, *args: int) -> int:
    a = (ctypes.c_uint64 * max(1, len(args)))(*args)
    return int(N.lib().taurus_hash(seed & (2**64 - 1), tag, len(args), ctypes.cast(a, ctypes.c_void_p)))


def build_csr(n: int, src: torch.Tensor, dst: torch.Tensor, stream=None):
    """taurus_build_csr: device edge list (int32) -> (row_off int64[n+1], col_dst int32[e])."""
    e = src.numel()
    row_off = torch.empty(n + 1, dtype=torch.int64, device=src.device)
    col_dst = torch.empty(max(e, 1), dtype=torch.int32, device=src.device)[:e]
    N.check(N.lib().taurus_build_csr(n, e, _dev_ptr(src, torch.int32, "src"), _dev_ptr(dst, torch.int32, "dst"),
                                     row_off.data_ptr(), col_dst.data_ptr() if e else None,
                                     _stream_ptr(stream)), "taurus_build_csr")
    return row_off, col_dst


NOALLOC_MAX_EDGES = N.NOALLOC_MAX_EDGES


def build_csr_noalloc(n: int, src: torch.Tensor, dst: torch.Tensor, row_off: torch.Tensor, col_dst: torch.Tensor,
                      stream=None) -> None:
    """taurus_build_csr_noalloc: the CSR build into caller-allocated row_off
    (int64[n+1]) and col_dst (int32[e]) with no device allocation by the
    library or by this wrapper; at most NOALLOC_MAX_EDGES edges."""
    e = src.numel()
    if row_off.numel() != n + 1 or col_dst.numel() != e:
        raise ValueError("row_off must hold n + 1 and col_dst e entries")
    N.check(N.lib().taurus_build_csr_noalloc(n, e, _dev_ptr(src, torch.int32, "src"),
                                             _dev_ptr(dst, torch.int32, "dst"),
                                             _dev_ptr(row_off, torch.int64, "row_off"),
                                             _dev_ptr(col_dst, torch.int32, "col_dst") if e else None,
                                             _stream_ptr(stream)), "taurus_build_csr_noalloc")


def _graph(n: int, row_off: torch.Tensor, col_dst: torch.Tensor) -> N.Graph:
    e = col_dst.numel()
    return N.Graph(n, e, _dev_ptr(row_off, torch.int64, "row_off"), _dev_ptr(col_dst, torch.int32, "col_dst") if e else None)


def reorder(n: int, row_off: torch.Tensor, col_dst: torch.Tensor, stream=None) -> torch.Tensor:
    """taurus_reorder: degree/BFS order, new_of_old int32[n] on the device."""
    g = _graph(n, row_off, col_dst)
    out = torch.empty(n, dtype=torch.int32, device=row_off.device)
    N.check(N.lib().taurus_reorder(ctypes.byref(g), out.data_ptr(), _stream_ptr(stream)), "taurus_reorder")
    return out


def reorder_rcm(n: int, row_off: torch.Tensor, col_dst: torch.Tensor, stream=None) -> torch.Tensor:
    """taurus_reorder_rcm: RCMK order of the symmetrised graph, new_of_old int32[n] on the device."""
    g = _graph(n, row_off, col_dst)
    out = torch.empty(n, dtype=torch.int32, device=row_off.device)
    N.check(N.lib().taurus_reorder_rcm(ctypes.byref(g), out.data_ptr(), _stream_ptr(stream)), "taurus_reorder_rcm")
    return out


class TaOrder(NamedTuple):
    """taurus_reorder_ta's outputs: the order and positions on the device, and
    per update (index 0 = the bootstrap) C(pi) and J(pi) on the host."""
    pi: torch.Tensor         # int32[n], new ID of each vertex
    positions: torch.Tensor  # float64[n], r after the last update made
    spans: np.ndarray        # int64[iterations + 1]
    disp: np.ndarray         # float64[iterations + 1]
    done: int                # updates made


def reorder_ta(n: int, row_off: torch.Tensor, col_dst: torch.Tensor, pi0: Optional[torch.Tensor] = None,
               iterations: int = 5, stream=None) -> TaOrder:
    """taurus_reorder_ta: topology-aware order (Alg. 1) from bootstrap pi0
    (identity if None)."""
    g = _graph(n, row_off, col_dst)
    out = torch.empty(n, dtype=torch.int32, device=row_off.device)
    pos = torch.empty(n, dtype=torch.float64, device=row_off.device)
    spans = np.zeros(iterations + 1, dtype=np.int64)
    disp = np.zeros(iterations + 1, dtype=np.float64)
    done = ctypes.c_int32(0)
    p0 = None if pi0 is None else _dev_ptr(pi0, torch.int32, "pi0")
    N.check(N.lib().taurus_reorder_ta(ctypes.byref(g), p0, iterations, out.data_ptr(), pos.data_ptr(),
                                      spans.ctypes.data, disp.ctypes.data, ctypes.byref(done),
                                      _stream_ptr(stream)), "taurus_reorder_ta")
    return TaOrder(out, pos, spans, disp, done.value)


def relabel_graph(n: int, row_off: torch.Tensor, col_dst: torch.Tensor, new_of_old: torch.Tensor, stream=None):
    """taurus_relabel_graph: CSR of the graph with vertex v renamed new_of_old[v]."""
    g = _graph(n, row_off, col_dst)
    e = col_dst.numel()
    r2 = torch.empty(n + 1, dtype=torch.int64, device=row_off.device)
    c2 = torch.empty(max(e, 1), dtype=torch.int32, device=row_off.device)[:e]
    N.check(N.lib().taurus_relabel_graph(ctypes.byref(g), _dev_ptr(new_of_old, torch.int32, "new_of_old"),
                                         r2.data_ptr(), c2.data_ptr() if e else None, _stream_ptr(stream)),
            "taurus_relabel_graph")
    return r2, c2


def permute_rows(x: torch.Tensor, new_of_old: torch.Tensor, inverse: bool = False, stream=None) -> torch.Tensor:
    """taurus_permute_rows: rows of x [n][...] into the new numbering
    (out[new_of_old[v]] = x[v]), or back (inverse: out[v] = x[new_of_old[v]])."""
    if not x.is_cuda or not x.is_contiguous():
        raise ValueError("x must be a contiguous device tensor")
    n = x.shape[0]
    out = torch.empty_like(x)
    row_bytes = x[0].numel() * x.element_size() if n else 0
    N.check(N.lib().taurus_permute_rows(x.data_ptr(), out.data_ptr(), n, row_bytes,
                                        _dev_ptr(new_of_old, torch.int32, "new_of_old"), int(inverse),
                                        _stream_ptr(stream)), "taurus_permute_rows")
    return out


def release_cached_memory(nbytes: int = 0) -> int:
    """taurus_release_cached_memory: hand the library's cached device blocks
    back to the runtime, smallest first, until at least nbytes are freed (0:
    all).  Returns the bytes freed."""
    r = N.lib().taurus_release_cached_memory(int(nbytes))
    if r < 0:
        raise N.TaurusError(int(r), "taurus_release_cached_memory", N.last_error())
    return int(r)


def alloc_device(shape, dtype, device) -> torch.Tensor:
    """torch.empty, handing back as much of the library's cached memory as
    the allocation lacks (and retrying) when the device is out of memory."""
    try:
        return torch.empty(shape, dtype=dtype, device=device)
    except torch.OutOfMemoryError:
        need = int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size()
        free, _ = torch.cuda.mem_get_info(device)
        release_cached_memory(max(need - free, 0) + (1 << 30))
        torch.cuda.empty_cache()
        return torch.empty(shape, dtype=dtype, device=device)


_hip = None


def alloc_pinned(shape, dtype) -> torch.Tensor:
    """Pinned host tensor of exactly this size (hipHostMalloc; torch's pinned
    allocator rounds large blocks up to a power of two, which matters where
    pinned memory is capped).  Freed when the last tensor viewing it goes."""
    import weakref
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipHostMalloc.restype = ctypes.c_int
        _hip.hipHostMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t, ctypes.c_uint]
        _hip.hipHostFree.restype = ctypes.c_int
        _hip.hipHostFree.argtypes = [ctypes.c_void_p]
    nbytes = max(1, int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size())
    p = ctypes.c_void_p()
    rc = _hip.hipHostMalloc(ctypes.byref(p), nbytes, 0)
    if rc != 0 or not p.value:
        raise MemoryError(f"hipHostMalloc({nbytes}) failed ({rc})")
    buf = (ctypes.c_uint8 * nbytes).from_address(p.value)
    weakref.finalize(buf, _hip.hipHostFree, p.value)
    t = torch.frombuffer(buf, dtype=torch.uint8)
    return t[:nbytes].view(dtype).view(shape) if shape else t.view(dtype)


# eviction policies of a budgeted layer (taurus_eviction)
EVICTION = {"pending": N.EVICT_PENDING, "random": N.EVICT_RANDOM, "fifo": N.EVICT_FIFO, "lru": N.EVICT_LRU}


class Plan:
    """taurus_plan_create / taurus_plan_destroy: the per-graph structures
    (exact chunk index, in-edge lists for sampling) for one chunk size,
    shared by the layers over it and built by the first layer that needs
    each."""

    def __init__(self, n: int, row_off: torch.Tensor, col_dst: torch.Tensor, chunk: int, stream=None):
        self._h = ctypes.c_void_p()
        e = col_dst.numel()
        self.graph = N.Graph(n, e, _dev_ptr(row_off, torch.int64, "row_off"), col_dst.data_ptr() if e else None)
        self.chunk = chunk
        self._keep = (row_off, col_dst)
        N.check(N.lib().taurus_plan_create(ctypes.byref(self.graph), chunk, _stream_ptr(stream),
                                           ctypes.byref(self._h)), "taurus_plan_create")

    @property
    def handle(self):
        return self._h.value

    def destroy(self) -> None:
        if self._h:
            N.lib().taurus_plan_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


class Layer:
    """One layer handle (taurus_layer_init ... taurus_layer_destroy)."""

    def __init__(self, n: int, row_off: torch.Tensor, col_dst: torch.Tensor, *, agg: int, d_in: int,
                 d_out: int, weight_cat: np.ndarray, bias: Optional[np.ndarray], out: torch.Tensor,
                 in_dtype: int = N.F32, out_dtype: int = N.F32, relu: bool = False, fanout: int = 0,
                 layer: int = 1, seed: int = 0, chunk: int = 65536, hbm_budget: int = 0,
                 hub_fraction: float = 0.0, stream=None, profile: int = 0, plan: "Plan" = None,
                 eviction: str = "pending", attn: Optional[np.ndarray] = None, d_hidden: int = 0,
                 weight2: Optional[np.ndarray] = None, bias2: Optional[np.ndarray] = None,
                 setup_stream=None):
        """setup_stream: a torch stream for the work the init enqueues (it
        then overlaps what `stream` still has queued, such as an earlier
        layer's chunks); the graph and plan must be ready on it."""
        self._h = ctypes.c_void_p()
        e = col_dst.numel()
        self.graph = N.Graph(n, e, _dev_ptr(row_off, torch.int64, "row_off"),
                             col_dst.data_ptr() if e else None)
        self._w = np.ascontiguousarray(weight_cat, dtype=np.float32)
        self._b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        self._a = None if attn is None else np.ascontiguousarray(attn, dtype=np.float32).reshape(2, d_out)
        self._w2 = None if weight2 is None else np.ascontiguousarray(weight2, dtype=np.float32)
        self._b2 = None if bias2 is None else np.ascontiguousarray(bias2, dtype=np.float32)
        # the library reads these host arrays at init with the sizes the
        # descriptor implies: a short array would be read past its end
        hidden = d_hidden if agg == N.GIN_MLP else d_out       # accumulator width
        width = 2 * d_out if agg == N.SAGE_MEAN else hidden     # transform columns
        sizes = [(self._w, d_in * width, "weight_cat"), (self._b, hidden, "bias"),
                 (self._a, 2 * d_out if agg == N.GAT_ATT else None, "attn"),
                 (self._w2, d_hidden * d_out if agg == N.GIN_MLP else None, "weight2"),
                 (self._b2, d_out if agg == N.GIN_MLP else None, "bias2")]
        for arr, want, name in sizes:
            if arr is not None and want is not None and arr.size != want:
                raise ValueError(f"{name} has {arr.size} values; this layer needs {want}")
        self.out = out
        out_ptr, out_on_host = _buf_ptr(out, _TORCH_DTYPE[out_dtype], "out")
        self.n, self.d_in, self.d_out, self.chunk, self.in_dtype = n, d_in, d_out, chunk, in_dtype
        self.desc = N.LayerDesc(
            agg=agg, d_in=d_in, d_out=d_out, in_dtype=in_dtype, out_dtype=out_dtype, relu=int(relu),
            weight=self._w.ctypes.data, bias=None if self._b is None else self._b.ctypes.data,
            fanout=fanout, layer=layer, seed=seed & (2**64 - 1), chunk=chunk, hbm_budget=hbm_budget,
            hub_fraction=hub_fraction, out=out_ptr, out_on_host=out_on_host,
            stream=_stream_ptr(stream), profile=int(profile), plan=plan.handle if plan is not None else None,
            eviction=EVICTION[eviction] if isinstance(eviction, str) else int(eviction),
            attn=None if self._a is None else self._a.ctypes.data, d_hidden=d_hidden,
            weight2=None if self._w2 is None else self._w2.ctypes.data,
            bias2=None if self._b2 is None else self._b2.ctypes.data,
            setup_stream=None if setup_stream is None else setup_stream.cuda_stream)
        self._keep = (row_off, col_dst, plan, setup_stream)
        N.check(N.lib().taurus_layer_init(ctypes.byref(self.graph), ctypes.byref(self.desc),
                                          ctypes.byref(self._h)), "taurus_layer_init")

    def push_chunk(self, begin: int, end: int, x: torch.Tensor) -> None:
        """taurus_push_chunk with x = rows [begin, end), on the device or in
        pinned host memory (then it must stay unchanged until the next call)."""
        ptr, on_host = _buf_ptr(x, _TORCH_DTYPE[self.in_dtype], "x")
        N.check(N.lib().taurus_push_chunk(self._h, begin, end, ptr, on_host), "taurus_push_chunk")

    def push_all(self, x: torch.Tensor, order: Optional[Sequence[int]] = None) -> None:
        """Stream every chunk of the full input x [n][d_in] (vertex order by default)."""
        nchunks = (self.n + self.chunk - 1) // self.chunk
        for j in (range(nchunks) if order is None else order):
            b, e = j * self.chunk, min((j + 1) * self.chunk, self.n)
            self.push_chunk(b, e, x[b:e])

    def stream(self, fill, ctx=None, threads: int = 2, ring: int = 0) -> dict:
        """taurus_stream_layer: the library's loader fills every chunk through
        fill (a C function address, or an N.FILL_FN callback) on `threads`
        host threads into a ring of pinned buffers and pushes them in order.
        ctx: a ctypes object (passed by address), an int address or None.
        Returns the loader's times."""
        fn = fill if isinstance(fill, int) else ctypes.cast(fill, ctypes.c_void_p).value
        if ctx is None or isinstance(ctx, int):
            cp = ctx
        else:
            cp = ctypes.addressof(ctx)
        st = N.StreamStats()
        N.check(N.lib().taurus_stream_layer(self._h, fn, cp, threads, ring, ctypes.byref(st)), "taurus_stream_layer")
        return st.as_dict()

    def finalize(self) -> dict:
        st = N.Stats()
        rc = N.lib().taurus_finalize(self._h, ctypes.byref(st))
        d = st.as_dict()
        if rc != N.OK:
            raise N.TaurusError(rc, "taurus_finalize", N.last_error())
        return d

    def reload_histogram(self, bins: int = 64) -> np.ndarray:
        """taurus_layer_reload_histogram: vertices reloaded exactly i times
        (i < bins - 1), then those reloaded bins - 1 times or more."""
        counts = np.zeros(bins, dtype=np.int64)
        N.check(N.lib().taurus_layer_reload_histogram(self._h, counts.ctypes.data, bins),
                "taurus_layer_reload_histogram")
        return counts

    def sampled_edges(self):
        """(mask_words uint64[ceil(e/64)], n_kept)."""
        words = np.zeros((self.graph.e + 63) // 64, dtype=np.uint64)
        kept = ctypes.c_int64()
        N.check(N.lib().taurus_sampled_edges(self._h, words.ctypes.data if words.size else None,
                                             ctypes.byref(kept)), "taurus_sampled_edges")
        return words, kept.value

    def destroy(self) -> None:
        if self._h:
            N.lib().taurus_layer_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def run_layers(n: int, row_off: torch.Tensor, col_dst: torch.Tensor, x: torch.Tensor, layers: list,
               *, chunk: int, stream=None, profile: bool = False, outs: Optional[list] = None):
    """Layer-wise inference: layer l's output is layer l+1's input.

    ``layers`` holds dicts with keys agg, d_in, d_out, weight_cat, bias,
    in_dtype, out_dtype, relu, fanout, layer, seed.  Returns (outputs, stats)."""
    h = x
    results, stats = [], []
    plan = Plan(n, row_off, col_dst, chunk, stream=stream)
    for i, spec in enumerate(layers):
        out = outs[i] if outs is not None else torch.empty(
            (n, spec["d_out"]), dtype=_TORCH_DTYPE[spec.get("out_dtype", N.F32)], device=x.device)
        L = Layer(n, row_off, col_dst, out=out, chunk=chunk, stream=stream, profile=profile, plan=plan, **spec)
        L.push_all(h)
        stats.append(L.finalize())
        L.destroy()
        results.append(out)
        h = out
    if plan is not None:
        plan.destroy()
    return results, stats
