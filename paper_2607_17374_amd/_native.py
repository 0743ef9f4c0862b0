"""ctypes binding of ``include/taurus.h``: argument marshalling only.

Every computation runs in the HIP library ``libtaurus.so``; this module
converts torch tensors to device pointers and Python values to the C
structures.  If the library is not built the import fails loudly: there is
no fallback path.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtaurus.so")

OK, E_INVALID, E_OOM, E_DEVICE, E_STATE, E_INCOMPLETE, E_BUDGET = 0, -1, -2, -3, -4, -5, -6
F32, BF16, F16 = 0, 1, 2
SAGE_MEAN, GCN_SYM, GIN_SUM, GAT_ATT, GIN_MLP = 0, 1, 2, 3, 4
EVICT_PENDING, EVICT_RANDOM, EVICT_FIFO, EVICT_LRU = 0, 1, 2, 3
NOALLOC_SCRATCH_BYTES, NOALLOC_MAX_EDGES = 32 << 20, 1 << 20

STATUS_NAMES = {OK: "OK", E_INVALID: "E_INVALID", E_OOM: "E_OOM", E_DEVICE: "E_DEVICE",
                E_STATE: "E_STATE", E_INCOMPLETE: "E_INCOMPLETE", E_BUDGET: "E_BUDGET"}


class TaurusError(RuntimeError):
    def __init__(self, status: int, call: str, message: str):
        super().__init__(f"{call}: {STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class Graph(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("e", ctypes.c_int64),
                ("row_off", ctypes.c_void_p), ("col_dst", ctypes.c_void_p)]


class LayerDesc(ctypes.Structure):
    _fields_ = [("agg", ctypes.c_int32), ("d_in", ctypes.c_int32), ("d_out", ctypes.c_int32),
                ("in_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32), ("relu", ctypes.c_int32),
                ("weight", ctypes.c_void_p), ("bias", ctypes.c_void_p),
                ("fanout", ctypes.c_int32), ("layer", ctypes.c_int32), ("seed", ctypes.c_uint64),
                ("chunk", ctypes.c_int64), ("hbm_budget", ctypes.c_int64), ("hub_fraction", ctypes.c_double),
                ("out", ctypes.c_void_p), ("out_on_host", ctypes.c_int32),
                ("stream", ctypes.c_void_p), ("profile", ctypes.c_int32), ("plan", ctypes.c_void_p),
                ("eviction", ctypes.c_int32), ("attn", ctypes.c_void_p), ("d_hidden", ctypes.c_int32),
                ("weight2", ctypes.c_void_p), ("bias2", ctypes.c_void_p), ("setup_stream", ctypes.c_void_p)]


class Stats(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int64) for name in (
        "n", "e", "messages", "self_terms", "pairs", "completed", "pending_left", "chunks",
        "chunks_pushed", "short_units", "wave_units", "split_segments", "evictions", "reloads",
        "h2d_bytes", "d2h_bytes", "device_bytes")] + [
        ("hub_message_share", ctypes.c_double), ("ms_init", ctypes.c_double), ("ms_index", ctypes.c_double),
        ("ms_gemm", ctypes.c_double),
        ("ms_self", ctypes.c_double), ("ms_scatter", ctypes.c_double), ("ms_fixup", ctypes.c_double),
        ("launches_gemm", ctypes.c_int64), ("launches_self", ctypes.c_int64),
        ("launches_scatter", ctypes.c_int64), ("launches_fixup", ctypes.c_int64),
        ("pool_rows", ctypes.c_int64), ("hub_rows", ctypes.c_int64),
        ("self_in_transform", ctypes.c_int64), ("self_fresh", ctypes.c_int64), ("self_last", ctypes.c_int64)]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_}


class StreamStats(ctypes.Structure):
    _fields_ = [("chunks", ctypes.c_int64), ("bytes", ctypes.c_int64), ("fill_seconds", ctypes.c_double),
                ("wait_seconds", ctypes.c_double), ("push_seconds", ctypes.c_double),
                ("wall_seconds", ctypes.c_double)]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_}


# the loader's fill callback: int fill(void* ctx, int64_t begin, int64_t end, void* dst)
FILL_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p)


# every function the header declares, with its C signature
SIGNATURES = {
    "taurus_last_error": (ctypes.c_char_p, []),
    "taurus_hash": (ctypes.c_uint64, [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32, ctypes.c_void_p]),
    "taurus_build_csr": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "taurus_build_csr_noalloc": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "taurus_layer_init": (ctypes.c_int, [ctypes.POINTER(Graph), ctypes.POINTER(LayerDesc),
                                         ctypes.POINTER(ctypes.c_void_p)]),
    "taurus_push_chunk": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                         ctypes.c_int32]),
    "taurus_finalize": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(Stats)]),
    "taurus_stream_layer": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                           ctypes.c_int32, ctypes.POINTER(StreamStats)]),
    "taurus_sampled_edges": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64)]),
    "taurus_layer_destroy": (None, [ctypes.c_void_p]),
    "taurus_layer_reload_histogram": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32]),
    "taurus_release_cached_memory": (ctypes.c_int64, [ctypes.c_int64]),
    "taurus_reorder": (ctypes.c_int, [ctypes.POINTER(Graph), ctypes.c_void_p, ctypes.c_void_p]),
    "taurus_reorder_rcm": (ctypes.c_int, [ctypes.POINTER(Graph), ctypes.c_void_p, ctypes.c_void_p]),
    "taurus_reorder_ta": (ctypes.c_int, [ctypes.POINTER(Graph), ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.POINTER(ctypes.c_int32), ctypes.c_void_p]),
    "taurus_relabel_graph": (ctypes.c_int, [ctypes.POINTER(Graph), ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_void_p, ctypes.c_void_p]),
    "taurus_permute_rows": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                           ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]),
    "taurus_plan_create": (ctypes.c_int, [ctypes.POINTER(Graph), ctypes.c_int64, ctypes.c_void_p,
                                          ctypes.POINTER(ctypes.c_void_p)]),
    "taurus_plan_destroy": (None, [ctypes.c_void_p]),
}

_lib = None


def lib():
    """Load libtaurus.so (raises if it was never built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run __graft_entry__.build() "
                              "(or python paper_2607_17374_amd/build.py) first")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(status: int, call: str) -> None:
    if status != OK:
        msg = lib().taurus_last_error()
        raise TaurusError(status, call, msg.decode() if msg else "")


def last_error() -> str:
    msg = lib().taurus_last_error()
    return msg.decode() if msg else ""
