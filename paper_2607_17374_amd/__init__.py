"""MI355X-native layer-wise broadcast GNN inference (Taurus, arXiv 2607.17374).

The compute lives in the HIP library ``libtaurus.so`` behind the C ABI of
``include/taurus.h``; this package holds its ctypes binding (``_native``)
and a thin torch-facing wrapper (``api``) that passes device pointers and
streams and loops over chunks and layers.
"""
from ._native import (F32, BF16, F16, SAGE_MEAN, GCN_SYM, GIN_SUM, GAT_ATT, GIN_MLP, TaurusError, lib)  # noqa: F401
from .api import (build_csr, Layer, Plan, hash_u64, run_layers, reorder, reorder_rcm, reorder_ta, release_cached_memory, alloc_device, relabel_graph,  # noqa: F401
                  permute_rows)
