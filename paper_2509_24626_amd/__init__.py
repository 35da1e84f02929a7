"""MI355X (gfx950) decode-step hot path of SparseServe's dynamic sparse
attention over a hierarchical HBM/DRAM KV cache (arXiv 2509.24626).

The computation lives in libsparseserve.so (HIP kernels for gfx950 and a
host-side block cache behind the C ABI in include/sparseserve.h);
`binding` is its ctypes binding and `harness` composes the calls into
decode-step layers (HBM-resident and hierarchical), using torch only for
device memory and streams.
"""
from . import binding  # noqa: F401
