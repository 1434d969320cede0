"""Hybrid sliding-window-attention paged KV attention for AMD MI355X (gfx950).

The compute lives in ``libhswa.so`` (hand-written HIP kernels behind a C ABI,
``include/hswa.h``); ``hswa`` is its Python binding and ``kvcache`` allocates
the dual pools and block tables with PyTorch device memory.
"""

from . import hswa  # noqa: F401
from .hswa import (Cache, HswaError, Layer, Shape, build_block_table, decode,  # noqa: F401
                   decode_split_len, decode_workspace_bytes, kv_append, load, page_bytes, prefill, ring_pages)
