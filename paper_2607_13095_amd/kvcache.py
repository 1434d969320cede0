"""Dual-pool KV cache allocation with PyTorch device memory.

One ``LayerKV`` holds the K and V pools and the device block table of one
layer ("KVCache Dual-Pool Design": a FULL pool sized for every position, an
SWA pool sized for a ring of ceil(W/PG)+1 pages per sequence). Block tables
are built by the library (``hswa_build_block_table``) from a caller-supplied
permutation of physical page ids. Pools can be filled with NaN so that any
read of a slot that was never written shows up in the output.
"""

from __future__ import annotations

from typing import Sequence

import numpy as np
import torch

from . import hswa


def pages_for(layer: hswa.Layer, page_size: int, final_lens: Sequence[int]) -> int:
    if layer.kind == "swa":
        return len(final_lens) * hswa.ring_pages(layer.window, page_size)
    return int(sum(-(-int(n) // page_size) for n in final_lens))


class LayerKV:
    def __init__(self, layer: hswa.Layer, shape: hswa.Shape, final_lens: Sequence[int], perm=None,
                 extra_pages: int = 0, fill: float = float("nan"), device="cuda", stride=None):
        self.layer, self.shape = layer, shape
        pg, hkv, d = shape.page_size, shape.num_kv_heads, shape.head_dim
        need = pages_for(layer, pg, final_lens)
        self.num_pages = max(1, need + int(extra_pages))
        if perm is None:
            perm = np.arange(self.num_pages)
        perm = np.asarray(perm, dtype=np.int32)
        if stride is None:
            stride = (hswa.ring_pages(layer.window, pg) if layer.kind == "swa"
                      else max(1, max(-(-int(n) // pg) for n in final_lens)))
        self.table_host = hswa.build_block_table(layer, pg, final_lens, perm, stride)
        self.block_table = torch.from_numpy(self.table_host).to(device)
        self.k_pool = torch.full(hswa.k_pool_shape(self.num_pages, hkv, pg, d), fill, dtype=torch.bfloat16,
                                 device=device)
        self.v_pool = torch.full(hswa.v_pool_shape(self.num_pages, hkv, pg, d), fill, dtype=torch.bfloat16,
                                 device=device)
        self.cache = hswa.Cache(self.k_pool, self.v_pool, self.block_table)

    def nbytes(self) -> int:
        return 2 * self.num_pages * hswa.page_bytes(self.shape)
