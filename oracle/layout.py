"""Integer rules of the dual-pool paged KV layout (the oracle).

TEST INFRASTRUCTURE ONLY: only tests, the smoke check and the benchmark's CPU
baseline may use this module.

Sources in the paper: "KVCache Dual-Pool Design" (separate FULL and SWA pools;
the SWA pool is sized for the window and evicts by window, so SWA storage is
O(W); the FULL index is authoritative with a FULL -> SWA mapping), and
"SWA-Aware Prefix Cache Tree" (out-of-window SWA release tied to chunk
completion and decode steps; evicted slots are never read).

Readings where the paper is silent:
  * SWA ring size R = ceil(W / PG) + 1 pages per sequence.
  * Logical page i of a sequence maps to ring entry i mod R, i.e. token position
    j lives in ring slot j mod (R * PG).
  * An append stores an SWA token at position j only when j >= L - R * PG, where
    L is the sequence length after the append; the ring then holds exactly the
    latest R * PG positions and no slot is written twice in one call.
  * Block tables are filled from a permutation of physical page ids, sequence
    by sequence: table[b][i] = perm[offset_b + i] for i < n_b, -1 elsewhere,
    with n_b = ceil(L_b_final / PG) for FULL and n_b = R for SWA.

Pool layout (one pool per layer and per K / V; the paper fixes none, this is
the library's own). Both pools hold a page-head as blocks of B = min(PG, 32)
consecutive keys:
  K pool: [num_pages][Hkv][PG/B][2][D/32][4][B/2][8]
          key k of a block sits in half (k // 4) % 2 at row 4 (k // 8) + k % 4;
          dim d in 32-dim slab d // 32, 8-dim piece (d // 8) % 4, element d % 8
  V pool: [num_pages][Hkv][PG/B][D][B]     (each block transposed)
A slot s addresses page s // PG, in-page offset s % PG.
"""

from __future__ import annotations

import numpy as np

FULL = "full"
SWA = "swa"


def ring_pages(window: int, page_size: int) -> int:
    """R = ceil(W / PG) + 1 ring pages per sequence for an SWA layer."""
    if window < 1 or page_size < 1:
        raise ValueError("window and page size must be positive")
    return -(-int(window) // int(page_size)) + 1


def pages_needed(kind: str, window, page_size: int, final_len: int) -> int:
    """Physical pages one sequence needs in a layer's pool."""
    if kind == FULL:
        return -(-int(final_len) // int(page_size))
    if kind == SWA:
        return ring_pages(window, page_size)
    raise ValueError(kind)


def build_block_table(kind, window, page_size, final_lens, perm, stride) -> np.ndarray:
    """Block table int32 [NS][stride] from a permutation of physical page ids."""
    final_lens = [int(x) for x in final_lens]
    need = [pages_needed(kind, window, page_size, n) for n in final_lens]
    if max(need, default=0) > stride:
        raise ValueError("table stride too small")
    perm = np.asarray(perm, dtype=np.int64)
    if sum(need) > perm.size:
        raise ValueError("not enough physical pages")
    table = np.full((len(final_lens), stride), -1, dtype=np.int32)
    off = 0
    for b, n in enumerate(need):
        table[b, :n] = perm[off:off + n]
        off += n
    return table


def slot_of(kind, window, page_size, table_row, pos: int, final_len: int) -> int:
    """Pool slot of token position ``pos`` of a sequence of length ``final_len``.

    Returns -1 for an SWA token that the ring does not keep.
    """
    pg = int(page_size)
    if kind == FULL:
        return int(table_row[pos // pg]) * pg + pos % pg
    r = ring_pages(window, pg)
    if pos < final_len - r * pg:
        return -1
    return int(table_row[(pos // pg) % r]) * pg + pos % pg


def slot_mapping(kind, window, page_size, table, start_pos, new_lens) -> np.ndarray:
    """int64 [T]: slot of every new token, sequences concatenated in order.

    Sequence b appends new_lens[b] tokens at positions start_pos[b] ... and has
    length start_pos[b] + new_lens[b] afterwards.
    """
    out = []
    for b, (s, n) in enumerate(zip(start_pos, new_lens)):
        s, n = int(s), int(n)
        final = s + n
        for pos in range(s, final):
            out.append(slot_of(kind, window, page_size, table[b], pos, final))
    return np.asarray(out, dtype=np.int64)


def key_block(page_size: int) -> int:
    """Keys per block of both pools: B = min(PG, 32)."""
    return min(int(page_size), 32)


def k_pool_shape(num_pages: int, num_kv_heads: int, page_size: int, head_dim: int):
    """[num_pages][Hkv][PG/B][2][D/32][4][B/2][8] (see the module header)."""
    b = key_block(page_size)
    if b < 8 or int(page_size) % b or int(head_dim) % 32:
        raise ValueError("the K layout needs PG >= 8 and head_dim a multiple of 32")
    return (int(num_pages), int(num_kv_heads), int(page_size) // b, 2, int(head_dim) // 32, 4, b // 2, 8)


def k_slot(k_pool_shape_, page: int, off: int):
    """Index (for numpy or torch) of the Hkv x D values of in-page offset
    `off` of `page` in a K pool of the given shape; the selection has shape
    [Hkv][D/32][4][8], i.e. the key's dims in order after a reshape to
    [Hkv][D]."""
    b = 2 * int(k_pool_shape_[6])
    k = int(off) % b
    half, row = (k // 4) % 2, 4 * (k // 8) + k % 4
    return (int(page), slice(None), int(off) // b, half, slice(None), slice(None), row, slice(None))


def k_rows(k_pool, page: int, off: int):
    """The [Hkv][D] K values stored for in-page offset `off` of `page`."""
    sel = k_pool[k_slot(k_pool.shape, page, off)]
    return sel.reshape(sel.shape[0], -1)


def apply_append(k_pool, v_pool, slots, k_new, v_new):
    """Expected pool content after an append (copies; bf16 bits as uint16).

    k_pool: [P][Hkv][PG/B][2][D/32][4][B/2][8]; v_pool: [P][Hkv][PG/B][D][B]
    (B = min(PG, 32); the module header gives the element order). k_new,
    v_new: [T][Hkv][D]. Tokens whose slot is -1 are not stored.
    """
    k_pool = np.array(k_pool, copy=True)
    v_pool = np.array(v_pool, copy=True)
    if k_pool.ndim != 8 or v_pool.ndim != 5:
        raise ValueError("k_pool is 8-D and v_pool 5-D")
    npg, hkv = k_pool.shape[:2]
    pg = k_pool.shape[2] * 2 * k_pool.shape[6]
    d = k_pool.shape[4] * 32
    if tuple(k_pool.shape) != k_pool_shape(npg, hkv, pg, d):
        raise ValueError("k_pool must be [P][Hkv][PG/B][2][D/32][4][B/2][8]")
    vb = v_pool.shape[4]
    if vb != key_block(pg) or v_pool.shape[2] * vb != pg:
        raise ValueError("v_pool blocks must hold min(PG, 32) keys")
    for t, s in enumerate(np.asarray(slots)):
        if s < 0:
            continue
        page, off = int(s) // pg, int(s) % pg
        k_pool[k_slot(k_pool.shape, page, off)] = np.asarray(k_new[t]).reshape(hkv, d // 32, 4, 8)
        v_pool[page, :, off // vb, :, off % vb] = v_new[t]
    return k_pool, v_pool


def ring_positions(window, page_size, length: int) -> dict:
    """Which position each SWA ring slot (entry, offset) holds after appends.

    Returns {(ring_entry, offset): position} for a sequence of ``length``
    tokens appended in any number of calls (the ring keeps the latest R*PG).
    """
    pg = int(page_size)
    r = ring_pages(window, pg)
    held = {}
    for pos in range(max(0, length - r * pg), length):
        held[((pos // pg) % r, pos % pg)] = pos
    return held


def page_bytes(num_kv_heads: int, page_size: int, head_dim: int, elem_bytes: int = 2) -> int:
    """Bytes of one page of one pool (K or V)."""
    return int(num_kv_heads) * int(page_size) * int(head_dim) * int(elem_bytes)


def layer_kv_bytes(kind, window, page_size, final_lens, num_kv_heads, head_dim) -> int:
    """K + V pool bytes one layer needs for a batch of sequences."""
    pages = sum(pages_needed(kind, window, page_size, n) for n in final_lens)
    return 2 * pages * page_bytes(num_kv_heads, page_size, head_dim)
