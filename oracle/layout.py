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
the library's own):
  K pool: [num_pages][Hkv][PG][D]          (key-major rows inside a page)
  V pool: [num_pages][Hkv][PG/VB][D][VB]   (blocks of VB = min(PG, 32) keys,
                                             each transposed)
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


def apply_append(k_pool, v_pool, slots, k_new, v_new):
    """Expected pool content after an append (copies; bf16 bits as uint16).

    k_pool: [P][Hkv][PG][D] (one row per slot). v_pool: [P][Hkv][PG/VB][D][VB]:
    the keys of a page in blocks of VB = min(PG, 32), each block stored with
    the dim index outer. k_new, v_new: [T][Hkv][D]. Tokens whose slot is -1 are
    not stored.
    """
    k_pool = np.array(k_pool, copy=True)
    v_pool = np.array(v_pool, copy=True)
    pg = k_pool.shape[2]
    vb = v_pool.shape[4]
    if vb != min(pg, 32) or v_pool.shape[2] * vb != pg:
        raise ValueError("v_pool blocks must hold min(PG, 32) keys")
    for t, s in enumerate(np.asarray(slots)):
        if s < 0:
            continue
        page, off = int(s) // pg, int(s) % pg
        k_pool[page, :, off, :] = k_new[t]
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
