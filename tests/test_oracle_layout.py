"""Pins for the layout oracle (CPU only): ring size, block tables, slot mapping,
pool content after appends, window safety of the ring and storage accounting.

The hand-worked cases use W = 4, PG = 2 (ring of R = 3 pages), the window size
of the paper's prefix-tree illustration ("SWA-Aware Prefix Cache Tree"); every
expected value below was worked out by hand from the rule stated in the test.
"""

import numpy as np
import pytest

from oracle import layout as Lo


def test_ring_pages_closed_form():
    assert Lo.ring_pages(128, 16) == 9          # ceil(128/16) + 1
    assert Lo.ring_pages(128, 64) == 3
    assert Lo.ring_pages(4, 2) == 3
    assert Lo.ring_pages(1, 16) == 2
    assert Lo.ring_pages(129, 64) == 4
    with pytest.raises(ValueError):
        Lo.ring_pages(0, 16)


def test_block_table_hand_worked():
    # FULL, PG = 2, final lengths 3 and 5 need 2 and 3 pages; perm handed out in order
    perm = [4, 0, 3, 1, 2, 5]
    t = Lo.build_block_table(Lo.FULL, None, 2, [3, 5], perm, 4)
    assert t.tolist() == [[4, 0, -1, -1], [3, 1, 2, -1]]
    assert t.dtype == np.int32
    # SWA, W = 4, PG = 2: R = 3 pages per sequence whatever the length
    t = Lo.build_block_table(Lo.SWA, 4, 2, [1, 100], [7, 6, 5, 4, 3, 2, 1, 0], 3)
    assert t.tolist() == [[7, 6, 5], [4, 3, 2]]
    with pytest.raises(ValueError):
        Lo.build_block_table(Lo.FULL, None, 2, [9], list(range(10)), 4)   # needs 5 > stride 4


def test_slot_mapping_swa_hand_worked():
    # W = 4, PG = 2, R = 3, ring row [10, 4, 7]; 9 tokens appended at once.
    # The ring keeps the latest R*PG = 6 positions 3..8; position j goes to
    # ring entry (j // 2) % 3 at offset j % 2:
    #   j=3: entry 1 -> page 4, off 1 -> slot 9     j=4: entry 2 -> page 7 -> 14
    #   j=5: 15    j=6: entry 0 -> page 10 -> 20    j=7: 21
    #   j=8: entry 1 -> page 4, off 0 -> slot 8     j=0,1,2: not kept (-1)
    table = np.array([[10, 4, 7]])
    got = Lo.slot_mapping(Lo.SWA, 4, 2, table, [0], [9])
    assert got.tolist() == [-1, -1, -1, 9, 14, 15, 20, 21, 8]
    # a decode step appends position 9 (length 10): entry 1 -> page 4, off 1 ->
    # slot 9, overwriting position 3, which is outside the window [6, 9]
    assert Lo.slot_mapping(Lo.SWA, 4, 2, table, [9], [1]).tolist() == [9]


def test_slot_mapping_full_hand_worked():
    table = np.array([[5, 2, -1], [0, 3, 1]])
    # seq 0: positions 1, 2, 3 -> (5*2+1, 2*2+0, 2*2+1); seq 1: position 4 -> 1*2+0
    got = Lo.slot_mapping(Lo.FULL, None, 2, table, [1, 4], [3, 1])
    assert got.tolist() == [11, 4, 5, 2]
    assert got.dtype == np.int64


def test_apply_append_hand_worked():
    """PG = 16 (blocks of B = 16 keys), D = 32 (one slab). Slot 21 = page 1,
    offset 5: bit 2 of 5 is set, so half 1, row 4 * (5 // 8) + 5 % 4 = 1;
    slot 0 = page 0, half 0, row 0; token 1 (slot -1) is dropped."""
    pg, hkv, d = 16, 1, 32
    kp = np.zeros(Lo.k_pool_shape(2, hkv, pg, d), dtype=np.uint16)
    assert kp.shape == (2, 1, 1, 2, 1, 4, 8, 8)
    vp = np.zeros((2, hkv, 1, d, pg), dtype=np.uint16)
    kn = np.arange(1, 1 + 3 * d, dtype=np.uint16).reshape(3, hkv, d)
    vn = kn + 1000
    k2, v2 = Lo.apply_append(kp, vp, [21, -1, 0], kn, vn)
    assert k2[1, 0, 0, 1, 0, :, 1, :].reshape(d).tolist() == kn[0, 0].tolist()
    assert k2[0, 0, 0, 0, 0, :, 0, :].reshape(d).tolist() == kn[2, 0].tolist()
    assert int(k2.sum()) == int(kn[0].sum()) + int(kn[2].sum())
    assert v2[1, 0, 0, :, 5].tolist() == vn[0, 0].tolist() and v2[0, 0, 0, :, 0].tolist() == vn[2, 0].tolist()
    assert Lo.k_rows(k2, 1, 5).tolist() == kn[0].tolist()


def test_k_layout_flat_offset_hand_worked():
    """PG = 32, D = 64: in-page offset 13 (binary 1101: half 1, row 4*1 + 1 = 5),
    dim 37 (slab 1, piece (37 // 8) % 4 = 0, element 5) sits at flat element
    ((((1 * 2 + 1) * 4 + 0) * 16 + 5) * 8 + 5 = 1581 of the page-head."""
    pg, hkv, d = 32, 1, 64
    kp = np.zeros(Lo.k_pool_shape(1, hkv, pg, d), dtype=np.uint16)
    kn = np.zeros((1, hkv, d), dtype=np.uint16)
    kn[0, 0, 37] = 777
    k2, _ = Lo.apply_append(kp, np.zeros((1, hkv, 1, d, 32), dtype=np.uint16), [13], kn, kn)
    flat = k2.reshape(pg * d)
    assert flat[1581] == 777 and int(flat.sum()) == 777


def test_k_layout_mfma_operand_runs():
    """PG = 64, D = 128: for 32-key block j, half h and slab t, the 16 keys
    32 j + 8 (r // 4) + 4 h + r % 4 (r < 16) with dims 32 t + 8 q + e are one
    contiguous 1 KiB run in the order of lane l = r + 16 q (16 bytes a lane)."""
    pg, hkv, d = 64, 1, 128
    kp = np.zeros(Lo.k_pool_shape(1, hkv, pg, d), dtype=np.uint16)
    kn = np.arange(pg * d, dtype=np.uint16).reshape(pg, hkv, d)  # value = 128 * key + dim
    k2, _ = Lo.apply_append(kp, np.zeros((1, hkv, 2, d, 32), dtype=np.uint16), list(range(pg)), kn, kn)
    flat = k2.reshape(pg * d)
    for j in range(2):
        for h in range(2):
            for t in range(4):
                run = flat[j * 4096 + h * 2048 + t * 512: j * 4096 + h * 2048 + (t + 1) * 512].reshape(64, 8)
                for lane in range(64):
                    r, q = lane % 16, lane // 16
                    key = 32 * j + 8 * (r // 4) + 4 * h + r % 4
                    assert run[lane].tolist() == [128 * key + 32 * t + 8 * q + e for e in range(8)]


@pytest.mark.parametrize("pg", [16, 32, 64, 256])
def test_k_layout_is_a_bijection(pg):
    """Every (key, dim) of a page-head lands on its own element: writing all
    keys with distinct values fills the page exactly once."""
    d = 128
    kp = np.zeros(Lo.k_pool_shape(1, 1, pg, d), dtype=np.int64)
    vals = np.arange(1, 1 + pg * d, dtype=np.int64).reshape(pg, 1, d)
    vb = min(pg, 32)
    k2, _ = Lo.apply_append(kp, np.zeros((1, 1, pg // vb, d, vb), dtype=np.int64), list(range(pg)), vals, vals)
    assert sorted(k2.reshape(-1).tolist()) == list(range(1, 1 + pg * d))
    for o in (0, pg // 2 + 5, pg - 1):
        assert Lo.k_rows(k2, 0, o).tolist() == vals[o].tolist()


def test_apply_append_v_blocks_hand_worked():
    """PG = 64: V is stored in two blocks of 32 keys; in-page offset 40 is key 8
    of block 1, so its dims sit at flat element 1*32*D + d*32 + 8 of the page."""
    pg, hkv, d = 64, 2, 32
    kp = np.zeros(Lo.k_pool_shape(3, hkv, pg, d), dtype=np.uint16)
    vp = np.zeros((3, hkv, 2, d, 32), dtype=np.uint16)
    kn = np.arange(1, 1 + hkv * d, dtype=np.uint16).reshape(1, hkv, d)
    _, v2 = Lo.apply_append(kp, vp, [2 * 64 + 40], kn, kn + 50)
    flat = v2.reshape(3, hkv, pg * d)
    for g in range(hkv):
        for dd in range(d):
            assert flat[2, g, 32 * d + dd * 32 + 8] == kn[0, g, dd] + 50
    assert int((v2 != 0).sum()) == hkv * d
    with pytest.raises(ValueError):
        Lo.apply_append(kp, np.zeros((3, hkv, d, pg), dtype=np.uint16)[..., None], [0], kn, kn)
    with pytest.raises(ValueError):
        Lo.apply_append(np.zeros((3, hkv, pg, d), dtype=np.uint16), vp, [0], kn, kn)


@pytest.mark.parametrize("window,pg", [(4, 2), (128, 16), (128, 64), (1, 16), (129, 64), (5, 4)])
def test_ring_invariants(window, pg):
    """Across appends of random sizes: no slot written twice in one call, every
    ring slot holds the latest position congruent to it modulo R*PG, and the
    window of every query position stays inside the ring (window safety)."""
    r = Lo.ring_pages(window, pg)
    ring_len = r * pg
    table = np.array([np.random.default_rng(0).permutation(50)[:r]])
    held = {}
    pos = 0
    rng = np.random.default_rng(window * 1000 + pg)
    for _ in range(40):
        n = int(rng.integers(1, 3 * ring_len))
        slots = Lo.slot_mapping(Lo.SWA, window, pg, table, [pos], [n])
        kept = slots[slots >= 0]
        assert len(set(kept.tolist())) == len(kept)             # one writer per slot
        assert len(kept) == min(n, ring_len) or pos + n <= ring_len
        for i, s in enumerate(slots):
            if s >= 0:
                held[int(s)] = pos + i
        pos += n
        # every written slot holds the latest position congruent to it
        for s, p in held.items():
            assert p > pos - 1 - ring_len and p <= pos - 1
        # window safety: the query at pos-1 needs [pos-W, pos-1]; all are held
        need = set(range(max(0, pos - window), pos))
        assert need <= set(held.values())
        assert Lo.ring_positions(window, pg, pos) == {
            ((p // pg) % r, p % pg): p for p in held.values() if p >= pos - ring_len}


def test_prefix_window_safety_for_chunks():
    """Before a chunk at prefix P the ring holds [P - R*PG, P); the earliest key a
    chunk query needs is P - W + 1, so reading the ring prefix is always safe."""
    for window, pg in ((128, 64), (128, 16), (4, 2), (1, 16)):
        r = Lo.ring_pages(window, pg)
        for P in (1, window - 1, window, window + 1, 3 * r * pg + 5):
            held = set(Lo.ring_positions(window, pg, P).values())
            need = set(range(max(0, P - window + 1), P))
            assert need <= held


def test_storage_closed_forms():
    hkv, d = 8, 128
    assert Lo.page_bytes(hkv, 64, d) == 128 * 1024               # one pool page
    assert Lo.page_bytes(1, 16, d) == 4 * 1024
    # SWA bytes are flat in context length: NS * R * 2 pools * page bytes
    flat = {Lo.layer_kv_bytes(Lo.SWA, 128, 64, [L] * 16, hkv, d) for L in (1, 1000, 131073, 10 ** 6)}
    assert flat == {16 * 3 * 2 * 128 * 1024}                     # 12 MiB
    # 70-layer stack at 16 x 131073 tokens: hybrid (10 FULL + 60 SWA) vs all FULL
    full = Lo.layer_kv_bytes(Lo.FULL, None, 64, [131073] * 16, hkv, d)
    assert full == 16 * 2049 * 2 * 128 * 1024                    # 8.59 GB per FULL layer
    swa = Lo.layer_kv_bytes(Lo.SWA, 128, 64, [131073] * 16, hkv, d)
    hybrid, all_full = 10 * full + 60 * swa, 70 * full
    assert hybrid / all_full == pytest.approx((60 * 3 + 10 * 2049) / (70 * 2049), rel=1e-15)
    assert 6.9 < all_full / hybrid < 7.0                         # the paper's "about 7x"


def test_planted_ring_mistake_is_caught(monkeypatch):
    """A ring that keeps only W positions (instead of R*PG) breaks the hand-worked
    slot list; a ring indexed by j % R breaks it too."""
    orig = Lo.ring_pages
    monkeypatch.setattr(Lo, "ring_pages", lambda w, pg: orig(w, pg) - 1)
    table = np.array([[10, 4, 7]])
    assert Lo.slot_mapping(Lo.SWA, 4, 2, table, [0], [9]).tolist() != [-1, -1, -1, 9, 14, 15, 20, 21, 8]
