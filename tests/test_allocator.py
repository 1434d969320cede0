"""The explicit-release dual-pool allocator (C ABI, host) against its reference
model: status codes, pages held per sequence and pool, and which logical pages
the FULL and SWA tables hold after every operation of seeded random serving
schedules; physical ids unique and in range; closed forms for the SWA pages a
long decode holds (flat in the context length); a hand-worked schedule."""

import numpy as np
import pytest

from oracle import allocator as OA
from paper_2607_13095_amd import hswa


def _check_state(alloc, model, cfg):
    full, swa = alloc.tables()
    ns, stride = cfg["max_seqs"], cfg["table_stride"]
    seen_f, seen_s = set(), set()
    for b in range(ns):
        if b in model.seqs:
            fu, su, _, _ = alloc.usage(b)
            want_full = model.full_pages_of(b)
            want_swa = model.swa_pages_of(b)
            assert fu == want_full and su == len(want_swa), (b, fu, su, want_full, want_swa)
            assert np.array_equal(full[b] >= 0, np.arange(stride) < want_full)
            assert set(np.nonzero(swa[b] >= 0)[0].tolist()) == want_swa
        else:
            assert (full[b] < 0).all() and (swa[b] < 0).all()
        for v in full[b][full[b] >= 0].tolist():
            assert 0 <= v < cfg["full_pages"] and v not in seen_f
            seen_f.add(v)
        for v in swa[b][swa[b] >= 0].tolist():
            assert 0 <= v < cfg["swa_pages"] and v not in seen_s
            seen_s.add(v)
    fu, su, ff, sf = alloc.usage(-1)
    assert (ff, sf) == (model.full_free(), model.swa_free())
    assert fu + ff == cfg["full_pages"] and su + sf == cfg["swa_pages"]


CONFIGS = [
    dict(page_size=4, window=6, full_pages=40, swa_pages=12, max_seqs=4, table_stride=16, release_every=2),
    dict(page_size=16, window=128, full_pages=200, swa_pages=60, max_seqs=6, table_stride=40, release_every=1),
    dict(page_size=64, window=128, full_pages=120, swa_pages=24, max_seqs=5, table_stride=30, release_every=8),
    dict(page_size=16, window=1, full_pages=60, swa_pages=8, max_seqs=3, table_stride=20, release_every=3),
]


@pytest.mark.parametrize("ci", range(len(CONFIGS)))
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_schedules_match_model(ci, seed):
    cfg = CONFIGS[ci]
    alloc = hswa.Allocator(**cfg)
    model = OA.DualPoolModel(**cfg)
    rng = np.random.default_rng([ci, seed])
    pg = cfg["page_size"]
    for _ in range(400):
        b = int(rng.integers(cfg["max_seqs"]))
        op = rng.choice(["admit", "chunk", "decode", "free", "bad"], p=[0.2, 0.25, 0.4, 0.1, 0.05])
        if op == "admit":
            length, chunk = int(rng.integers(0, 6 * pg * 4)), int(rng.integers(1, 4 * pg))
            assert alloc.admit(b, length, chunk) == model.admit(b, length, chunk)
        elif op in ("chunk", "decode"):
            if b not in model.seqs:
                assert alloc.extend(b, 5) == model.extend(b, 5) == OA.INVALID
                continue
            cur = model.seqs[b]["len"]
            new = cur + (1 if op == "decode" else int(rng.integers(1, 3 * pg)))
            st = alloc.extend(b, new)
            assert st == model.extend(b, new), (op, b, cur, new)
            if st == 0:
                got = alloc.step_end(b, op == "decode")
                _, want = model.step_end(b, op == "decode")
                assert got == want
        elif op == "free":
            if b in model.seqs:
                alloc.free(b)
                model.free(b)
        else:
            assert alloc.extend(b, -1) == OA.INVALID if b in model.seqs else True
            assert alloc.admit(b, -1, 1) == OA.INVALID
        _check_state(alloc, model, cfg)
    alloc.close()


@pytest.mark.parametrize("pg,w", [(16, 128), (64, 128), (4, 6), (16, 1), (64, 200)])
def test_decode_swa_pages_closed_form(pg, w):
    """Releasing every step, after the step that makes the length L the SWA pool
    holds exactly the pages of positions [max(0, L-W+1), L): flat in L."""
    stride = 4096 // pg + 2
    alloc = hswa.Allocator(pg, w, stride + 4, 64, 1, stride, 1)
    assert alloc.admit(0, 0, 1) == 0
    bound = -(-(w - 1) // pg) + 1
    for L in range(1, 4097):
        assert alloc.extend(0, L) == 0
        alloc.step_end(0, True)
        lo = max(0, L - w + 1)
        want = (L - 1) // pg - lo // pg + 1
        _, su, _, _ = alloc.usage(0)
        assert su == want and su <= bound, (L, su, want)
    alloc.free(0)
    assert alloc.usage(-1)[:2] == (0, 0)


def test_hand_worked_schedule():
    # PG = 4, W = 6, release every 2 decode steps.
    a = hswa.Allocator(4, 6, 100, 100, 1, 16, 2)
    assert a.admit(0, 11, 8) == 0
    # chunk of 11 tokens: stored positions max(0, 11 - 6) = 5 .. 10 -> SWA
    # logical pages 1 (4..7) and 2 (8..11); FULL pages 0, 1, 2
    assert a.extend(0, 11) == 0
    full, swa = a.tables()
    assert (full[0][:4] >= 0).tolist() == [True, True, True, False]
    assert (swa[0][:4] >= 0).tolist() == [False, True, True, False]
    assert a.step_end(0, False) == 0  # nothing wholly before position 6 is held
    # decode 11 -> length 12: window of the next query [7, 12]: page 1 (4..7) still needed
    assert a.extend(0, 12) == 0 and a.step_end(0, True) == 0
    # decode 12 -> length 13: window [8, 13]; second decode step -> release page 1
    assert a.extend(0, 13) == 0 and a.step_end(0, True) == 1
    full, swa = a.tables()
    assert (swa[0][:5] >= 0).tolist() == [False, False, True, True, False]
    assert (full[0][:5] >= 0).tolist() == [True, True, True, True, False]


def test_admission_checks_both_pools():
    a = hswa.Allocator(16, 128, 10, 4, 4, 64, 1)
    assert a.admit(0, 200, 64) == -3          # FULL needs 13 pages, has 10
    assert a.admit(0, 160, 64) == -3          # FULL 10 fits, SWA needs ceil(min(160, 192)/16)+1 = 11 > 4
    assert a.admit(0, 48, 16) == 0            # FULL 3, SWA ceil(48/16)+1 = 4
    a2 = hswa.Allocator(16, 128, 100, 4, 4, 64, 1)
    assert a2.admit(0, 160, 64) == -3         # SWA needs ceil(min(160, 192)/16)+1 = 11 > 4
    assert a2.admit(0, 30, 16) == 0           # SWA ceil(30/16)+1 = 3 <= 4
    assert a2.admit(0, 30, 16) == -1          # slot in use
    a2.free(0)
    assert a2.admit(0, 30, 16) == 0


def test_invalid_config():
    with pytest.raises(hswa.HswaError):
        hswa.Allocator(0, 128, 10, 10, 1, 8, 1)
    with pytest.raises(hswa.HswaError):
        hswa.Allocator(16, 128, 10, 10, 1, 8, 0)
