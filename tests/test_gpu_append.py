"""GPU parity of hswa_kv_append: slot mapping and pool bytes are bit-exact
against the layout oracle, including ring-wrap eviction for SWA layers."""

import numpy as np
import pytest
import torch

import synth
from oracle import layout as OL
from paper_2607_13095_amd import hswa
from tests.hswa_testlib import append_history, make_layer, SeqHistory, to_bits

pytestmark = pytest.mark.gpu

NAN_BITS = None


def _check_pools(kv, exp_k, exp_v):
    got_k, got_v = to_bits(kv.k_pool), to_bits(kv.v_pool)
    assert np.array_equal(got_k, exp_k)
    assert np.array_equal(got_v, exp_v)


# (kind, window, page size, Hkv, list of append calls: per call, per seq: (start, end))
CASES = [
    ("full", 0, 16, 1, [[(0, 37), (0, 16), (0, 1)]]),
    ("full", 0, 64, 8, [[(0, 130), (0, 64)], [(130, 131), (64, 200)]]),
    ("swa", 4, 16, 2, [[(0, 9), (0, 40)], [(9, 10), (40, 41)], [(10, 50), (41, 42)]]),
    ("swa", 128, 16, 1, [[(0, 512)]]),
    ("swa", 128, 64, 8, [[(0, 300), (0, 129), (0, 5)], [(300, 301), (129, 130), (5, 6)], [(301, 700), (130, 140), (6, 7)]]),
    ("swa", 1, 16, 1, [[(0, 33)], [(33, 34)]]),
    ("swa", 129, 64, 8, [[(0, 1000)], [(1000, 1008)], [(1008, 1017)]]),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_append_bit_exact(gpu_lib, case):
    kind, window, pg, hkv, calls = CASES[case]
    print(f"[append] case={case} kind={kind} W={window} PG={pg} Hkv={hkv}", flush=True)
    shape = hswa.Shape(hkv * 2, hkv, 128, pg)
    ns = len(calls[0])
    final = [max(c[b][1] for c in calls) for b in range(ns)]
    layer, kv = make_layer(kind, window, shape, final, (100, case))
    hist = SeqHistory(final, hkv, 128, 100, case)
    exp_k, exp_v = to_bits(kv.k_pool), to_bits(kv.v_pool)
    okind = OL.SWA if kind == "swa" else OL.FULL
    for call in calls:
        starts = [s for s, _ in call]
        ends = [e for _, e in call]
        slots = append_history(layer, shape, kv, hist, starts, ends)
        exp_slots = OL.slot_mapping(okind, window or None, pg, kv.table_host, starts,
                                    [e - s for s, e in call])
        assert np.array_equal(slots, exp_slots), "slot mapping differs from the oracle"
        kn = np.concatenate([hist.k[b][s:e] for b, (s, e) in enumerate(call)])
        vn = np.concatenate([hist.v[b][s:e] for b, (s, e) in enumerate(call)])
        exp_k, exp_v = OL.apply_append(exp_k, exp_v, exp_slots, kn, vn)
        torch.cuda.synchronize()
        _check_pools(kv, exp_k, exp_v)
    # the oracle's view of which ring slot holds which position agrees as well
    if kind == "swa":
        r = OL.ring_pages(window, pg)
        for b in range(ns):
            for (entry, off), pos in OL.ring_positions(window, pg, final[b]).items():
                page = kv.table_host[b][entry]
                assert np.array_equal(OL.k_rows(to_bits(kv.k_pool), page, off), hist.k[b][pos])
        assert r == hswa.ring_pages(window, pg)


def test_append_empty_and_noop(gpu_lib):
    shape = hswa.Shape(8, 1, 128, 16)
    layer, kv = make_layer("full", 0, shape, [16], (101,))
    before = to_bits(kv.k_pool)
    empty = torch.empty((0, 1, 128), dtype=torch.bfloat16, device="cuda")
    hswa.kv_append(layer, shape, kv.cache, empty, empty, torch.tensor([0, 0], dtype=torch.int32, device="cuda"),
                   torch.tensor([0], dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    assert np.array_equal(before, to_bits(kv.k_pool))
