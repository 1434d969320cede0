"""Pins from text fixtures under tests/golden/: figures the paper states
(layer mix, window, the ~1/7 compute and ~7x KV capacity ratios) and a
hand-worked SWA ring slot mapping."""

import os

import numpy as np
import pytest

from oracle import attention as OA
from oracle import layout as OL

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _figures():
    out = {}
    with open(os.path.join(GOLDEN, "paper_figures.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                k, v = (x.strip() for x in line.split("="))
                out[k] = float(v)
    return out


def test_paper_layer_mix():
    f = _figures()
    assert f["layers_full"] + f["layers_swa"] == f["layers_total"]


def test_paper_kv_capacity_ratio():
    """All-FULL vs hybrid KV bytes of the paper's layer mix at a long context
    (16 sequences x 131073 tokens, 8 KV heads, page size 64)."""
    f = _figures()
    nf, ns_, w = int(f["layers_full"]), int(f["layers_swa"]), int(f["swa_window"])
    lens = [131073] * 16
    full = OL.layer_kv_bytes(OL.FULL, None, 64, lens, 8, 128)
    swa = OL.layer_kv_bytes(OL.SWA, w, 64, lens, 8, 128)
    ratio = (nf + ns_) * full / (nf * full + ns_ * swa)
    assert ratio == pytest.approx(f["kv_capacity_ratio"], rel=0.02)


def test_paper_compute_ratio():
    """Attention pairs of a long causal prefill (L = 131072): hybrid vs all-FULL."""
    f = _figures()
    nf, ns_, w = int(f["layers_full"]), int(f["layers_swa"]), int(f["swa_window"])
    L = 131072
    full_pairs = sum(OA.visible_key_count(p, None) for p in range(0, L, 64)) * 64
    swa_pairs = sum(OA.visible_key_count(p, w) for p in range(0, L, 64)) * 64
    ratio = (nf * full_pairs + ns_ * swa_pairs) / ((nf + ns_) * full_pairs)
    assert ratio == pytest.approx(f["compute_ratio"], rel=0.02)


def test_hand_worked_ring_slots():
    with open(os.path.join(GOLDEN, "ring_slots_w4_pg2.txt")) as fh:
        lines = [l.split("#", 1)[0].strip() for l in fh]
    lines = [l for l in lines if l]
    row = np.array([[int(x) for x in lines[0].split("=")[1].split()]])
    assert OL.ring_pages(4, 2) == row.shape[1]
    for l in lines[1:]:
        head, slots = l.split("slots =")
        kv = dict(t.split("=") for t in head.split()[1:])
        got = OL.slot_mapping(OL.SWA, 4, 2, row, [int(kv["start"])], [int(kv["count"])])
        assert got.tolist() == [int(x) for x in slots.split()]
