"""Slot reuse order of the layerwise prefetch schedule (host logic)."""

import pytest

from paper_2607_13095_amd.prefetch import slot_schedule


def test_slot_schedule_reuse_order():
    s = slot_schedule(["swa", "swa", "full", "swa", "full", "swa", "full"], 2)
    # slots alternate within each kind; a slot's previous user is two same-kind layers back
    assert s == [(0, -1), (1, -1), (0, -1), (0, 0), (1, -1), (1, 1), (0, 2)]


@pytest.mark.parametrize("depth", [1, 2, 3])
def test_slot_schedule_previous_user_is_depth_back(depth):
    kinds = ["swa" if l % 7 != 6 else "full" for l in range(70)]
    s = slot_schedule(kinds, depth)
    for l, (slot, prev) in enumerate(s):
        same = [j for j in range(l) if kinds[j] == kinds[l]]
        assert slot == len(same) % depth
        assert prev == (same[-depth] if len(same) >= depth else -1)
        if prev >= 0:
            assert s[prev][0] == slot


def test_slot_schedule_rejects_zero_depth():
    with pytest.raises(ValueError):
        slot_schedule(["swa"], 0)
