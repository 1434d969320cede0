"""The window-safe prefix cache tree (C ABI, host) against its reference model
(a dictionary of cached prefixes): matched FULL length, window-safe length and
matched slots, SWA releases, segment evictions and token counts over seeded
random operation sequences on small alphabets (heavy prefix sharing, node
splits); hand-worked cases of the clipping rule."""

import numpy as np
import pytest

from oracle import prefix as OP
from paper_2607_13095_amd import hswa


def _rand_seq(rng, alphabet, lo, hi, base=None):
    n = int(rng.integers(lo, hi))
    if base is not None and len(base) and rng.random() < 0.7:  # share a prefix with an earlier sequence
        k = int(rng.integers(0, len(base) + 1))
        return list(base[:k]) + [int(x) for x in rng.integers(0, alphabet, max(0, n - k))]
    return [int(x) for x in rng.integers(0, alphabet, n)]


@pytest.mark.parametrize("window", [1, 2, 4, 7, 128])
@pytest.mark.parametrize("seed", [0, 1])
def test_random_ops_match_model(window, seed):
    rng = np.random.default_rng([window, seed])
    tree, model = hswa.PrefixTree(window), OP.PrefixModel(window)
    seqs = []
    slot = 0
    for _ in range(600):
        op = rng.choice(["insert", "match", "release", "evict"], p=[0.3, 0.4, 0.15, 0.15])
        base = seqs[int(rng.integers(len(seqs)))] if seqs else None
        toks = _rand_seq(rng, 3, 0, 40, base)
        if op == "insert":
            n = len(toks)
            full = np.arange(slot, slot + n)
            swa = np.where(rng.random(n) < 0.8, np.arange(slot, slot + n), -1)
            full = np.where(rng.random(n) < 0.95, full, -1)
            slot += n
            tree.insert(toks, full, swa)
            model.insert(toks, full, swa)
            seqs.append(toks)
        elif op == "match":
            fl, sl, fs, ss = tree.match(toks)
            mfl, msl, mfs, mss = model.match(toks)
            assert (fl, sl) == (mfl, msl), (toks, fl, sl, mfl, msl)
            assert fs.tolist() == mfs and ss.tolist() == mss
        elif op == "release":
            upto = int(rng.integers(0, len(toks) + 2))
            assert tree.release_swa(toks, upto) == model.release_swa(toks, upto)
        else:
            keep = int(rng.integers(0, len(toks) + 1))
            assert tree.evict(toks, keep) == model.evict(toks, keep), (toks, keep)
        _, ntok, nswa = tree.stats()
        assert (ntok, nswa) == model.stats()
    tree.close()


def test_window_safe_clipping_hand_worked():
    W = 4
    t = hswa.PrefixTree(W)
    toks = [11, 12, 13, 14, 15, 16, 17, 18]
    full = list(range(100, 108))
    # SWA slots released for positions 0..4, held for 5, 6, 7 (the tail W - 1)
    swa = [-1, -1, -1, -1, -1, 205, 206, 207]
    t.insert(toks, full, swa)
    fl, sl, fs, ss = t.match(toks + [19, 20])
    assert (fl, sl) == (8, 8)  # a new query at 8 reads keys 5, 6, 7: all held
    assert fs.tolist() == full and ss.tolist() == swa
    # a request sharing only the first 7 tokens: P = 7 needs keys 4, 5, 6 -> 4 is gone
    fl, sl, _, _ = t.match(toks[:7] + [99])
    assert (fl, sl) == (7, 0)
    # drop SWA up to position 6: nothing window-safe except the empty prefix
    assert t.release_swa(toks, 6) == 1
    assert t.match(toks)[:2] == (8, 0)
    # a FULL hole stops the match itself
    t.insert(toks, full[:3] + [-1] + full[4:], [200 + i for i in range(8)])
    assert t.match(toks)[:2] == (3, 3)
    # evicting from position 5 on leaves 5 cached tokens
    assert t.evict(toks, 5) == 3
    assert t.stats()[1] == 5


def test_window_one_never_clips():
    t = hswa.PrefixTree(1)
    t.insert([1, 2, 3], [0, 1, 2], [-1, -1, -1])
    assert t.match([1, 2, 3, 4])[:2] == (3, 3)  # W = 1 reads no earlier key
