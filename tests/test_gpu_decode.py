"""GPU parity of hswa_decode against the fp64 oracle over the contiguous
history: SWA single pass over the ring, FULL split-KV with log-sum-exp merge,
edge positions around page, window, ring and split boundaries, GQA groups
from 1 to 32, and page sizes 16 and 64."""

import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from paper_2607_13095_amd import hswa
from tests.hswa_testlib import (SeqHistory, append_history, assert_close, i32, make_layer, to_dev, to_f64)

pytestmark = pytest.mark.gpu


def run_decode(kind, window, pg, hq, hkv, ctxs, seed, fill=float("nan"), perm_seed=None):
    """Cache c_b tokens, append the token at c_b, decode it; returns (gpu, ref)."""
    ns = len(ctxs)
    final = [c + 1 for c in ctxs]
    shape = hswa.Shape(hq, hkv, 128, pg)
    layer, kv = make_layer(kind, window, shape, final, perm_seed or seed, fill=fill)
    hist = SeqHistory(final, hkv, 128, *seed)
    append_history(layer, shape, kv, hist, [0] * ns, ctxs)
    append_history(layer, shape, kv, hist, ctxs, final)
    qbits = synth.normal_bf16((ns, hq, 128), *seed, synth.TAG_QDEC)
    out = torch.empty((ns, hq, 128), dtype=torch.bfloat16, device="cuda")
    maxc = max(final)
    wsb = hswa.decode_workspace_bytes(shape, ns, maxc)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device="cuda") if kind == "full" else None
    hswa.decode(layer, shape, kv.cache, to_dev(qbits), i32(final), maxc, out, workspace=ws)
    torch.cuda.synchronize()
    gpu = to_f64(out)
    qf = OA.bf16_bits_to_f64(qbits)
    w = window if kind == "swa" else None
    ref = np.stack([OA.decode(qf[b], OA.bf16_bits_to_f64(hist.k[b]), OA.bf16_bits_to_f64(hist.v[b]), w)
                    for b in range(ns)])
    return gpu, ref


SWA_CTX = [0, 1, 15, 16, 17, 63, 64, 65, 126, 127, 128, 129, 143, 144, 145, 191, 192, 193, 1000, 4097]


@pytest.mark.parametrize("pg", [16, 64])
@pytest.mark.parametrize("window", [1, 2, 127, 128, 129])
def test_decode_swa_edges(gpu_lib, pg, window):
    print(f"[decode-swa] pg={pg} W={window}", flush=True)
    gpu, ref = run_decode("swa", window, pg, 64, 8, SWA_CTX, (200, pg, window))
    assert_close(gpu, ref, f"swa W={window} PG={pg}")


@pytest.mark.parametrize("hq,hkv", [(8, 8), (8, 1), (16, 1), (32, 1), (64, 8)])
def test_decode_groups(gpu_lib, hq, hkv):
    print(f"[decode-groups] hq={hq} hkv={hkv}", flush=True)
    ctxs = [5, 200, 777, 2048, 3000]
    for kind, window in (("swa", 128), ("full", 0)):
        gpu, ref = run_decode(kind, window, 64, hq, hkv, ctxs, (201, hq, hkv))
        assert_close(gpu, ref, f"{kind} hq={hq} hkv={hkv}")


def test_decode_window_one_is_exact_value(gpu_lib):
    """W = 1: the output is V at the query's own position, bit for bit."""
    ctxs = [0, 3, 64, 191, 192, 500]
    shape_hq, shape_hkv = 16, 2
    gpu, ref = run_decode("swa", 1, 16, shape_hq, shape_hkv, ctxs, (202,))
    assert np.array_equal(gpu, ref)


@pytest.mark.parametrize("pg", [16, 64])
def test_decode_full_split_boundaries(gpu_lib, pg):
    """Contexts around multiples of split_len, as one batch and one sequence at
    a time. Alone, a sequence of few chunks gets spans of exactly split_len
    keys, so KV head 0's pieces are [s * split_len, (s + 1) * split_len): then a
    last piece holding only the newest key, quarter pieces and exact
    boundaries all occur; in the batch the span cuts fall elsewhere."""
    shape = hswa.Shape(64, 8, 128, pg)
    ns = 12
    maxc = 5000
    sl = hswa.decode_split_len(shape, ns, maxc)
    assert sl % 256 == 0 and sl > 0
    tl = sl // 4
    ctxs = [sl - 2, sl - 1, sl, 2 * sl - 1, 2 * sl, sl + tl - 1, sl + tl, 2 * sl + 3 * tl, tl - 1, 3 * sl - 2,
            3 * sl - 1, maxc - 1]
    assert len(ctxs) == ns and max(c + 1 for c in ctxs) == maxc and maxc > sl
    print(f"[decode-full-split] pg={pg} split_len={sl}", flush=True)
    gpu, ref = run_decode("full", 0, pg, 64, 8, ctxs, (203, pg))
    assert_close(gpu, ref, f"full split PG={pg}")
    for c in ctxs:
        if c + 1 <= hswa.decode_split_len(shape, 1, c + 1):
            continue  # one pass
        gpu, ref = run_decode("full", 0, pg, 64, 8, [c], (203, pg, c))
        assert_close(gpu, ref, f"full split PG={pg} alone, context {c + 1}")


def test_decode_full_long(gpu_lib):
    ctxs = [1, 100, 32767, 20000, 8191]
    gpu, ref = run_decode("full", 0, 64, 64, 8, ctxs, (204,))
    assert_close(gpu, ref, "full long")


def test_decode_context_clamp_and_empty(gpu_lib):
    """context_lens < 1 give zero rows; ns = 0 is a no-op."""
    shape = hswa.Shape(8, 1, 128, 16)
    layer, kv = make_layer("full", 0, shape, [64, 64], (205,))
    q = torch.zeros((2, 8, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.full((2, 8, 128), 7.0, dtype=torch.bfloat16, device="cuda")
    hswa.decode(layer, shape, kv.cache, q, i32([0, -3]), 64, out)
    torch.cuda.synchronize()
    assert torch.count_nonzero(out).item() == 0


def test_decode_full_spans_cross_short_segments(gpu_lib):
    """FULL split over a batch of many short and some long contexts: the spans
    (about 16 chunks here) cross (sequence, head) segments of 1-13 chunks, so
    some segments are covered whole by one wave (output written directly) and
    others are cut into pieces merged by log-sum-exp."""
    rng = np.random.default_rng(206)
    ctxs = [int(x) for x in rng.integers(0, 420, size=100)] + [6000] * 12
    rng.shuffle(ctxs)
    shape = hswa.Shape(64, 16, 128, 64)
    sl = hswa.decode_split_len(shape, len(ctxs), max(ctxs) + 1)
    assert max(ctxs) + 1 > sl  # the split path
    print(f"[decode-full-spans] ns={len(ctxs)} split_len={sl}", flush=True)
    gpu, ref = run_decode("full", 0, 64, 64, 16, ctxs, (206,))
    assert_close(gpu, ref, "full spans over short segments")


def test_decode_full_split_with_empty_contexts(gpu_lib):
    """context_lens < 1 inside a split batch: those rows are zero, the span walk
    skips them, and every other row matches the oracle."""
    ctxs = [700, 0, 5000, 3, 0, 2500, 64, 4095]
    ns = len(ctxs)
    final = [c + 1 for c in ctxs]
    shape = hswa.Shape(64, 8, 128, 16)
    seed = (207,)
    layer, kv = make_layer("full", 0, shape, final, seed)
    hist = SeqHistory(final, 8, 128, *seed)
    append_history(layer, shape, kv, hist, [0] * ns, ctxs)
    append_history(layer, shape, kv, hist, ctxs, final)
    qbits = synth.normal_bf16((ns, 64, 128), *seed, synth.TAG_QDEC)
    lens = [0 if i in (1, 4) else f for i, f in enumerate(final)]
    lens[6] = -5
    maxc = max(final)
    out = torch.full((ns, 64, 128), 3.0, dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(max(1, hswa.decode_workspace_bytes(shape, ns, maxc)), dtype=torch.uint8, device="cuda")
    assert maxc > hswa.decode_split_len(shape, ns, maxc)
    print(f"[decode-full-empty] lens={lens}", flush=True)
    hswa.decode(layer, shape, kv.cache, to_dev(qbits), i32(lens), maxc, out, workspace=ws)
    torch.cuda.synchronize()
    gpu = to_f64(out)
    qf = OA.bf16_bits_to_f64(qbits)
    for b in range(ns):
        if lens[b] < 1:
            assert np.all(gpu[b] == 0.0), b
        else:
            ref = OA.decode(qf[b], OA.bf16_bits_to_f64(hist.k[b]), OA.bf16_bits_to_f64(hist.v[b]), None)
            assert_close(gpu[b], ref, f"full split with empty contexts, row {b}")
    # every context empty on the split path: no wave has work, the merge zeroes every row
    out.fill_(3.0)
    hswa.decode(layer, shape, kv.cache, to_dev(qbits), i32([0] * ns), maxc, out, workspace=ws)
    torch.cuda.synchronize()
    assert torch.count_nonzero(out).item() == 0


def test_decode_full_one_long_sequence_many_pieces(gpu_lib):
    """One 70000-key sequence: its eight head segments are each cut into more
    than 64 pieces (the merge takes them in several 64-wide passes)."""
    ctxs = [69999]
    shape = hswa.Shape(64, 8, 128, 64)
    sl = hswa.decode_split_len(shape, 1, 70000)
    assert 70000 / sl > 64
    print(f"[decode-full-one-long] split_len={sl}", flush=True)
    gpu, ref = run_decode("full", 0, 64, 64, 8, ctxs, (208,))
    assert_close(gpu, ref, "full one long sequence")
