"""GPU parity of multi-query decode (hswa_decode_multi, the verification shape
of multi-token prediction: several new tokens per sequence, causal among
themselves) against the fp64 oracle: FULL layers with split-KV pieces whose
last piece holds keys only the later queries see, SWA windows per query,
GQA groups 1 to 16, and agreement with single-query decode."""

import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from paper_2607_13095_amd import hswa
from tests.hswa_testlib import SeqHistory, append_history, assert_close, i32, make_layer, to_dev, to_f64

pytestmark = pytest.mark.gpu

D = 128


def run_multi(kind, window, pg, hq, hkv, ctxs, nq, seed, ctx_override=None, scale=None):
    """ctxs: cached tokens before the nq new ones; returns (gpu, ref) [ns, nq, hq, D]."""
    ns = len(ctxs)
    final = [c + nq for c in ctxs]
    shape = hswa.Shape(hq, hkv, D, pg, scale=scale)
    layer, kv = make_layer(kind, window, shape, final, seed)
    hist = SeqHistory(final, hkv, D, *seed)
    append_history(layer, shape, kv, hist, [0] * ns, ctxs)
    append_history(layer, shape, kv, hist, ctxs, final)
    qbits = synth.normal_bf16((ns, nq, hq, D), *seed, synth.TAG_QDEC)
    lens = ctx_override if ctx_override is not None else final
    maxc = max(max(lens), 1)
    out = torch.full((ns, nq, hq, D), 7.0, dtype=torch.bfloat16, device="cuda")
    wsb = hswa.decode_multi_workspace_bytes(shape, ns, nq, maxc)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device="cuda")
    hswa.decode_multi(layer, shape, kv.cache, to_dev(qbits), i32(lens), maxc, out, workspace=ws)
    torch.cuda.synchronize()
    w = window if kind == "swa" else None
    ref = np.zeros((ns, nq, hq, D))
    for b in range(ns):
        L = lens[b]
        pos = np.arange(L - nq, L)
        ok = pos >= 0
        if ok.any():
            ref[b][ok] = OA.masked_attention(OA.bf16_bits_to_f64(qbits[b][ok]), OA.bf16_bits_to_f64(hist.k[b][:L]),
                                             OA.bf16_bits_to_f64(hist.v[b][:L]), pos[ok], w, shape.scale)
    return to_f64(out), ref, (layer, shape, kv, qbits, lens, maxc)


@pytest.mark.parametrize("nq", [2, 4, 7])
@pytest.mark.parametrize("kind,window", [("full", 0), ("swa", 128), ("swa", 5), ("swa", 1)])
def test_decode_multi(gpu_lib, nq, kind, window):
    print(f"[decode-multi] nq={nq} {kind} W={window}", flush=True)
    ctxs = [0, 1, 62, 63, 200, 1000, 3000]
    gpu, ref, _ = run_multi(kind, window, 64, 64, 8, ctxs, nq, (900, nq, window))
    assert_close(gpu, ref, f"decode multi nq={nq} {kind} W={window}")


@pytest.mark.parametrize("hq,hkv", [(8, 8), (16, 1), (32, 4)])
def test_decode_multi_groups(gpu_lib, hq, hkv):
    print(f"[decode-multi-groups] hq={hq} hkv={hkv}", flush=True)
    for kind, window in (("full", 0), ("swa", 128)):
        gpu, ref, _ = run_multi(kind, window, 16, hq, hkv, [5, 300, 2500], 4, (901, hq, hkv))
        assert_close(gpu, ref, f"decode multi groups {kind} hq={hq} hkv={hkv}")


def test_decode_multi_split_tail(gpu_lib):
    """FULL split with final contexts (c + nq) one past a multiple of split_len,
    quarter offsets, an exact multiple, one below three and the max, as one
    batch and one sequence at a time. Alone, KV head 0's spans are split_len
    keys from position 0, so a final context of s * split_len + 1 leaves a last
    piece holding only the newest key, which the first three queries do not
    see (their partials carry weight 0 in the merge)."""
    nq, ns, maxc = 4, 7, 6000
    shape = hswa.Shape(64, 8, D, 64)
    sl = hswa.decode_split_len(shape, ns, maxc)
    tl = sl // 4
    finals = [sl + 1, 2 * sl + 1, 3 * sl + 2 * tl + 1, 2 * sl + 3 * tl + 2, sl, 3 * sl - 1, maxc]
    ctxs = [f - nq for f in finals]
    gpu, ref, _ = run_multi("full", 0, 64, 64, 8, ctxs, nq, (902,))
    assert_close(gpu, ref, f"decode multi split tail, split_len {sl}")
    for f in finals:
        sl1 = hswa.decode_split_len(shape, 1, f)
        if f <= sl1:
            continue  # one pass
        gpu, ref, _ = run_multi("full", 0, 64, 64, 8, [f - nq], nq, (902, f))
        assert_close(gpu, ref, f"decode multi split tail alone, final {f}, split_len {sl1}")


def test_decode_multi_split_no_visible_key(gpu_lib):
    """Split path (max context above one piece) with a sequence whose context
    is below num_queries: its first queries see no key and get zero rows from
    the merge (every partial has log-sum-exp -inf)."""
    gpu, ref, _ = run_multi("full", 0, 64, 64, 8, [0, 6000], 4, (905,), ctx_override=[2, 6004])
    assert np.all(gpu[0][:2] == 0) and np.all(gpu[0][2:] != 0)
    assert_close(gpu, ref, "decode multi split, no visible key")


def test_decode_multi_one_equals_decode(gpu_lib):
    gpu, ref, (layer, shape, kv, qbits, lens, maxc) = run_multi("full", 0, 64, 64, 8, [100, 5000, 20000], 1, (903,))
    assert_close(gpu, ref, "decode multi nq=1")
    out = torch.empty((3, 64, D), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(max(1, hswa.decode_workspace_bytes(shape, 3, maxc)), dtype=torch.uint8, device="cuda")
    hswa.decode(layer, shape, kv.cache, to_dev(qbits[:, 0]), i32(lens), maxc, out, workspace=ws)
    torch.cuda.synchronize()
    assert np.array_equal(to_f64(out), gpu[:, 0])


def test_decode_multi_short_context_zero_rows(gpu_lib):
    """context_lens below num_queries: queries at negative positions get zero rows."""
    gpu, ref, _ = run_multi("full", 0, 16, 16, 2, [3, 3], 4, (904,), ctx_override=[2, 4])
    assert np.all(gpu[0][:2] == 0) and np.all(gpu[0][2:] != 0)
    assert_close(gpu, ref, "decode multi short")


@pytest.mark.parametrize("pg,window,nq", [(16, 128, 17), (16, 5, 28), (64, 128, 64)])
def test_decode_multi_swa_largest_legal_count(gpu_lib, pg, window, nq):
    """The largest query count an SWA ring accepts, R * PG - W + 1 (capped at
    64): the first query's window reaches back to the oldest position the ring
    still holds once all nq tokens are appended. One more is rejected."""
    print(f"[decode-multi-limit] pg={pg} W={window} nq={nq}", flush=True)
    assert nq == min(64, hswa.ring_pages(window, pg) * pg - window + 1)
    gpu, ref, (layer, shape, kv, qbits, lens, maxc) = run_multi("swa", window, pg, 16, 2, [0, 3, 150, 1000, 4097],
                                                                nq, (906, pg, window))
    assert_close(gpu, ref, f"decode multi SWA W={window} PG={pg} nq={nq}")
    if nq < 64:
        q = torch.zeros((5, nq + 1, 16, D), dtype=torch.bfloat16, device="cuda")
        out = torch.empty_like(q)
        with pytest.raises(hswa.HswaError) as e:
            hswa.decode_multi(layer, shape, kv.cache, q, i32(lens), maxc, out)
        assert e.value.status == -2


@pytest.mark.parametrize("scale", [1.0, 4.0])
@pytest.mark.parametrize("kind,window", [("full", 0), ("swa", 128), ("swa", 5)])
def test_decode_multi_large_scale(gpu_lib, scale, kind, window):
    """Scales above ln 2: columns whose wave sees none of their keys in a chunk
    keep a finite running maximum (exp2 units) and give no NaN; single-query
    decode too (nq = 1), on the one-pass and the split path."""
    print(f"[decode-multi-scale] scale={scale} {kind} W={window}", flush=True)
    ctxs = [0, 1, 63, 200, 3000, 9000]
    for nq in (1, 4):
        gpu, ref, _ = run_multi(kind, window, 64, 64, 8, ctxs, nq, (907, nq), scale=scale)
        assert_close(gpu, ref, f"decode multi nq={nq} {kind} W={window} scale {scale}")
