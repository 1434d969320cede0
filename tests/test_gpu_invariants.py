"""GPU invariants of the paged hybrid-SWA path.

* physical page placement does not change any output bit (splits are in
  logical positions);
* unused, stale and out-of-window cache slots never reach an output: filling
  them with NaN or with +-3e38 garbage gives bit-identical results ("SWA-Aware
  Prefix Cache Tree": evicted or overwritten SWA slots must never be read);
* W >= L makes the SWA kernels agree with the FULL kernels;
* a chunk longer than the ring, prefilled then appended, leaves a ring from
  which the next decode still matches the oracle over the whole history;
* decode at c equals the last row of a prefill over c + 1 tokens.
"""

import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from oracle import layout as OL
from paper_2607_13095_amd import hswa
from tests.hswa_testlib import (SeqHistory, append_history, assert_close, i32, make_layer, to_dev, to_f64)
from tests.test_gpu_decode import run_decode
from tests.test_gpu_prefill import run_prefill

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kind,window", [("full", 0), ("swa", 128), ("swa", 5)])
def test_page_permutation_bit_identical(gpu_lib, kind, window):
    ctxs = [0, 70, 1000, 5000, 191]
    a, _ = run_decode(kind, window, 16, 64, 8, ctxs, (400,), perm_seed=(401,))
    b, _ = run_decode(kind, window, 16, 64, 8, ctxs, (400,), perm_seed=(402,))
    assert np.array_equal(a, b)
    pa, _, _ = run_prefill(kind, window, 64, 64, 8, [0, 300, 129], [100, 200, 64], (403,), perm_seed=(404,))
    pb, _, _ = run_prefill(kind, window, 64, 64, 8, [0, 300, 129], [100, 200, 64], (403,), perm_seed=(405,))
    assert np.array_equal(pa, pb)


@pytest.mark.parametrize("kind,window", [("full", 0), ("swa", 128), ("swa", 3)])
def test_poisoned_unused_slots_bit_identical(gpu_lib, kind, window):
    ctxs = [0, 15, 63, 64, 1000, 4099]
    a, ref = run_decode(kind, window, 64, 64, 8, ctxs, (410,), fill=float("nan"))
    b, _ = run_decode(kind, window, 64, 64, 8, ctxs, (410,), fill=3e38)
    c, _ = run_decode(kind, window, 64, 64, 8, ctxs, (410,), fill=-3e38)
    assert np.array_equal(a, b) and np.array_equal(a, c)
    assert_close(a, ref, "poisoned decode")
    pa, pref, _ = run_prefill(kind, window, 16, 8, 1, [0, 33, 500], [40, 17, 300], (411,), fill=float("nan"))
    pb, _, _ = run_prefill(kind, window, 16, 8, 1, [0, 33, 500], [40, 17, 300], (411,), fill=3e38)
    assert np.array_equal(pa, pb)
    assert_close(pa, pref, "poisoned prefill")


def test_poisoned_stale_ring_slots(gpu_lib):
    """Overwrite every ring slot outside the decode window with NaN after the
    appends: the decode output does not change by a single bit."""
    window, pg, hq, hkv = 128, 16, 16, 2
    ctxs = [130, 143, 144, 145, 700]
    ns = len(ctxs)
    final = [c + 1 for c in ctxs]
    shape = hswa.Shape(hq, hkv, 128, pg)
    layer, kv = make_layer("swa", window, shape, final, (420,))
    hist = SeqHistory(final, hkv, 128, 420)
    append_history(layer, shape, kv, hist, [0] * ns, ctxs)
    append_history(layer, shape, kv, hist, ctxs, final)
    qbits = synth.normal_bf16((ns, hq, 128), 420, synth.TAG_QDEC)
    out1 = torch.empty((ns, hq, 128), dtype=torch.bfloat16, device="cuda")
    hswa.decode(layer, shape, kv.cache, to_dev(qbits), i32(final), max(final), out1)
    torch.cuda.synchronize()
    poisoned = 0
    for b, L in enumerate(final):
        for (entry, off), pos in OL.ring_positions(window, pg, L).items():
            if pos < L - window:  # held by the ring but outside the window of the query at L-1
                page = int(kv.table_host[b][entry])
                kv.k_pool[OL.k_slot(kv.k_pool.shape, page, off)] = float("nan")
                vb = hswa.v_block(pg)
                kv.v_pool[page, :, off // vb, :, off % vb] = float("nan")
                poisoned += 1
    assert poisoned > 0
    out2 = torch.empty_like(out1)
    hswa.decode(layer, shape, kv.cache, to_dev(qbits), i32(final), max(final), out2)
    torch.cuda.synchronize()
    assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))


def test_window_ge_len_matches_full(gpu_lib):
    ctxs = [0, 100, 1000, 3000]
    s, _ = run_decode("swa", 100000, 64, 64, 8, ctxs, (430,))
    f, ref = run_decode("full", 0, 64, 64, 8, ctxs, (430,))
    assert_close(s, f, "decode SWA(W>=L) vs FULL")
    ps, _, _ = run_prefill("swa", 100000, 64, 64, 8, [0, 500], [300, 200], (431,))
    pf, _, _ = run_prefill("full", 0, 64, 64, 8, [0, 500], [300, 200], (431,))
    assert_close(ps, pf, "prefill SWA(W>=L) vs FULL")


@pytest.mark.parametrize("pg", [16, 64])
def test_ring_eviction_then_decode(gpu_lib, pg):
    """Prefill a 2048-token chunk over an 8192-token prefix on an SWA layer,
    append it (wrapping the ring many times), then decode the next token."""
    window, hq, hkv = 128, 64, 8
    P, C = 8192, 2048
    gpu, ref, (layer, shape, kv, hist, kn, vn) = run_prefill("swa", window, pg, hq, hkv, [P], [C], (440, pg))
    assert_close(gpu, ref, "chunk prefill")
    # the chunk is appended after the prefill (the order the API requires)
    hswa.kv_append(layer, shape, kv.cache, to_dev(kn), to_dev(vn), i32([0, C]), i32([P]))
    # decode the token at position P + C (its K/V drawn now)
    L = P + C + 1
    knew = synth.normal_bf16((1, hkv, 128), 441, synth.TAG_KDEC)
    vnew = synth.normal_bf16((1, hkv, 128), 441, synth.TAG_VDEC)
    hswa.kv_append(layer, shape, kv.cache, to_dev(knew), to_dev(vnew), i32([0, 1]), i32([P + C]))
    qbits = synth.normal_bf16((1, hq, 128), 441, synth.TAG_QDEC)
    out = torch.empty((1, hq, 128), dtype=torch.bfloat16, device="cuda")
    hswa.decode(layer, shape, kv.cache, to_dev(qbits), i32([L]), L, out)
    torch.cuda.synchronize()
    kf = OA.bf16_bits_to_f64(np.concatenate([hist.k[0], knew]))
    vf = OA.bf16_bits_to_f64(np.concatenate([hist.v[0], vnew]))
    dref = OA.decode(OA.bf16_bits_to_f64(qbits[0]), kf, vf, window)
    assert_close(to_f64(out)[0], dref, "decode after ring eviction")
    # the ring holds R*PG positions, flat in the context length
    assert kv.num_pages == hswa.ring_pages(window, pg) + 3


def test_decode_equals_last_prefill_row(gpu_lib):
    for kind, window in (("full", 0), ("swa", 128)):
        c = 777
        gpu_p, _, (layer, shape, kv, hist, kn, vn) = run_prefill(kind, window, 64, 64, 8, [0], [c + 1], (450,))
        # decode the same query over the same history through the cache
        hswa.kv_append(layer, shape, kv.cache, to_dev(kn), to_dev(vn), i32([0, c + 1]), i32([0]))
        qbits = synth.normal_bf16((c + 1, 64, 128), 450, synth.TAG_Q)[-1:]
        out = torch.empty((1, 64, 128), dtype=torch.bfloat16, device="cuda")
        ws = torch.empty(max(1, hswa.decode_workspace_bytes(shape, 1, c + 1)), dtype=torch.uint8, device="cuda")
        hswa.decode(layer, shape, kv.cache, to_dev(qbits), i32([c + 1]), c + 1, out, workspace=ws)
        torch.cuda.synchronize()
        assert_close(to_f64(out)[0], gpu_p[-1], f"decode vs last prefill row ({kind})")
