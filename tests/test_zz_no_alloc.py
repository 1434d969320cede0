"""hswa_decode_noalloc (the decode entry point that allocates nothing: its FULL
split partials live in the library's fixed device array) against hswa_decode
with a caller workspace, through the C ABI: identical outputs on two calls in
a row, the second with a smaller batch and shorter contexts, for a FULL layer
on the split path and an SWA layer; spot rows also against the oracle."""

import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from paper_2607_13095_amd import hswa
from tests.hswa_testlib import SeqHistory, append_history, assert_close, i32, make_layer, to_dev, to_f64

pytestmark = pytest.mark.gpu

D = 128


def _setup(kind, ctxs, seed):
    shape = hswa.Shape(64, 8, D, 64)
    final = [c + 1 for c in ctxs]
    layer, kv = make_layer(kind, 128, shape, final, seed)
    hist = SeqHistory(final, 8, D, *seed)
    append_history(layer, shape, kv, hist, [0] * len(ctxs), final)
    q = synth.normal_bf16((len(ctxs), 64, D), *seed, synth.TAG_QDEC)
    return shape, layer, kv, hist, q, final


def _both(shape, layer, kv, q, final):
    ns, maxc = len(final), max(final)
    lens = i32(final)
    qd = to_dev(q)
    ref_out = torch.full((ns, 64, D), 7.0, dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(max(1, hswa.decode_workspace_bytes(shape, ns, maxc)), dtype=torch.uint8, device="cuda")
    hswa.decode(layer, shape, kv.cache, qd, lens, maxc, ref_out, workspace=ws)
    out = torch.full((ns, 64, D), 7.0, dtype=torch.bfloat16, device="cuda")
    hswa.decode_noalloc(layer, shape, kv.cache, qd, lens, maxc, out)
    torch.cuda.synchronize()
    return to_f64(out), to_f64(ref_out)


@pytest.mark.parametrize("kind", ["full", "swa"])
def test_decode_noalloc_matches_decode(gpu_lib, kind):
    runs = [([int(x) for x in synth.rng_of(1200).integers(1024, 20000, 24)], (1200, 1)),
            ([int(x) for x in synth.rng_of(1201).integers(300, 4000, 5)], (1200, 2))]
    for i, (ctxs, seed) in enumerate(runs):
        print(f"[noalloc] {kind} call {i}: ns={len(ctxs)} max ctx={max(ctxs)}", flush=True)
        shape, layer, kv, hist, q, final = _setup(kind, ctxs, seed)
        if kind == "full":  # both calls take the split path, i.e. use the scratch array
            need = hswa.decode_workspace_bytes(shape, len(final), max(final))
            assert 0 < need <= hswa.NOALLOC_SCRATCH_BYTES
        got, ref = _both(shape, layer, kv, q, final)
        assert np.array_equal(got, ref), f"noalloc differs from decode ({kind}, call {i})"
        w = 128 if kind == "swa" else None
        for b in (0, len(ctxs) - 1):
            o = OA.decode(OA.bf16_bits_to_f64(q[b]), OA.bf16_bits_to_f64(hist.k[b]), OA.bf16_bits_to_f64(hist.v[b]), w)
            assert_close(got[b], o, f"noalloc {kind} call {i} seq {b}")
        del kv
        torch.cuda.empty_cache()
