"""HIP-graph capture of the decode and prefill calls (the library enqueues
kernels only: no allocation, no memset): a captured step (kv_append + decode
for an SWA and a FULL layer) and a captured chunked prefill are replayed
several times, with eager work of the program and synchronizations between the
replays, and every replay's outputs are compared bit for bit with the eager
call's outputs, which are themselves checked against the fp64 oracle."""

import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from paper_2607_13095_amd import hswa
from tests.hswa_testlib import SeqHistory, append_history, assert_close, i32, make_layer, to_dev, to_f64

pytestmark = pytest.mark.gpu

D = 128


def _capture(fn):
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()  # warm-up on a side stream, as graph capture expects
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def test_graph_decode_step_replays(gpu_lib):
    print("[graph] decode step: SWA + FULL append and decode", flush=True)
    hq, hkv, pg, W = 32, 4, 64, 128
    ctxs = [5, 300, 4100, 9000]
    ns = len(ctxs)
    final = [c + 1 for c in ctxs]
    shape = hswa.Shape(hq, hkv, D, pg)
    maxc = max(final)
    layers = []
    for li, (kind, w) in enumerate((("swa", W), ("full", 0))):
        layer, kv = make_layer(kind, w, shape, final, (1100, li))
        hist = SeqHistory(final, hkv, D, 1100, li)
        append_history(layer, shape, kv, hist, [0] * ns, ctxs)
        kn = to_dev(np.stack([hist.k[b][c] for b, c in enumerate(ctxs)]))
        vn = to_dev(np.stack([hist.v[b][c] for b, c in enumerate(ctxs)]))
        qbits = synth.normal_bf16((ns, hq, D), 1100, li, synth.TAG_QDEC)
        ws = torch.empty(max(1, hswa.decode_workspace_bytes(shape, ns, maxc)), dtype=torch.uint8, device="cuda")
        layers.append(dict(kind=kind, w=w, layer=layer, kv=kv, hist=hist, kn=kn, vn=vn, qbits=qbits, q=to_dev(qbits),
                           ws=ws, out=torch.empty((ns, hq, D), dtype=torch.bfloat16, device="cuda")))
    cu1, start, lens = i32(np.arange(ns + 1)), i32(ctxs), i32(final)

    def step():
        for L in layers:
            hswa.kv_append(L["layer"], shape, L["kv"].cache, L["kn"], L["vn"], cu1, start)
            hswa.decode(L["layer"], shape, L["kv"].cache, L["q"], lens, maxc, L["out"], workspace=L["ws"])

    step()
    torch.cuda.synchronize()
    eager = [L["out"].clone() for L in layers]
    for L, e in zip(layers, eager):
        qf = OA.bf16_bits_to_f64(L["qbits"])
        ref = np.stack([OA.decode(qf[b], OA.bf16_bits_to_f64(L["hist"].k[b]), OA.bf16_bits_to_f64(L["hist"].v[b]),
                                  L["w"] if L["kind"] == "swa" else None) for b in range(ns)])
        assert_close(to_f64(e), ref, f"eager decode {L['kind']}")
    g = _capture(step)
    for rep in range(4):
        for L in layers:
            L["out"].fill_(float("nan"))  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for L, e in zip(layers, eager):
            assert torch.equal(L["out"].view(torch.int16), e.view(torch.int16)), f"replay {rep} {L['kind']}"
        step()  # an eager step between replays
        torch.cuda.synchronize()


def test_graph_prefill_replays(gpu_lib):
    print("[graph] chunked prefill, SWA and FULL", flush=True)
    hq, hkv, pg, W = 16, 2, 64, 128
    prefixes, chunks = [0, 700, 3000], [300, 129, 64]
    ns = len(prefixes)
    final = [p + c for p, c in zip(prefixes, chunks)]
    shape = hswa.Shape(hq, hkv, D, pg)
    T = sum(chunks)
    cu, pre = i32(synth.cu_seqlens(chunks)), i32(prefixes)
    for li, (kind, w) in enumerate((("swa", W), ("full", 0))):
        layer, kv = make_layer(kind, w, shape, final, (1200, li))
        hist = SeqHistory(final, hkv, D, 1200, li)
        append_history(layer, shape, kv, hist, [0] * ns, prefixes)
        kn = to_dev(np.concatenate([hist.k[b][p:p + c] for b, (p, c) in enumerate(zip(prefixes, chunks))]))
        vn = to_dev(np.concatenate([hist.v[b][p:p + c] for b, (p, c) in enumerate(zip(prefixes, chunks))]))
        qbits = synth.normal_bf16((T, hq, D), 1200, li, synth.TAG_Q)
        q = to_dev(qbits)
        out = torch.empty((T, hq, D), dtype=torch.bfloat16, device="cuda")

        # the prefill alone (it only reads the cache): replaying an append as
        # well would move the SWA ring past the prefix window it reads
        def call():
            hswa.prefill(layer, shape, kv.cache, q, kn, vn, cu, pre, max(chunks), out)

        call()
        torch.cuda.synchronize()
        eager = out.clone()
        qf = OA.bf16_bits_to_f64(qbits)
        refs, off = [], 0
        for b, (p, c) in enumerate(zip(prefixes, chunks)):
            refs.append(OA.prefill(qf[off:off + c], OA.bf16_bits_to_f64(hist.k[b]), OA.bf16_bits_to_f64(hist.v[b]), p,
                                   w if kind == "swa" else None))
            off += c
        assert_close(to_f64(eager), np.concatenate(refs), f"eager prefill {kind}")
        g = _capture(call)
        for rep in range(4):
            out.fill_(float("nan"))
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), f"replay {rep} {kind}"
            call()
            torch.cuda.synchronize()


_CAPTURE_FIRST = r"""
import numpy as np, torch, sys
sys.path.insert(0, '.')
import synth
from paper_2607_13095_amd import hswa
from tests.hswa_testlib import SeqHistory, append_history, i32, make_layer, to_dev, to_f64
ctxs = [700, 3000, 5000]
ns, hq, hkv, D = 3, 32, 4, 128
final = [c + 1 for c in ctxs]
maxc = max(final)
shape = hswa.Shape(hq, hkv, D, 64)
assert maxc > hswa.decode_split_len(shape, ns, maxc)
layer, kv = make_layer("full", 0, shape, final, (1102,))
hist = SeqHistory(final, hkv, D, 1102)
append_history(layer, shape, kv, hist, [0] * ns, final)
q = to_dev(synth.normal_bf16((ns, hq, D), 1102, synth.TAG_QDEC))
ws = torch.empty(max(1, hswa.decode_workspace_bytes(shape, ns, maxc)), dtype=torch.uint8, device="cuda")
out = torch.zeros((ns, hq, D), dtype=torch.bfloat16, device="cuda")
lens = i32(final)
torch.cuda.synchronize()
g = torch.cuda.CUDAGraph()
with torch.cuda.graph(g):  # the process's first decode call
    hswa.decode(layer, shape, kv.cache, q, lens, maxc, out, workspace=ws)
outs = []
for _ in range(3):
    out.zero_()
    g.replay()
    torch.cuda.synchronize()
    outs.append(to_f64(out))
eager = torch.empty_like(out)
hswa.decode(layer, shape, kv.cache, q, lens, maxc, eager, workspace=ws)
torch.cuda.synchronize()
ref = to_f64(eager)
assert np.abs(ref).max() > 0
assert all(np.array_equal(o, ref) for o in outs)
print("CAPTURE-FIRST OK", flush=True)
"""


def test_graph_capture_is_first_decode_call(gpu_lib):
    """A FULL (split) decode captured before the process has made any eager
    decode call: the device's resident wave count, looked up on first use,
    must be obtainable inside a capture. Runs in a fresh child process."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    print("[graph] capture as the first decode call (child process)", flush=True)
    r = subprocess.run([sys.executable, "-c", _CAPTURE_FIRST], cwd=root, capture_output=True, text=True, timeout=200)
    assert r.returncode == 0 and "CAPTURE-FIRST OK" in r.stdout, (r.returncode, r.stdout[-2000:], r.stderr[-3000:])
