"""GPU parity of serving schedules whose block tables come from the
explicit-release dual-pool allocator: sequences are admitted, prefilled in
chunks, decoded for a number of steps and freed, while others reuse their
pages (pools start NaN-filled, so reused pages hold stale keys of other
sequences). Every prefill and decode output of a FULL layer and of an SWA layer
over the explicit-release table (HSWA_LAYER_SWA_PAGED) is compared with the
fp64 oracle over each sequence's whole history: released pages are never read
and a page that changes owner never leaks into a result."""

import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from paper_2607_13095_amd import hswa
from tests.hswa_testlib import assert_close, i32, to_dev, to_f64

pytestmark = pytest.mark.gpu

D = 128


def _pools(num_pages, hkv, pg):
    k = torch.full(hswa.k_pool_shape(num_pages, hkv, pg, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    v = torch.full(hswa.v_pool_shape(num_pages, hkv, pg, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    return k, v


@pytest.mark.parametrize("pg,window,release_every", [(16, 128, 3), (64, 128, 1), (16, 40, 8)])
def test_allocator_serving_schedule(gpu_lib, pg, window, release_every):
    print(f"[allocator] pg={pg} W={window} N={release_every}", flush=True)
    hq, hkv, slots, stride = 16, 2, 3, 64
    full_pages, swa_pages = slots * stride, slots * (-(-(window + 300) // pg) + 2)
    alloc = hswa.Allocator(pg, window, full_pages, swa_pages, slots, stride, release_every)
    shape = hswa.Shape(hq, hkv, D, pg)
    kf, vf = _pools(full_pages, hkv, pg)
    ks, vs = _pools(swa_pages, hkv, pg)
    full_layer, swa_layer = hswa.Layer.full(), hswa.Layer.swa_paged(window)
    rng = synth.rng_of(700, pg, window)
    hist = {}       # slot -> (K bits, V bits) of the whole sequence so far
    plan = {}       # slot -> remaining work: ("chunk", n) / ("decode", n)
    seq_id = 0
    checked = 0
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")

    def tables(b):
        f, s = alloc.tables()
        return (hswa.Cache(kf, vf, torch.from_numpy(f[b:b + 1].copy()).cuda()),
                hswa.Cache(ks, vs, torch.from_numpy(s[b:b + 1].copy()).cuda()))

    for step in range(70):
        b = step % slots
        if b not in plan:  # admit a new request into this slot
            prompt = int(rng.integers(40, 700))
            chunk = int(rng.integers(24, 260))
            if alloc.admit(b, prompt, chunk) != 0:
                continue
            seq_id += 1
            total = prompt + int(rng.integers(4, 30))
            hist[b] = (synth.normal_bf16((total, hkv, D), 700, seq_id, synth.TAG_K),
                       synth.normal_bf16((total, hkv, D), 700, seq_id, synth.TAG_V))
            plan[b] = {"len": 0, "prompt": prompt, "chunk": chunk, "total": total, "id": seq_id}
        st = plan[b]
        L = st["len"]
        kh, vh = hist[b]
        if L < st["prompt"]:  # one prefill chunk
            C = min(st["chunk"], st["prompt"] - L)
            assert alloc.extend(b, L + C) == 0
            cf, cs = tables(b)
            q = synth.normal_bf16((C, hq, D), 700, st["id"], L, synth.TAG_Q)
            kn, vn = to_dev(kh[L:L + C]), to_dev(vh[L:L + C])
            cu, pre = i32([0, C]), i32([L])
            for layer, cache, w in ((full_layer, cf, None), (swa_layer, cs, window)):
                out = torch.empty((C, hq, D), dtype=torch.bfloat16, device="cuda")
                hswa.prefill(layer, shape, cache, to_dev(q), kn, vn, cu, pre, C, out)
                hswa.kv_append(layer, shape, cache, kn, vn, cu, pre)
                torch.cuda.synchronize()
                ref = OA.prefill(OA.bf16_bits_to_f64(q), OA.bf16_bits_to_f64(kh[:L + C]),
                                 OA.bf16_bits_to_f64(vh[:L + C]), L, w)
                assert_close(to_f64(out), ref, f"prefill seq {st['id']} [{L}, {L + C}) {layer.kind}")
                checked += 1
            alloc.step_end(b, False)
            st["len"] = L + C
        elif L < st["total"]:  # one decode step
            assert alloc.extend(b, L + 1) == 0
            cf, cs = tables(b)
            q = synth.normal_bf16((1, hq, D), 700, st["id"], L, synth.TAG_QDEC)
            kn, vn = to_dev(kh[L:L + 1]), to_dev(vh[L:L + 1])
            for layer, cache, w in ((full_layer, cf, None), (swa_layer, cs, window)):
                hswa.kv_append(layer, shape, cache, kn, vn, i32([0, 1]), i32([L]))
                out = torch.empty((1, hq, D), dtype=torch.bfloat16, device="cuda")
                hswa.decode(layer, shape, cache, to_dev(q), i32([L + 1]), L + 1, out, workspace=ws)
                torch.cuda.synchronize()
                ref = OA.decode(OA.bf16_bits_to_f64(q[0]), OA.bf16_bits_to_f64(kh[:L + 1]),
                                OA.bf16_bits_to_f64(vh[:L + 1]), w)
                assert_close(to_f64(out)[0], ref, f"decode seq {st['id']} at {L} {layer.kind}")
                checked += 1
            alloc.step_end(b, True)
            st["len"] = L + 1
        else:  # request end
            alloc.free(b)
            del plan[b], hist[b]
        # SWA usage stays at window (+ chunk) size whatever the length
        _, su, _, _ = alloc.usage(-1)
        assert su <= swa_pages
    assert checked > 60 and seq_id > slots  # pages were handed to later requests
    alloc.close()
