"""Prefill and decode of disjoint sequences of one layer, issued on two HIP
streams at once (the prefill chain on one, the decode chain on the other),
give bit-identical results to the same calls in order on one stream: the
library keeps no state that concurrent calls on one device could share,
besides the documented per-device constant. One layer of each kind, a few
prefill chunks over cached prefixes and 64 single-token decodes; each step
also appends its new keys, and the appends are idempotent (the same keys to
the same slots), except that a chunk longer than the SWA ring's spare slots
overwrites prefix keys; every step therefore first re-stores the prefill
sequences' prefixes, so every run sees the same cache. The serial outputs are
checked against the fp64 oracle on sampled rows as well."""

import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from paper_2607_13095_amd import hswa
from tests.hswa_testlib import SeqHistory, append_history, assert_close, i32, make_layer, to_bits, to_dev, to_f64

pytestmark = pytest.mark.gpu

PREFIX = [1900, 0, 777, 3000]
CHUNK = [512, 300, 129, 64]


@pytest.mark.parametrize("kind,window", [("full", 0), ("swa", 128)])
def test_two_streams_match_serial(gpu_lib, kind, window):
    print(f"[streams] kind={kind} W={window}", flush=True)
    hq, hkv, d, pg = 64, 8, 128, 64
    rng = np.random.default_rng(99)
    ndec = 64
    dctx = rng.integers(1, 6000, ndec).tolist()  # context after the appended token
    npf = len(PREFIX)
    final = [p + c for p, c in zip(PREFIX, CHUNK)] + dctx
    shape = hswa.Shape(hq, hkv, d, pg)
    layer, kv = make_layer(kind, window, shape, final, (71, window))
    hist = SeqHistory(final, hkv, d, 71, window)
    # cached state: prefill sequences up to their prefix, decode sequences up to ctx - 1
    append_history(layer, shape, kv, hist, [0] * len(final), PREFIX + [c - 1 for c in dctx])
    cp = hswa.Cache(kv.k_pool, kv.v_pool, kv.block_table[:npf])
    cd = hswa.Cache(kv.k_pool, kv.v_pool, kv.block_table[npf:])
    T = sum(CHUNK)
    qbits = synth.normal_bf16((T, hq, d), 71, window, synth.TAG_Q)
    qp = to_dev(qbits)
    kp = to_dev(np.concatenate([hist.k[b][p:p + c] for b, (p, c) in enumerate(zip(PREFIX, CHUNK))]))
    vp = to_dev(np.concatenate([hist.v[b][p:p + c] for b, (p, c) in enumerate(zip(PREFIX, CHUNK))]))
    qdbits = synth.normal_bf16((ndec, hq, d), 71, window, synth.TAG_QDEC)
    qd = to_dev(qdbits)
    kd = to_dev(np.stack([hist.k[npf + i][c - 1] for i, c in enumerate(dctx)]))
    vd = to_dev(np.stack([hist.v[npf + i][c - 1] for i, c in enumerate(dctx)]))
    cup, prep = i32(synth.cu_seqlens(CHUNK)), i32(PREFIX)
    cud, startd, lensd = i32(np.arange(ndec + 1)), i32([c - 1 for c in dctx]), i32(dctx)
    maxd = max(dctx)
    ws = torch.empty(max(1, hswa.decode_workspace_bytes(shape, ndec, maxd)), dtype=torch.uint8, device="cuda")

    kpre = to_dev(np.concatenate([hist.k[b][:p] for b, p in enumerate(PREFIX)]))
    vpre = to_dev(np.concatenate([hist.v[b][:p] for b, p in enumerate(PREFIX)]))
    cupre, zero = i32(synth.cu_seqlens(PREFIX)), i32([0] * npf)

    def restore():  # the prefill sequences' cached prefixes, as before any step
        hswa.kv_append(layer, shape, cp, kpre, vpre, cupre, zero)

    def prefill(out):
        hswa.prefill(layer, shape, cp, qp, kp, vp, cup, prep, max(CHUNK), out)
        hswa.kv_append(layer, shape, cp, kp, vp, cup, prep)

    def decode(out):
        hswa.kv_append(layer, shape, cd, kd, vd, cud, startd)
        hswa.decode(layer, shape, cd, qd, lensd, maxd, out, workspace=ws)

    op = torch.full((T, hq, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    od = torch.full((ndec, hq, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    restore()
    prefill(op)
    decode(od)
    torch.cuda.synchronize()
    ref_p, ref_d = to_bits(op), to_bits(od)

    # serial outputs against the oracle on sampled rows
    w = window if kind == "swa" else None
    off = 0
    for b, (p, c) in enumerate(zip(PREFIX, CHUNK)):
        rows = np.unique(np.r_[0, c - 1, rng.integers(0, c, 6)])
        full = OA.prefill(OA.bf16_bits_to_f64(qbits[off:off + c]), OA.bf16_bits_to_f64(hist.k[b]),
                          OA.bf16_bits_to_f64(hist.v[b]), p, w, shape.scale)
        assert_close(to_f64(op[off:off + c])[rows], full[rows], f"serial prefill seq {b}")
        off += c
    for i in rng.integers(0, ndec, 8):
        c = dctx[i]
        ref = OA.decode(OA.bf16_bits_to_f64(qdbits[i]), OA.bf16_bits_to_f64(hist.k[npf + i][:c]),
                        OA.bf16_bits_to_f64(hist.v[npf + i][:c]), w, shape.scale)
        assert_close(to_f64(od[i]), ref, f"serial decode seq {i}")

    side = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    outs = []
    for rep in range(3):  # back to back, no host synchronisation between reps
        op2 = torch.full_like(op, float("nan"))
        od2 = torch.full_like(od, float("nan"))
        restore()
        side.wait_stream(main)
        with torch.cuda.stream(side):
            decode(od2)
        prefill(op2)
        main.wait_stream(side)
        outs.append((op2, od2))
    torch.cuda.synchronize()
    for rep, (op2, od2) in enumerate(outs):
        assert np.array_equal(to_bits(op2), ref_p), f"prefill rep {rep} differs from the serial run"
        assert np.array_equal(to_bits(od2), ref_d), f"decode rep {rep} differs from the serial run"
