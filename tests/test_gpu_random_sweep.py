"""Seeded random sweep of the compute calls against the fp64 oracle, over
combinations the hand-picked cases do not pair: page sizes 16-256, GQA groups
1-16, scales from 0.02 to 1.5 (the running maximum then moves in large steps
in exp2 units), SWA windows from 1 to beyond the context (so the window is
served by each of the three prefill kernels: the persistent run kernel, the
per-tile window kernel and the general one), prefixes that do not align
with pages or tiles, and decode batches whose context mixes do or do not
split. Every case prints its parameters before it runs, and every output row
is compared (decode) or all rows of every sequence (prefill)."""

import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from paper_2607_13095_amd import hswa
from tests.hswa_testlib import SeqHistory, append_history, assert_close, i32, make_layer, to_dev, to_f64

pytestmark = pytest.mark.gpu

D = 128


def draw_shape(rng):
    pg = int(rng.choice([16, 32, 64, 128, 256]))
    group = int(rng.choice([1, 2, 4, 8, 16]))
    hkv = int(rng.choice([1, 2, 4]))
    scale = float(1 / np.sqrt(D)) if rng.random() < 0.5 else float(np.exp(rng.uniform(np.log(0.02), np.log(1.5))))
    return pg, group * hkv, hkv, scale


def draw_layer(rng, maxlen):
    if rng.random() < 0.35:
        return "full", 0
    # windows from 1 to past the longest context, log-uniform
    return "swa", int(np.exp(rng.uniform(0, np.log(max(2, 2 * maxlen)))))


@pytest.mark.parametrize("seed", range(32))
def test_random_prefill(gpu_lib, seed):
    rng = np.random.default_rng(9000 + seed)
    pg, hq, hkv, scale = draw_shape(rng)
    ns = int(rng.integers(1, 5))
    prefixes = [int(x) for x in rng.integers(0, 1500, ns)]
    chunks = [int(x) for x in rng.integers(1, 400, ns)]
    kind, window = draw_layer(rng, max(p + c for p, c in zip(prefixes, chunks)))
    print(f"[sweep-prefill] seed={seed} kind={kind} W={window} pg={pg} hq={hq} hkv={hkv} scale={scale:.4f} "
          f"P={prefixes} C={chunks}", flush=True)
    final = [p + c for p, c in zip(prefixes, chunks)]
    shape = hswa.Shape(hq, hkv, D, pg, scale=scale)
    layer, kv = make_layer(kind, window, shape, final, (9000, seed))
    hist = SeqHistory(final, hkv, D, 9000, seed)
    append_history(layer, shape, kv, hist, [0] * ns, prefixes)
    T = sum(chunks)
    qbits = synth.normal_bf16((T, hq, D), 9000, seed, synth.TAG_Q)
    kn = np.concatenate([hist.k[b][p:p + c] for b, (p, c) in enumerate(zip(prefixes, chunks))])
    vn = np.concatenate([hist.v[b][p:p + c] for b, (p, c) in enumerate(zip(prefixes, chunks))])
    out = torch.full((T, hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    hswa.prefill(layer, shape, kv.cache, to_dev(qbits), to_dev(kn), to_dev(vn), i32(synth.cu_seqlens(chunks)),
                 i32(prefixes), max(chunks), out)
    torch.cuda.synchronize()
    gpu = to_f64(out)
    qf = OA.bf16_bits_to_f64(qbits)
    w = window if kind == "swa" else None
    off = 0
    for b, (p, c) in enumerate(zip(prefixes, chunks)):
        ref = OA.prefill(qf[off:off + c], OA.bf16_bits_to_f64(hist.k[b]), OA.bf16_bits_to_f64(hist.v[b]), p, w, scale)
        assert_close(gpu[off:off + c], ref, f"prefill seed {seed} seq {b}")
        off += c


@pytest.mark.parametrize("seed", range(32))
def test_random_decode(gpu_lib, seed):
    rng = np.random.default_rng(9100 + seed)
    pg, hq, hkv, scale = draw_shape(rng)
    ns = int(rng.integers(1, 33))
    # a mix of tiny and long contexts (cached tokens before the new one)
    ctxs = [int(x) for x in np.where(rng.random(ns) < 0.3, rng.integers(0, 40, ns), rng.integers(40, 12000, ns))]
    kind, window = draw_layer(rng, max(ctxs) + 1)
    fused = bool(rng.random() < 0.5)
    print(f"[sweep-decode] seed={seed} kind={kind} W={window} pg={pg} hq={hq} hkv={hkv} scale={scale:.4f} "
          f"ns={ns} fused={fused} ctx max {max(ctxs)}", flush=True)
    final = [c + 1 for c in ctxs]
    shape = hswa.Shape(hq, hkv, D, pg, scale=scale)
    layer, kv = make_layer(kind, window, shape, final, (9100, seed))
    hist = SeqHistory(final, hkv, D, 9100, seed)
    append_history(layer, shape, kv, hist, [0] * ns, ctxs)
    qbits = synth.normal_bf16((ns, hq, D), 9100, seed, synth.TAG_QDEC)
    out = torch.full((ns, hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    maxc = max(final)
    wsb = hswa.decode_workspace_bytes(shape, ns, maxc)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device="cuda")
    if fused:
        kd = to_dev(np.stack([hist.k[b][c] for b, c in enumerate(ctxs)]))
        vd = to_dev(np.stack([hist.v[b][c] for b, c in enumerate(ctxs)]))
        hswa.decode_append(layer, shape, kv.cache, to_dev(qbits), kd, vd, i32(final), maxc, out, workspace=ws)
    else:
        append_history(layer, shape, kv, hist, ctxs, final)
        hswa.decode(layer, shape, kv.cache, to_dev(qbits), i32(final), maxc, out, workspace=ws)
    torch.cuda.synchronize()
    gpu = to_f64(out)
    qf = OA.bf16_bits_to_f64(qbits)
    w = window if kind == "swa" else None
    ref = np.stack([OA.decode(qf[b], OA.bf16_bits_to_f64(hist.k[b]), OA.bf16_bits_to_f64(hist.v[b]), w, scale)
                    for b in range(ns)])
    assert_close(gpu, ref, f"decode seed {seed}")


@pytest.mark.parametrize("seed", range(24))
def test_random_decode_multi(gpu_lib, seed):
    rng = np.random.default_rng(9200 + seed)
    pg, hq, hkv, scale = draw_shape(rng)
    ns = int(rng.integers(1, 17))
    ctxs = [int(x) for x in rng.integers(0, 9000, ns)]
    kind, window = draw_layer(rng, max(ctxs) + 8)
    nq = int(rng.integers(1, 9))
    if kind == "swa":  # a ring keeps R * PG positions: query 0 still needs its window after nq appends
        nq = max(1, min(nq, hswa.ring_pages(window, pg) * pg - window + 1))
    print(f"[sweep-multi] seed={seed} kind={kind} W={window} pg={pg} hq={hq} hkv={hkv} scale={scale:.4f} "
          f"ns={ns} nq={nq} ctx max {max(ctxs)}", flush=True)
    final = [c + nq for c in ctxs]
    shape = hswa.Shape(hq, hkv, D, pg, scale=scale)
    layer, kv = make_layer(kind, window, shape, final, (9200, seed))
    hist = SeqHistory(final, hkv, D, 9200, seed)
    append_history(layer, shape, kv, hist, [0] * ns, ctxs)
    append_history(layer, shape, kv, hist, ctxs, final)
    qbits = synth.normal_bf16((ns, nq, hq, D), 9200, seed, synth.TAG_QDEC)
    maxc = max(final)
    out = torch.full((ns, nq, hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    wsb = hswa.decode_multi_workspace_bytes(shape, ns, nq, maxc)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device="cuda")
    hswa.decode_multi(layer, shape, kv.cache, to_dev(qbits), i32(final), maxc, out, workspace=ws)
    torch.cuda.synchronize()
    gpu = to_f64(out)
    qf = OA.bf16_bits_to_f64(qbits)
    w = window if kind == "swa" else None
    for b, c in enumerate(ctxs):
        ref = OA.prefill(qf[b], OA.bf16_bits_to_f64(hist.k[b]), OA.bf16_bits_to_f64(hist.v[b]), c, w, scale)
        assert_close(gpu[b], ref, f"multi seed {seed} seq {b}")


@pytest.mark.parametrize("seed", range(24))
def test_random_append(gpu_lib, seed):
    """Random batches of append calls (empty and single-token appends
    included): the slot mapping and every byte of both pools, NaN-filled at
    the start, match the layout oracle after every call."""
    from oracle import layout as OL
    from tests.hswa_testlib import to_bits

    rng = np.random.default_rng(9300 + seed)
    pg = int(rng.choice([16, 32, 64, 128, 256]))
    hkv = int(rng.choice([1, 2, 4, 8]))
    ns = int(rng.integers(1, 7))
    ncalls = int(rng.integers(1, 5))
    calls, pos = [], [0] * ns
    for _ in range(ncalls):
        call = []
        for b in range(ns):
            n = int(rng.choice([0, 1, int(rng.integers(1, 700))]))
            call.append((pos[b], pos[b] + n))
            pos[b] += n
        calls.append(call)
    final = [max(1, p) for p in pos]
    kind, window = draw_layer(rng, max(final))
    print(f"[sweep-append] seed={seed} kind={kind} W={window} pg={pg} hkv={hkv} ns={ns} calls={ncalls} "
          f"final={final}", flush=True)
    shape = hswa.Shape(hkv, hkv, D, pg)
    layer, kv = make_layer(kind, window, shape, final, (9300, seed))
    hist = SeqHistory(final, hkv, D, 9300, seed)
    exp_k, exp_v = to_bits(kv.k_pool), to_bits(kv.v_pool)
    okind = OL.SWA if kind == "swa" else OL.FULL
    for ci, call in enumerate(calls):
        starts = [s for s, _ in call]
        slots = append_history(layer, shape, kv, hist, starts, [e for _, e in call])
        exp_slots = OL.slot_mapping(okind, window or None, pg, kv.table_host, starts, [e - s for s, e in call])
        assert np.array_equal(slots, exp_slots), f"slot mapping differs, call {ci}"
        if len(exp_slots):
            kn = np.concatenate([hist.k[b][s:e] for b, (s, e) in enumerate(call)])
            vn = np.concatenate([hist.v[b][s:e] for b, (s, e) in enumerate(call)])
            exp_k, exp_v = OL.apply_append(exp_k, exp_v, exp_slots, kn, vn)
        torch.cuda.synchronize()
        assert np.array_equal(to_bits(kv.k_pool), exp_k), f"K pool differs after call {ci}"
        assert np.array_equal(to_bits(kv.v_pool), exp_v), f"V pool differs after call {ci}"
