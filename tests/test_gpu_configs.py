"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times, against the fp64 oracle.

  * swa_prefill_512 (1 SWA layer, no cache, 8 q / 1 kv heads, PG 16): every
    output, every slot of the mapping and the pool content after the append.
  * decode_b64 (64 sequences, contexts 1K-32K, SWA + FULL): the benchmark's own
    step (append + decode of both layers); every output.
  * chunked_prefill_4x8k (4 x (8192 cached + 2048 new), SWA + FULL): the
    benchmark's own prefill calls; every output of both layers.
  * stack70 shapes (16 sequences at a 131072-token context): one FULL and one
    SWA layer at full size, sampled sequences; and the 70-layer stack (FULL iff
    layer % 7 == 6) at small contexts, every output of every layer.
  * mixed_step (8 chunks of 4096 over prefixes U[0, 65536] plus 256 decodes with
    log-normal contexts, one pool per layer shared by both calls): sampled
    prefill rows and decode sequences.

Large inputs are drawn on the GPU by the seeded generator; the oracle reads
host copies of those same bf16 inputs. For an SWA query the oracle may be given
a suffix of the history that still holds its whole window: attention is
invariant under a shift of positions and keys outside the window have zero
weight, so the result is the same as over the whole history.
"""

import os

import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from oracle import layout as OL
from paper_2607_13095_amd import hswa
from paper_2607_13095_amd.kvcache import LayerKV, pages_for
from tests.hswa_testlib import assert_close, i32, to_bits, to_dev, to_f64

pytestmark = pytest.mark.gpu

D = 128


def _f64(t):
    return to_f64(t)


def _say(msg):
    print(msg, flush=True)


# ---------------------------------------------------------------------------
# swa_prefill_512
# ---------------------------------------------------------------------------

def test_cfg_swa_prefill_512(gpu_lib):
    wl = synth.swa_prefill_512()
    _say(f"[cfg] {wl.name}")
    C, W, pg = wl.new[0], wl.window, wl.page_size
    shape = hswa.Shape(wl.hq, wl.hkv, D, pg)
    layer = hswa.Layer.swa(W)
    npages = pages_for(layer, pg, [C])
    kv = LayerKV(layer, shape, [C], perm=synth.page_permutation(npages, wl.seed, 0))
    q = synth.normal_bf16((C, wl.hq, D), wl.seed, 0, 0, synth.TAG_Q)
    k = synth.normal_bf16((C, wl.hkv, D), wl.seed, 0, 0, synth.TAG_K)
    v = synth.normal_bf16((C, wl.hkv, D), wl.seed, 0, 0, synth.TAG_V)
    out = torch.full((C, wl.hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    cu, pre = i32([0, C]), i32([0])
    hswa.prefill(layer, shape, kv.cache, to_dev(q), to_dev(k), to_dev(v), cu, pre, C, out)
    slots = torch.empty(C, dtype=torch.int64, device="cuda")
    hswa.kv_append(layer, shape, kv.cache, to_dev(k), to_dev(v), cu, pre, slot_mapping_out=slots)
    torch.cuda.synchronize()

    ref = OA.prefill(OA.bf16_bits_to_f64(q), OA.bf16_bits_to_f64(k), OA.bf16_bits_to_f64(v), 0, W)
    assert_close(_f64(out), ref, wl.name)

    table = OL.build_block_table("swa", W, pg, [C], synth.page_permutation(npages, wl.seed, 0), kv.table_host.shape[1])
    assert np.array_equal(table, kv.table_host)
    want = OL.slot_mapping("swa", W, pg, table, [0], [C])
    got = slots.cpu().numpy()
    assert np.array_equal(got, want)
    assert int((want >= 0).sum()) == OL.ring_pages(W, pg) * pg  # the ring keeps the last R * PG tokens
    kp = to_bits(kv.k_pool)
    vp = to_bits(kv.v_pool)
    for t in np.nonzero(want >= 0)[0]:
        s = int(want[t])
        assert np.array_equal(OL.k_rows(kp, s // pg, s % pg), k[t])
        vb = hswa.v_block(pg)
        assert np.array_equal(vp[s // pg, :, (s % pg) // vb, :, (s % pg) % vb], v[t])


# ---------------------------------------------------------------------------
# decode_b64: the benchmark's own step
# ---------------------------------------------------------------------------

def test_cfg_decode_b64_bench_step(gpu_lib):
    import bench

    wl = synth.decode_b64()
    _say(f"[cfg] {wl.name}")
    db = bench.DecodeBench(wl)
    db.step()
    torch.cuda.synchronize()
    ctx = np.asarray(wl.prefix)
    sample = range(wl.ns)
    for L in db.layers:
        out = _f64(L["out"])
        q = _f64(L["q"])
        w = wl.window if L["kind"] == "swa" else None
        for b in sample:
            lo, hi = int(L["cu"][b]), int(L["cu"][b + 1])
            if w is not None:
                lo = max(lo, hi - 4 * wl.window)  # a suffix that holds the whole window
            kh = np.concatenate([_f64(L["k_hist"][lo:hi]), _f64(L["k_new"][b:b + 1])])
            vh = np.concatenate([_f64(L["v_hist"][lo:hi]), _f64(L["v_new"][b:b + 1])])
            ref = OA.decode(q[b], kh, vh, w)
            assert_close(out[b], ref, f"{wl.name} {L['kind']} seq {b} ctx {ctx[b]}")


# ---------------------------------------------------------------------------
# chunked_prefill_4x8k: the benchmark's own prefill calls
# ---------------------------------------------------------------------------

def _oracle_workers():
    return max(1, min(16, len(os.sched_getaffinity(0))))


def test_cfg_chunked_prefill_bench_calls(gpu_lib):
    """Every output of both layers (4 x 2048 rows x 64 heads each) against the
    oracle. The oracle runs once per (sequence, KV head) over that KV head's 8
    query heads (the GQA group), the tasks spread over a thread pool with one
    BLAS thread each; an SWA task sees the suffix of the history that holds
    every window of its queries."""
    import bench
    from concurrent.futures import ThreadPoolExecutor
    from threadpoolctl import threadpool_limits

    wl = synth.chunked_prefill_4x8k()
    _say(f"[cfg] {wl.name}")
    pb = bench.PrefillBench(wl)
    P, C = np.asarray(wl.prefix), np.asarray(wl.new)
    cuP, cuC = synth.cu_seqlens(P), synth.cu_seqlens(C)
    G = wl.hq // wl.hkv
    for li, L in enumerate(pb.layers):
        pb.call(L)
        torch.cuda.synchronize()
        # the cached prefix was drawn with these seeds and appended at set-up
        kp = _f64(synth.torch_normal_bf16((int(P.sum()), wl.hkv, D), "cuda", wl.seed, li, 0, synth.TAG_K))
        vp = _f64(synth.torch_normal_bf16((int(P.sum()), wl.hkv, D), "cuda", wl.seed, li, 0, synth.TAG_V))
        kn, vn, q, out = _f64(L["kn"]), _f64(L["vn"]), _f64(L["q"]), _f64(L["out"])
        w = wl.window if L["kind"] == "swa" else None

        def task(bg):
            b, g = bg
            p, c = int(P[b]), int(C[b])
            kh = np.concatenate([kp[cuP[b]:cuP[b + 1], g:g + 1], kn[cuC[b]:cuC[b + 1], g:g + 1]])
            vh = np.concatenate([vp[cuP[b]:cuP[b + 1], g:g + 1], vn[cuC[b]:cuC[b + 1], g:g + 1]])
            lo = 0 if w is None else max(0, p - w + 1)  # the first query's window start
            heads = slice(g * G, (g + 1) * G)
            ref = OA.masked_attention(q[cuC[b]:cuC[b + 1], heads], kh[lo:], vh[lo:], np.arange(p, p + c) - lo, w)
            assert_close(out[cuC[b]:cuC[b + 1], heads], ref, f"{wl.name} {L['kind']} seq {b} kv head {g}")
            return b, g

        tasks = [(b, g) for b in range(wl.ns) for g in range(wl.hkv)]
        with threadpool_limits(1), ThreadPoolExecutor(_oracle_workers()) as ex:
            done = list(ex.map(task, tasks))
        assert len(done) == len(tasks)
        _say(f"[cfg] {wl.name} {L['kind']}: all {int(C.sum())} rows x {wl.hq} heads checked")
        del kp, vp, kn, vn, q, out
    del pb
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# stack70 shapes
# ---------------------------------------------------------------------------

def _decode_layer(kind, wl, ctx, li, hist_from=None):
    """Pools of one layer holding positions [hist_from[b], ctx[b]) of every
    sequence, then one decode step (append the token at ctx[b], decode it)."""
    ns, pg, W = len(ctx), wl.page_size, wl.window
    shape = hswa.Shape(wl.hq, wl.hkv, D, pg)
    layer = hswa.Layer.swa(W) if kind == "swa" else hswa.Layer.full()
    final = [c + 1 for c in ctx]
    npages = pages_for(layer, pg, final)
    kv = LayerKV(layer, shape, final, perm=synth.page_permutation(npages, wl.seed, li))
    start = [0] * ns if hist_from is None else list(hist_from)
    n = [c - s for c, s in zip(ctx, start)]
    kh = synth.torch_normal_bf16((sum(n), wl.hkv, D), "cuda", wl.seed, li, 0, synth.TAG_K)
    vh = synth.torch_normal_bf16((sum(n), wl.hkv, D), "cuda", wl.seed, li, 0, synth.TAG_V)
    hswa.kv_append(layer, shape, kv.cache, kh, vh, i32(synth.cu_seqlens(n)), i32(start))
    kn = synth.torch_normal_bf16((ns, wl.hkv, D), "cuda", wl.seed, li, 0, synth.TAG_KDEC)
    vn = synth.torch_normal_bf16((ns, wl.hkv, D), "cuda", wl.seed, li, 0, synth.TAG_VDEC)
    q = synth.torch_normal_bf16((ns, wl.hq, D), "cuda", wl.seed, li, 0, synth.TAG_QDEC)
    hswa.kv_append(layer, shape, kv.cache, kn, vn, i32(np.arange(ns + 1)), i32(ctx))
    out = torch.empty((ns, wl.hq, D), dtype=torch.bfloat16, device="cuda")
    maxc = max(final)
    ws = torch.empty(max(1, hswa.decode_workspace_bytes(shape, ns, maxc)), dtype=torch.uint8, device="cuda")
    hswa.decode(layer, shape, kv.cache, q, i32(final), maxc, out, workspace=ws)
    torch.cuda.synchronize()
    return dict(kv=kv, kh=kh, vh=vh, kn=kn, vn=vn, q=q, out=out, cu=synth.cu_seqlens(n))


def _check_decode_layer(kind, wl, r, seqs, what):
    w = wl.window if kind == "swa" else None
    out, q = _f64(r["out"]), _f64(r["q"])
    for b in seqs:
        lo, hi = int(r["cu"][b]), int(r["cu"][b + 1])
        kh = np.concatenate([_f64(r["kh"][lo:hi]), _f64(r["kn"][b:b + 1])])
        vh = np.concatenate([_f64(r["vh"][lo:hi]), _f64(r["vn"][b:b + 1])])
        assert_close(out[b], OA.decode(q[b], kh, vh, w), f"{what} seq {b}")


@pytest.mark.parametrize("kind", ["full", "swa"])
def test_cfg_stack70_full_size_layer(gpu_lib, kind):
    wl = synth.stack70_decode()
    _say(f"[cfg] {wl.name} {kind} layer at full size")
    ctx = list(wl.prefix)
    li = 6 if kind == "full" else 0
    # SWA: only the last 4096 positions are appended (the ring keeps 192 of them)
    hist_from = None if kind == "full" else [c - 4096 for c in ctx]
    r = _decode_layer(kind, wl, ctx, li, hist_from)
    if kind == "swa":
        assert r["kv"].nbytes() == wl.ns * OL.ring_pages(wl.window, wl.page_size) * 2 * OL.page_bytes(
            wl.hkv, wl.page_size, D)
    _check_decode_layer(kind, wl, r, [0, 3, 7, 11, 15], f"{wl.name} {kind}")


def test_cfg_stack70_dispatch(gpu_lib):
    """70 layers, FULL iff layer % 7 == 6, at small contexts: every output."""
    base = synth.stack70_decode()
    wl = synth.Workload("stack70_small", base.seed, base.hq, base.hkv, D, base.page_size, base.window,
                        base.layers, [100, 300, 700, 1100], [1] * 4, "decode")
    _say(f"[cfg] {wl.name}: {wl.layers.count('full')} FULL + {wl.layers.count('swa')} SWA layers")
    assert wl.layers.count("full") == 10 and all((k == "full") == (l % 7 == 6) for l, k in enumerate(wl.layers))
    for li, kind in enumerate(wl.layers):
        r = _decode_layer(kind, wl, list(wl.prefix), li)
        _check_decode_layer(kind, wl, r, range(4), f"layer {li} {kind}")
        del r


# ---------------------------------------------------------------------------
# mixed_step
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("kind", ["full", "swa"])
def test_cfg_mixed_step(gpu_lib, kind):
    wl = synth.mixed_step()
    _say(f"[cfg] {wl.name} {kind}")
    li = 1 if kind == "full" else 0
    dm = np.asarray(wl.decode_mask)
    P, C = np.asarray(wl.prefix), np.asarray(wl.new)
    pre_idx, dec_idx = np.nonzero(~dm)[0], np.nonzero(dm)[0]
    assert np.all(pre_idx < dec_idx.min())  # chunks first, then decodes
    npre = len(pre_idx)
    pg, W = wl.page_size, wl.window
    shape = hswa.Shape(wl.hq, wl.hkv, D, pg)
    layer = hswa.Layer.swa(W) if kind == "swa" else hswa.Layer.full()
    final = (P + C).tolist()
    npages = pages_for(layer, pg, final)
    kv = LayerKV(layer, shape, final, perm=synth.page_permutation(npages, wl.seed, li))
    # one pool and one block table for all sequences; history = the whole final length
    cuF = synth.cu_seqlens(final)
    kh = synth.torch_normal_bf16((int(cuF[-1]), wl.hkv, D), "cuda", wl.seed, li, 0, synth.TAG_K)
    vh = synth.torch_normal_bf16((int(cuF[-1]), wl.hkv, D), "cuda", wl.seed, li, 0, synth.TAG_V)
    # cached prefixes
    idx = torch.cat([torch.arange(int(cuF[b]), int(cuF[b]) + int(P[b]), device="cuda") for b in range(wl.ns)])
    hswa.kv_append(layer, shape, kv.cache, kh[idx].contiguous(), vh[idx].contiguous(),
                   i32(synth.cu_seqlens(P)), i32(np.zeros(wl.ns)))
    # the new tokens of every sequence, in batch order
    idx = torch.cat([torch.arange(int(cuF[b]) + int(P[b]), int(cuF[b + 1]), device="cuda") for b in range(wl.ns)])
    kn, vn = kh[idx].contiguous(), vh[idx].contiguous()
    cuN = synth.cu_seqlens(C)
    Tp = int(cuN[npre])
    qp = synth.torch_normal_bf16((Tp, wl.hq, D), "cuda", wl.seed, li, 1, synth.TAG_Q)
    qd = synth.torch_normal_bf16((len(dec_idx), wl.hq, D), "cuda", wl.seed, li, 1, synth.TAG_QDEC)
    # prefill of the chunks over their cached prefixes (rows 0..npre-1 of the table)
    cache_p = hswa.Cache(kv.k_pool, kv.v_pool, kv.block_table[:npre])
    outp = torch.empty((Tp, wl.hq, D), dtype=torch.bfloat16, device="cuda")
    hswa.prefill(layer, shape, cache_p, qp, kn[:Tp], vn[:Tp], i32(cuN[:npre + 1]), i32(P[:npre]), int(C.max()), outp)
    # append every new token (chunks and decode tokens), then decode
    hswa.kv_append(layer, shape, kv.cache, kn, vn, i32(cuN), i32(P))
    cache_d = hswa.Cache(kv.k_pool, kv.v_pool, kv.block_table[npre:])
    outd = torch.empty((len(dec_idx), wl.hq, D), dtype=torch.bfloat16, device="cuda")
    dfinal = (P[dec_idx] + 1).tolist()
    maxc = max(dfinal)
    ws = torch.empty(max(1, hswa.decode_workspace_bytes(shape, len(dec_idx), maxc)), dtype=torch.uint8, device="cuda")
    hswa.decode(layer, shape, cache_d, qd, i32(dfinal), maxc, outd, workspace=ws)
    torch.cuda.synchronize()

    w = W if kind == "swa" else None
    rng = synth.rng_of(wl.seed, 99, li)
    for b in range(npre):
        c, p = int(C[b]), int(P[b])
        rows = np.array(sorted({0, 63, 64, c - 1} | {int(x) for x in rng.integers(0, c, 6)}))
        lo = int(cuF[b]) if w is None else max(int(cuF[b]), int(cuF[b]) + p + int(rows.min()) - W + 1)
        off = lo - int(cuF[b])
        kf, vf = _f64(kh[lo:int(cuF[b + 1])]), _f64(vh[lo:int(cuF[b + 1])])
        ref = OA.masked_attention(_f64(qp[int(cuN[b]) + rows]), kf, vf, p + rows - off, w)
        assert_close(_f64(outp[int(cuN[b]) + rows]), ref, f"mixed prefill {kind} seq {b} P={p}")
    order = np.argsort(P[dec_idx])
    sample = sorted(set([int(order[0]), int(order[-1])] + [int(x) for x in rng.choice(len(dec_idx), 30, replace=False)]))
    outd64, qd64 = _f64(outd), _f64(qd)
    for i in sample:
        b = int(dec_idx[i])
        lo, hi = int(cuF[b]), int(cuF[b + 1])
        if w is not None:
            lo = max(lo, hi - 4 * W)
        ref = OA.decode(qd64[i], _f64(kh[lo:hi]), _f64(vh[lo:hi]), w)
        assert_close(outd64[i], ref, f"mixed decode {kind} seq {b} ctx {int(P[b])}")
