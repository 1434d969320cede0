"""Benchmark of the hybrid-SWA paged attention hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--no-prefill]

Workload (the decode configuration the headline metric is quoted on):
  64 sequences, cached contexts uniform in [1024, 32768], one SWA layer
  (W = 128) and one FULL layer, 64 query / 8 KV heads, head dim 128, bf16,
  page size 64, pages placed by a seeded permutation. One step appends one new
  token per sequence to both layers (hswa_kv_append) and decodes it
  (hswa_decode): the whole decode hot path. Inputs are resident in HBM before
  the timed region.

Also measured (same run, reported under "prefill"): chunked prefill of 4
sequences with an 8192-token cached prefix and a 2048-token chunk, one SWA and
one FULL layer (hswa_prefill then hswa_kv_append).

value = algorithmic decode bytes (K and V of every visible key read once per
(sequence, KV head, layer), plus q and o) / step time. The roofline entry is
for the FULL-layer decode call (split-KV kernel + log-sum-exp merge), timed with
HIP events on the stream it runs on, inside the timed region.
The CPU baseline is the fp64 oracle on a bounded sample of the same workload.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2516.6

# Bytes moved between L2 and memory per call, from rocprofv3 --pmc FETCH_SIZE and
# --pmc WRITE_SIZE runs of this script with --copy-calibration, each counter
# scaled by what it reads for the plain 1 GiB copy (FETCH_SIZE reads 524,300 KiB
# for 1 GiB read: x2.0; WRITE_SIZE reads 1,048,576 KiB for 1 GiB written: x1.0).
# A figure holds only for the kernel sources it was taken on (SHA-256 below);
# once they change the benchmark reports null until it is measured again.
MEASURED_TRAFFIC = {
    "decode_full": {"sources": ["decode.hip", "hswa_common.h", "hswa_launch.h"],
                    "sha256": "a3f66ed9d3e531aac9d80aa9c69110a213dbcd93cc88299e96a6bacde1a87893",
                    "fetch_bytes": 4100957394, "write_bytes": 34749121},
    "prefill_full": {"sources": ["prefill.hip", "hswa_common.h", "hswa_launch.h"],
                     "sha256": "0f480bc1173720a12440ca104f61931cab2c2ffbe7cd6fb8b16772aa08ca3a76",
                     "fetch_bytes": 453118809, "write_bytes": 134217728},
}


def sources_sha256(names):
    import hashlib

    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2607_13095_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(key):
    """HBM-side bytes per call of a kernel, or None if its sources changed."""
    t = MEASURED_TRAFFIC[key]
    if sources_sha256(t["sources"]) != t["sha256"]:
        return None
    return int(t["fetch_bytes"] + t["write_bytes"])


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--roofline-only", action="store_true",
                    help="only the decode step and the prefill calls the roofline entries time (for counter runs)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target oracle time for the CPU baseline")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 1 GiB device copy three times (reference for HBM byte counters)")
    return ap.parse_args()


COPY_BYTES = 1 << 30


def copy_calibration():
    """A plain device-to-device copy of COPY_BYTES, three times: under
    rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE its readings give the factor that
    turns the counters into bytes."""
    import torch

    src = torch.ones(COPY_BYTES // 2, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"[bench] copy calibration: 3 x {COPY_BYTES} bytes copied")
    del src, dst
    torch.cuda.empty_cache()


# ----------------------------------------------------------------------------
# decode workload
# ----------------------------------------------------------------------------

class DecodeBench:
    def __init__(self, wl, nq=1):
        import torch

        import synth
        from paper_2607_13095_amd import hswa
        from paper_2607_13095_amd.kvcache import LayerKV, pages_for

        self.wl, self.nq = wl, int(nq)
        dev = "cuda"
        hq, hkv, d, pg, W = wl.hq, wl.hkv, wl.head_dim, wl.page_size, wl.window
        ns = wl.ns
        self.ctx = np.asarray(wl.prefix, dtype=np.int64)          # cached tokens c_b
        self.final = (self.ctx + nq).tolist()                      # context incl. the nq new tokens
        self.shape = hswa.Shape(hq, hkv, d, pg)
        self.maxc = int(max(self.final))
        i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32), device=dev)  # noqa: E731
        self.layers = []
        for li, kind in enumerate(wl.layers):
            layer = hswa.Layer.swa(W) if kind == "swa" else hswa.Layer.full()
            npages = pages_for(layer, pg, self.final)
            kv = LayerKV(layer, self.shape, self.final, perm=synth.page_permutation(npages, wl.seed, li))
            # history: positions [0, c_b] of every sequence, drawn on the GPU
            T = int(self.ctx.sum())
            k_hist = synth.torch_normal_bf16((T, hkv, d), dev, wl.seed, li, 0, synth.TAG_K)
            v_hist = synth.torch_normal_bf16((T, hkv, d), dev, wl.seed, li, 0, synth.TAG_V)
            cu = synth.cu_seqlens(self.ctx)
            hswa.kv_append(layer, self.shape, kv.cache, k_hist, v_hist, i32(cu), i32(np.zeros(ns)))
            k_new = synth.torch_normal_bf16((ns * nq, hkv, d), dev, wl.seed, li, 0, synth.TAG_KDEC)
            v_new = synth.torch_normal_bf16((ns * nq, hkv, d), dev, wl.seed, li, 0, synth.TAG_VDEC)
            qshape = (ns, hq, d) if nq == 1 else (ns, nq, hq, d)
            q = synth.torch_normal_bf16(qshape, dev, wl.seed, li, 0, synth.TAG_QDEC)
            out = torch.empty(qshape, dtype=torch.bfloat16, device=dev)
            wsb = hswa.decode_multi_workspace_bytes(self.shape, ns, nq, self.maxc) if kind == "full" else 0
            ws = torch.empty(max(1, wsb), dtype=torch.uint8, device=dev)
            self.layers.append(dict(kind=kind, layer=layer, kv=kv, k_hist=k_hist, v_hist=v_hist, cu=cu,
                                    k_new=k_new, v_new=v_new, q=q, out=out, ws=ws))
        self.cu1 = i32(np.arange(ns + 1) * nq)
        self.start = i32(self.ctx)
        self.ctx_lens = i32(self.final)
        torch.cuda.synchronize()
        # algorithmic bytes
        row = hkv * d * 2 * 2                                      # K + V bytes per key
        qo = 2 * ns * nq * hq * d * 2
        self.bytes = {}
        for L in self.layers:
            if L["kind"] == "full":
                keys = int(np.sum(self.ctx + nq))
            else:
                keys = int(np.sum(np.minimum(W + nq - 1, self.ctx + nq)))
            self.bytes[L["kind"]] = keys * row + qo
        self.append_bytes = len(self.layers) * ns * nq * hkv * d * 2 * 2 * 2   # read + write

    def step(self):
        from paper_2607_13095_amd import hswa

        for L in self.layers:
            hswa.kv_append(L["layer"], self.shape, L["kv"].cache, L["k_new"], L["v_new"], self.cu1, self.start)
            self.decode(L)

    def decode(self, L):
        from paper_2607_13095_amd import hswa

        fn = hswa.decode if self.nq == 1 else hswa.decode_multi
        fn(L["layer"], self.shape, L["kv"].cache, L["q"], self.ctx_lens, self.maxc, L["out"], workspace=L["ws"])

    def time_kind_back_to_back(self, kind, reps):
        """Mean time of one layer kind's decode call over reps calls issued back
        to back between one pair of HIP events on the current stream."""
        import torch

        L = next(x for x in self.layers if x["kind"] == kind)
        self.decode(L)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(reps):
            self.decode(L)
        b.record()
        b.synchronize()
        return a.elapsed_time(b) / reps

    def time_kind(self, kind, reps=20):
        """Event timing of one layer kind's decode call alone (median of reps)."""
        import torch

        L = next(x for x in self.layers if x["kind"] == kind)
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            self.decode(L)
            b.record()
            b.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts))

    def cpu_baseline(self, target_s):
        """fp64 oracle over the sequences (both layers) until ~target_s seconds of
        oracle time. When a whole pass would take less, each oracle call is
        repeated (the count estimated from the first sequence's share of the
        keys), so the rate is measured over about target_s seconds."""
        import math

        from oracle import attention as OA

        threads = _blas_threads()
        done_bytes, t_total, nseq, reps = 0, 0.0, 0, 1
        row = self.wl.hkv * self.wl.head_dim * 2 * 2
        qo = 2 * self.wl.hq * self.wl.head_dim * 2
        W = self.wl.window

        def keys(c):  # keys both layers read for a sequence with c cached tokens
            return sum(c + 1 if L["kind"] == "full" else min(W, c + 1) for L in self.layers)

        for b in range(self.wl.ns):
            for L in self.layers:
                c = int(self.ctx[b])
                lo = int(L["cu"][b])
                window = W if L["kind"] == "swa" else None
                first = 0 if window is None else max(0, c + 1 - window)
                # host copies of exactly the inputs the GPU read (untimed)
                k = _host_f64(L["k_hist"][lo + first:lo + c])
                v = _host_f64(L["v_hist"][lo + first:lo + c])
                k = np.concatenate([k, _host_f64(L["k_new"][b:b + 1])])
                v = np.concatenate([v, _host_f64(L["v_new"][b:b + 1])])
                q = _host_f64(L["q"][b])
                for _ in range(reps):
                    t0 = time.perf_counter()
                    OA.decode(q, k, v, window, self.shape.scale)
                    t_total += time.perf_counter() - t0
                    done_bytes += k.shape[0] * row + qo
            nseq += 1
            if b == 0:
                est_pass = t_total * sum(keys(int(c)) for c in self.ctx) / keys(int(self.ctx[0]))
                reps = max(1, min(20, math.ceil(target_s / est_pass)))
            if t_total >= target_s:
                break
        return {"value": done_bytes / t_total / 1e9, "unit": "GB/s", "cores": threads, "kind": "oracle",
                "sample": f"first {nseq} of {self.wl.ns} sequences, both layers, each oracle call after the "
                          f"first sequence's repeated {reps}x, fp64 numpy oracle, {t_total:.1f} s of oracle time"}


def _host_f64(t):
    import torch

    from oracle import attention as OA

    return OA.bf16_bits_to_f64(t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16))


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info

        info = threadpool_info()
        return int(max((i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"), default=1))
    except Exception:
        return 1


# ----------------------------------------------------------------------------
# prefill workload
# ----------------------------------------------------------------------------

class PrefillBench:
    def __init__(self, wl):
        import torch

        import synth
        from paper_2607_13095_amd import hswa
        from paper_2607_13095_amd.kvcache import LayerKV, pages_for

        self.wl = wl
        dev = "cuda"
        hq, hkv, d, pg, W = wl.hq, wl.hkv, wl.head_dim, wl.page_size, wl.window
        ns = wl.ns
        P = np.asarray(wl.prefix, dtype=np.int64)
        C = np.asarray(wl.new, dtype=np.int64)
        self.P, self.C = P, C
        final = (P + C).tolist()
        self.shape = hswa.Shape(hq, hkv, d, pg)
        i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32), device=dev)  # noqa: E731
        T = int(C.sum())
        self.maxc = int(C.max())
        self.cu = i32(synth.cu_seqlens(C))
        self.pre = i32(P)
        self.layers = []
        for li, kind in enumerate(wl.layers):
            layer = hswa.Layer.swa(W) if kind == "swa" else hswa.Layer.full()
            npages = pages_for(layer, pg, final)
            kv = LayerKV(layer, self.shape, final, perm=synth.page_permutation(npages, wl.seed, li))
            kp = synth.torch_normal_bf16((int(P.sum()), hkv, d), dev, wl.seed, li, 0, synth.TAG_K)
            vp = synth.torch_normal_bf16((int(P.sum()), hkv, d), dev, wl.seed, li, 0, synth.TAG_V)
            hswa.kv_append(layer, self.shape, kv.cache, kp, vp, i32(synth.cu_seqlens(P)), i32(np.zeros(ns)))
            del kp, vp
            q = synth.torch_normal_bf16((T, hq, d), dev, wl.seed, li, 1, synth.TAG_Q)
            kn = synth.torch_normal_bf16((T, hkv, d), dev, wl.seed, li, 1, synth.TAG_K)
            vn = synth.torch_normal_bf16((T, hkv, d), dev, wl.seed, li, 1, synth.TAG_V)
            out = torch.empty((T, hq, d), dtype=torch.bfloat16, device=dev)
            self.layers.append(dict(kind=kind, layer=layer, kv=kv, q=q, kn=kn, vn=vn, out=out))
        torch.cuda.synchronize()
        self.flops, self.bytes = {}, {}
        for L in self.layers:
            pairs = 0
            for p, c in zip(P, C):
                if L["kind"] == "full":
                    pairs += int(c * p + c * (c + 1) // 2)
                else:
                    pos = np.arange(p, p + c)
                    pairs += int(np.minimum(W, pos + 1).sum())
            self.flops[L["kind"]] = 4 * d * hq * pairs
            keys = int((P + C).sum()) if L["kind"] == "full" else int(
                sum(min(int(p), W - 1) + int(c) for p, c in zip(P, C)))
            self.bytes[L["kind"]] = keys * hkv * d * 4 + 2 * T * hq * d * 2

    def call(self, L):
        from paper_2607_13095_amd import hswa

        hswa.prefill(L["layer"], self.shape, L["kv"].cache, L["q"], L["kn"], L["vn"], self.cu, self.pre, self.maxc,
                     L["out"])

    def time_kind(self, kind, reps=20, warmup=10):
        import torch

        L = next(x for x in self.layers if x["kind"] == kind)
        for _ in range(warmup):
            self.call(L)
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            self.call(L)
            b.record()
            b.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts))


def allocator_report(wl, reps=20):
    """SWA layer of the decode workload over explicit-release tables from the
    dual-pool allocator (HSWA_LAYER_SWA_PAGED): pages held per sequence, host
    cost of one decode step's allocator calls, and the decode call's time."""
    import time

    import torch

    import synth
    from paper_2607_13095_amd import hswa

    hq, hkv, d, pg, W = wl.hq, wl.hkv, wl.head_dim, wl.page_size, wl.window
    ns = wl.ns
    ctx = np.asarray(wl.prefix, dtype=np.int64)
    stride = int(-(-(int(ctx.max()) + 2) // pg))
    swa_pages = ns * (-(-(W + 1) // pg) + 2)
    alloc = hswa.Allocator(pg, W, ns * stride, swa_pages, ns, stride, 1)
    shape = hswa.Shape(hq, hkv, d, pg)
    layer = hswa.Layer.swa_paged(W)
    for b in range(ns):
        assert alloc.admit(b, int(ctx[b]), 1) == 0 and alloc.extend(b, int(ctx[b])) == 0
    _, swa_tab = alloc.tables()
    kp = torch.full(hswa.k_pool_shape(swa_pages, hkv, pg, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    vp = torch.full(hswa.v_pool_shape(swa_pages, hkv, pg, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    cache = hswa.Cache(kp, vp, torch.from_numpy(swa_tab).cuda())
    i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32), device="cuda")  # noqa: E731
    # the last W positions of every sequence (earlier ones are not held and would be dropped)
    lo = np.maximum(ctx - W, 0)
    n = ctx - lo
    kh = synth.torch_normal_bf16((int(n.sum()), hkv, d), "cuda", wl.seed, 9, 0, synth.TAG_K)
    vh = synth.torch_normal_bf16((int(n.sum()), hkv, d), "cuda", wl.seed, 9, 0, synth.TAG_V)
    hswa.kv_append(layer, shape, cache, kh, vh, i32(synth.cu_seqlens(n)), i32(lo))
    # one decode step: host allocator calls, then append + decode on the GPU
    t0 = time.perf_counter()
    for b in range(ns):
        assert alloc.extend(b, int(ctx[b]) + 1) == 0
    _, swa_tab = alloc.tables()
    for b in range(ns):
        alloc.step_end(b, True)
    host_us = (time.perf_counter() - t0) * 1e6
    cache = hswa.Cache(kp, vp, torch.from_numpy(swa_tab).cuda())
    kn = synth.torch_normal_bf16((ns, hkv, d), "cuda", wl.seed, 9, 0, synth.TAG_KDEC)
    q = synth.torch_normal_bf16((ns, hq, d), "cuda", wl.seed, 9, 0, synth.TAG_QDEC)
    hswa.kv_append(layer, shape, cache, kn, kn, i32(np.arange(ns + 1)), i32(ctx))
    out = torch.empty((ns, hq, d), dtype=torch.bfloat16, device="cuda")
    lens, maxc = i32(ctx + 1), int(ctx.max()) + 1
    for _ in range(3):
        hswa.decode(layer, shape, cache, q, lens, maxc, out)
    ts = []
    for _ in range(reps):
        a, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        hswa.decode(layer, shape, cache, q, lens, maxc, out)
        b_.record()
        b_.synchronize()
        ts.append(a.elapsed_time(b_))
    per_seq = [alloc.usage(b)[1] for b in range(ns)]
    full_used = alloc.usage(-1)[0]
    alloc.close()
    return {"layer": "SWA over explicit-release tables", "swa_paged_decode_ms": round(float(np.median(ts)), 5),
            "swa_pages_per_seq": [int(min(per_seq)), int(max(per_seq))],
            "swa_pages_per_seq_bound": int(-(-(W - 1) // pg) + 1),
            "full_pages_held": int(full_used), "host_us_per_decode_step": round(host_us, 1)}


def prefetch_report(pb, layers=70, depth=2, reps=3):
    """Layerwise host-to-device prefetch on the chunked-prefill workload: a
    70-layer stack (FULL iff layer % 7 == 6) whose layer pools are loaded from
    pinned host memory into a ring of `depth` device slots per kind. Times the
    stack with data resident (attention only), with copy-then-compute per
    layer on one stream, and with the copies on a stream running ahead."""
    import torch

    from paper_2607_13095_amd import hswa
    from paper_2607_13095_amd.prefetch import LayerPlan, LayerwisePrefetch

    kinds = ["full" if l % 7 == 6 else "swa" for l in range(layers)]
    by_kind = {L["kind"]: L for L in pb.layers}
    host, rings = {}, {}
    for k, L in by_kind.items():
        kp, vp = L["kv"].k_pool, L["kv"].v_pool
        host[k] = (torch.empty(kp.shape, dtype=kp.dtype, pin_memory=True),
                   torch.empty(vp.shape, dtype=vp.dtype, pin_memory=True))
        host[k][0].copy_(kp)
        host[k][1].copy_(vp)
        rings[k] = [(torch.empty_like(kp), torch.empty_like(vp)) for _ in range(depth)]
    plans = [LayerPlan(k, host[k]) for k in kinds]
    h2d_bytes = sum(sum(t.numel() * t.element_size() for t in host[k]) for k in kinds)

    def compute(l, slot):
        L = by_kind[kinds[l]]
        cache = hswa.Cache(slot[0], slot[1], L["kv"].block_table)
        hswa.prefill(L["layer"], pb.shape, cache, L["q"], L["kn"], L["vn"], pb.cu, pb.pre, pb.maxc, L["out"])

    def resident(l, _slot):
        pb.call(by_kind[kinds[l]])

    pf = LayerwisePrefetch(rings, depth)

    def timed(fn):
        fn()  # warm-up
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts))

    t_att = timed(lambda: [resident(l, None) for l in range(layers)])
    t_serial = timed(lambda: pf.run(plans, compute, overlap=False))
    t_over = timed(lambda: pf.run(plans, compute, overlap=True))
    copy_ms = max(t_serial - t_att, 1e-6)
    return {"layers": layers, "depth": depth, "h2d_bytes_per_stack": int(h2d_bytes),
            "attention_only_ms": round(t_att, 3), "copy_then_compute_ms": round(t_serial, 3),
            "layerwise_prefetch_ms": round(t_over, 3),
            "h2d_gbs_serial": round(h2d_bytes / (copy_ms * 1e-3) / 1e9, 1),
            "copy_hidden_frac": round((t_serial - t_over) / copy_ms, 3)}


def prefix_tree_report(window=128, convs=128, turns=8, turn_len=512, seed=11):
    """Window-safe prefix matching on a synthetic multi-turn workload: every
    conversation grows turn by turn; after each turn the SWA slots before the
    window of the next query are released (FULL slots stay). Continuing
    requests match their whole history; requests that branch from an earlier
    turn find FULL KV but no intact window there and are clipped. Reports host
    cost per insert / match and the matched lengths."""
    import time

    from paper_2607_13095_amd import hswa

    rng = np.random.default_rng(seed)
    tree = hswa.PrefixTree(window)
    hist = [[] for _ in range(convs)]
    t_ins = t_match = t_rel = 0.0
    n_ins = n_match = 0
    cont_full = cont_safe = br_full = br_safe = 0
    slot = 0
    for t in range(turns):
        for c in range(convs):
            toks = hist[c] + [int(x) for x in rng.integers(0, 32000, turn_len)]
            t0 = time.perf_counter()
            fl, sl, _, _ = tree.match(toks)
            t_match += time.perf_counter() - t0
            n_match += 1
            cont_full += fl
            cont_safe += sl
            n = len(toks)
            slots = np.arange(slot, slot + n, dtype=np.int64)
            slot += n
            t0 = time.perf_counter()
            tree.insert(toks, slots, slots)
            t_ins += time.perf_counter() - t0
            n_ins += 1
            t0 = time.perf_counter()
            tree.release_swa(toks, n - window + 1)
            t_rel += time.perf_counter() - t0
            hist[c] = toks
    # branch requests: regenerate from the middle of an earlier turn
    for c in range(convs):
        cut = int(rng.integers(1, turns)) * turn_len - 7
        fl, sl, _, _ = tree.match(hist[c][:cut] + [1, 2, 3])
        br_full += fl
        br_safe += sl
    nodes, toks, swa_valid = tree.stats()
    tree.close()
    return {"window": window, "conversations": convs, "turns": turns, "turn_tokens": turn_len,
            "cached_tokens": toks, "tokens_with_swa_slot": swa_valid, "nodes": nodes,
            "continuing_hit_full": cont_full, "continuing_hit_window_safe": cont_safe,
            "branch_hit_full": br_full, "branch_hit_window_safe": br_safe,
            "host_us_per_match": round(t_match / n_match * 1e6, 1),
            "host_us_per_insert": round(t_ins / n_ins * 1e6, 1),
            "host_us_per_release": round(t_rel / n_ins * 1e6, 1)}


def stack70_report(steps=5, warmup=2):
    """The 70-layer hybrid decode step (10 FULL + 60 SWA layers, 16 sequences at
    a 131072-token context): every layer's pools hold its own synthetic KV
    (86 GB of FULL pages, 12 MiB per SWA layer), and one step appends the new
    token and decodes it in every layer. Timed eagerly and as a replayed graph
    of the step, plus per-kind parts; also reports the pool bytes per kind."""
    import torch

    import synth
    from paper_2607_13095_amd import hswa
    from paper_2607_13095_amd.kvcache import LayerKV, pages_for

    wl = synth.stack70_decode()
    dev = "cuda"
    hq, hkv, d, pg, W = wl.hq, wl.hkv, wl.head_dim, wl.page_size, wl.window
    ns = wl.ns
    ctx = np.asarray(wl.prefix, dtype=np.int64)
    final = (ctx + 1).tolist()
    maxc = int(max(final))
    shape = hswa.Shape(hq, hkv, d, pg)
    i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32), device=dev)  # noqa: E731
    ring = hswa.ring_pages(W, pg)
    ws = torch.empty(max(1, hswa.decode_workspace_bytes(shape, ns, maxc)), dtype=torch.uint8, device=dev)
    layers = []
    for li, kind in enumerate(wl.layers):
        layer = hswa.Layer.swa(W) if kind == "swa" else hswa.Layer.full()
        kv = LayerKV(layer, shape, final, perm=synth.page_permutation(pages_for(layer, pg, final), wl.seed, li))
        # cached history: every position for FULL (four sequences at a time),
        # the positions the ring keeps for SWA
        first = np.zeros(ns, dtype=np.int64) if kind == "full" else np.maximum(0, ctx - ring * pg)
        for b0 in range(0, ns, 4):
            sl = slice(b0, min(ns, b0 + 4))
            lens = ctx[sl] - first[sl]
            T = int(lens.sum())
            kh = synth.torch_normal_bf16((T, hkv, d), dev, wl.seed, li, b0, synth.TAG_K)
            vh = synth.torch_normal_bf16((T, hkv, d), dev, wl.seed, li, b0, synth.TAG_V)
            sub = hswa.Cache(kv.k_pool, kv.v_pool, kv.block_table[sl])
            hswa.kv_append(layer, shape, sub, kh, vh, i32(synth.cu_seqlens(lens)), i32(first[sl]))
            del kh, vh
        layers.append(dict(kind=kind, layer=layer, kv=kv,
                           k_new=synth.torch_normal_bf16((ns, hkv, d), dev, wl.seed, li, 0, synth.TAG_KDEC),
                           v_new=synth.torch_normal_bf16((ns, hkv, d), dev, wl.seed, li, 0, synth.TAG_VDEC),
                           q=synth.torch_normal_bf16((ns, hq, d), dev, wl.seed, li, 0, synth.TAG_QDEC),
                           out=torch.empty((ns, hq, d), dtype=torch.bfloat16, device=dev)))
    torch.cuda.synchronize()
    cu1, start, lens_dev = i32(np.arange(ns + 1)), i32(ctx), i32(final)

    def run(kinds):
        for L in layers:
            if L["kind"] in kinds:
                hswa.kv_append(L["layer"], shape, L["kv"].cache, L["k_new"], L["v_new"], cu1, start)
                hswa.decode(L["layer"], shape, L["kv"].cache, L["q"], lens_dev, maxc, L["out"], workspace=ws)

    def timed(fn, n):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(n):
            fn()
        b.record()
        b.synchronize()
        return a.elapsed_time(b) / n

    step_ms = timed(lambda: run(("full", "swa")), steps)
    full_ms = timed(lambda: run(("full",)), steps)
    swa_ms = timed(lambda: run(("swa",)), steps)
    graph_ms = None
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run(("full", "swa"))
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        run(("full", "swa"))
    graph_ms = timed(g.replay, steps)
    row, qo = hkv * d * 2 * 2, 2 * ns * hq * d * 2
    nfull = sum(1 for L in layers if L["kind"] == "full")
    nswa = len(layers) - nfull
    full_bytes = nfull * (int(np.sum(ctx + 1)) * row + qo)
    swa_bytes = nswa * (int(np.sum(np.minimum(W, ctx + 1))) * row + qo)
    page_b = hswa.page_bytes(shape)
    rep = {
        "workload": wl.name, "layers": len(layers), "full_layers": nfull, "swa_layers": nswa,
        "step_ms": round(step_ms, 4), "graph_step_ms": round(graph_ms, 4),
        "step_gbs": round((full_bytes + swa_bytes) / (step_ms * 1e-3) / 1e9, 1),
        "graph_step_gbs": round((full_bytes + swa_bytes) / (graph_ms * 1e-3) / 1e9, 1),
        "frac_hbm": round((full_bytes + swa_bytes) / (min(step_ms, graph_ms) * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "full_layers_ms": round(full_ms, 4), "full_gbs": round(full_bytes / (full_ms * 1e-3) / 1e9, 1),
        "swa_layers_ms": round(swa_ms, 4), "swa_gbs": round(swa_bytes / (swa_ms * 1e-3) / 1e9, 1),
        "algorithmic_bytes": full_bytes + swa_bytes,
        "pool_bytes_per_full_layer": 2 * pages_for(hswa.Layer.full(), pg, final) * page_b,
        "pool_bytes_per_swa_layer": 2 * pages_for(hswa.Layer.swa(W), pg, final) * page_b,
    }
    del layers, ws, g
    torch.cuda.empty_cache()
    return rep


def mixed_report(reps=10, warmup=3):
    """Mixed prefill + decode step of one SWA and one FULL layer: 8 chunks of
    4096 tokens over cached prefixes uniform in [0, 65536], plus 256 decodes with
    log-normal contexts. Per layer the step runs the chunks' prefill and append,
    then the decodes' append and decode. Reports each call's rate and the step
    time against the sum of the calls' rooflines."""
    import torch

    import synth
    from paper_2607_13095_amd import hswa
    from paper_2607_13095_amd.kvcache import LayerKV, pages_for

    wl = synth.mixed_step()
    dev = "cuda"
    hq, hkv, d, pg, W = wl.hq, wl.hkv, wl.head_dim, wl.page_size, wl.window
    pre = np.asarray(wl.prefix, dtype=np.int64)
    new = np.asarray(wl.new, dtype=np.int64)
    is_dec = np.asarray(wl.decode_mask, dtype=bool)
    npf = int((~is_dec).sum())
    final = (pre + new).tolist()
    shape = hswa.Shape(hq, hkv, d, pg)
    i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32), device=dev)  # noqa: E731
    ring = hswa.ring_pages(W, pg)
    Tp = int(new[:npf].sum())
    ndec = int(is_dec.sum())
    dec_lens = (pre[npf:] + 1)
    maxd = int(dec_lens.max())
    ws = torch.empty(max(1, hswa.decode_workspace_bytes(shape, ndec, maxd)), dtype=torch.uint8, device=dev)
    layers = []
    for li, kind in enumerate(wl.layers):
        layer = hswa.Layer.swa(W) if kind == "swa" else hswa.Layer.full()
        kv = LayerKV(layer, shape, final, perm=synth.page_permutation(pages_for(layer, pg, final), wl.seed, li))
        first = np.zeros(len(pre), dtype=np.int64) if kind == "full" else np.maximum(0, pre - ring * pg)
        for b0 in range(0, len(pre), 32):
            sl = slice(b0, min(len(pre), b0 + 32))
            lens = pre[sl] - first[sl]
            T = int(lens.sum())
            if T == 0:
                continue
            kh = synth.torch_normal_bf16((T, hkv, d), dev, wl.seed, li, b0, synth.TAG_K)
            vh = synth.torch_normal_bf16((T, hkv, d), dev, wl.seed, li, b0, synth.TAG_V)
            sub = hswa.Cache(kv.k_pool, kv.v_pool, kv.block_table[sl])
            hswa.kv_append(layer, shape, sub, kh, vh, i32(synth.cu_seqlens(lens)), i32(first[sl]))
            del kh, vh
        layers.append(dict(
            kind=kind, layer=layer, kv=kv,
            cp=hswa.Cache(kv.k_pool, kv.v_pool, kv.block_table[:npf]),
            cd=hswa.Cache(kv.k_pool, kv.v_pool, kv.block_table[npf:]),
            qp=synth.torch_normal_bf16((Tp, hq, d), dev, wl.seed, li, 1, synth.TAG_Q),
            kp=synth.torch_normal_bf16((Tp, hkv, d), dev, wl.seed, li, 1, synth.TAG_K),
            vp=synth.torch_normal_bf16((Tp, hkv, d), dev, wl.seed, li, 1, synth.TAG_V),
            op=torch.empty((Tp, hq, d), dtype=torch.bfloat16, device=dev),
            qd=synth.torch_normal_bf16((ndec, hq, d), dev, wl.seed, li, 2, synth.TAG_QDEC),
            kd=synth.torch_normal_bf16((ndec, hkv, d), dev, wl.seed, li, 2, synth.TAG_KDEC),
            vd=synth.torch_normal_bf16((ndec, hkv, d), dev, wl.seed, li, 2, synth.TAG_VDEC),
            od=torch.empty((ndec, hq, d), dtype=torch.bfloat16, device=dev)))
    torch.cuda.synchronize()
    cup, prep = i32(synth.cu_seqlens(new[:npf])), i32(pre[:npf])
    cud, startd, lensd = i32(np.arange(ndec + 1)), i32(pre[npf:]), i32(dec_lens)
    maxchunk = int(new[:npf].max())

    def prefill(L):
        hswa.prefill(L["layer"], shape, L["cp"], L["qp"], L["kp"], L["vp"], cup, prep, maxchunk, L["op"])
        hswa.kv_append(L["layer"], shape, L["cp"], L["kp"], L["vp"], cup, prep)

    def decode(L):
        hswa.kv_append(L["layer"], shape, L["cd"], L["kd"], L["vd"], cud, startd)
        hswa.decode(L["layer"], shape, L["cd"], L["qd"], lensd, maxd, L["od"], workspace=ws)

    def step():
        for L in layers:
            prefill(L)
            decode(L)

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        b.synchronize()
        return a.elapsed_time(b) / reps

    by = {L["kind"]: L for L in layers}
    t = {f"{what}_{k}": timed(lambda f=f, L=L: f(L)) for k, L in by.items()
         for what, f in (("prefill", prefill), ("decode", decode))}
    step_ms = timed(step)
    row, hd = hkv * d * 2 * 2, 4 * d * hq
    flops, pbytes, dbytes = {}, {}, {}
    for k in by:
        pairs = 0
        for p_, c_ in zip(pre[:npf], new[:npf]):
            pos = np.arange(p_, p_ + c_)
            pairs += int((pos + 1).sum()) if k == "full" else int(np.minimum(W, pos + 1).sum())
        flops[k] = hd * pairs
        keys = int(np.sum(pre[:npf] + new[:npf])) if k == "full" else int(
            sum(min(int(p_), W - 1) + int(c_) for p_, c_ in zip(pre[:npf], new[:npf])))
        pbytes[k] = keys * row + 2 * Tp * hq * d * 2
        dkeys = int(np.sum(dec_lens)) if k == "full" else int(np.sum(np.minimum(W, dec_lens)))
        dbytes[k] = dkeys * row + 2 * ndec * hq * d * 2
    roof = sum(max(flops[k] / (MFMA_BF16_PEAK_TFLOPS * 1e12), pbytes[k] / (HBM_PEAK_GBS * 1e9)) +
               dbytes[k] / (HBM_PEAK_GBS * 1e9) for k in by) * 1e3
    rep = {
        "workload": wl.name, "step_ms": round(step_ms, 4), "roofline_sum_ms": round(roof, 4),
        "frac_of_roofline": round(roof / step_ms, 4),
        "prefill_full_ms": round(t["prefill_full"], 4),
        "prefill_full_tflops": round(flops["full"] / (t["prefill_full"] * 1e-3) / 1e12, 1),
        "prefill_swa_ms": round(t["prefill_swa"], 4),
        "decode_full_ms": round(t["decode_full"], 4),
        "decode_full_gbs": round(dbytes["full"] / (t["decode_full"] * 1e-3) / 1e9, 1),
        "decode_swa_ms": round(t["decode_swa"], 4),
        "note": "prefill and decode call times include their kv_append",
    }
    del layers, ws
    torch.cuda.empty_cache()
    return rep


def extra_reports(wl, full_avg):
    """Multi-query decode, window-safe prefix tree and explicit-release allocator reports."""
    import torch

    log("[bench] multi-query decode (1 + 3 queries per sequence)")
    mt = DecodeBench(wl, nq=4)
    for _ in range(3):
        mt.step()
    torch.cuda.synchronize()
    mt_full = mt.time_kind_back_to_back("full", 20)
    mt_swa = mt.time_kind_back_to_back("swa", 20)
    mtp = {"queries_per_seq": 4, "full_ms": round(mt_full, 5), "swa_ms": round(mt_swa, 5),
           "full_gbs": round(mt.bytes["full"] / (mt_full * 1e-3) / 1e9, 1),
           "full_ms_vs_one_query": round(mt_full / full_avg, 3)}
    log(f"[bench] multi-query decode: {mtp}")
    del mt
    torch.cuda.empty_cache()

    log("[bench] window-safe prefix tree")
    prefix_rep = prefix_tree_report()
    log(f"[bench] prefix tree: {prefix_rep}")

    log("[bench] explicit-release allocator")
    alloc_rep = allocator_report(wl)
    log(f"[bench] allocator: {alloc_rep}")

    log("[bench] 70-layer hybrid decode step (16 x 131072 context)")
    stack = stack70_report()
    log(f"[bench] stack70: {stack}")

    log("[bench] mixed prefill + decode step")
    mixed = mixed_report()
    log(f"[bench] mixed: {mixed}")

    return mtp, prefix_rep, alloc_rep, stack, mixed


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (run with --gpus 1)",
              file=sys.stderr)
        sys.exit(2)
    import torch

    import synth
    from paper_2607_13095_amd import hswa

    hswa.load()
    torch.cuda.set_device(0)
    if args.copy_calibration:
        copy_calibration()

    wl = synth.decode_b64()
    log(f"[bench] setting up {wl.name}")
    db = DecodeBench(wl)
    for _ in range(args.warmup):
        db.step()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        db.step()
    stop.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    ms_step = total_ms / args.steps
    dec_bytes = sum(db.bytes.values())
    value = dec_bytes / (ms_step * 1e-3) / 1e9
    # The roofline kernel alone: FULL-layer decode calls back to back on the
    # stream they run on, one HIP event pair around them (no host gap per call).
    full_avg = db.time_kind_back_to_back("full", max(args.steps, 10))
    full_gbs = db.bytes["full"] / (full_avg * 1e-3) / 1e9
    swa_ms = db.time_kind("swa")
    log(f"[bench] decode step {ms_step:.4f} ms; FULL decode {full_avg:.4f} ms ({full_gbs:.0f} GB/s); "
        f"SWA decode {swa_ms:.4f} ms")

    prefill = None
    if not args.no_prefill:
        pw = synth.chunked_prefill_4x8k()
        log(f"[bench] setting up {pw.name}")
        pb = PrefillBench(pw)
        f_ms = pb.time_kind("full")
        s_ms = pb.time_kind("swa")
        f_tf = pb.flops["full"] / (f_ms * 1e-3) / 1e12
        s_gbs = pb.bytes["swa"] / (s_ms * 1e-3) / 1e9
        prefill = {
            "workload": pw.name, "full_ms": round(f_ms, 4), "full_tflops": round(f_tf, 2),
            "full_frac_mfma": round(f_tf / MFMA_BF16_PEAK_TFLOPS, 4),
            "swa_ms": round(s_ms, 4), "swa_gbs": round(s_gbs, 1), "swa_frac_hbm": round(s_gbs / HBM_PEAK_GBS, 4),
            "swa_tflops": round(pb.flops["swa"] / (s_ms * 1e-3) / 1e12, 2),
            "roofline": {"bound": "mfma", "achieved": round(f_tf, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(f_tf / MFMA_BF16_PEAK_TFLOPS, 4),
                         "traffic": measured_traffic("prefill_full"), "algorithmic_bytes": pb.bytes["full"],
                         "algorithmic_flops": pb.flops["full"]},
        }
        log(f"[bench] prefill FULL {f_ms:.3f} ms = {f_tf:.1f} TFLOP/s; SWA {s_ms:.3f} ms = {s_gbs:.0f} GB/s")
        if not args.roofline_only:
            log("[bench] layerwise prefetch (70-layer prefill stack, prefix from pinned host memory)")
            prefill["prefetch"] = prefetch_report(pb)
            log(f"[bench] prefetch: {prefill['prefetch']}")
        del pb
        torch.cuda.empty_cache()

    mtp = prefix_rep = alloc_rep = stack = mixed = cpu = None
    if args.roofline_only:
        args.no_cpu_baseline = True
    else:
        mtp, prefix_rep, alloc_rep, stack, mixed = extra_reports(wl, full_avg)

    if not args.no_cpu_baseline:
        log("[bench] CPU baseline (oracle)")
        cpu = db.cpu_baseline(args.cpu_seconds)


    line = {
        "metric": "decode attn HBM GB/s (% peak) + prefill attn TFLOP/s (% MFMA), W=128",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "sequences": wl.ns, "context": "uniform [1024, 32768] cached tokens",
                   "layers": "1 SWA (W=128) + 1 FULL", "q_heads": wl.hq, "kv_heads": wl.hkv,
                   "head_dim": wl.head_dim, "page_size": wl.page_size, "frac_hbm": round(value / HBM_PEAK_GBS, 4),
                   "decode_bytes": dec_bytes, "full_decode_ms": round(full_avg, 5),
                   "swa_decode_ms": round(swa_ms, 5)},
        "roofline": {"bound": "hbm", "achieved": round(full_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(full_gbs / HBM_PEAK_GBS, 4), "traffic": measured_traffic("decode_full"),
                     "algorithmic_bytes": db.bytes["full"],
                     "kernel": "FULL-layer decode call: decode_kernel<true,true> + decode_merge_kernel"},
        "prefill": prefill,
        "multi_query_decode": mtp,
        "allocator": alloc_rep,
        "prefix_tree": prefix_rep,
        "stack70_decode": stack,
        "mixed_step": mixed,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
