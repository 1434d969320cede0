"""Benchmark of the hybrid-SWA paged attention hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--no-prefill]
                    [--roofline-only] [--prefill-only] [--copy-calibration]

Headline workload (the largest configuration that fits one GPU): a 70-layer
hybrid decode step, 60 SWA layers (W = 128) and 10 FULL layers (FULL iff
layer % 7 == 6), 16 sequences at a 131072-token cached context, 64 query / 8 KV
heads, head dim 128, bf16, page size 64, pages placed by a seeded permutation.
One step stores one new token per sequence in every layer and decodes it
(hswa_decode_append: one launch for an SWA layer, the append kernel then the
split decode for a FULL layer). Every layer's pools hold their own synthetic KV
(86 GB of FULL pages, 12 MiB per SWA layer), resident in HBM before the timed
region. value = algorithmic decode bytes of the step (K and V of every visible
key read once per (sequence, KV head, layer), plus q and o) / step time.

The roofline entry is the FULL-layer decode call of that step (split-KV kernel
+ log-sum-exp merge), timed back to back with HIP events on the stream it runs
on. Per-call timings elsewhere are medians with p10 / p90 over calls each
preceded (outside the events) by a 1 GiB device write that evicts the
memory-side cache.

Also measured in the same run: the 64-sequence decode (contexts 1K-32K), the
512-token SWA prefill (8 / 1 heads, page size 16), chunked prefill (4 x (8192
cached + 2048 new), timed calls are hswa_prefill alone), layerwise prefetch,
multi-query decode, the explicit-release allocator, the window-safe prefix
tree and the mixed prefill + decode step. The CPU baselines time the fp64
oracle on bounded samples of the same workloads on the host's cores.
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
FLUSH_BYTES = 1 << 30  # a write this large evicts the 256 MB memory-side cache

# Bytes moved between L2 and memory per call, from rocprofv3 --pmc FETCH_SIZE and
# --pmc WRITE_SIZE runs of this script with --roofline-only --copy-calibration,
# each counter scaled by what it reads for the plain 1 GiB copy (FETCH_SIZE
# reads 524,300 KiB for 1 GiB read: x2.0; WRITE_SIZE reads 1,048,576 KiB for
# 1 GiB written: x1.0). A figure holds only for the kernel sources it was taken
# on (SHA-256 below); once they change the benchmark reports null until it is
# measured again.
MEASURED_TRAFFIC = {
    "decode_full_stack70": {"sources": ["decode.hip", "hswa_common.h", "hswa_launch.h"],
                            "sha256": "33e861862964a2599c57b8f8b62732bb38b9230475ce145bad52e97f5f5aaef7",
                            "fetch_bytes": 8609499338, "write_bytes": 5574682},
    "prefill_full": {"sources": ["prefill.hip", "hswa_common.h", "hswa_launch.h"],
                     "sha256": "09c415c25425ca9092c56d08c06cfb6cdf7ea89fd23249c800f47ff74d31818f",
                     "fetch_bytes": 453240070, "write_bytes": 141568870},
    "prefill_swa": {"sources": ["prefill_run.hip", "hswa_common.h", "hswa_launch.h"],
                    "sha256": "1ab52ecfb56b32547d74b3a6bf166c7dc311a3e9828d48afb8205e14c9a02211",
                    "fetch_bytes": 184794072, "write_bytes": 149292872},
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
    if not t["sha256"] or sources_sha256(t["sources"]) != t["sha256"]:
        return None
    return int(t["fetch_bytes"] + t["write_bytes"])


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--roofline-only", action="store_true",
                    help="only the headline step and the prefill calls the roofline entries time (for counter runs)")
    ap.add_argument("--prefill-only", action="store_true",
                    help="only the chunked-prefill calls (FULL and SWA, timed back to back) and their power and "
                         "clock telemetry; prints a JSON line with that entry alone (for counter runs)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target oracle time of the headline CPU baseline")
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
# timing helpers
# ----------------------------------------------------------------------------

class MallFlush:
    """Writes FLUSH_BYTES of device memory (a fill kernel) so that the next
    call starts with nothing of its inputs in the memory-side cache."""

    def __init__(self):
        import torch

        self.buf = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")
        self.k = 0

    def __call__(self):
        self.k += 1
        self.buf.fill_(float(self.k))


def time_calls(fn, flush, reps=20, warmup=3):
    """Per-call event timing: median, p10 and p90 (ms) over `reps` calls, each
    preceded by a memory-side cache flush outside the events."""
    import torch

    for _ in range(warmup):
        fn()
    ts = []
    for _ in range(reps):
        flush()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        b.synchronize()
        ts.append(a.elapsed_time(b))
    ts = np.asarray(ts)
    return {"ms_median": round(float(np.median(ts)), 5), "ms_p10": round(float(np.percentile(ts, 10)), 5),
            "ms_p90": round(float(np.percentile(ts, 90)), 5), "reps": reps, "mall_flushed": True}


def power_telemetry(fn, seconds=1.2):
    """Socket power and reported gfx clock while `fn` runs back to back for
    about `seconds` (amdsmi, polled every 5 ms from a host thread; the SMU's
    metrics table lags by a few hundred ms, so only the second half of the
    window counts). None where amdsmi is not usable."""
    import threading

    import torch

    try:
        import amdsmi

        amdsmi.amdsmi_init()
    except Exception as e:  # no SMU access on this host
        log(f"[bench] power telemetry unavailable: {e!r}")
        return None
    try:
        h = amdsmi.amdsmi_get_processor_handles()[0]
        cap_w = amdsmi.amdsmi_get_power_cap_info(h)["power_cap"] / 1e6
        samples, stop = [], threading.Event()

        def poll():
            while not stop.is_set():
                m = amdsmi.amdsmi_get_gpu_metrics_info(h)
                samples.append((time.perf_counter(), float(np.mean(m["current_gfxclks"])),
                                float(m["current_socket_power"])))
                time.sleep(0.005)

        th = threading.Thread(target=poll)
        th.start()
        t0 = time.perf_counter()
        calls = 0
        while time.perf_counter() - t0 < seconds:
            for _ in range(20):
                fn()
            calls += 20
            torch.cuda.synchronize()
        t1 = time.perf_counter()
        stop.set()
        th.join()
        s = np.asarray([x for x in samples if (t0 + t1) / 2 <= x[0] <= t1])
        if len(s) == 0:
            return None
        return {"socket_power_w": round(float(s[:, 2].mean()), 1), "power_cap_w": round(cap_w, 1),
                "gfxclk_mhz_reported": round(float(s[:, 1].mean()), 1), "samples": int(len(s)), "calls": calls,
                "note": "amdsmi metrics over the second half of ~1 s of back-to-back calls (the SMU's reported "
                        "clock; rocprofv3's GRBM_GUI_ACTIVE per XCD over the kernel time gives the effective one)"}
    except Exception as e:
        log(f"[bench] power telemetry failed: {e!r}")
        return None
    finally:
        amdsmi.amdsmi_shut_down()


def time_back_to_back(fn, reps, warmup=2):
    """Mean time (ms) of `reps` calls issued back to back between one pair of
    HIP events on the current stream (no host gap per call)."""
    import torch

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


def rate(nbytes=None, flops=None, ms=None):
    out = {}
    if nbytes is not None:
        gbs = nbytes / (ms * 1e-3) / 1e9
        out.update(gbs=round(gbs, 1), frac_hbm=round(gbs / HBM_PEAK_GBS, 4))
    if flops is not None:
        tf = flops / (ms * 1e-3) / 1e12
        out.update(tflops=round(tf, 2), frac_mfma=round(tf / MFMA_BF16_PEAK_TFLOPS, 4))
    if nbytes is not None and flops is not None:
        # the binding roofline: the larger of the two floors, over the time
        floor_ms = max(flops / (MFMA_BF16_PEAK_TFLOPS * 1e12), nbytes / (HBM_PEAK_GBS * 1e9)) * 1e3
        out.update(frac_binding=round(floor_ms / ms, 4))
    return out


# ----------------------------------------------------------------------------
# CPU description
# ----------------------------------------------------------------------------

def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _blas_info():
    try:
        from threadpoolctl import threadpool_info

        return [{"library": i.get("internal_api"), "version": i.get("version"), "threads": i.get("num_threads")}
                for i in threadpool_info() if i.get("user_api") == "blas"]
    except Exception:
        return []


def _blas_threads():
    info = _blas_info()
    return int(max((i["threads"] or 1 for i in info), default=1))


def _host_cores():
    return len(os.sched_getaffinity(0))


def _host_f64(t):
    import torch

    from oracle import attention as OA

    return OA.bf16_bits_to_f64(t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16))


# ----------------------------------------------------------------------------
# headline: the 70-layer hybrid decode step
# ----------------------------------------------------------------------------

class Stack70Bench:
    """The 70-layer hybrid decode step (10 FULL + 60 SWA layers, 16 sequences
    at a 131072-token context): every layer's pools hold their own synthetic KV
    and one step appends the new token and decodes it in every layer."""

    def __init__(self):
        import torch

        import synth
        from paper_2607_13095_amd import hswa
        from paper_2607_13095_amd.kvcache import LayerKV, pages_for

        self.wl = wl = synth.stack70_decode()
        dev = "cuda"
        hq, hkv, d, pg, W = wl.hq, wl.hkv, wl.head_dim, wl.page_size, wl.window
        ns = wl.ns
        self.ctx = ctx = np.asarray(wl.prefix, dtype=np.int64)
        final = (ctx + 1).tolist()
        self.maxc = int(max(final))
        self.shape = shape = hswa.Shape(hq, hkv, d, pg)
        i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32), device=dev)  # noqa: E731
        self.ring = ring = hswa.ring_pages(W, pg)
        self.ws = torch.empty(max(1, hswa.decode_workspace_bytes(shape, ns, self.maxc)), dtype=torch.uint8,
                              device=dev)
        self.layers = []
        for li, kind in enumerate(wl.layers):
            layer = hswa.Layer.swa(W) if kind == "swa" else hswa.Layer.full()
            kv = LayerKV(layer, shape, final, perm=synth.page_permutation(pages_for(layer, pg, final), wl.seed, li))
            # cached history: every position for FULL (four sequences at a time),
            # the positions the ring keeps for SWA
            first = self.first_cached(kind)
            for b0 in range(0, ns, 4):
                sl = slice(b0, min(ns, b0 + 4))
                kh, vh, lens = self.history(li, kind, b0)
                sub = hswa.Cache(kv.k_pool, kv.v_pool, kv.block_table[sl])
                hswa.kv_append(layer, shape, sub, kh, vh, i32(synth.cu_seqlens(lens)), i32(first[sl]))
                del kh, vh
            self.layers.append(dict(
                li=li, kind=kind, layer=layer, kv=kv,
                k_new=synth.torch_normal_bf16((ns, hkv, d), dev, wl.seed, li, 0, synth.TAG_KDEC),
                v_new=synth.torch_normal_bf16((ns, hkv, d), dev, wl.seed, li, 0, synth.TAG_VDEC),
                q=synth.torch_normal_bf16((ns, hq, d), dev, wl.seed, li, 0, synth.TAG_QDEC),
                out=torch.empty((ns, hq, d), dtype=torch.bfloat16, device=dev)))
        torch.cuda.synchronize()
        self.cu1, self.start, self.lens = i32(np.arange(ns + 1)), i32(ctx), i32(final)
        row, qo = hkv * d * 2 * 2, 2 * ns * hq * d * 2
        self.nfull = sum(1 for L in self.layers if L["kind"] == "full")
        self.nswa = len(self.layers) - self.nfull
        self.full_layer_bytes = int(np.sum(ctx + 1)) * row + qo
        self.swa_layer_bytes = int(np.sum(np.minimum(W, ctx + 1))) * row + qo
        self.bytes = self.nfull * self.full_layer_bytes + self.nswa * self.swa_layer_bytes
        page_b = hswa.page_bytes(shape)
        self.pool_bytes = {"full_layer": 2 * pages_for(hswa.Layer.full(), pg, final) * page_b,
                           "swa_layer": 2 * pages_for(hswa.Layer.swa(W), pg, final) * page_b}

    def first_cached(self, kind):
        if kind == "full":
            return np.zeros(self.wl.ns, dtype=np.int64)
        return np.maximum(0, self.ctx - self.ring * self.wl.page_size)

    def history(self, li, kind, b0):
        """The seeded cached K / V of sequences b0 .. b0+3 of layer li (device)."""
        import synth

        wl = self.wl
        first = self.first_cached(kind)
        sl = slice(b0, min(wl.ns, b0 + 4))
        lens = self.ctx[sl] - first[sl]
        T = int(lens.sum())
        kh = synth.torch_normal_bf16((T, wl.hkv, wl.head_dim), "cuda", wl.seed, li, b0, synth.TAG_K)
        vh = synth.torch_normal_bf16((T, wl.hkv, wl.head_dim), "cuda", wl.seed, li, b0, synth.TAG_V)
        return kh, vh, lens

    def append(self, L):
        from paper_2607_13095_amd import hswa

        hswa.kv_append(L["layer"], self.shape, L["kv"].cache, L["k_new"], L["v_new"], self.cu1, self.start)

    def decode(self, L):
        from paper_2607_13095_amd import hswa

        hswa.decode(L["layer"], self.shape, L["kv"].cache, L["q"], self.lens, self.maxc, L["out"], workspace=self.ws)

    def step_layer(self, L):
        """One layer's step: store the new token and decode it (one call)."""
        from paper_2607_13095_amd import hswa

        hswa.decode_append(L["layer"], self.shape, L["kv"].cache, L["q"], L["k_new"], L["v_new"], self.lens,
                           self.maxc, L["out"], workspace=self.ws)

    def run(self, kinds=("full", "swa")):
        for L in self.layers:
            if L["kind"] in kinds:
                self.step_layer(L)

    def graph(self, kinds):
        """The step (or one kind's layers) captured as one HIP graph."""
        import torch

        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self.run(kinds)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            self.run(kinds)
        return g

    def cpu_baseline(self, target_s):
        """fp64 oracle on the host cores over a sample of the step: every
        sequence of SWA layer 0, then the sequences of the FULL layers in order
        until about target_s seconds of oracle time. Inputs are regenerated on
        the GPU from their seeds and copied to the host (untimed)."""
        from oracle import attention as OA

        wl = self.wl
        W = wl.window
        done_bytes, t_total, pairs = 0, 0.0, []
        row, qo = wl.hkv * wl.head_dim * 2 * 2, 2 * wl.hq * wl.head_dim * 2
        order = [L for L in self.layers if L["kind"] == "swa"][:1] + [L for L in self.layers if L["kind"] == "full"]
        for L in order:
            window = W if L["kind"] == "swa" else None
            first = self.first_cached(L["kind"])
            for b0 in range(0, wl.ns, 4):
                kh, vh, lens = self.history(L["li"], L["kind"], b0)
                cu = np.concatenate([[0], np.cumsum(lens)])
                for i in range(len(lens)):
                    b = b0 + i
                    c = int(self.ctx[b])
                    lo = 0 if window is None else max(0, c + 1 - window) - int(first[b])
                    k = np.concatenate([_host_f64(kh[int(cu[i]) + lo:int(cu[i + 1])]), _host_f64(L["k_new"][b:b + 1])])
                    v = np.concatenate([_host_f64(vh[int(cu[i]) + lo:int(cu[i + 1])]), _host_f64(L["v_new"][b:b + 1])])
                    q = _host_f64(L["q"][b])
                    t0 = time.perf_counter()
                    OA.decode(q, k, v, window, self.shape.scale)
                    t_total += time.perf_counter() - t0
                    done_bytes += k.shape[0] * row + qo
                    pairs.append((L["li"], b))
                    del k, v
                    if L["kind"] == "full" and t_total >= target_s:
                        break
                del kh, vh
                if L["kind"] == "full" and t_total >= target_s:
                    break
            if t_total >= target_s:
                break
        nfull = sum(1 for li, _ in pairs if self.layers[li]["kind"] == "full")
        return {"value": round(done_bytes / t_total / 1e9, 4), "unit": "GB/s", "cores": _blas_threads(),
                "kind": "oracle", "cpu_model": _cpu_model(), "host_cores": _host_cores(), "blas": _blas_info(),
                "sample": f"stack70 decode: the 16 sequences of SWA layer 0 and {nfull} (FULL layer, sequence) "
                          f"decodes at a 131073-token context, each an fp64 numpy oracle call over the "
                          f"sequence's contiguous history (inputs regenerated from their seeds, untimed); "
                          f"{t_total:.1f} s of oracle time, {done_bytes / 1e9:.2f} GB of algorithmic bytes"}


# ----------------------------------------------------------------------------
# decode_b64 (64 sequences, contexts uniform in [1024, 32768])
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
            if self.nq == 1:  # store the new token and decode it in one call
                hswa.decode_append(L["layer"], self.shape, L["kv"].cache, L["q"], L["k_new"], L["v_new"],
                                   self.ctx_lens, self.maxc, L["out"], workspace=L["ws"])
            else:
                hswa.kv_append(L["layer"], self.shape, L["kv"].cache, L["k_new"], L["v_new"], self.cu1, self.start)
                self.decode(L)

    def decode(self, L):
        from paper_2607_13095_amd import hswa

        fn = hswa.decode if self.nq == 1 else hswa.decode_multi
        fn(L["layer"], self.shape, L["kv"].cache, L["q"], self.ctx_lens, self.maxc, L["out"], workspace=L["ws"])

    def kind(self, kind):
        return next(x for x in self.layers if x["kind"] == kind)

    def cpu_baseline(self, target_s):
        """fp64 oracle over the sequences (both layers), in order, until about
        target_s seconds of oracle time."""
        from oracle import attention as OA

        done_bytes, t_total, nseq = 0, 0.0, 0
        row = self.wl.hkv * self.wl.head_dim * 2 * 2
        qo = 2 * self.wl.hq * self.wl.head_dim * 2
        W = self.wl.window
        for b in range(self.wl.ns):
            for L in self.layers:
                c = int(self.ctx[b])
                lo = int(L["cu"][b])
                window = W if L["kind"] == "swa" else None
                first = 0 if window is None else max(0, c + 1 - window)
                k = np.concatenate([_host_f64(L["k_hist"][lo + first:lo + c]), _host_f64(L["k_new"][b:b + 1])])
                v = np.concatenate([_host_f64(L["v_hist"][lo + first:lo + c]), _host_f64(L["v_new"][b:b + 1])])
                q = _host_f64(L["q"][b])
                t0 = time.perf_counter()
                OA.decode(q, k, v, window, self.shape.scale)
                t_total += time.perf_counter() - t0
                done_bytes += k.shape[0] * row + qo
            nseq += 1
            if t_total >= target_s:
                break
        return {"value": round(done_bytes / t_total / 1e9, 4), "unit": "GB/s", "cores": _blas_threads(),
                "kind": "oracle", "sample": f"first {nseq} of {self.wl.ns} sequences, both layers, one fp64 "
                                            f"oracle call each, {t_total:.1f} s of oracle time"}


# ----------------------------------------------------------------------------
# chunked prefill (4 x (8192 cached + 2048 new))
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
            self.layers.append(dict(li=li, kind=kind, layer=layer, kv=kv, q=q, kn=kn, vn=vn, out=out))
        torch.cuda.synchronize()
        self.flops, self.bytes = {}, {}
        for L in self.layers:
            self.flops[L["kind"]] = 4 * d * hq * self.pairs(L["kind"])
            keys = int((P + C).sum()) if L["kind"] == "full" else int(
                sum(min(int(p), W - 1) + int(c) for p, c in zip(P, C)))
            self.bytes[L["kind"]] = keys * hkv * d * 4 + 2 * T * hq * d * 2

    def pairs(self, kind, rows=None):
        """Allowed (query, key) pairs of a layer kind; `rows` restricts each
        sequence to the chunk rows it lists."""
        W = self.wl.window
        total = 0
        for p, c in zip(self.P, self.C):
            pos = p + (np.arange(c) if rows is None else np.asarray(rows))
            total += int((pos + 1).sum()) if kind == "full" else int(np.minimum(W, pos + 1).sum())
        return total

    def call(self, L):
        from paper_2607_13095_amd import hswa

        hswa.prefill(L["layer"], self.shape, L["kv"].cache, L["q"], L["kn"], L["vn"], self.cu, self.pre, self.maxc,
                     L["out"])

    def kind(self, kind):
        return next(x for x in self.layers if x["kind"] == kind)

    def cpu_baseline(self, full_rows=512, workers=None):
        """fp64 oracle rates on the host cores, one task per (sequence, KV head)
        (the oracle over that KV head's query heads), the tasks spread over a
        thread pool of `workers` with one BLAS thread each. SWA: the whole layer
        (each task sees the suffix of the history that holds its windows).
        FULL: the last `full_rows` rows of every chunk (the longest ones) of
        half of the tasks, then extrapolated by algorithmic flops."""
        from concurrent.futures import ThreadPoolExecutor

        import synth
        from oracle import attention as OA
        from threadpoolctl import threadpool_limits

        wl = self.wl
        workers = workers or max(1, min(16, _host_cores()))
        G, W = wl.hq // wl.hkv, wl.window
        cuP, cuC = synth.cu_seqlens(self.P), synth.cu_seqlens(self.C)
        res = {}
        for L in self.layers:
            kind = L["kind"]
            kp = _host_f64(synth.torch_normal_bf16((int(self.P.sum()), wl.hkv, wl.head_dim), "cuda", wl.seed,
                                                   L["li"], 0, synth.TAG_K))
            vp = _host_f64(synth.torch_normal_bf16((int(self.P.sum()), wl.hkv, wl.head_dim), "cuda", wl.seed,
                                                   L["li"], 0, synth.TAG_V))
            kn, vn, q = _host_f64(L["kn"]), _host_f64(L["vn"]), _host_f64(L["q"])
            rows = None if kind == "swa" else np.arange(int(self.C.min()) - full_rows, int(self.C.min()))
            tasks = [(b, g) for b in range(wl.ns) for g in range(wl.hkv)]
            if kind == "full":
                tasks = tasks[: len(tasks) // 2]
            inputs = []
            for b, g in tasks:
                p, c = int(self.P[b]), int(self.C[b])
                kh = np.concatenate([kp[cuP[b]:cuP[b + 1], g:g + 1], kn[cuC[b]:cuC[b + 1], g:g + 1]])
                vh = np.concatenate([vp[cuP[b]:cuP[b + 1], g:g + 1], vn[cuC[b]:cuC[b + 1], g:g + 1]])
                r = np.arange(c) if rows is None else rows
                lo = 0 if kind == "full" else max(0, p + int(r[0]) - W + 1)
                inputs.append((q[cuC[b] + r, g * G:(g + 1) * G], kh[lo:], vh[lo:], p + r - lo))
            window = W if kind == "swa" else None
            with threadpool_limits(1), ThreadPoolExecutor(workers) as ex:
                t0 = time.perf_counter()
                list(ex.map(lambda a: OA.masked_attention(a[0], a[1], a[2], a[3], window, self.shape.scale), inputs))
                dt = time.perf_counter() - t0
            frac_tasks = len(tasks) / (wl.ns * wl.hkv)
            flops = 4 * wl.head_dim * wl.hq * self.pairs(kind, rows) * frac_tasks
            entry = {"gflops": round(flops / dt / 1e9, 3), "seconds": round(dt, 2), "threads": workers}
            if kind == "swa":
                entry.update(gbs=round(self.bytes["swa"] / dt / 1e9, 4), sample="whole layer (measured)")
            else:
                entry.update(extrapolated_layer_seconds=round(dt * self.flops["full"] / flops, 1),
                             sample=f"{len(tasks)} of {wl.ns * wl.hkv} (sequence, KV head) tasks, the last "
                                    f"{full_rows} rows of each chunk; whole-layer time extrapolated by flops")
            res[kind] = entry
            del kp, vp, kn, vn, q, inputs
        return {"kind": "oracle", "unit": "GFLOP/s", "cores": workers, **res}


# ----------------------------------------------------------------------------
# swa_prefill_512 (one SWA layer, no cache, 8 / 1 heads, page size 16)
def prefix_sweep_report(prefixes=(0, 16384, 65536, 262144, 1048576), chunk=16384):
    """FULL-layer prefill of one 16K-token chunk (64 / 8 heads, PG 64) over
    cached prefixes from 0 to 1M: time, TFLOP/s and tokens/s against the empty
    prefix. Context for the paper's prefill-throughput-vs-prefix figure, which
    is end to end (the rest of its model costs the same per token at any
    prefix); this is the FULL layer's attention alone, whose work grows with
    the prefix, so its tokens/s falls much further. The prefix's keys are
    synthetic values in the pages, drawn once for the longest prefix."""
    import torch

    import synth
    from paper_2607_13095_amd import hswa
    from paper_2607_13095_amd.kvcache import LayerKV, pages_for

    hq, hkv, d, pg = 64, 8, 128, 64
    shape = hswa.Shape(hq, hkv, d, pg)
    layer = hswa.Layer.full()
    final = [max(prefixes) + chunk]
    kv = LayerKV(layer, shape, final, perm=synth.page_permutation(pages_for(layer, pg, final), 17, 0))
    i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32), device="cuda")  # noqa: E731
    P = max(prefixes)
    step_keys = 1 << 18
    for s0 in range(0, P, step_keys):  # the cached keys, a quarter million at a time
        n = min(step_keys, P - s0)
        kh = synth.torch_normal_bf16((n, hkv, d), "cuda", 17, 0, s0, synth.TAG_K)
        vh = synth.torch_normal_bf16((n, hkv, d), "cuda", 17, 0, s0, synth.TAG_V)
        hswa.kv_append(layer, shape, kv.cache, kh, vh, i32([0, n]), i32([s0]))
        del kh, vh
    q = synth.torch_normal_bf16((chunk, hq, d), "cuda", 17, 1, 0, synth.TAG_Q)
    kn = synth.torch_normal_bf16((chunk, hkv, d), "cuda", 17, 1, 0, synth.TAG_K)
    vn = synth.torch_normal_bf16((chunk, hkv, d), "cuda", 17, 1, 0, synth.TAG_V)
    out = torch.empty((chunk, hq, d), dtype=torch.bfloat16, device="cuda")
    cu = i32([0, chunk])
    rows = []
    for p0 in prefixes:
        pre = i32([p0])

        def call():
            hswa.prefill(layer, shape, kv.cache, q, kn, vn, cu, pre, chunk, out)

        # ~40 calls' worth of an empty-prefix call to warm up (the clock ramp),
        # at least 2 calls; fewer timed calls for the long prefixes (0.5 s at 1M)
        reps = 20 if p0 <= 65536 else 3
        warm = max(2, min(40, (40 * 16) // (p0 // 1024 + 16)))
        ms = time_back_to_back(call, reps, warmup=warm)
        pairs = chunk * p0 + chunk * (chunk + 1) // 2
        flops = 4 * d * hq * pairs
        nbytes = (p0 + chunk) * hkv * d * 4 + 2 * chunk * hq * d * 2
        rows.append({"prefix": p0, "ms": round(ms, 4), "tokens_per_s": round(chunk / (ms * 1e-3), 1),
                     **rate(nbytes, flops, ms)})
    base = rows[0]["tokens_per_s"]
    for r in rows:
        r["tokens_per_s_vs_empty_prefix"] = round(r["tokens_per_s"] / base, 5)
    del kv, q, kn, vn, out
    torch.cuda.empty_cache()
    return {"workload": "prefill_16k_chunk_vs_prefix", "layer": "FULL, 64/8 heads, PG 64", "chunk": chunk,
            "rows": rows,
            "paper_context": "the paper's end-to-end prefill throughput at a 1M prefix is about 0.12x its "
                             "throughput near an empty prefix (other hardware, whole model)"}


# ----------------------------------------------------------------------------

def swa512_report(flush, cpu=True):
    """The 512-token SWA prefill (then its append) of one 8 / 1-head layer over
    a ring of 9 pages of 16 tokens: a few microseconds of work, so its time is
    launch latency; reported for completeness."""
    import torch

    import synth
    from paper_2607_13095_amd import hswa
    from paper_2607_13095_amd.kvcache import LayerKV, pages_for

    wl = synth.swa_prefill_512()
    C, W, pg, d = wl.new[0], wl.window, wl.page_size, wl.head_dim
    shape = hswa.Shape(wl.hq, wl.hkv, d, pg)
    layer = hswa.Layer.swa(W)
    kv = LayerKV(layer, shape, [C], perm=synth.page_permutation(pages_for(layer, pg, [C]), wl.seed, 0))
    qb = synth.normal_bf16((C, wl.hq, d), wl.seed, 0, 0, synth.TAG_Q)
    kb = synth.normal_bf16((C, wl.hkv, d), wl.seed, 0, 0, synth.TAG_K)
    vb = synth.normal_bf16((C, wl.hkv, d), wl.seed, 0, 0, synth.TAG_V)
    dev = lambda x: torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()  # noqa: E731
    q, k, v = dev(qb), dev(kb), dev(vb)
    out = torch.empty((C, wl.hq, d), dtype=torch.bfloat16, device="cuda")
    cu, pre = (torch.tensor(x, dtype=torch.int32, device="cuda") for x in ([0, C], [0]))

    def prefill():
        hswa.prefill(layer, shape, kv.cache, q, k, v, cu, pre, C, out)

    def step():
        prefill()
        hswa.kv_append(layer, shape, kv.cache, k, v, cu, pre)

    pos = np.arange(C)
    pairs = int(np.minimum(W, pos + 1).sum())
    flops = 4 * d * wl.hq * pairs
    nbytes = 2 * C * wl.hq * d * 2 + 2 * C * wl.hkv * d * 2
    t = time_calls(prefill, flush)
    b2b = time_back_to_back(prefill, 50)
    rep = {"workload": wl.name, "prefill": t, "prefill_back_to_back_ms": round(b2b, 5),
           "prefill_and_append": time_calls(step, flush), "algorithmic_flops": flops, "algorithmic_bytes": nbytes,
           **rate(nbytes, flops, b2b), "note": "microseconds of work: bound by launch latency"}
    if cpu:
        from oracle import attention as OA

        qf, kf, vf = (OA.bf16_bits_to_f64(x) for x in (qb, kb, vb))
        ts = []
        for _ in range(5):
            t0 = time.perf_counter()
            OA.prefill(qf, kf, vf, 0, W, shape.scale)
            ts.append(time.perf_counter() - t0)
        tm = float(np.median(ts))
        rep["cpu_baseline"] = {"kind": "oracle", "seconds": round(tm, 4), "gflops": round(flops / tm / 1e9, 3),
                               "gbs": round(nbytes / tm / 1e9, 4), "cores": _blas_threads(),
                               "sample": "whole workload, median of 5 oracle calls"}
    return rep


# ----------------------------------------------------------------------------
# widening reports
# ----------------------------------------------------------------------------

def allocator_report(wl, reps=20):
    """SWA layer of the decode workload over explicit-release tables from the
    dual-pool allocator (HSWA_LAYER_SWA_PAGED): pages held per sequence, host
    cost of one decode step's allocator calls, and the decode call's time."""
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
    ms = time_back_to_back(lambda: hswa.decode(layer, shape, cache, q, lens, maxc, out), reps)
    per_seq = [alloc.usage(b)[1] for b in range(ns)]
    full_used = alloc.usage(-1)[0]
    alloc.close()
    return {"layer": "SWA over explicit-release tables", "swa_paged_decode_ms": round(ms, 5),
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


def mixed_report(reps=10, warmup=3):
    """Mixed prefill + decode step of one SWA and one FULL layer: 8 chunks of
    4096 tokens over cached prefixes uniform in [0, 65536], plus 256 decodes with
    log-normal contexts. Per layer the step runs the chunks' prefill and append,
    then the decodes' append and decode. Reports each call's rate and the step
    time against the sum of the calls' rooflines (one stream) and against the
    larger of the prefill and decode rooflines (the bound if the two ran
    overlapped on two streams), and the step run that way: the prefill chain
    on the current stream, the decode chain on a second one."""
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

    # The same step with the prefill chain (every layer's prefill + append) on
    # the current stream and the decode chain on a second stream of the same
    # (default) priority: the two touch disjoint sequences, so a serving loop
    # may overlap them; the decode's memory traffic then runs beside the
    # prefill's matrix work wherever the scheduler gives it CUs.
    side = torch.cuda.Stream()

    def step_two_streams():
        main = torch.cuda.current_stream()
        side.wait_stream(main)
        with torch.cuda.stream(side):
            for L in layers:
                decode(L)
        for L in layers:
            prefill(L)
        main.wait_stream(side)

    by = {L["kind"]: L for L in layers}
    t = {f"{what}_{k}": time_back_to_back(lambda f=f, L=L: f(L), reps, warmup) for k, L in by.items()
         for what, f in (("prefill", prefill), ("decode", decode))}
    step_ms = time_back_to_back(step, reps, warmup)
    step2_ms = time_back_to_back(step_two_streams, reps, warmup)
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
    pre_roof = sum(max(flops[k] / (MFMA_BF16_PEAK_TFLOPS * 1e12), pbytes[k] / (HBM_PEAK_GBS * 1e9)) for k in by) * 1e3
    dec_roof = sum(dbytes[k] / (HBM_PEAK_GBS * 1e9) for k in by) * 1e3
    rep = {
        "workload": wl.name, "step_ms": round(step_ms, 4),
        "roofline_sum_ms": round(pre_roof + dec_roof, 4), "frac_of_roofline": round((pre_roof + dec_roof) / step_ms, 4),
        "roofline_two_stream_ms": round(max(pre_roof, dec_roof), 4),
        "frac_of_two_stream_roofline": round(max(pre_roof, dec_roof) / step_ms, 4),
        "step_two_streams_ms": round(step2_ms, 4),
        "frac_of_two_stream_roofline_overlapped": round(max(pre_roof, dec_roof) / step2_ms, 4),
        "prefill_full_ms": round(t["prefill_full"], 4),
        "prefill_full_tflops": round(flops["full"] / (t["prefill_full"] * 1e-3) / 1e12, 1),
        "prefill_swa_ms": round(t["prefill_swa"], 4),
        "decode_full_ms": round(t["decode_full"], 4),
        "decode_full_gbs": round(dbytes["full"] / (t["decode_full"] * 1e-3) / 1e9, 1),
        "decode_swa_ms": round(t["decode_swa"], 4),
        "note": "back-to-back means; prefill and decode call times include their kv_append",
    }
    del layers, ws
    torch.cuda.empty_cache()
    return rep


# ----------------------------------------------------------------------------
# main
# ----------------------------------------------------------------------------

def headline(args, flush):
    """The 70-layer step: K timed steps after W warm-ups (the contract), the
    FULL decode call's roofline, per-kind parts, graph replays."""
    import torch

    log("[bench] setting up stack70_decode (86 GB of FULL pages)")
    st = Stack70Bench()
    for _ in range(args.warmup):
        st.run()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        st.run()
    stop.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(stop) / args.steps
    value = st.bytes / (ms_step * 1e-3) / 1e9
    log(f"[bench] stack70 step {ms_step:.4f} ms = {value:.0f} GB/s")
    # the roofline kernel: one FULL layer's decode calls back to back
    Lf = next(L for L in st.layers if L["kind"] == "full")
    full_avg = time_back_to_back(lambda: st.decode(Lf), max(args.steps, 10))
    full_gbs = st.full_layer_bytes / (full_avg * 1e-3) / 1e9
    log(f"[bench] stack70 FULL decode call {full_avg:.4f} ms = {full_gbs:.0f} GB/s")
    rep = {"step_ms": round(ms_step, 5), "full_decode_call_ms": round(full_avg, 5), "full_decode_gbs": round(full_gbs, 1)}
    if not args.roofline_only:
        Ls = next(L for L in st.layers if L["kind"] == "swa")
        rep["full_decode_call"] = time_calls(lambda: st.decode(Lf), flush, reps=10)
        rep["swa_decode_call"] = time_calls(lambda: st.decode(Ls), flush)
        rep["swa_decode_call_back_to_back_ms"] = round(time_back_to_back(lambda: st.decode(Ls), 50), 5)
        rep["swa_step_call"] = time_calls(lambda: st.step_layer(Ls), flush)
        rep["swa_step_call_back_to_back_ms"] = round(time_back_to_back(lambda: st.step_layer(Ls), 50), 5)
        full_ms = time_back_to_back(lambda: st.run(("full",)), 3)
        swa_ms = time_back_to_back(lambda: st.run(("swa",)), 10)
        g_step = st.graph(("full", "swa"))
        graph_ms = time_back_to_back(g_step.replay, args.steps)
        del g_step
        g_swa = st.graph(("swa",))
        graph_swa_ms = time_back_to_back(g_swa.replay, 20)
        del g_swa
        swa_bytes = st.nswa * st.swa_layer_bytes
        rep.update({
            "graph_step_ms": round(graph_ms, 5), **{f"graph_step_{k}": v for k, v in rate(st.bytes, ms=graph_ms).items()},
            "full_layers_ms": round(full_ms, 4), **{f"full_layers_{k}": v for k, v in
                                                    rate(st.nfull * st.full_layer_bytes, ms=full_ms).items()},
            "swa_layers_ms": round(swa_ms, 4), "swa_layers_graph_ms": round(graph_swa_ms, 4),
            **{f"swa_layers_graph_{k}": v for k, v in rate(swa_bytes, ms=graph_swa_ms).items()},
        })
        log(f"[bench] stack70 parts: {rep}")
    cpu = None
    if not args.no_cpu_baseline and not args.roofline_only:
        log("[bench] CPU baseline: oracle on a sample of the 70-layer step")
        cpu = st.cpu_baseline(args.cpu_seconds)
        log(f"[bench] CPU baseline: {cpu}")
    out = dict(st=st, ms_step=ms_step, value=value, full_avg=full_avg, full_gbs=full_gbs, rep=rep, cpu=cpu)
    return out


def prefill_section(args, flush):
    """The chunked-prefill entry: FULL and SWA calls timed back to back (the
    FULL one is the MFMA roofline entry), their power and clock telemetry, and
    (outside --roofline-only / --prefill-only) the flushed per-call timings,
    the layerwise prefetch and the prefill CPU baseline."""
    import torch

    import synth

    pw = synth.chunked_prefill_4x8k()
    log(f"[bench] setting up {pw.name}")
    pb = PrefillBench(pw)
    Lf, Ls = pb.kind("full"), pb.kind("swa")
    # The clock settles over the first ~20 FULL calls (~50 ms of matrix-core
    # load): time the calls after 40 untimed ones (the SWA call after 200).
    f_ms = time_back_to_back(lambda: pb.call(Lf), 20, warmup=40)
    s_ms = time_back_to_back(lambda: pb.call(Ls), 20, warmup=200)
    f_tf = pb.flops["full"] / (f_ms * 1e-3) / 1e12
    prefill = {
        "workload": pw.name, "full_ms": round(f_ms, 4), **{f"full_{k}": v for k, v in
                                                          rate(pb.bytes["full"], pb.flops["full"], f_ms).items()},
        "swa_ms": round(s_ms, 4), **{f"swa_{k}": v for k, v in rate(pb.bytes["swa"], pb.flops["swa"], s_ms).items()},
        "swa_traffic": measured_traffic("prefill_swa"), "swa_algorithmic_bytes": pb.bytes["swa"],
        "roofline": {"bound": "mfma", "achieved": round(f_tf, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(f_tf / MFMA_BF16_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic("prefill_full"), "algorithmic_bytes": pb.bytes["full"],
                     "algorithmic_flops": pb.flops["full"], "kernel": "prefill_kernel (FULL layer call)"},
    }
    log(f"[bench] prefill FULL {f_ms:.3f} ms = {f_tf:.1f} TFLOP/s; SWA {s_ms:.4f} ms")
    if not args.roofline_only:
        # the power and clock this MFMA-bound call runs at differ from box to
        # box, and so does its rate
        prefill["full_power"] = power_telemetry(lambda: pb.call(Lf))
        log(f"[bench] FULL prefill power: {prefill['full_power']}")
    if not args.roofline_only and not args.prefill_only:
        prefill["full_call"] = time_calls(lambda: pb.call(Lf), flush)
        prefill["swa_call"] = time_calls(lambda: pb.call(Ls), flush)
        log("[bench] layerwise prefetch (70-layer prefill stack, prefix from pinned host memory)")
        prefill["prefetch"] = prefetch_report(pb)
        log(f"[bench] prefetch: {prefill['prefetch']}")
        if not args.no_cpu_baseline:
            log("[bench] prefill CPU baseline")
            prefill["cpu_baseline"] = pb.cpu_baseline()
            log(f"[bench] prefill CPU baseline: {prefill['cpu_baseline']}")
    del pb
    torch.cuda.empty_cache()
    return prefill


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
    flush = MallFlush()

    if args.prefill_only:
        prefill = prefill_section(args, flush)
        print(json.dumps({"metric": "prefill attn TFLOP/s (% MFMA), W=128", "value": prefill["roofline"]["achieved"],
                          "unit": "TFLOP/s", "n_gpus": 1, "higher_is_better": True, "dtype": "bf16",
                          "data": "synthetic", "config": {"workload": prefill["workload"]}, "prefill": prefill}),
              flush=True)
        return

    h = headline(args, flush)
    st = h["st"]
    wl = st.wl
    stack = {"workload": wl.name, "layers": len(st.layers), "full_layers": st.nfull, "swa_layers": st.nswa,
             "algorithmic_bytes": st.bytes, "pool_bytes_per_full_layer": st.pool_bytes["full_layer"],
             "pool_bytes_per_swa_layer": st.pool_bytes["swa_layer"], **h["rep"]}
    full_layer_bytes = st.full_layer_bytes
    del h["st"], st
    torch.cuda.empty_cache()

    decode_b64 = None
    if not args.roofline_only:
        dw = synth.decode_b64()
        log(f"[bench] setting up {dw.name}")
        db = DecodeBench(dw)
        d_step = time_back_to_back(db.step, 20, warmup=5)
        d_full = time_back_to_back(lambda: db.decode(db.kind("full")), 20)
        decode_b64 = {
            "workload": dw.name, "step_ms": round(d_step, 5),
            **{f"step_{k}": v for k, v in rate(sum(db.bytes.values()), ms=d_step).items()},
            "full_decode_ms": round(d_full, 5), **{f"full_{k}": v for k, v in rate(db.bytes["full"], ms=d_full).items()},
            "full_decode_call": time_calls(lambda: db.decode(db.kind("full")), flush),
            "swa_decode_call": time_calls(lambda: db.decode(db.kind("swa")), flush),
            "swa_decode_back_to_back_ms": round(time_back_to_back(lambda: db.decode(db.kind("swa")), 50), 5),
            "decode_bytes": db.bytes,
        }
        if not args.no_cpu_baseline:
            decode_b64["cpu_baseline"] = db.cpu_baseline(5.0)
        log(f"[bench] decode_b64: {decode_b64}")
        mtp_wl = dw
        del db
        torch.cuda.empty_cache()

    swa512 = None
    if not args.roofline_only:
        log("[bench] swa_prefill_512")
        swa512 = swa512_report(flush, cpu=not args.no_cpu_baseline)
        log(f"[bench] swa_prefill_512: {swa512}")

    prefill = None if args.no_prefill else prefill_section(args, flush)
    prefix_sweep = None
    if not args.no_prefill and not args.roofline_only:
        log("[bench] FULL prefill of a 16K chunk over prefixes 0 .. 1M")
        prefix_sweep = prefix_sweep_report()
        log(f"[bench] prefix sweep: {[(r['prefix'], r['ms'], r.get('frac_mfma')) for r in prefix_sweep['rows']]}")

    mtp = prefix_rep = alloc_rep = mixed = None
    if not args.roofline_only:
        log("[bench] multi-query decode (1 + 3 queries per sequence)")
        mt = DecodeBench(mtp_wl, nq=4)
        mt_full = time_back_to_back(lambda: mt.decode(mt.kind("full")), 20, warmup=3)
        mt_swa = time_back_to_back(lambda: mt.decode(mt.kind("swa")), 20, warmup=3)
        mtp = {"queries_per_seq": 4, "full_ms": round(mt_full, 5), "swa_ms": round(mt_swa, 5),
               "full_gbs": round(mt.bytes["full"] / (mt_full * 1e-3) / 1e9, 1),
               "full_ms_vs_one_query": round(mt_full / decode_b64["full_decode_ms"], 3)}
        log(f"[bench] multi-query decode: {mtp}")
        del mt
        torch.cuda.empty_cache()
        log("[bench] window-safe prefix tree")
        prefix_rep = prefix_tree_report()
        log("[bench] explicit-release allocator")
        alloc_rep = allocator_report(mtp_wl)
        log("[bench] mixed prefill + decode step")
        mixed = mixed_report()
        log(f"[bench] mixed: {mixed}")

    ms_step, value = h["ms_step"], h["value"]
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
        "config": {"workload": wl.name, "sequences": wl.ns, "context": "131072 cached tokens",
                   "layers": "70: 60 SWA (W=128) + 10 FULL (FULL iff layer % 7 == 6)", "q_heads": wl.hq,
                   "kv_heads": wl.hkv, "head_dim": wl.head_dim, "page_size": wl.page_size,
                   "frac_hbm": round(value / HBM_PEAK_GBS, 4), "decode_bytes": stack["algorithmic_bytes"]},
        "roofline": {"bound": "hbm", "achieved": round(h["full_gbs"], 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(h["full_gbs"] / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic("decode_full_stack70"), "algorithmic_bytes": full_layer_bytes,
                     "kernel": "FULL-layer decode call of the 70-layer step: decode_kernel<true,true,1> + "
                               "decode_merge_kernel"},
        "stack70_decode": stack,
        "decode_b64": decode_b64,
        "swa_prefill_512": swa512,
        "prefill": prefill,
        "prefill_vs_prefix": prefix_sweep,
        "multi_query_decode": mtp,
        "allocator": alloc_rep,
        "prefix_tree": prefix_rep,
        "mixed_step": mixed,
        "cpu_baseline": h["cpu"],
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
