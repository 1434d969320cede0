"""GPU parity of hswa_prefill against the fp64 oracle: chunks over cached
prefixes of many lengths (aligned and not), FULL and SWA windows from 1 to
beyond the context, GQA groups 1 to 64, page sizes 16 and 64, several
sequences of mixed lengths in one call."""

import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from paper_2607_13095_amd import hswa
from tests.hswa_testlib import (SeqHistory, append_history, assert_close, i32, make_layer, to_dev, to_f64)

pytestmark = pytest.mark.gpu


def run_prefill(kind, window, pg, hq, hkv, prefixes, chunks, seed, fill=float("nan"), perm_seed=None,
                max_chunk=None, scale=None):
    ns = len(prefixes)
    final = [p + c for p, c in zip(prefixes, chunks)]
    shape = hswa.Shape(hq, hkv, 128, pg, scale=scale)
    layer, kv = make_layer(kind, window, shape, final, perm_seed or seed, fill=fill)
    hist = SeqHistory(final, hkv, 128, *seed)
    append_history(layer, shape, kv, hist, [0] * ns, prefixes)
    T = sum(chunks)
    qbits = synth.normal_bf16((T, hq, 128), *seed, synth.TAG_Q)
    kn = np.concatenate([hist.k[b][p:p + c] for b, (p, c) in enumerate(zip(prefixes, chunks))])
    vn = np.concatenate([hist.v[b][p:p + c] for b, (p, c) in enumerate(zip(prefixes, chunks))])
    out = torch.full((T, hq, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
    hswa.prefill(layer, shape, kv.cache, to_dev(qbits), to_dev(kn), to_dev(vn), i32(synth.cu_seqlens(chunks)),
                 i32(prefixes), max_chunk or max(chunks), out)
    torch.cuda.synchronize()
    gpu = to_f64(out)
    qf = OA.bf16_bits_to_f64(qbits)
    w = window if kind == "swa" else None
    refs, off = [], 0
    for b, (p, c) in enumerate(zip(prefixes, chunks)):
        refs.append(OA.prefill(qf[off:off + c], OA.bf16_bits_to_f64(hist.k[b]), OA.bf16_bits_to_f64(hist.v[b]), p, w,
                               shape.scale))
        off += c
    return gpu, np.concatenate(refs), (layer, shape, kv, hist, kn, vn)


PREFIXES = [0, 1, 127, 128, 200, 64, 0]
CHUNKS = [1, 15, 16, 17, 300, 129, 256]


@pytest.mark.parametrize("pg", [16, 64])
@pytest.mark.parametrize("kind,window", [("full", 0), ("swa", 1), ("swa", 4), ("swa", 128), ("swa", 129),
                                         ("swa", 100000)])
def test_prefill_mixed_batch(gpu_lib, pg, kind, window):
    print(f"[prefill] pg={pg} kind={kind} W={window}", flush=True)
    gpu, ref, _ = run_prefill(kind, window, pg, 64, 8, PREFIXES, CHUNKS, (300, pg, window))
    assert_close(gpu, ref, f"prefill {kind} W={window} PG={pg}")


@pytest.mark.parametrize("hq,hkv", [(8, 8), (8, 1), (16, 1), (64, 1), (32, 4)])
def test_prefill_groups(gpu_lib, hq, hkv):
    print(f"[prefill-groups] hq={hq} hkv={hkv}", flush=True)
    for kind, window in (("full", 0), ("swa", 128)):
        gpu, ref, _ = run_prefill(kind, window, 16, hq, hkv, [0, 300], [200, 77], (301, hq, hkv))
        assert_close(gpu, ref, f"prefill groups {kind} hq={hq} hkv={hkv}")


@pytest.mark.parametrize("hq,hkv", [(32, 32), (64, 16)])
def test_prefill_many_kv_heads(gpu_lib, hq, hkv):
    """More KV heads than the configs' 8: chunk rows of Hkv * 256 bytes, read by
    the full-chunk-tile buffer loads at per-lane row offsets, and page-heads of
    Hkv * PG * 256 bytes for the interior tiles (PG 64); FULL, and SWA with a
    window that takes the FULL kernel's masked path."""
    print(f"[prefill-many-kv] hq={hq} hkv={hkv}", flush=True)
    for kind, window in (("full", 0), ("swa", 1000)):
        gpu, ref, _ = run_prefill(kind, window, 64, hq, hkv, [0, 130, 1100], [300, 200, 129], (308, hq, hkv))
        assert_close(gpu, ref, f"prefill many KV heads {kind} hq={hq} hkv={hkv}")


def test_prefill_long_chunk_over_prefix(gpu_lib):
    """A 2048-token chunk over a 1000-token prefix, FULL and SWA (wraps the ring)."""
    for kind, window in (("full", 0), ("swa", 128)):
        gpu, ref, _ = run_prefill(kind, window, 64, 64, 8, [1000, 3], [2048, 700], (302,))
        assert_close(gpu, ref, f"long chunk {kind}")


def test_prefill_empty_chunks(gpu_lib):
    """Sequences with an empty chunk in the batch are skipped; max_chunk_len 0 is a no-op."""
    gpu, ref, _ = run_prefill("full", 0, 16, 8, 1, [5, 0, 40], [3, 0, 20], (303,))
    assert_close(gpu, ref, "empty chunk in batch")


@pytest.mark.parametrize("scale", [1.0, 4.0])
def test_prefill_large_scale(gpu_lib, scale):
    """Scales above ln 2 (scale * log2 e > 1, e.g. queries that arrive
    pre-scaled): the running maximum starts finite in exp2 units, so a column
    whose first tile is wholly masked (SWA rows whose window starts past the
    workgroup's first tile) gets no NaN. The 512-token SWA prefill (8 / 1 heads,
    PG 16) and a chunk over a cached prefix at 64 / 8 heads, PG 64."""
    print(f"[prefill-scale] scale={scale}", flush=True)
    gpu, ref, _ = run_prefill("swa", 128, 16, 8, 1, [0], [512], (304, 1), scale=scale)
    assert_close(gpu, ref, f"swa prefill 512, scale {scale}")
    for kind, window in (("swa", 128), ("full", 0)):
        gpu, ref, _ = run_prefill(kind, window, 64, 64, 8, [1000, 3], [2048, 700], (304, 2), scale=scale)
        assert_close(gpu, ref, f"{kind} prefill over a prefix, scale {scale}")


@pytest.mark.parametrize("hq,hkv,window", [(64, 8, 129), (64, 8, 130), (128, 8, 145), (128, 8, 146),
                                           (32, 8, 512), (32, 8, 513), (64, 8, 33)])
def test_prefill_window_kernel_boundaries(gpu_lib, hq, hkv, window):
    """SWA prefill takes one of three kernels: with a GQA group G >= 8 and
    W + 256 / G - 1 <= 160 the persistent one over runs of tiles, otherwise up
    to W = 512 the per-tile windowed one, and beyond that the FULL-style one.
    Each side of both limits, over prefixes that put window starts before,
    across and after the prefix / chunk boundary (PG 16 and 64), against the
    oracle."""
    print(f"[prefill-boundaries] hq={hq} hkv={hkv} W={window}", flush=True)
    for pg in (16, 64):
        gpu, ref, _ = run_prefill("swa", window, pg, hq, hkv, [0, 37, 300, 1000], [700, 333, 64, 900],
                                  (305, hq, window, pg))
        assert_close(gpu, ref, f"prefill W={window} hq={hq} hkv={hkv} PG={pg}")
