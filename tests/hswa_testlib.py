"""Helpers for the GPU parity tests: moving seeded bf16 inputs between numpy
(the oracle's side) and torch device tensors (the library's side), building a
filled paged cache through the library, and the tolerance check.

The tolerance is the one fixed for bf16 inputs with fp32 accumulation:
|gpu - ref| <= 1e-2 + 1e-2 * |ref| element-wise, plus a relative-L2 check of
1e-2 per output tensor.
"""

from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import attention as OA
from paper_2607_13095_amd import hswa
from paper_2607_13095_amd.kvcache import LayerKV, pages_for

ATOL = 1e-2
RTOL = 1e-2


def to_dev(bits: np.ndarray) -> torch.Tensor:
    """uint16 bf16 bit patterns -> bf16 device tensor (bit-exact)."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def to_bits(t: torch.Tensor) -> np.ndarray:
    """bf16 device tensor -> uint16 bit patterns on the host."""
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def to_f64(t: torch.Tensor) -> np.ndarray:
    return OA.bf16_bits_to_f64(to_bits(t))


def i32(x) -> torch.Tensor:
    return torch.as_tensor(np.asarray(x, dtype=np.int32)).cuda()


def assert_close(gpu: np.ndarray, ref: np.ndarray, what: str = ""):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite output"
    err = np.abs(gpu - ref)
    bound = ATOL + RTOL * np.abs(ref)
    bad = err > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} elements outside tolerance, max err "
                           f"{err.max():.3e} at {np.unravel_index(np.argmax(err - bound), err.shape)}")
    rel = np.linalg.norm(gpu - ref) / max(np.linalg.norm(ref), 1e-30)
    assert rel <= 1e-2, f"{what}: relative L2 error {rel:.3e}"


class SeqHistory:
    """Contiguous bf16 K/V history of every sequence of one layer (host bits)."""

    def __init__(self, lens, hkv, d, *seed):
        self.k = [synth.normal_bf16((n, hkv, d), *seed, b, synth.TAG_K) for b, n in enumerate(lens)]
        self.v = [synth.normal_bf16((n, hkv, d), *seed, b, synth.TAG_V) for b, n in enumerate(lens)]

    def rows(self, b, lo, hi):
        return self.k[b][lo:hi], self.v[b][lo:hi]


def make_layer(kind: str, window: int, shape: hswa.Shape, final_lens, seed, extra_pages=3, fill=float("nan")):
    """A layer's pools with a seeded page permutation (spare pages included)."""
    layer = hswa.Layer.swa(window) if kind == "swa" else hswa.Layer.full()
    total = pages_for(layer, shape.page_size, final_lens) + extra_pages
    perm = synth.page_permutation(total, *seed)
    return layer, LayerKV(layer, shape, final_lens, perm=perm, extra_pages=extra_pages, fill=fill)


def append_history(layer, shape, kv: LayerKV, hist: SeqHistory, starts, ends):
    """Append positions [starts[b], ends[b]) of every sequence in one call."""
    ks, vs, lens = [], [], []
    for b, (s, e) in enumerate(zip(starts, ends)):
        k, v = hist.rows(b, s, e)
        ks.append(k)
        vs.append(v)
        lens.append(e - s)
    hkv, d = shape.num_kv_heads, shape.head_dim
    kn = np.concatenate(ks) if ks else np.zeros((0, hkv, d), np.uint16)
    vn = np.concatenate(vs) if vs else np.zeros((0, hkv, d), np.uint16)
    slots = torch.empty(max(1, kn.shape[0]), dtype=torch.int64, device="cuda")
    hswa.kv_append(layer, shape, kv.cache, to_dev(kn), to_dev(vn), i32(synth.cu_seqlens(lens)), i32(starts),
                   slot_mapping_out=slots)
    return slots[:kn.shape[0]].cpu().numpy()
