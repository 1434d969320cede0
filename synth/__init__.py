"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds no attention, slot-mapping or block-table arithmetic: it only
draws numbers (bf16 q/k/v, sequence lengths, page permutations) and describes
the workload shapes. Both the GPU path's tests and the oracle receive exactly
the arrays produced here.

Recipe (same for every workload):
  * q, k, v are i.i.d. N(0, 1), drawn in float32 and rounded to bf16 with
    round-to-nearest-even; the bf16 bit patterns are the inputs.
  * every draw has its own seed, derived from (workload seed, layer, sequence,
    tag) through numpy's SeedSequence, so a sample of sequences can be
    regenerated without drawing the rest.
  * physical page ids of a pool are a seeded permutation of [0, num_pages).
  * lengths follow the workload: uniform integers, inclusive, not page aligned;
    log-normal decode contexts use ln c ~ N(ln median, 1), clipped, floored.
"""

from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np

FULL = "full"
SWA = "swa"

# Tags that separate the independent draws of one (workload, layer, sequence).
TAG_Q, TAG_K, TAG_V, TAG_QDEC, TAG_KDEC, TAG_VDEC = 1, 2, 3, 4, 5, 6
TAG_PERM, TAG_LENS = 7, 8


def seed_of(*keys: int) -> np.random.SeedSequence:
    return np.random.SeedSequence([int(k) & 0xFFFFFFFF for k in keys])


def rng_of(*keys: int) -> np.random.Generator:
    return np.random.default_rng(seed_of(*keys))


def torch_seed_of(*keys: int) -> int:
    return int(seed_of(*keys).generate_state(1, dtype=np.uint64)[0] & 0x7FFFFFFFFFFFFFFF)


def f32_to_bf16_bits(x) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even); uint16 bits."""
    u = np.ascontiguousarray(np.asarray(x, dtype=np.float32)).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def normal_bf16(shape, *keys: int) -> np.ndarray:
    """i.i.d. N(0,1) drawn in float32 from the seed ``keys``; bf16 bit patterns."""
    x = rng_of(*keys).standard_normal(size=shape, dtype=np.float32)
    return f32_to_bf16_bits(x)


def page_permutation(num_pages: int, *keys: int) -> np.ndarray:
    return rng_of(*keys, TAG_PERM).permutation(int(num_pages)).astype(np.int64)


def torch_normal_bf16(shape, device, *keys: int):
    """Large draws on the GPU: N(0,1) in float32 from a seeded torch generator,
    rounded to bf16 by torch (round to nearest even). Host copies of the result
    are what the oracle reads."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(torch_seed_of(*keys))
    x = torch.randn(tuple(shape), generator=gen, device=device, dtype=torch.float32)
    return x.to(torch.bfloat16)


# ----------------------------------------------------------------------------
# Workload descriptions
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Workload:
    """One synthetic workload.

    Every sequence b has ``prefix[b]`` cached tokens and appends ``new[b]`` new
    tokens (new[b] == 1 for a decode sequence). ``layers`` lists the layer
    kinds; SWA layers use ``window``.
    """
    name: str
    seed: int
    hq: int
    hkv: int
    head_dim: int
    page_size: int
    window: int
    layers: List[str]
    prefix: List[int]
    new: List[int]
    mode: str  # "prefill" | "decode" | "mixed"
    decode_mask: Optional[List[bool]] = None  # mixed: which sequences decode

    @property
    def ns(self) -> int:
        return len(self.prefix)

    @property
    def final_lens(self) -> List[int]:
        return [p + n for p, n in zip(self.prefix, self.new)]


def _uniform_ints(n, lo, hi, *keys):
    return [int(x) for x in rng_of(*keys, TAG_LENS).integers(lo, hi + 1, size=n)]


def _lognormal_ints(n, median, sigma, lo, hi, *keys):
    z = rng_of(*keys, TAG_LENS).standard_normal(size=n)
    c = np.floor(np.exp(math.log(median) + sigma * z))
    return [int(x) for x in np.clip(c, lo, hi)]


def swa_prefill_512() -> Workload:
    """One SWA layer, no cache: 1 sequence of 512 tokens, 8 q / 1 kv heads,
    D = 128, W = 128, page size 16 (ring of 9 pages)."""
    return Workload("swa_prefill_512", 1, 8, 1, 128, 16, 128, [SWA], [0], [512], "prefill")


def decode_b64() -> Workload:
    """Decode, one SWA + one FULL layer: 64 sequences with contexts uniform in
    [1024, 32768], 64 q / 8 kv heads, D = 128, page size 64, one new token each."""
    ctx = _uniform_ints(64, 1024, 32768, 2)
    return Workload("decode_b64_ctx1k-32k", 2, 64, 8, 128, 64, 128, [SWA, FULL], ctx, [1] * 64, "decode")


def chunked_prefill_4x8k() -> Workload:
    """Chunked prefill, one SWA + one FULL layer: 4 sequences with an 8192-token
    cached prefix and a 2048-token new chunk, 64 q / 8 kv heads, page size 64."""
    return Workload("prefill_4x(8192+2048)", 3, 64, 8, 128, 64, 128, [SWA, FULL], [8192] * 4, [2048] * 4, "prefill")


def stack70_decode() -> Workload:
    """70-layer decode step: every 7th layer FULL (10 FULL, 60 SWA), 16
    sequences at a 131072-token context, 64 q / 8 kv heads, page size 64."""
    layers = [FULL if (l % 7) == 6 else SWA for l in range(70)]
    return Workload("stack70_decode_b16_ctx128k", 4, 64, 8, 128, 64, 128, layers, [131072] * 16, [1] * 16, "decode")


def mixed_step() -> Workload:
    """Mixed prefill + decode, one SWA + one FULL layer: 8 chunks of 4096 tokens
    with cached prefixes uniform in [0, 65536] plus 256 decodes with log-normal
    contexts (median 8192, sigma 1, clipped to [2048, 65536])."""
    pre = _uniform_ints(8, 0, 65536, 5, 0)
    dec = _lognormal_ints(256, 8192, 1.0, 2048, 65536, 5, 1)
    return Workload("mixed_8x4096+256dec", 5, 64, 8, 128, 64, 128, [SWA, FULL],
                    pre + dec, [4096] * 8 + [1] * 256, "mixed",
                    decode_mask=[False] * 8 + [True] * 256)


WORKLOADS = {
    "swa_prefill_512": swa_prefill_512,
    "decode_b64": decode_b64,
    "chunked_prefill_4x8k": chunked_prefill_4x8k,
    "stack70_decode": stack70_decode,
    "mixed_step": mixed_step,
}


def cu_seqlens(lens: Sequence[int]) -> np.ndarray:
    return np.concatenate([[0], np.cumsum(np.asarray(lens, dtype=np.int64))]).astype(np.int32)
