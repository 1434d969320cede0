"""fp64 masked softmax attention over a contiguous KV history (the oracle).

TEST INFRASTRUCTURE ONLY: only tests, the smoke check and the benchmark's CPU
baseline may use this module.

What is computed (plain definition; paging, ring buffers, tile skipping and
split-KV in the GPU path only reorder this exact computation):

    For one sequence with contiguous history K, V of shape [L, Hkv, D] (position
    j stored at row j, including positions a GPU ring has already evicted), a
    query q at absolute position p and query head h sees KV head g = h // G,
    G = Hq / Hkv, and the keys j with lo(p) <= j <= p, where
        lo(p) = 0                      for a FULL (global) layer,
        lo(p) = max(0, p - W + 1)      for an SWA layer of window W.
    s_j = scale * <q, K[j, g]> on allowed keys, -inf elsewhere;
    o   = sum_j softmax(s)_j * V[j, g].

Sources: the paper's "Introduction" and "Compute Analysis" (SWA layers attend
only inside a local window, FULL layers attend globally, interleaved), and
"KVCache Dual-Pool Design" / "SWA-Aware Prefix Cache Tree" (SWA keeps only the
in-window KV; evicted or overwritten slots must never contribute).

Readings where the paper is silent (each one is pinned by a CPU test):
  * W counts the query itself: keys [p - W + 1, p] (W = 1 gives V at p).
  * scale is a parameter; the default is 1/sqrt(D).
  * consecutive query heads share a KV head: g = h // G.
  * no positional term, sink, soft-cap or bias inside attention.
"""

from __future__ import annotations

import numpy as np

FULL = "full"
SWA = "swa"


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact conversion of bf16 bit patterns (uint16) to float64.

    A bf16 value is the upper half of an IEEE binary32; shifting its 16 bits into
    the high half of a 32-bit word gives that binary32 exactly.
    """
    u16 = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16))
    return (u16.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def default_scale(head_dim: int) -> float:
    return 1.0 / np.sqrt(float(head_dim))


def kv_head_of(h, group: int):
    """KV head that query head ``h`` reads (consecutive query heads share one)."""
    return h // group


def allowed_mask(q_pos, num_keys: int, window) -> np.ndarray:
    """Boolean mask [len(q_pos), num_keys]: key j is visible to the query at p.

    ``window`` is None for a FULL layer, else the SWA window W >= 1.
    """
    p = np.asarray(q_pos, dtype=np.int64)[:, None]
    j = np.arange(num_keys, dtype=np.int64)[None, :]
    causal = j <= p
    if window is None:
        return causal
    return causal & (j >= p - (int(window) - 1))


def masked_attention(q, k, v, q_pos, window, scale=None) -> np.ndarray:
    """Attention of queries at absolute positions ``q_pos`` over a history.

    q: [Tq, Hq, D]; k, v: [L, Hkv, D] (row j = position j); q_pos: [Tq] ints in
    [0, L). Returns float64 [Tq, Hq, D]. Inputs are converted to float64.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    tq, hq, d = q.shape
    num_keys, hkv, dk = k.shape
    if dk != d or v.shape != k.shape:
        raise ValueError("q, k, v head dims / shapes disagree")
    if hq % hkv:
        raise ValueError("query heads must be a multiple of KV heads")
    q_pos = np.asarray(q_pos, dtype=np.int64)
    if q_pos.shape != (tq,):
        raise ValueError("one position per query row")
    if tq and (q_pos.min() < 0 or q_pos.max() >= num_keys):
        raise ValueError("query position outside the history")
    if scale is None:
        scale = default_scale(d)
    group = hq // hkv
    if tq == 0:
        return np.zeros((0, hq, d), dtype=np.float64)

    mask = allowed_mask(q_pos, num_keys, window)          # [Tq, L]
    out = np.zeros((tq, hq, d), dtype=np.float64)
    for h in range(hq):
        g = kv_head_of(h, group)
        s = scale * (q[:, h, :] @ k[:, g, :].T)              # [Tq, L]
        s = np.where(mask, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        e = np.exp(s - m)                                   # exp(-inf) = 0
        w = e / e.sum(axis=1, keepdims=True)
        out[:, h, :] = w @ v[:, g, :]
    return out


def prefill(q_chunk, k_hist, v_hist, prefix_len: int, window, scale=None):
    """Chunked prefill: the C new queries sit at positions prefix_len .. L-1.

    k_hist, v_hist hold the whole history [L, Hkv, D] with L = prefix_len + C
    (the cached prefix followed by the new chunk's keys).
    """
    c = np.asarray(q_chunk).shape[0]
    if prefix_len + c != np.asarray(k_hist).shape[0]:
        raise ValueError("history length must be prefix_len + chunk length")
    pos = np.arange(prefix_len, prefix_len + c, dtype=np.int64)
    return masked_attention(q_chunk, k_hist, v_hist, pos, window, scale)


def decode(q_new, k_hist, v_hist, window, scale=None):
    """Decode: one query per sequence, at the last position L-1 of the history.

    q_new: [Hq, D]; returns [Hq, D].
    """
    num_keys = np.asarray(k_hist).shape[0]
    q1 = np.asarray(q_new)[None]
    return masked_attention(q1, k_hist, v_hist, [num_keys - 1], window, scale)[0]


def visible_key_count(p: int, window) -> int:
    """Number of keys the query at position p sees."""
    return p + 1 if window is None else min(int(window), p + 1)
