"""Pins for the fp64 attention oracle (CPU only).

Each check compares the oracle against something other than itself: a
pure-Python brute force with its own loops, torch's scaled_dot_product_attention
in float64 with an explicit boolean mask, closed forms (W = 1, zero query,
single key, two keys), and invariants (W >= L equals FULL, translation,
GQA head repetition, chunk splitting, decode = last prefill row, a spike key
just outside the window). ``test_planted_mistakes_are_caught`` plants plausible
mistakes in the oracle and checks that these pins catch every one.
"""

import math

import numpy as np
import pytest
import torch

from oracle import attention as A

RTOL = 1e-12


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _brute(q, k, v, q_pos, window, scale):
    """Pure-Python loops, no max subtraction, its own window test."""
    tq, hq, d = q.shape
    L, hkv, _ = k.shape
    grp = hq // hkv
    out = np.zeros_like(q)
    for t in range(tq):
        p = int(q_pos[t])
        for h in range(hq):
            g = h // grp
            num = [0.0] * d
            den = 0.0
            for j in range(L):
                if j > p:
                    continue
                if window is not None and p - j >= window:
                    continue
                s = scale * sum(q[t, h, x] * k[j, g, x] for x in range(d))
                e = math.exp(s)
                den += e
                for x in range(d):
                    num[x] += e * v[j, g, x]
            for x in range(d):
                out[t, h, x] = num[x] / den
    return out


def _sdpa(q, k, v, q_pos, window, scale):
    """torch SDPA in float64 with an explicit boolean mask, KV heads repeated."""
    tq, hq, d = q.shape
    L, hkv, _ = k.shape
    grp = hq // hkv
    p = torch.as_tensor(np.asarray(q_pos))[:, None]
    j = torch.arange(L)[None, :]
    mask = j <= p
    if window is not None:
        mask &= (p - j) < window
    qt = torch.as_tensor(q).permute(1, 0, 2)                       # [hq, tq, d]
    kt = torch.as_tensor(k).permute(1, 0, 2).repeat_interleave(grp, dim=0)
    vt = torch.as_tensor(v).permute(1, 0, 2).repeat_interleave(grp, dim=0)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)
    return o.permute(1, 0, 2).numpy()


# --------------------------------------------------------------------------
# pin suite: every function returns a list of failure strings (empty = pass)
# --------------------------------------------------------------------------

def pin_brute_force():
    fails = []
    case = 0
    for d in (1, 4):
        for hq, hkv in ((1, 1), (2, 1), (4, 2)):
            for L in (1, 2, 5, 9, 12):
                for window in (None, 1, 2, 3, 7, 20):
                    case += 1
                    q = _rand((3, hq, d), case)
                    k = _rand((L, hkv, d), case + 1000)
                    v = _rand((L, hkv, d), case + 2000)
                    pos = np.random.default_rng(case).integers(0, L, size=3)
                    scale = 0.37 + 0.1 * d
                    got = A.masked_attention(q, k, v, pos, window, scale)
                    ref = _brute(q, k, v, pos, window, scale)
                    if not np.allclose(got, ref, rtol=RTOL, atol=1e-13):
                        fails.append(f"brute d={d} hq={hq} hkv={hkv} L={L} W={window}")
    return fails


def pin_sdpa():
    fails = []
    for i, (hq, hkv, L, window) in enumerate([(8, 2, 40, None), (8, 2, 40, 5), (4, 4, 33, 1),
                                              (8, 1, 64, 16), (6, 3, 50, 49)]):
        d = 16
        q = _rand((L, hq, d), 10 + i)
        k = _rand((L, hkv, d), 20 + i)
        v = _rand((L, hkv, d), 30 + i)
        pos = np.arange(L)
        scale = 1.0 / math.sqrt(d)
        got = A.masked_attention(q, k, v, pos, window, scale)
        ref = _sdpa(q, k, v, pos, window, scale)
        if not np.allclose(got, ref, rtol=1e-11, atol=1e-12):
            fails.append(f"sdpa hq={hq} hkv={hkv} L={L} W={window}")
    return fails


def pin_window_one_returns_own_value():
    fails = []
    L, hq, hkv, d = 17, 4, 2, 8
    q, k, v = _rand((L, hq, d), 1), _rand((L, hkv, d), 2), _rand((L, hkv, d), 3)
    got = A.masked_attention(q, k, v, np.arange(L), 1)
    for p in range(L):
        for h in range(hq):
            if not np.array_equal(got[p, h], v[p, h // 2]):
                fails.append(f"W=1 p={p} h={h}")
    return fails


def pin_zero_query_is_window_mean():
    """q = 0 gives uniform weights, so o is the mean of exactly the visible keys."""
    fails = []
    L, hq, hkv, d = 23, 2, 1, 5
    k, v = _rand((L, hkv, d), 4), _rand((L, hkv, d), 5)
    q = np.zeros((L, hq, d))
    for window in (None, 1, 2, 3, 8, 22, 23, 40):
        got = A.masked_attention(q, k, v, np.arange(L), window)
        for p in range(L):
            lo = 0 if window is None else max(0, p - window + 1)
            ref = v[lo:p + 1, 0].mean(axis=0)
            if not np.allclose(got[p, 0], ref, rtol=RTOL, atol=1e-14):
                fails.append(f"mean W={window} p={p}")
    return fails


def pin_single_key():
    q, k, v = _rand((1, 3, 6), 6), _rand((1, 1, 6), 7), _rand((1, 1, 6), 8)
    fails = []
    for window in (None, 1, 128):
        got = A.masked_attention(q, k, v, [0], window)
        if not all(np.array_equal(got[0, h], v[0, 0]) for h in range(3)):
            fails.append(f"L=1 W={window}")
    return fails


def pin_two_keys_closed_form():
    """Two visible keys: o = v0 + sigmoid(s1 - s0) * (v1 - v0), s_j = scale<q,k_j>."""
    fails = []
    d = 3
    q = np.array([[[0.5, -1.0, 2.0]]])
    k = np.array([[[1.0, 0.0, 0.0]], [[0.0, 1.0, 1.0]]])
    v = np.array([[[1.0, 2.0, 3.0]], [[-1.0, 0.0, 5.0]]])
    scale = 0.75
    s0, s1 = scale * 0.5, scale * 1.0            # <q,k0> = 0.5, <q,k1> = 1.0
    w1 = 1.0 / (1.0 + math.exp(s0 - s1))
    ref = v[0, 0] + w1 * (v[1, 0] - v[0, 0])
    got = A.masked_attention(q, k, v, [1], None, scale)[0, 0]
    if not np.allclose(got, ref, rtol=1e-14, atol=0):
        fails.append("two keys")
    # default scale is 1/sqrt(D): D = 4 gives scale 1/2
    q4 = np.array([[[2.0, 0.0, 0.0, 0.0]]])
    k4 = np.array([[[0.0, 0.0, 0.0, 0.0]], [[1.0, 0.0, 0.0, 0.0]]])
    v4 = np.array([[[0.0, 0.0, 0.0, 0.0]], [[1.0, 1.0, 1.0, 1.0]]])
    w1 = 1.0 / (1.0 + math.exp(-1.0))              # s1 - s0 = (1/2) * 2 = 1
    got = A.masked_attention(q4, k4, v4, [1], None)[0, 0]
    if not np.allclose(got, np.full(4, w1), rtol=1e-14, atol=0):
        fails.append("two keys, default scale")
    return fails


def pin_spike_outside_window():
    """A key that would dominate the softmax, one position outside the window,
    must not change the result; one position inside, it must dominate."""
    fails = []
    d, W, p = 8, 5, 12
    rng = np.random.default_rng(9)
    k = rng.standard_normal((p + 1, 1, d)) * 0.01
    v = rng.standard_normal((p + 1, 1, d))
    q = np.ones((1, 1, d))
    for j_spike, inside in ((p - W, False), (p - W + 1, True)):
        k2 = k.copy()
        k2[j_spike, 0] = 50.0
        got = A.masked_attention(q, k2, v, [p], W, 1.0)[0, 0]
        base = A.masked_attention(q, k, v, [p], W, 1.0)[0, 0]
        if inside and not np.allclose(got, v[j_spike, 0], atol=1e-12):
            fails.append("spike inside not dominant")
        if not inside and not np.array_equal(got, base):
            fails.append("spike outside leaked")
    # the future key just after p must never count either (causality)
    k3 = k.copy()
    v3 = v.copy()
    extra_k = np.full((1, 1, d), 50.0)
    extra_v = rng.standard_normal((1, 1, d))
    got = A.masked_attention(q, np.concatenate([k3, extra_k]), np.concatenate([v3, extra_v]), [p], None, 1.0)
    base = A.masked_attention(q, k3, v3, [p], None, 1.0)
    if not np.array_equal(got, base):
        fails.append("future key leaked")
    return fails


def pin_window_ge_len_is_full():
    fails = []
    L, hq, hkv, d = 30, 4, 2, 8
    q, k, v = _rand((L, hq, d), 11), _rand((L, hkv, d), 12), _rand((L, hkv, d), 13)
    full = A.masked_attention(q, k, v, np.arange(L), None)
    for window in (L, L + 1, 10 * L):
        if not np.array_equal(A.masked_attention(q, k, v, np.arange(L), window), full):
            fails.append(f"W={window} != FULL")
    # and a window smaller than L must differ somewhere
    if np.allclose(A.masked_attention(q, k, v, np.arange(L), L - 5), full):
        fails.append("small window equals FULL")
    return fails


def pin_translation():
    """SWA at position p equals FULL attention over the slice [p-W+1, p]."""
    fails = []
    L, hq, hkv, d, W = 40, 4, 1, 8, 7
    q, k, v = _rand((L, hq, d), 14), _rand((L, hkv, d), 15), _rand((L, hkv, d), 16)
    swa = A.masked_attention(q, k, v, np.arange(L), W)
    for p in range(L):
        lo = max(0, p - W + 1)
        ref = A.masked_attention(q[p:p + 1], k[lo:p + 1], v[lo:p + 1], [p - lo], None)[0]
        if not np.allclose(swa[p], ref, rtol=RTOL, atol=1e-14):
            fails.append(f"translation p={p}")
    return fails


def pin_gqa_repeat():
    fails = []
    L, hq, hkv, d = 20, 8, 2, 8
    q, k, v = _rand((L, hq, d), 17), _rand((L, hkv, d), 18), _rand((L, hkv, d), 19)
    grp = hq // hkv
    krep, vrep = np.repeat(k, grp, axis=1), np.repeat(v, grp, axis=1)
    for window in (None, 4):
        a = A.masked_attention(q, k, v, np.arange(L), window)
        b = A.masked_attention(q, krep, vrep, np.arange(L), window)
        if not np.allclose(a, b, rtol=RTOL, atol=1e-14):
            fails.append(f"gqa W={window}")
    return fails


def pin_chunked_and_decode():
    """prefill(P, C) equals the last C rows of a one-shot prefill over P + C
    tokens; decode at c equals the last row of a prefill over c + 1 tokens."""
    fails = []
    L, hq, hkv, d = 37, 4, 2, 8
    q, k, v = _rand((L, hq, d), 20), _rand((L, hkv, d), 21), _rand((L, hkv, d), 22)
    for window in (None, 6):
        whole = A.prefill(q, k, v, 0, window)
        for P in (0, 1, 5, 20, 36):
            part = A.prefill(q[P:], k, v, P, window)
            if not np.allclose(part, whole[P:], rtol=RTOL, atol=1e-14):
                fails.append(f"chunk P={P} W={window}")
        dec = A.decode(q[L - 1], k, v, window)
        if not np.allclose(dec, whole[L - 1], rtol=RTOL, atol=1e-14):
            fails.append(f"decode W={window}")
    return fails


PINS = [pin_brute_force, pin_sdpa, pin_window_one_returns_own_value, pin_zero_query_is_window_mean,
        pin_single_key, pin_two_keys_closed_form, pin_spike_outside_window, pin_window_ge_len_is_full,
        pin_translation, pin_gqa_repeat, pin_chunked_and_decode]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    assert pin() == []


def test_bf16_conversion_exact():
    bits = np.array([0x0000, 0x8000, 0x3F80, 0xBF80, 0x4049, 0x7F7F, 0x0001, 0x7F80], dtype=np.uint16)
    ref = [0.0, -0.0, 1.0, -1.0, 3.140625, 3.3895313892515355e38, 9.183549615799121e-41, np.inf]
    got = A.bf16_bits_to_f64(bits)
    assert got.tolist() == ref
    assert np.signbit(got[1])


# --------------------------------------------------------------------------
# planted mistakes: each must be caught by at least one pin
# --------------------------------------------------------------------------

def _mask_off_by_one(q_pos, num_keys, window):
    p = np.asarray(q_pos)[:, None]
    j = np.arange(num_keys)[None, :]
    m = j <= p
    return m if window is None else m & (j >= p - window)


def _mask_not_causal(q_pos, num_keys, window):
    p = np.asarray(q_pos)[:, None]
    j = np.arange(num_keys)[None, :]
    m = np.ones((p.shape[0], num_keys), dtype=bool)
    return m if window is None else m & (j >= p - window + 1)


def _mask_window_ignored(q_pos, num_keys, window):
    p = np.asarray(q_pos)[:, None]
    return np.arange(num_keys)[None, :] <= p


def _head_modulo(h, group):
    return h % group


MUTANTS = {
    "window_off_by_one": ("allowed_mask", _mask_off_by_one),
    "not_causal": ("allowed_mask", _mask_not_causal),
    "window_ignored": ("allowed_mask", _mask_window_ignored),
    "gqa_head_modulo": ("kv_head_of", _head_modulo),
    "scale_dropped": ("default_scale", lambda d: 1.0),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_planted_mistakes_are_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(A, attr, fn)
    caught = []
    for pin in PINS:
        try:
            if pin():
                caught.append(pin.__name__)
        except Exception as e:  # a crash also counts as caught
            caught.append(f"{pin.__name__}:{type(e).__name__}")
    assert caught, f"planted mistake {name} escaped every pin"


def test_planted_value_transpose_is_caught(monkeypatch):
    """Using K in place of V for the weighted sum must be caught."""
    orig = A.masked_attention

    def wrong(q, k, v, q_pos, window, scale=None):
        return orig(q, k, k, q_pos, window, scale)

    monkeypatch.setattr(A, "masked_attention", wrong)
    assert any(pin() for pin in (pin_brute_force, pin_sdpa))
