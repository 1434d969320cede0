"""The C ABI on the CPU: the library loads, exports every function that
include/hswa.h declares, its host helpers agree bit-exactly with the layout
oracle, and argument validation returns the documented status codes before
any device work (no GPU is touched by these tests)."""

import ctypes
import os
import re

import numpy as np
import pytest

from oracle import layout as OL
from paper_2607_13095_amd import hswa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x1000  # a non-null pointer value; validation must fail before any use


def _declared():
    text = open(os.path.join(ROOT, "include", "hswa.h")).read()
    return sorted(set(re.findall(r"\b(hswa_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    lib = hswa.load()
    names = _declared()
    assert len(names) >= 9
    for n in names:
        assert hasattr(lib, n), f"{n} is declared in hswa.h but not exported"
    assert sorted(hswa.EXPORTS) == names


def test_status_strings():
    lib = hswa.load()
    for code, name in hswa.STATUS.items():
        assert lib.hswa_status_string(code).decode() == name


@pytest.mark.parametrize("window,pg", [(1, 16), (128, 16), (128, 64), (129, 64), (4, 2), (1000, 256)])
def test_ring_pages_matches_oracle(window, pg):
    assert hswa.ring_pages(window, pg) == OL.ring_pages(window, pg)


def test_ring_pages_invalid():
    assert hswa.ring_pages(0, 16) == -1 and hswa.ring_pages(5, 0) == -1


@pytest.mark.parametrize("seed", range(6))
def test_block_table_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    pg = int(rng.choice([16, 64]))
    lens = rng.integers(0, 5000, size=int(rng.integers(1, 9))).tolist()
    for kind, window in (("full", 0), ("swa", int(rng.integers(1, 300)))):
        layer = hswa.Layer(kind, window)
        okind = OL.SWA if kind == "swa" else OL.FULL
        need = sum(OL.pages_needed(okind, window, pg, n) for n in lens)
        perm = rng.permutation(need + 7)
        stride = max(OL.pages_needed(okind, window, pg, n) for n in lens) + int(rng.integers(0, 3))
        got = hswa.build_block_table(layer, pg, lens, perm, stride)
        ref = OL.build_block_table(okind, window, pg, lens, perm, stride)
        assert np.array_equal(got, ref)


def test_block_table_capacity_errors():
    with pytest.raises(hswa.HswaError) as e:
        hswa.build_block_table(hswa.Layer.full(), 16, [100], np.arange(100), 4)   # needs 7 > 4
    assert e.value.status == -3
    with pytest.raises(hswa.HswaError) as e:
        hswa.build_block_table(hswa.Layer.full(), 16, [100], np.arange(3), 8)     # perm too short
    assert e.value.status == -3
    with pytest.raises(hswa.HswaError) as e:
        hswa.build_block_table(hswa.Layer.swa(0), 16, [100], np.arange(30), 8)    # W < 1
    assert e.value.status == -1


def test_page_bytes():
    assert hswa.page_bytes(hswa.Shape(64, 8, 128, 64)) == OL.page_bytes(8, 64, 128) == 131072
    assert hswa.page_bytes(hswa.Shape(8, 1, 128, 16)) == 4096


def _shape(hq=64, hkv=8, d=128, pg=64, scale=0.088):
    return hswa._Shape(hq, hkv, d, pg, scale)


def _cache(stride=8, pages=10):
    return hswa._Cache(FAKE, FAKE, pages, FAKE, stride)


def _decode(layer, shape, cache, ns=2, maxc=100, ws=None, wsb=0, q=FAKE, ctx=FAKE, out=FAKE):
    lib = hswa.load()
    return lib.hswa_decode(layer, ctypes.byref(shape), ctypes.byref(cache) if cache is not None else None,
                           q, ctx, ns, maxc, ws, wsb, out, None)


FULL, SWA128 = hswa._Layer(0, 0), hswa._Layer(1, 128)


@pytest.mark.parametrize("shape,code", [
    (_shape(d=64), -2), (_shape(d=256), -2),            # head_dim must be 128
    (_shape(hq=12, hkv=8), -1),                         # Hq % Hkv != 0
    (_shape(hq=24, hkv=8), -2),                         # group 3 does not divide 128
    (_shape(pg=48), -2), (_shape(pg=8), -2), (_shape(pg=512), -2),
    (_shape(scale=0.0), -1), (_shape(scale=float("nan")), -1),
    (_shape(hq=0), -1),
    (_shape(hq=8192, hkv=8192), -2),                   # more than 4096 KV heads
])
def test_decode_shape_validation(shape, code):
    assert _decode(FULL, shape, _cache()) == code


def test_decode_argument_validation():
    sh = _shape()
    assert _decode(hswa._Layer(1, 0), sh, _cache()) == -1          # SWA window < 1
    assert _decode(hswa._Layer(7, 0), sh, _cache()) == -1          # unknown kind
    assert _decode(FULL, sh, None) == -1                           # null cache
    assert _decode(FULL, sh, _cache(), q=None) == -1               # null q
    assert _decode(FULL, sh, _cache(), maxc=0) == -1               # max context < 1
    assert _decode(FULL, sh, _cache(stride=1), maxc=100) == -3     # 64-token table for 100 tokens
    assert _decode(SWA128, sh, _cache(stride=2)) == -3             # ring needs 3 entries
    # a FULL decode long enough to split needs a workspace of the advertised size
    need = hswa.load().hswa_decode_workspace_bytes(ctypes.byref(sh), 4, 100000)
    assert need > 0
    assert _decode(FULL, sh, _cache(stride=2000), ns=4, maxc=100000, ws=None) == -1
    assert _decode(FULL, sh, _cache(stride=2000), ns=4, maxc=100000, ws=FAKE, wsb=need - 1) == -3


def test_prefill_and_append_validation():
    lib = hswa.load()
    sh = _shape()
    ca = _cache()
    st = lib.hswa_prefill(FULL, ctypes.byref(sh), ctypes.byref(ca), None, FAKE, FAKE, FAKE, FAKE, 1, 10, 10, FAKE, None)
    assert st == -1
    st = lib.hswa_prefill(FULL, ctypes.byref(_shape(d=64)), ctypes.byref(ca), FAKE, FAKE, FAKE, FAKE, FAKE, 1, 10, 10,
                          FAKE, None)
    assert st == -2
    st = lib.hswa_prefill(FULL, ctypes.byref(sh), ctypes.byref(ca), FAKE, FAKE, FAKE, FAKE, FAKE, -1, 10, 10, FAKE, None)
    assert st == -1
    # empty work is accepted without touching anything
    assert lib.hswa_prefill(FULL, ctypes.byref(sh), ctypes.byref(ca), None, None, None, None, None, 0, 0, 0, None,
                            None) == 0
    st = lib.hswa_kv_append(SWA128, ctypes.byref(sh), ctypes.byref(ca), None, FAKE, FAKE, FAKE, 1, 5, None, None)
    assert st == -1
    st = lib.hswa_kv_append(SWA128, ctypes.byref(sh), ctypes.byref(_cache(stride=2)), FAKE, FAKE, FAKE, FAKE, 1, 5,
                            None, None)
    assert st == -3
    assert lib.hswa_kv_append(FULL, ctypes.byref(sh), ctypes.byref(ca), None, None, None, None, 0, 0, None, None) == 0


def test_workspace_and_split_len_host_helpers():
    sh = hswa.Shape(64, 8, 128, 64)
    for ns, maxc in ((64, 32769), (16, 131073), (1, 300), (4, 10240)):
        sl = hswa.decode_split_len(sh, ns, maxc)
        assert sl >= 256 and sl % 256 == 0
        splits = -(-maxc // sl)
        wsb = hswa.decode_workspace_bytes(sh, ns, maxc)
        if splits == 1:
            assert wsb == 0
        else:
            assert wsb >= ns * 64 * splits * (128 + 1) * 4
    assert hswa.decode_split_len(hswa.Shape(64, 8, 64, 64), 4, 100) == -1


def _decode_multi(layer, shape, cache, nq, ns=2, maxc=300):
    lib = hswa.load()
    return lib.hswa_decode_multi(layer, ctypes.byref(shape), ctypes.byref(cache), FAKE, FAKE, ns, nq, maxc, FAKE,
                                 1 << 30, FAKE, None)


def test_decode_multi_swa_query_limit():
    """The first of nq new queries reads the W - 1 keys before it; a ring of R
    pages keeps the latest R * PG positions, so an SWA ring layer accepts
    nq <= R * PG - W + 1 and an explicit-release table (which stores the last
    W positions of one extend) nq <= W. Beyond: HSWA_ERR_UNSUPPORTED before any
    device work."""
    sh16 = _shape(pg=16)
    ring16 = OL.ring_pages(128, 16) * 16            # 144 positions held
    assert ring16 - 128 + 1 == 17
    assert _decode_multi(SWA128, sh16, _cache(stride=9), 18) == -2
    assert _decode_multi(SWA128, sh16, _cache(stride=9), 64) == -2
    assert _decode_multi(hswa._Layer(1, 5), sh16, _cache(stride=2), 29) == -2    # R = 2: 32 - 5 + 1 = 28
    # SWA_PAGED: nq <= W
    assert _decode_multi(hswa._Layer(2, 4), sh16, _cache(stride=32), 5) == -2
    assert _decode_multi(hswa._Layer(2, 1), sh16, _cache(stride=32), 2) == -2
    # the limits do not apply to FULL layers, nor at PG 64 / W 128 (65 > 64 queries)
    assert _decode_multi(FULL, sh16, _cache(stride=32), 65) == -1    # 65 > 64: the general limit
    for layer, cache, nq in ((SWA128, _cache(stride=3), 64), (hswa._Layer(2, 128), _cache(stride=8), 64)):
        # legal counts pass validation; a null q then stops the call before any device work
        lib = hswa.load()
        sh = _shape()
        st = lib.hswa_decode_multi(layer, ctypes.byref(sh), ctypes.byref(cache), None, FAKE, 2, nq, 300, FAKE,
                                   1 << 30, FAKE, None)
        assert st == -1
    lib = hswa.load()
    st = lib.hswa_decode_multi(SWA128, ctypes.byref(sh16), ctypes.byref(_cache(stride=9)), None, FAKE, 2, 17, 300,
                               FAKE, 1 << 30, FAKE, None)
    assert st == -1                                   # 17 is legal at PG 16: reaches the null-q check


def test_binding_rejects_pools_that_disagree_with_the_shape():
    """The binding checks pools and table against the shape before any call."""
    import torch

    sh = hswa.Shape(64, 8, 128, 64)

    class T:  # stands in for device tensors: only .shape is read by the check
        def __init__(self, *shape):
            self.shape = torch.Size(shape)

    def cache(hkv=8, pg=64, d=128, rows=4):
        c = hswa.Cache.__new__(hswa.Cache)
        c.v_pool = T(10, hkv, pg // min(pg, 32), d, min(pg, 32))
        c.block_table = T(rows, 5)
        return c

    hswa._check_cache(sh, cache(), 4)
    for bad, ns in ((cache(hkv=4), 4), (cache(pg=16), 4), (cache(d=64), 4), (cache(rows=3), 4)):
        with pytest.raises(ValueError):
            hswa._check_cache(sh, bad, ns)


def test_decode_noalloc_validation():
    """The allocation-free decode validates like hswa_decode and rejects a FULL
    call whose split partials exceed its fixed array, before any device work."""
    lib = hswa.load()
    sh = _shape()

    def call(layer, cache, ns, maxc, q=FAKE):
        return lib.hswa_decode_noalloc(layer, ctypes.byref(sh), ctypes.byref(cache), q, FAKE, ns, maxc, FAKE, None)

    need = lib.hswa_decode_workspace_bytes(ctypes.byref(sh), 256, 65537)
    assert need > hswa.NOALLOC_SCRATCH_BYTES
    assert call(FULL, _cache(stride=1100), 256, 65537) == -3
    fits = lib.hswa_decode_workspace_bytes(ctypes.byref(sh), 64, 32769)
    assert 0 < fits <= hswa.NOALLOC_SCRATCH_BYTES
    assert call(FULL, _cache(stride=600), 64, 32769, q=None) == -1    # fits: reaches the null-q check
    assert call(FULL, _cache(stride=1), 2, 100) == -3                 # table too short, as hswa_decode
    assert call(hswa._Layer(1, 0), _cache(), 2, 100) == -1            # SWA window < 1
    assert call(SWA128, _cache(stride=3), 2, 100, q=None) == -1


def test_decode_append_validation():
    """The fused decode step validates like hswa_decode and also needs the new
    token's K and V rows; every failure returns before any device work."""
    lib = hswa.load()
    sh = _shape()

    def call(layer, cache, ns, maxc, q=FAKE, k=FAKE, v=FAKE, ws=None, wsb=0):
        return lib.hswa_decode_append(layer, ctypes.byref(sh), ctypes.byref(cache), q, k, v, FAKE, ns, maxc, ws, wsb,
                                      FAKE, None)

    assert call(SWA128, _cache(stride=3), 2, 100, k=None) == -1
    assert call(SWA128, _cache(stride=3), 2, 100, v=None) == -1
    assert call(SWA128, _cache(stride=3), 2, 100, q=None) == -1
    assert call(SWA128, _cache(stride=2), 2, 100) == -3               # ring needs 3 entries (PG 64)
    assert call(FULL, _cache(stride=1), 2, 100) == -3                 # table too short, as hswa_decode
    assert call(hswa._Layer(1, 0), _cache(), 2, 100) == -1            # SWA window < 1
    assert call(FULL, _cache(stride=600), 64, 32769) == -1            # split FULL without a workspace
    assert call(SWA128, _cache(stride=3), 0, 100) == 0                # nothing to do
