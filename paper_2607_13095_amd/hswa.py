"""Python binding of libhswa (ctypes): argument marshalling only.

Every call checks device, dtype, contiguity and sizes of the torch tensors it
is given, passes their device pointers and the current HIP stream to the C ABI
(``include/hswa.h``) and raises ``HswaError`` on a non-OK status. All compute
runs in the library's HIP kernels; there is no fallback of any kind: if
``libhswa.so`` is not built, ``load()`` raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# HSWA_LIB names another build of the same library (the host-sanitizer build)
LIB_PATH = os.environ.get("HSWA_LIB") or os.path.join(_PKG, "libhswa.so")

HSWA_LAYER_FULL = 0
HSWA_LAYER_SWA = 1
HSWA_LAYER_SWA_PAGED = 2

STATUS = {0: "HSWA_OK", -1: "HSWA_ERR_INVALID_ARG", -2: "HSWA_ERR_UNSUPPORTED", -3: "HSWA_ERR_CAPACITY",
          -4: "HSWA_ERR_LAUNCH"}

EXPORTS = ["hswa_ring_pages", "hswa_page_bytes", "hswa_build_block_table", "hswa_kv_append", "hswa_prefill",
           "hswa_decode_workspace_bytes", "hswa_decode_split_len", "hswa_decode", "hswa_status_string",
           "hswa_allocator_create", "hswa_allocator_destroy", "hswa_allocator_admit", "hswa_allocator_extend",
           "hswa_allocator_step_end", "hswa_allocator_free", "hswa_allocator_tables", "hswa_allocator_usage",
           "hswa_prefix_tree_create", "hswa_prefix_tree_destroy", "hswa_prefix_tree_insert",
           "hswa_prefix_tree_match", "hswa_prefix_tree_release_swa", "hswa_prefix_tree_evict",
           "hswa_prefix_tree_stats", "hswa_decode_multi_workspace_bytes", "hswa_decode_multi",
           "hswa_decode_noalloc", "hswa_decode_append"]

# bytes of the library's fixed device array behind hswa_decode_noalloc
NOALLOC_SCRATCH_BYTES = 128 << 20


class HswaError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {STATUS.get(status, status)}")
        self.status = status


class _Layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("window", ctypes.c_int32)]


class _Shape(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("scale", ctypes.c_float)]


class _AllocConfig(ctypes.Structure):
    _fields_ = [("page_size", ctypes.c_int32), ("window", ctypes.c_int32), ("full_pages", ctypes.c_int64),
                ("swa_pages", ctypes.c_int64), ("max_seqs", ctypes.c_int32), ("table_stride", ctypes.c_int32),
                ("release_every", ctypes.c_int32)]


class _Cache(ctypes.Structure):
    _fields_ = [("k_pool", ctypes.c_void_p), ("v_pool", ctypes.c_void_p), ("num_pages", ctypes.c_int64),
                ("block_table", ctypes.c_void_p), ("table_stride", ctypes.c_int32)]


_lib = None


def load():
    """Load libhswa.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2607_13095_amd.build_lib`")
    # torch first: its HIP runtime must be the one the library binds to, so that
    # streams and device pointers are shared (loading the library first would
    # bring in a second HIP runtime next to torch's own copy).
    import torch  # noqa: F401

    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    LP, SP, CP = _Layer, ctypes.POINTER(_Shape), ctypes.POINTER(_Cache)
    sig = {
        "hswa_ring_pages": (I32, [I32, I32]),
        "hswa_page_bytes": (I64, [SP]),
        "hswa_build_block_table": (ctypes.c_int, [LP, I32, I32, P, P, I64, P, I32]),
        "hswa_kv_append": (ctypes.c_int, [LP, SP, CP, P, P, P, P, I32, I32, P, P]),
        "hswa_prefill": (ctypes.c_int, [LP, SP, CP, P, P, P, P, P, I32, I32, I32, P, P]),
        "hswa_decode_workspace_bytes": (SZ, [SP, I32, I32]),
        "hswa_decode_split_len": (I32, [SP, I32, I32]),
        "hswa_decode": (ctypes.c_int, [LP, SP, CP, P, P, I32, I32, P, SZ, P, P]),
        "hswa_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "hswa_decode_multi_workspace_bytes": (SZ, [SP, I32, I32, I32]),
        "hswa_decode_multi": (ctypes.c_int, [LP, SP, CP, P, P, I32, I32, I32, P, SZ, P, P]),
        "hswa_decode_noalloc": (ctypes.c_int, [LP, SP, CP, P, P, I32, I32, P, P]),
        "hswa_decode_append": (ctypes.c_int, [LP, SP, CP, P, P, P, P, I32, I32, P, SZ, P, P]),
        "hswa_allocator_create": (ctypes.c_int, [ctypes.POINTER(_AllocConfig), ctypes.POINTER(P)]),
        "hswa_allocator_destroy": (None, [P]),
        "hswa_allocator_admit": (ctypes.c_int, [P, I32, I64, I32]),
        "hswa_allocator_extend": (ctypes.c_int, [P, I32, I64]),
        "hswa_allocator_step_end": (ctypes.c_int, [P, I32, I32, P]),
        "hswa_allocator_free": (ctypes.c_int, [P, I32]),
        "hswa_allocator_tables": (ctypes.c_int, [P, P, P]),
        "hswa_allocator_usage": (ctypes.c_int, [P, I32, P, P, P, P]),
        "hswa_prefix_tree_create": (ctypes.c_int, [I32, ctypes.POINTER(P)]),
        "hswa_prefix_tree_destroy": (None, [P]),
        "hswa_prefix_tree_insert": (ctypes.c_int, [P, P, I64, P, P]),
        "hswa_prefix_tree_match": (ctypes.c_int, [P, P, I64, P, P, P, P]),
        "hswa_prefix_tree_release_swa": (ctypes.c_int, [P, P, I64, I64, P]),
        "hswa_prefix_tree_evict": (ctypes.c_int, [P, P, I64, I64, P]),
        "hswa_prefix_tree_stats": (ctypes.c_int, [P, P, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    _lib = lib
    return lib


# ---------------------------------------------------------------------------
# argument objects
# ---------------------------------------------------------------------------

class Layer:
    """Layer-kind flag {SWA(W), FULL}; "swa_paged" is an SWA layer over an
    explicit-release (FULL-indexed) SWA block table from ``Allocator``."""

    _KINDS = {"full": HSWA_LAYER_FULL, "swa": HSWA_LAYER_SWA, "swa_paged": HSWA_LAYER_SWA_PAGED}

    def __init__(self, kind: str, window: int = 0):
        if kind not in self._KINDS:
            raise ValueError(kind)
        self.kind, self.window = kind, int(window)

    @classmethod
    def full(cls):
        return cls("full")

    @classmethod
    def swa(cls, window: int):
        return cls("swa", window)

    @classmethod
    def swa_paged(cls, window: int):
        return cls("swa_paged", window)

    def c(self):
        key = (self.kind, self.window)
        if getattr(self, "_ck", None) != key:
            self._c, self._ck = _Layer(self._KINDS[self.kind], self.window), key
        return self._c


class Shape:
    def __init__(self, num_q_heads, num_kv_heads, head_dim=128, page_size=64, scale=None):
        self.num_q_heads, self.num_kv_heads = int(num_q_heads), int(num_kv_heads)
        self.head_dim, self.page_size = int(head_dim), int(page_size)
        self.scale = float(1.0 / np.sqrt(head_dim) if scale is None else scale)

    def c(self):
        key = (self.num_q_heads, self.num_kv_heads, self.head_dim, self.page_size, self.scale)
        if getattr(self, "_ck", None) != key:
            self._c, self._ck = _Shape(*key), key
        return self._c


def _ptr(t, name, dtypes, numel=None):
    torch = _torch()
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must live on the GPU")
    if t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype} not in {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, needs {numel}")
    return t.data_ptr()


_TORCH = None


def _torch():
    global _TORCH
    if _TORCH is None:
        import torch

        _TORCH = torch
    return _TORCH


def _bf16():
    return (_torch().bfloat16,)


def _i32():
    return (_torch().int32,)


V_BLOCK_MAX = 32


def v_block(page_size: int) -> int:
    """Keys per transposed V block: VB = min(PG, 32)."""
    return min(int(page_size), V_BLOCK_MAX)


def v_pool_shape(num_pages: int, num_kv_heads: int, page_size: int, head_dim: int = 128):
    vb = v_block(page_size)
    return (int(num_pages), int(num_kv_heads), int(page_size) // vb, int(head_dim), vb)


def k_pool_shape(num_pages: int, num_kv_heads: int, page_size: int, head_dim: int = 128):
    """[num_pages, Hkv, PG/B, 2, D/32, 4, B/2, 8] with B = min(PG, 32): per block
    of B keys, two halves (in-block offset bit 2 clear / set) of D/32 slabs of
    [4 dim pieces][B/2 keys][8 dims] (the element order is in include/hswa.h)."""
    b = v_block(page_size)
    return (int(num_pages), int(num_kv_heads), int(page_size) // b, 2, int(head_dim) // 32, 4, b // 2, 8)


class Cache:
    """One layer's K pool, V pool and block table (device tensors).

    k_pool: bf16 k_pool_shape(num_pages, Hkv, PG, D); v_pool: bf16
    [num_pages, Hkv, PG/B, D, B] with B = min(PG, 32) (see include/hswa.h);
    block_table: int32 [ns, stride].
    """

    def __init__(self, k_pool, v_pool, block_table):
        if k_pool.dim() != 8 or v_pool.dim() != 5 or block_table.dim() != 2:
            raise ValueError("k_pool is 8-D, v_pool 5-D, the block table 2-D")
        npg, hkv, d, vb = v_pool.shape[0], v_pool.shape[1], v_pool.shape[3], v_pool.shape[4]
        pg = v_pool.shape[2] * vb
        if tuple(v_pool.shape) != v_pool_shape(npg, hkv, pg, d):
            raise ValueError("v_pool must be [num_pages, Hkv, PG/B, D, B] with B = min(PG, 32)")
        if tuple(k_pool.shape) != k_pool_shape(npg, hkv, pg, d):
            raise ValueError("k_pool must be k_pool_shape(num_pages, Hkv, PG, D)")
        self.k_pool, self.v_pool, self.block_table = k_pool, v_pool, block_table
        self.num_pages, self.stride = int(npg), int(block_table.shape[1])

    def c(self):
        # the tensors are fixed at construction: the struct is built (and the
        # tensors checked) once
        if getattr(self, "_c", None) is None:
            self._c = _Cache(_ptr(self.k_pool, "k_pool", _bf16()), _ptr(self.v_pool, "v_pool", _bf16()),
                             self.num_pages, _ptr(self.block_table, "block_table", _i32()), self.stride)
        return self._c


def _check_cache(shape: Shape, cache: Cache, ns: int):
    """The pools and the table must match the shape the kernels are told."""
    key = (shape.num_kv_heads, shape.page_size, shape.head_dim, ns)
    if getattr(cache, "_checked", None) == key:
        return
    v = cache.v_pool.shape
    if int(v[1]) != shape.num_kv_heads:
        raise ValueError(f"pools hold {int(v[1])} KV heads, shape says {shape.num_kv_heads}")
    if int(v[2]) * int(v[4]) != shape.page_size:
        raise ValueError(f"pool page size {int(v[2]) * int(v[4])} != shape page size {shape.page_size}")
    if int(v[3]) != shape.head_dim:
        raise ValueError(f"pool head dim {int(v[3])} != shape head dim {shape.head_dim}")
    if int(cache.block_table.shape[0]) < ns:
        raise ValueError(f"block table has {int(cache.block_table.shape[0])} rows for {ns} sequences")
    cache._checked = key


def _stream(stream):
    torch = _torch()
    if stream is None:
        try:  # the current stream's handle without building a Stream object
            return ctypes.c_void_p(torch._C._cuda_getCurrentRawStream(torch._C._cuda_getDevice()))
        except AttributeError:
            return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _check(status, where):
    if status != 0:
        raise HswaError(status, where)


# ---------------------------------------------------------------------------
# host helpers
# ---------------------------------------------------------------------------

def ring_pages(window: int, page_size: int) -> int:
    return int(load().hswa_ring_pages(int(window), int(page_size)))


def page_bytes(shape: Shape) -> int:
    sh = shape.c()
    return int(load().hswa_page_bytes(ctypes.byref(sh)))


def build_block_table(layer: Layer, page_size: int, final_lens: Sequence[int], perm, stride: int) -> np.ndarray:
    """Host block table int32 [ns, stride] from a page permutation."""
    lens = np.ascontiguousarray(np.asarray(final_lens, dtype=np.int32))
    perm = np.ascontiguousarray(np.asarray(perm, dtype=np.int32))
    out = np.empty((lens.size, int(stride)), dtype=np.int32)
    st = load().hswa_build_block_table(layer.c(), int(page_size), int(lens.size), lens.ctypes.data,
                                       perm.ctypes.data if perm.size else None, int(perm.size), out.ctypes.data,
                                       int(stride))
    _check(st, "hswa_build_block_table")
    return out


def decode_workspace_bytes(shape: Shape, ns: int, max_context_len: int) -> int:
    sh = shape.c()
    return int(load().hswa_decode_workspace_bytes(ctypes.byref(sh), int(ns), int(max_context_len)))


def decode_split_len(shape: Shape, ns: int, max_context_len: int) -> int:
    sh = shape.c()
    return int(load().hswa_decode_split_len(ctypes.byref(sh), int(ns), int(max_context_len)))


# ---------------------------------------------------------------------------
# device calls
# ---------------------------------------------------------------------------

def kv_append(layer: Layer, shape: Shape, cache: Cache, k_new, v_new, cu_seqlens, start_pos,
              slot_mapping_out=None, stream=None):
    """Append k_new / v_new [T, Hkv, D] (bf16) to the pools; see hswa_kv_append."""
    torch = _torch()
    ns = int(cu_seqlens.numel()) - 1
    t = int(k_new.shape[0]) if k_new.dim() else 0
    row = shape.num_kv_heads * shape.head_dim
    args = (_ptr(k_new, "k_new", _bf16(), t * row), _ptr(v_new, "v_new", _bf16(), t * row),
            _ptr(cu_seqlens, "cu_seqlens", _i32(), ns + 1), _ptr(start_pos, "start_pos", _i32(), ns))
    slots = _ptr(slot_mapping_out, "slot_mapping_out", (torch.int64,), t) if slot_mapping_out is not None else None
    _check_cache(shape, cache, ns)
    sh, ca = shape.c(), cache.c()
    st = load().hswa_kv_append(layer.c(), ctypes.byref(sh), ctypes.byref(ca), *args, ns, t, slots, _stream(stream))
    _check(st, "hswa_kv_append")


def prefill(layer: Layer, shape: Shape, cache: Cache, q, k_new, v_new, cu_seqlens, prefix_lens,
            max_chunk_len: int, out, stream=None):
    """Chunked prefill; q, out [T, Hq, D], k_new / v_new [T, Hkv, D]; see hswa_prefill."""
    ns = int(cu_seqlens.numel()) - 1
    t = int(q.shape[0])
    qrow, krow = shape.num_q_heads * shape.head_dim, shape.num_kv_heads * shape.head_dim
    args = (_ptr(q, "q", _bf16(), t * qrow), _ptr(k_new, "k_new", _bf16(), t * krow),
            _ptr(v_new, "v_new", _bf16(), t * krow), _ptr(cu_seqlens, "cu_seqlens", _i32(), ns + 1),
            _ptr(prefix_lens, "prefix_lens", _i32(), ns))
    o = _ptr(out, "out", _bf16(), t * qrow)
    _check_cache(shape, cache, ns)
    sh, ca = shape.c(), cache.c()
    st = load().hswa_prefill(layer.c(), ctypes.byref(sh), ctypes.byref(ca), *args, ns, t, int(max_chunk_len), o,
                             _stream(stream))
    _check(st, "hswa_prefill")


def decode_multi_workspace_bytes(shape: Shape, ns: int, num_queries: int, max_context_len: int) -> int:
    sh = shape.c()
    return int(load().hswa_decode_multi_workspace_bytes(ctypes.byref(sh), int(ns), int(num_queries),
                                                        int(max_context_len)))


def decode_multi(layer: Layer, shape: Shape, cache: Cache, q, context_lens, max_context_len: int, out,
                 workspace=None, stream=None):
    """Multi-query decode; q, out [NS, nq, Hq, D]; see hswa_decode_multi."""
    torch = _torch()
    if q.dim() != 4:
        raise ValueError("q must be [NS, num_queries, Hq, D]")
    ns, nq = int(q.shape[0]), int(q.shape[1])
    if int(context_lens.numel()) != ns:
        raise ValueError("one context length per sequence")
    row = nq * shape.num_q_heads * shape.head_dim
    qp = _ptr(q, "q", _bf16(), ns * row)
    cp = _ptr(context_lens, "context_lens", _i32(), ns)
    o = _ptr(out, "out", _bf16(), ns * row)
    wp, wbytes = None, 0
    if workspace is not None:
        wp = _ptr(workspace, "workspace", (torch.uint8, torch.float32, torch.int32))
        wbytes = workspace.numel() * workspace.element_size()
    _check_cache(shape, cache, ns)
    sh, ca = shape.c(), cache.c()
    st = load().hswa_decode_multi(layer.c(), ctypes.byref(sh), ctypes.byref(ca), qp, cp, ns, nq,
                                  int(max_context_len), wp, wbytes, o, _stream(stream))
    _check(st, "hswa_decode_multi")


def decode(layer: Layer, shape: Shape, cache: Cache, q, context_lens, max_context_len: int, out,
           workspace=None, stream=None):
    """Decode one query per sequence; q, out [NS, Hq, D]; see hswa_decode."""
    torch = _torch()
    ns = int(context_lens.numel())
    qrow = shape.num_q_heads * shape.head_dim
    qp = _ptr(q, "q", _bf16(), ns * qrow)
    cp = _ptr(context_lens, "context_lens", _i32(), ns)
    o = _ptr(out, "out", _bf16(), ns * qrow)
    wp, wbytes = None, 0
    if workspace is not None:
        wp = _ptr(workspace, "workspace", (torch.uint8, torch.float32, torch.int32))
        wbytes = workspace.numel() * workspace.element_size()
    _check_cache(shape, cache, ns)
    sh, ca = shape.c(), cache.c()
    st = load().hswa_decode(layer.c(), ctypes.byref(sh), ctypes.byref(ca), qp, cp, ns, int(max_context_len), wp,
                            wbytes, o, _stream(stream))
    _check(st, "hswa_decode")


def decode_append(layer: Layer, shape: Shape, cache: Cache, q, k_new, v_new, context_lens, max_context_len: int,
                  out, workspace=None, stream=None):
    """One decode step: store every sequence's new token (k_new / v_new
    [NS, Hkv, D]) at position context_lens[b] - 1, then decode q [NS, Hq, D]
    there; see hswa_decode_append."""
    torch = _torch()
    ns = int(context_lens.numel())
    qrow, krow = shape.num_q_heads * shape.head_dim, shape.num_kv_heads * shape.head_dim
    qp = _ptr(q, "q", _bf16(), ns * qrow)
    kp = _ptr(k_new, "k_new", _bf16(), ns * krow)
    vp = _ptr(v_new, "v_new", _bf16(), ns * krow)
    cp = _ptr(context_lens, "context_lens", _i32(), ns)
    o = _ptr(out, "out", _bf16(), ns * qrow)
    wp, wbytes = None, 0
    if workspace is not None:
        wp = _ptr(workspace, "workspace", (torch.uint8, torch.float32, torch.int32))
        wbytes = workspace.numel() * workspace.element_size()
    _check_cache(shape, cache, ns)
    sh, ca = shape.c(), cache.c()
    st = load().hswa_decode_append(layer.c(), ctypes.byref(sh), ctypes.byref(ca), qp, kp, vp, cp, ns,
                                   int(max_context_len), wp, wbytes, o, _stream(stream))
    _check(st, "hswa_decode_append")


def decode_noalloc(layer: Layer, shape: Shape, cache: Cache, q, context_lens, max_context_len: int, out,
                   stream=None):
    """Decode without a workspace (the library's fixed device array holds the
    split partials); q, out [NS, Hq, D]; see hswa_decode_noalloc."""
    ns = int(context_lens.numel())
    qrow = shape.num_q_heads * shape.head_dim
    qp = _ptr(q, "q", _bf16(), ns * qrow)
    cp = _ptr(context_lens, "context_lens", _i32(), ns)
    o = _ptr(out, "out", _bf16(), ns * qrow)
    _check_cache(shape, cache, ns)
    sh, ca = shape.c(), cache.c()
    st = load().hswa_decode_noalloc(layer.c(), ctypes.byref(sh), ctypes.byref(ca), qp, cp, ns, int(max_context_len),
                                    o, _stream(stream))
    _check(st, "hswa_decode_noalloc")


# ---------------------------------------------------------------------------
# explicit-release dual-pool allocator (host object)
# ---------------------------------------------------------------------------

class Allocator:
    """Host page allocator of one FULL pool and one SWA pool (see
    hswa_allocator_* in include/hswa.h); tables come back as numpy int32."""

    def __init__(self, page_size, window, full_pages, swa_pages, max_seqs, table_stride, release_every=1):
        self._lib = load()
        self.cfg = _AllocConfig(int(page_size), int(window), int(full_pages), int(swa_pages), int(max_seqs),
                                int(table_stride), int(release_every))
        h = ctypes.c_void_p()
        _check(self._lib.hswa_allocator_create(ctypes.byref(self.cfg), ctypes.byref(h)), "hswa_allocator_create")
        self._h = h

    def close(self):
        if self._h:
            self._lib.hswa_allocator_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def admit(self, seq, length, chunk):
        """Returns the status (0 = admitted, HSWA_ERR_CAPACITY = -3 = a pool is short)."""
        return int(self._lib.hswa_allocator_admit(self._h, int(seq), int(length), int(chunk)))

    def extend(self, seq, new_len):
        return int(self._lib.hswa_allocator_extend(self._h, int(seq), int(new_len)))

    def step_end(self, seq, decode_step):
        n = ctypes.c_int32(0)
        _check(self._lib.hswa_allocator_step_end(self._h, int(seq), int(bool(decode_step)), ctypes.byref(n)),
               "hswa_allocator_step_end")
        return int(n.value)

    def free(self, seq):
        _check(self._lib.hswa_allocator_free(self._h, int(seq)), "hswa_allocator_free")

    def tables(self):
        ns, st = self.cfg.max_seqs, self.cfg.table_stride
        full = np.empty((ns, st), dtype=np.int32)
        swa = np.empty((ns, st), dtype=np.int32)
        _check(self._lib.hswa_allocator_tables(self._h, full.ctypes.data, swa.ctypes.data), "hswa_allocator_tables")
        return full, swa

    def usage(self, seq=-1):
        """(full_used, swa_used, full_free, swa_free) for one sequence or all."""
        v = [ctypes.c_int64(0) for _ in range(4)]
        _check(self._lib.hswa_allocator_usage(self._h, int(seq), *[ctypes.byref(x) for x in v]),
               "hswa_allocator_usage")
        return tuple(int(x.value) for x in v)


# ---------------------------------------------------------------------------
# window-safe prefix cache tree (host object)
# ---------------------------------------------------------------------------

def _i32_arr(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def _i64_arr(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.int64))


class PrefixTree:
    """Radix tree with per-token FULL and SWA slots (hswa_prefix_tree_*)."""

    def __init__(self, window):
        self._lib = load()
        h = ctypes.c_void_p()
        _check(self._lib.hswa_prefix_tree_create(int(window), ctypes.byref(h)), "hswa_prefix_tree_create")
        self._h, self.window = h, int(window)

    def close(self):
        if self._h:
            self._lib.hswa_prefix_tree_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def insert(self, tokens, full_slots, swa_slots):
        t, f, s = _i32_arr(tokens), _i64_arr(full_slots), _i64_arr(swa_slots)
        if not (t.size == f.size == s.size):
            raise ValueError("one slot per token")
        _check(self._lib.hswa_prefix_tree_insert(self._h, t.ctypes.data, t.size, f.ctypes.data, s.ctypes.data),
               "hswa_prefix_tree_insert")

    def match(self, tokens):
        """(full_len, safe_len, full_slots[:full_len], swa_slots[:full_len])."""
        t = _i32_arr(tokens)
        fo = np.full(max(1, t.size), -2, dtype=np.int64)
        so = np.full(max(1, t.size), -2, dtype=np.int64)
        fl, sl = ctypes.c_int64(0), ctypes.c_int64(0)
        _check(self._lib.hswa_prefix_tree_match(self._h, t.ctypes.data, t.size, ctypes.byref(fl), ctypes.byref(sl),
                                                fo.ctypes.data, so.ctypes.data), "hswa_prefix_tree_match")
        n = int(fl.value)
        return n, int(sl.value), fo[:n].copy(), so[:n].copy()

    def release_swa(self, tokens, upto):
        t = _i32_arr(tokens)
        r = ctypes.c_int64(0)
        _check(self._lib.hswa_prefix_tree_release_swa(self._h, t.ctypes.data, t.size, int(upto), ctypes.byref(r)),
               "hswa_prefix_tree_release_swa")
        return int(r.value)

    def evict(self, tokens, keep):
        t = _i32_arr(tokens)
        r = ctypes.c_int64(0)
        _check(self._lib.hswa_prefix_tree_evict(self._h, t.ctypes.data, t.size, int(keep), ctypes.byref(r)),
               "hswa_prefix_tree_evict")
        return int(r.value)

    def stats(self):
        """(nodes, cached tokens, tokens with a valid SWA slot)."""
        v = [ctypes.c_int64(0) for _ in range(3)]
        _check(self._lib.hswa_prefix_tree_stats(self._h, *[ctypes.byref(x) for x in v]), "hswa_prefix_tree_stats")
        return tuple(int(x.value) for x in v)
