"""CPU oracle for the paged-KV host<->pool transfer (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline leg
may import this package.  It wraps ``kvoracle.c`` (plain C99 loops, one memcpy
per token row) through ctypes and shares nothing with the HIP path.

Strata, Sec. 4.2 and Sec. 4.2.1 (Fig. 6): a GPU-assisted I/O job moves each
small chunk from a source to a destination, and converting between the
transfer-friendly host layout and the layer-first paged pool costs one extra
offset computation per chunk.  With R = row bytes, P = page size:

    slot(t)  = page_idx[t // P] * P + t % P
    host row = ((layer * 2 + kv) * host_tokens + t) * R      (kv: 0 = K, 1 = V)
    load:    pool[kv][layer][slot(t)] = host row;   offload: the inverse.

Pool images are numpy ``uint8`` arrays shaped ``(L, S, R)`` (one for K, one for
V, or one ``(2, L, S, R)`` array); host chunks are flat ``uint8`` arrays of at
least ``L * 2 * host_tokens * R`` bytes.  Parity is pinned by the tests in
``tests/test_oracle_pins.py`` (identity table, numpy fancy indexing, brute
force by the inverse mapping, round trip, sentinels, hand-worked example).
"""
from __future__ import annotations

import ctypes
import os
from typing import Iterable, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# KVO_ORACLE_LIB lets the pin tests run against a deliberately broken copy
# of the oracle (to show that the pins catch plausible mistakes).
_LIB_PATH = os.environ.get("KVO_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

TOKEN_MAJOR = 0
PAGE_FIRST = 1
HEAD_MAJOR = 2

OK = 0
EINVAL = -1
ERANGE = -2
EDUP = -3
ENOMEM = -4
_NAMES = {EINVAL: "EINVAL", ERANGE: "ERANGE", EDUP: "EDUP", ENOMEM: "ENOMEM"}


class OracleError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"oracle {what} failed: {_NAMES.get(code, code)}")
        self.code = code


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        if _LIB_PATH != _b.LIB:
            raise FileNotFoundError(_LIB_PATH)
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    i32, i64, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
    lib.kvo_host_row_offset.restype = i64
    lib.kvo_host_row_offset.argtypes = [i32, i32, i64, i64, i64]
    lib.kvo_expand_slots.restype = ctypes.c_int
    lib.kvo_expand_slots.argtypes = [vp, i32, i64, i64, vp]
    for name in ("kvo_load_slab", "kvo_offload_slab"):
        f = getattr(lib, name)
        f.restype = ctypes.c_int
        f.argtypes = [vp, i64, i32, i64, vp, i64, vp]
    for name in ("kvo_load_batch", "kvo_offload_batch"):
        f = getattr(lib, name)
        f.restype = ctypes.c_int
        f.argtypes = [vp, vp, i32, i64, i32, i64, i32, vp, vp, vp, vp, i32, i32]
    for name in ("kvo_load_layout", "kvo_offload_layout"):
        f = getattr(lib, name)
        f.restype = ctypes.c_int
        f.argtypes = [vp, vp, i32, i64, i32, i64, i32, i32, i32, vp, vp, vp, vp, i32, i32]
    lib.kvo_host_row_offset_page_first.restype = i64
    lib.kvo_host_row_offset_page_first.argtypes = [i32, i32, i32, i32, i64, i64]
    lib.kvo_host_seg_offset_head_major.restype = i64
    lib.kvo_host_seg_offset_head_major.argtypes = [i32, i32, i32, i32, i64, i64, i64]
    _lib = lib
    return lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _check(rc: int, what: str) -> None:
    if rc != OK:
        raise OracleError(rc, what)


def host_row_offset(layer: int, kv: int, host_tokens: int, token: int, row_bytes: int) -> int:
    """Byte offset of host row (layer, kv, token) in a layer-major chunk."""
    return int(_load().kvo_host_row_offset(layer, kv, host_tokens, token, row_bytes))


def host_row_offset_page_first(layer: int, kv: int, num_layers: int, page_size: int, token: int,
                               row_bytes: int) -> int:
    """Byte offset of host row (layer, kv, token) in a page-first chunk."""
    return int(_load().kvo_host_row_offset_page_first(layer, kv, num_layers, page_size, token, row_bytes))


def host_seg_offset_head_major(layer: int, kv: int, head: int, num_heads: int, host_tokens: int, token: int,
                               seg_bytes: int) -> int:
    """Byte offset of head `head` of row (layer, kv, token) in a head-major chunk."""
    return int(_load().kvo_host_seg_offset_head_major(layer, kv, head, num_heads, host_tokens, token,
                                                        seg_bytes))


def host_chunk_bytes(layout: int, num_layers: int, host_tokens: int, row_bytes: int, page_size: int) -> int:
    """Bytes of one context's host chunk in a layout."""
    if layout == PAGE_FIRST:
        return -(-host_tokens // page_size) * page_size * num_layers * 2 * row_bytes
    return num_layers * 2 * host_tokens * row_bytes


def expand_slots(page_idx: np.ndarray, page_size: int, num_tokens: int, num_slots: int) -> np.ndarray:
    """Pool slot of each context token t < num_tokens (page-offset expansion)."""
    pidx = np.ascontiguousarray(page_idx, dtype=np.int32)
    out = np.empty(max(num_tokens, 0), dtype=np.int64)
    rc = _load().kvo_expand_slots(_ptr(pidx), page_size, num_tokens, num_slots, _ptr(out))
    _check(rc, "expand_slots")
    return out


def load_slab(pool_slab: np.ndarray, page_size: int, host_slab: np.ndarray,
              num_tokens: int, page_idx: np.ndarray) -> None:
    """One (layer, kv) slab: pool_slab is (S, R) uint8, host_slab rows t = 0.."""
    assert pool_slab.dtype == np.uint8 and pool_slab.ndim == 2 and pool_slab.flags.c_contiguous
    assert host_slab.dtype == np.uint8 and host_slab.flags.c_contiguous
    assert host_slab.size >= num_tokens * pool_slab.shape[1]
    pidx = np.ascontiguousarray(page_idx, dtype=np.int32)
    rc = _load().kvo_load_slab(_ptr(pool_slab), pool_slab.shape[0], page_size, pool_slab.shape[1],
                               _ptr(host_slab), num_tokens, _ptr(pidx))
    _check(rc, "load_slab")


def offload_slab(pool_slab: np.ndarray, page_size: int, host_slab: np.ndarray,
                 num_tokens: int, page_idx: np.ndarray) -> None:
    assert pool_slab.dtype == np.uint8 and pool_slab.ndim == 2 and pool_slab.flags.c_contiguous
    assert host_slab.dtype == np.uint8 and host_slab.flags.c_contiguous
    assert host_slab.size >= num_tokens * pool_slab.shape[1]
    pidx = np.ascontiguousarray(page_idx, dtype=np.int32)
    rc = _load().kvo_offload_slab(_ptr(pool_slab), pool_slab.shape[0], page_size, pool_slab.shape[1],
                                  _ptr(host_slab), num_tokens, _ptr(pidx))
    _check(rc, "offload_slab")


Span = Tuple[np.ndarray, int, int, np.ndarray]   # (host uint8, host_tokens, num_tokens, page_idx)


def _layer_ptrs(pool: np.ndarray):
    assert pool.dtype == np.uint8 and pool.ndim == 3 and pool.flags.c_contiguous
    return (ctypes.c_void_p * pool.shape[0])(*[_ptr(pool[i]) for i in range(pool.shape[0])])


def _batch(fn, k_pool, v_pool, page_size, spans: Sequence[Span], layer_begin, layer_end, what,
           layout=None, num_heads=1):
    assert k_pool.shape == v_pool.shape
    num_layers, num_slots, row_bytes = k_pool.shape
    n = len(spans)
    keep = []
    hosts = (ctypes.c_void_p * max(n, 1))()
    pidxs = (ctypes.c_void_p * max(n, 1))()
    htok = np.zeros(max(n, 1), dtype=np.int64)
    ntok = np.zeros(max(n, 1), dtype=np.int64)
    for i, (host, host_tokens, num_tokens, page_idx) in enumerate(spans):
        assert host.dtype == np.uint8 and host.flags.c_contiguous
        assert host.size >= host_chunk_bytes(layout or TOKEN_MAJOR, num_layers, host_tokens, row_bytes, page_size)
        p = np.ascontiguousarray(page_idx, dtype=np.int32)
        keep.append(p)
        hosts[i] = _ptr(host)
        pidxs[i] = _ptr(p) if p.size else None
        htok[i] = host_tokens
        ntok[i] = num_tokens
    if layout is None:
        rc = fn(_layer_ptrs(k_pool), _layer_ptrs(v_pool), num_layers, num_slots, page_size, row_bytes,
                n, hosts, _ptr(htok), _ptr(ntok), pidxs, layer_begin, layer_end)
    else:
        rc = fn(_layer_ptrs(k_pool), _layer_ptrs(v_pool), num_layers, num_slots, page_size, row_bytes,
                num_heads, layout, n, hosts, _ptr(htok), _ptr(ntok), pidxs, layer_begin, layer_end)
    _check(rc, what)


def load(k_pool: np.ndarray, v_pool: np.ndarray, page_size: int, spans: Iterable[Span],
         layer_begin: int = 0, layer_end: int | None = None) -> None:
    """Load host chunks into the (L, S, R) K and V pool images, in place."""
    layer_end = k_pool.shape[0] if layer_end is None else layer_end
    _batch(_load().kvo_load_batch, k_pool, v_pool, page_size, list(spans), layer_begin, layer_end, "load")


def offload(k_pool: np.ndarray, v_pool: np.ndarray, page_size: int, spans: Iterable[Span],
            layer_begin: int = 0, layer_end: int | None = None) -> None:
    """Offload pool rows into the host chunks, in place."""
    layer_end = k_pool.shape[0] if layer_end is None else layer_end
    _batch(_load().kvo_offload_batch, k_pool, v_pool, page_size, list(spans), layer_begin, layer_end,
           "offload")


def load_layout(k_pool: np.ndarray, v_pool: np.ndarray, page_size: int, spans: Iterable[Span], layout: int,
                num_heads: int = 1, layer_begin: int = 0, layer_end: int | None = None) -> None:
    """Load host chunks in any layout (TOKEN_MAJOR, PAGE_FIRST, HEAD_MAJOR)."""
    layer_end = k_pool.shape[0] if layer_end is None else layer_end
    _batch(_load().kvo_load_layout, k_pool, v_pool, page_size, list(spans), layer_begin, layer_end,
           "load_layout", layout, num_heads)


def offload_layout(k_pool: np.ndarray, v_pool: np.ndarray, page_size: int, spans: Iterable[Span], layout: int,
                   num_heads: int = 1, layer_begin: int = 0, layer_end: int | None = None) -> None:
    """Offload into host chunks in any layout."""
    layer_end = k_pool.shape[0] if layer_end is None else layer_end
    _batch(_load().kvo_offload_layout, k_pool, v_pool, page_size, list(spans), layer_begin, layer_end,
           "offload_layout", layout, num_heads)


def load_layout_layer(k_slab: np.ndarray, v_slab: np.ndarray, page_size: int, spans: Iterable[Span], layout: int,
                      num_layers: int, layer: int, num_heads: int = 1) -> None:
    """One layer of load_layout: loads layer `layer` of each span's chunk (a
    context of num_layers layers in any layout) into the (S, R) K and V slab
    images of that layer, in place.  The same C routine as load_layout, run
    over the layer range [layer, layer + 1) with every layer's pool pointer
    aimed at the two slabs; only `layer` is touched, so a whole-pool check can
    build its expected image one layer at a time."""
    assert k_slab.shape == v_slab.shape and k_slab.ndim == 2
    for sl in (k_slab, v_slab):
        assert sl.dtype == np.uint8 and sl.flags.c_contiguous
    num_slots, row_bytes = k_slab.shape
    spans = list(spans)
    n = len(spans)
    keep = []
    hosts = (ctypes.c_void_p * max(n, 1))()
    pidxs = (ctypes.c_void_p * max(n, 1))()
    htok = np.zeros(max(n, 1), dtype=np.int64)
    ntok = np.zeros(max(n, 1), dtype=np.int64)
    for i, (host, host_tokens, num_tokens, page_idx) in enumerate(spans):
        assert host.dtype == np.uint8 and host.flags.c_contiguous
        assert host.size >= host_chunk_bytes(layout, num_layers, host_tokens, row_bytes, page_size)
        p = np.ascontiguousarray(page_idx, dtype=np.int32)
        keep.append(p)
        hosts[i] = _ptr(host)
        pidxs[i] = _ptr(p) if p.size else None
        htok[i] = host_tokens
        ntok[i] = num_tokens
    kp = (ctypes.c_void_p * num_layers)(*([_ptr(k_slab)] * num_layers))
    vp = (ctypes.c_void_p * num_layers)(*([_ptr(v_slab)] * num_layers))
    rc = _load().kvo_load_layout(kp, vp, num_layers, num_slots, page_size, row_bytes, num_heads, layout, n, hosts,
                                 _ptr(htok), _ptr(ntok), pidxs, layer, layer + 1)
    _check(rc, "load_layout_layer")
