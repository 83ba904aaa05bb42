"""ctypes binding of libkvio.so (include/kvio.h), argument marshalling only.

Every transfer step runs in the HIP kernels of libkvio.so; this module only
packs arguments.  Importing it loads torch first so that libkvio.so binds to
the same HIP runtime as torch (device memory and streams come from torch).
There is no fallback: if the library is missing or fails to load, importing
this module raises.

Names follow the C ABI (kvio_load, kvio_offload, kvio_load_layer, ...).
Pointers are Python ints (``tensor.data_ptr()``); streams are
``torch.cuda.Stream`` objects, raw ``hipStream_t`` ints, or None (the default
stream); events are ``torch.cuda.Event`` objects or raw ints (a torch event
that was never recorded has no HIP event yet; it is recorded once on the
current stream first, then by the library after its launch).
"""
from __future__ import annotations

import ctypes
import os
from typing import Iterable, Optional, Sequence, Tuple, Union

import numpy as np
import torch  # noqa: F401  (binds the HIP runtime before libkvio.so loads)

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libkvio.so")

# kvio_status
KVIO_OK = 0
KVIO_EINVAL = -1
KVIO_ERANGE = -2
KVIO_EALIGN = -3
KVIO_ENOTMAPPED = -4
KVIO_EHIP = -5
KVIO_ENOMEM = -6
KVIO_EIO = -7

# host chunk layouts
KVIO_HOST_TOKEN_MAJOR = 0
KVIO_HOST_PAGE_FIRST = 1
KVIO_HOST_HEAD_MAJOR = 2
# launch flags
KVIO_LAUNCH_CACHED = 0x1
KVIO_LAUNCH_NO_LDS = 0x2
KVIO_LAUNCH_STAGED = 0x4
# disk store layouts
KVIO_DISK_PAGE_FIRST = 0
KVIO_DISK_LAYER_FIRST = 1
# pinned host memory flags
KVIO_HOST_COHERENT = 0x0
KVIO_HOST_NONCOHERENT = 0x1
KVIO_MAX_SPANS_PER_LAUNCH = 64
KVIO_NOALLOC_MAX_LAYERS = 128


class kvio_launch(ctypes.Structure):
    _fields_ = [("workgroups", ctypes.c_int32), ("threads", ctypes.c_int32),
                ("tile_kib", ctypes.c_int32), ("flags", ctypes.c_int32)]


class kvio_pool_desc(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("elem_bytes", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("host_layout", ctypes.c_int32),
                ("num_slots", ctypes.c_int64),
                ("k_layers", ctypes.POINTER(ctypes.c_void_p)),
                ("v_layers", ctypes.POINTER(ctypes.c_void_p)),
                ("load_launch", kvio_launch), ("offload_launch", kvio_launch),
                ("staging_bytes", ctypes.c_int64)]


class kvio_span(ctypes.Structure):
    _fields_ = [("host", ctypes.c_void_p), ("host_tokens", ctypes.c_int64),
                ("num_tokens", ctypes.c_int64), ("page_idx", ctypes.c_void_p)]


class kvio_request(ctypes.Structure):
    _fields_ = [("load_tokens", ctypes.c_int64), ("compute_tokens", ctypes.c_int64),
                ("context", ctypes.c_int64), ("transient_matches", ctypes.c_int64)]


class kvio_batch_policy(ctypes.Structure):
    _fields_ = [("max_tokens", ctypes.c_int64), ("max_requests", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("loading_bound_ratio", ctypes.c_double),
                ("delay_hit_threshold", ctypes.c_int64)]


class kvio_disk_store(ctypes.Structure):
    _fields_ = [("fd", ctypes.c_int32), ("disk_layout", ctypes.c_int32), ("num_disk_pages", ctypes.c_int64),
                ("num_layers", ctypes.c_int32), ("page_size", ctypes.c_int32), ("row_bytes", ctypes.c_int64)]


class KvioError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{kvio_strerror(status)}: {detail}")
        self.status = status
        self.detail = detail


def _load_library() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "(or python paper_2508_18572_amd/_build.py)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, st = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_int
    sig = {
        "kvio_pool_create": [ctypes.POINTER(kvio_pool_desc), ctypes.POINTER(vp)],
        "kvio_pool_destroy": [vp],
        "kvio_load": [vp, ctypes.POINTER(kvio_span), i32, i32, i32, vp],
        "kvio_offload": [vp, ctypes.POINTER(kvio_span), i32, i32, i32, vp],
        "kvio_load_layer": [vp, ctypes.POINTER(kvio_span), i32, i32, vp, vp],
        "kvio_check": [vp],
        "kvio_naive_load": [vp, ctypes.POINTER(kvio_span), i32, i32, i32, vp],
        "kvio_naive_offload": [vp, ctypes.POINTER(kvio_span), i32, i32, i32, vp],
        "kvio_memcpy": [vp, vp, ctypes.c_size_t, vp],
        "kvio_kernel_memcpy": [vp, vp, ctypes.c_size_t, vp],
        "kvio_host_alloc": [ctypes.c_size_t, ctypes.c_uint32, ctypes.POINTER(vp)],
        "kvio_host_free": [vp],
        "kvio_stream_create": [ctypes.POINTER(ctypes.c_uint32), ctypes.c_uint32, ctypes.POINTER(vp)],
        "kvio_stream_destroy": [vp],
        "kvio_disk_prefetch": [ctypes.POINTER(kvio_disk_store), ctypes.POINTER(i64), i32, vp, i64, i32, i32],
        "kvio_disk_store_pages": [ctypes.POINTER(kvio_disk_store), ctypes.POINTER(i64), i32, vp, i64, i32, i32],
        "kvio_disk_prefetch_start": [ctypes.POINTER(kvio_disk_store), ctypes.POINTER(i64), i32, vp, i64, i32, i32,
                                     ctypes.POINTER(vp)],
        "kvio_disk_prefetch_progress": [vp, ctypes.POINTER(i32)],
        "kvio_disk_prefetch_finish": [vp, i32, ctypes.POINTER(ctypes.c_uint8), ctypes.POINTER(i32)],
        "kvio_load_noalloc": [ctypes.POINTER(kvio_pool_desc), ctypes.POINTER(kvio_span), i32, i32, i32, vp],
        "kvio_schedule_round": [ctypes.POINTER(kvio_request), i32, ctypes.POINTER(kvio_batch_policy),
                                ctypes.POINTER(i32), ctypes.POINTER(i32), ctypes.POINTER(i32),
                                ctypes.POINTER(i32)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = st
    lib.kvio_strerror.argtypes = [st]
    lib.kvio_strerror.restype = ctypes.c_char_p
    lib.kvio_last_error.argtypes = []
    lib.kvio_last_error.restype = ctypes.c_char_p
    return lib


_lib = _load_library()

# Exported symbols of the C ABI (checked by the CPU tests against include/kvio.h).
EXPORTS = ("kvio_pool_create", "kvio_pool_destroy", "kvio_load", "kvio_offload", "kvio_load_layer",
           "kvio_check", "kvio_naive_load", "kvio_naive_offload", "kvio_memcpy", "kvio_host_alloc",
           "kvio_host_free", "kvio_stream_create", "kvio_stream_destroy", "kvio_schedule_round",
           "kvio_disk_prefetch", "kvio_disk_store_pages", "kvio_disk_prefetch_start", "kvio_disk_prefetch_progress",
           "kvio_disk_prefetch_finish", "kvio_load_noalloc", "kvio_kernel_memcpy",
           "kvio_strerror", "kvio_last_error")


def kvio_strerror(status: int) -> str:
    return _lib.kvio_strerror(status).decode()


def kvio_last_error() -> str:
    return _lib.kvio_last_error().decode()


def _check(status: int) -> None:
    if status != KVIO_OK:
        raise KvioError(status, kvio_last_error())


def _stream(s) -> Optional[int]:
    if s is None:
        return None
    if isinstance(s, int):
        return s or None
    return s.cuda_stream or None


def _event(e) -> Optional[int]:
    if e is None:
        return None
    if isinstance(e, int):
        return e or None
    if not e.cuda_event:
        # torch creates the HIP event at its first record; record it once (on
        # the current stream) so that there is a handle for the library to
        # record after its launch
        e.record()
    return e.cuda_event


SpanLike = Union[kvio_span, Tuple[int, int, int, int]]


def make_spans(spans: Iterable[SpanLike]):
    """Pack spans given as kvio_span or (host_ptr, host_tokens, num_tokens, page_idx_ptr)."""
    items = list(spans)
    arr = (kvio_span * max(len(items), 1))()
    for i, sp in enumerate(items):
        if isinstance(sp, kvio_span):
            arr[i] = sp
        else:
            host, host_tokens, num_tokens, page_idx = sp
            arr[i] = kvio_span(host, host_tokens, num_tokens, page_idx)
    return arr, len(items)


def launch(workgroups: int = 0, threads: int = 0, tile_kib: int = 0, flags: int = 0) -> kvio_launch:
    return kvio_launch(workgroups, threads, tile_kib, flags)


def kvio_pool_create(num_layers: int, num_kv_heads: int, head_dim: int, elem_bytes: int,
                     page_size: int, num_slots: int, k_layers: Sequence[int], v_layers: Sequence[int],
                     load_launch: Optional[kvio_launch] = None,
                     offload_launch: Optional[kvio_launch] = None,
                     host_layout: int = KVIO_HOST_TOKEN_MAJOR, staging_bytes: int = 0) -> int:
    """Create a pool handle; k_layers / v_layers are device pointers (ints)."""
    d, _keep = pool_desc(num_layers, num_kv_heads, head_dim, elem_bytes, page_size, num_slots, k_layers, v_layers,
                         load_launch, offload_launch, host_layout, staging_bytes)
    h = ctypes.c_void_p()
    _check(_lib.kvio_pool_create(ctypes.byref(d), ctypes.byref(h)))
    return h.value


def pool_desc(num_layers: int, num_kv_heads: int, head_dim: int, elem_bytes: int, page_size: int,
              num_slots: int, k_layers: Sequence[int], v_layers: Sequence[int],
              load_launch: Optional[kvio_launch] = None, offload_launch: Optional[kvio_launch] = None,
              host_layout: int = KVIO_HOST_TOKEN_MAJOR, staging_bytes: int = 0):
    """A kvio_pool_desc; returns (desc, keep), where `keep` holds the pointer
    arrays the description points into (keep it alive while desc is used)."""
    kt = (ctypes.c_void_p * len(k_layers))(*k_layers)
    vt = (ctypes.c_void_p * len(v_layers))(*v_layers)
    d = kvio_pool_desc(num_layers, num_kv_heads, head_dim, elem_bytes, page_size, host_layout,
                       num_slots, ctypes.cast(kt, ctypes.POINTER(ctypes.c_void_p)),
                       ctypes.cast(vt, ctypes.POINTER(ctypes.c_void_p)),
                       load_launch or kvio_launch(), offload_launch or kvio_launch(), staging_bytes)
    return d, (kt, vt)


def kvio_load_noalloc(desc: "kvio_pool_desc", spans: Iterable[SpanLike], layer_begin: int, layer_end: int,
                      stream=None) -> None:
    """kvio_load from a pool description, allocating nothing (static device
    scratch shared by every call on a GPU)."""
    arr, n = make_spans(spans)
    _check(_lib.kvio_load_noalloc(ctypes.byref(desc), arr, n, layer_begin, layer_end, _stream(stream)))


def kvio_pool_destroy(pool: int) -> None:
    _check(_lib.kvio_pool_destroy(pool))


def kvio_load(pool: int, spans: Iterable[SpanLike], layer_begin: int, layer_end: int, stream=None) -> None:
    arr, n = make_spans(spans)
    _check(_lib.kvio_load(pool, arr, n, layer_begin, layer_end, _stream(stream)))


def kvio_offload(pool: int, spans: Iterable[SpanLike], layer_begin: int, layer_end: int, stream=None) -> None:
    arr, n = make_spans(spans)
    _check(_lib.kvio_offload(pool, arr, n, layer_begin, layer_end, _stream(stream)))


def kvio_load_layer(pool: int, spans: Iterable[SpanLike], layer: int, stream=None, done=None) -> None:
    arr, n = make_spans(spans)
    _check(_lib.kvio_load_layer(pool, arr, n, layer, _stream(stream), _event(done)))


def kvio_check(pool: int) -> None:
    _check(_lib.kvio_check(pool))


def kvio_naive_load(pool: int, spans: Iterable[SpanLike], layer_begin: int, layer_end: int,
                    stream=None) -> None:
    arr, n = make_spans(spans)
    _check(_lib.kvio_naive_load(pool, arr, n, layer_begin, layer_end, _stream(stream)))


def kvio_naive_offload(pool: int, spans: Iterable[SpanLike], layer_begin: int, layer_end: int,
                       stream=None) -> None:
    arr, n = make_spans(spans)
    _check(_lib.kvio_naive_offload(pool, arr, n, layer_begin, layer_end, _stream(stream)))


def kvio_memcpy(dst: int, src: int, nbytes: int, stream=None) -> None:
    _check(_lib.kvio_memcpy(dst, src, nbytes, _stream(stream)))


def kvio_kernel_memcpy(dst: int, src: int, nbytes: int, stream=None) -> None:
    _check(_lib.kvio_kernel_memcpy(dst, src, nbytes, _stream(stream)))


def kvio_host_alloc(nbytes: int, flags: int = KVIO_HOST_COHERENT) -> int:
    p = ctypes.c_void_p()
    _check(_lib.kvio_host_alloc(nbytes, flags, ctypes.byref(p)))
    return p.value


def kvio_host_free(ptr: int) -> None:
    _check(_lib.kvio_host_free(ptr))


def kvio_stream_create(cu_mask=None) -> int:
    """Raw hipStream_t (int).  cu_mask: None for an ordinary non-blocking stream,
    or a sequence of CU indices the stream's kernels may use."""
    out = ctypes.c_void_p()
    if cu_mask is None:
        _check(_lib.kvio_stream_create(None, 0, ctypes.byref(out)))
    else:
        cus = sorted(set(int(c) for c in cu_mask))
        words = (ctypes.c_uint32 * (cus[-1] // 32 + 1 if cus else 1))()
        for c in cus:
            words[c // 32] |= 1 << (c % 32)
        _check(_lib.kvio_stream_create(words, len(words), ctypes.byref(out)))
    return out.value


def kvio_stream_destroy(stream: int) -> None:
    _check(_lib.kvio_stream_destroy(stream))


class Stream:
    """A kvio_stream_create stream wrapped for torch (torch.cuda.ExternalStream)."""

    def __init__(self, cu_mask=None):
        self.handle = kvio_stream_create(cu_mask)
        self.torch = torch.cuda.ExternalStream(self.handle)

    @property
    def cuda_stream(self) -> int:
        return self.handle

    def close(self) -> None:
        if self.handle:
            torch.cuda.synchronize()
            kvio_stream_destroy(self.handle)
            self.handle = 0


def kvio_schedule_round(requests, max_tokens: int, max_requests: int, loading_bound_ratio: float = 0.0,
                        delay_hit_threshold: int = -1):
    """One scheduling round over `requests`, a sequence of (load_tokens,
    compute_tokens, context or -1, transient_matches).  Returns (batch, next
    queue) as lists of indices into `requests`."""
    n = len(requests)
    arr = (kvio_request * max(n, 1))()
    for i, (load, comp, ctx, match) in enumerate(requests):
        arr[i] = kvio_request(load, comp, -1 if ctx is None else ctx, match)
    pol = kvio_batch_policy(max_tokens, max_requests, 0, loading_bound_ratio, delay_hit_threshold)
    b = (ctypes.c_int32 * max(n, 1))()
    q = (ctypes.c_int32 * max(n, 1))()
    nb, nq = ctypes.c_int32(), ctypes.c_int32()
    _check(_lib.kvio_schedule_round(arr, n, ctypes.byref(pol), b, ctypes.byref(nb), q, ctypes.byref(nq)))
    return list(b[:nb.value]), list(q[:nq.value])


def _disk_args(fd, disk_layout, num_disk_pages, num_layers, page_size, row_bytes, disk_pages):
    st = kvio_disk_store(fd, disk_layout, num_disk_pages, num_layers, page_size, row_bytes)
    pages = (ctypes.c_int64 * max(len(disk_pages), 1))(*[int(p) for p in disk_pages])
    return st, pages


def kvio_disk_prefetch(fd: int, disk_layout: int, num_disk_pages: int, num_layers: int, page_size: int,
                       row_bytes: int, disk_pages, host_ptr: int, host_tokens: int,
                       host_layout: int = KVIO_HOST_TOKEN_MAJOR, threads: int = 8) -> None:
    """Read a context's disk pages into the host chunk at host_ptr."""
    st, pages = _disk_args(fd, disk_layout, num_disk_pages, num_layers, page_size, row_bytes, disk_pages)
    _check(_lib.kvio_disk_prefetch(ctypes.byref(st), pages, len(disk_pages), host_ptr, host_tokens,
                                   host_layout, threads))


def kvio_disk_store_pages(fd: int, disk_layout: int, num_disk_pages: int, num_layers: int, page_size: int,
                          row_bytes: int, disk_pages, host_ptr: int, host_tokens: int,
                          host_layout: int = KVIO_HOST_TOKEN_MAJOR, threads: int = 8) -> None:
    """Write a context's pages from the host chunk at host_ptr to the disk pages."""
    st, pages = _disk_args(fd, disk_layout, num_disk_pages, num_layers, page_size, row_bytes, disk_pages)
    _check(_lib.kvio_disk_store_pages(ctypes.byref(st), pages, len(disk_pages), host_ptr, host_tokens,
                                      host_layout, threads))


class DiskPrefetch:
    """A background prefetch of a context's disk pages into a host chunk
    (kvio_disk_prefetch_start); finish() stops it (cancel=True) or waits for
    it, and returns which context pages arrived in full."""

    def __init__(self, fd: int, disk_layout: int, num_disk_pages: int, num_layers: int, page_size: int,
                 row_bytes: int, disk_pages, host_ptr: int, host_tokens: int,
                 host_layout: int = KVIO_HOST_TOKEN_MAJOR, threads: int = 8):
        self._st, self._pages = _disk_args(fd, disk_layout, num_disk_pages, num_layers, page_size, row_bytes,
                                           disk_pages)
        self.n_pages = len(disk_pages)
        h = ctypes.c_void_p()
        _check(_lib.kvio_disk_prefetch_start(ctypes.byref(self._st), self._pages, self.n_pages, host_ptr,
                                             host_tokens, host_layout, threads, ctypes.byref(h)))
        self._h = h

    def progress(self) -> int:
        n = ctypes.c_int32()
        _check(_lib.kvio_disk_prefetch_progress(self._h, ctypes.byref(n)))
        return n.value

    def finish(self, cancel: bool = False) -> np.ndarray:
        """Bool array: page j arrived in full.  A failed read raises KvioError
        whose `page_done` attribute holds the same array."""
        if self._h is None:
            raise RuntimeError("prefetch already finished")
        done = (ctypes.c_uint8 * max(self.n_pages, 1))()
        n = ctypes.c_int32()
        st = _lib.kvio_disk_prefetch_finish(self._h, 1 if cancel else 0, done, ctypes.byref(n))
        self._h = None
        page_done = np.frombuffer(bytes(done), np.uint8)[:self.n_pages].astype(bool)
        if st != KVIO_OK:
            err = KvioError(st, kvio_last_error())
            err.page_done = page_done
            raise err
        assert int(page_done.sum()) == n.value
        return page_done

    def __del__(self):
        if getattr(self, "_h", None) is not None and _lib is not None:
            _lib.kvio_disk_prefetch_finish(self._h, 1, None, None)


class HostBuffer:
    """Pinned, device-mapped host memory from kvio_host_alloc, with a numpy view."""

    def __init__(self, nbytes: int, flags: int = KVIO_HOST_COHERENT):
        self.nbytes = nbytes
        self.ptr = kvio_host_alloc(nbytes, flags)
        self.array = np.ctypeslib.as_array((ctypes.c_uint8 * nbytes).from_address(self.ptr))

    def free(self) -> None:
        if self.ptr:
            self.array = None
            kvio_host_free(self.ptr)
            self.ptr = 0

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.free()


class KVPool:
    """A pool handle over a torch tensor shaped (2, L, S, H, D): K then V, each
    layer a token-major (S, H, D) array of 16-bit elements.

    load_launch / offload_launch shape each direction (see launch(); a
    KVIO_LAUNCH_STAGED flag stages that direction through HBM slots of
    staging_bytes / 4 each, 0 = the library default); host_layout names the
    layout of the host chunks this handle moves (KVIO_HOST_*)."""

    def __init__(self, pool: "torch.Tensor", page_size: int,
                 load_launch: Optional[kvio_launch] = None, offload_launch: Optional[kvio_launch] = None,
                 host_layout: int = KVIO_HOST_TOKEN_MAJOR, staging_bytes: int = 0):
        assert pool.is_cuda and pool.is_contiguous() and pool.dim() == 5 and pool.shape[0] == 2
        _, L, S, H, D = pool.shape
        self.tensor = pool
        self.num_layers, self.num_slots, self.page_size = L, S, page_size
        self.row_bytes = H * D * pool.element_size()
        self.handle = kvio_pool_create(L, H, D, pool.element_size(), page_size, S,
                                       [pool[0, l].data_ptr() for l in range(L)],
                                       [pool[1, l].data_ptr() for l in range(L)],
                                       load_launch, offload_launch, host_layout, staging_bytes)

    def load(self, spans, layer_begin=0, layer_end=None, stream=None):
        kvio_load(self.handle, spans, layer_begin, self.num_layers if layer_end is None else layer_end, stream)

    def offload(self, spans, layer_begin=0, layer_end=None, stream=None):
        kvio_offload(self.handle, spans, layer_begin, self.num_layers if layer_end is None else layer_end,
                     stream)

    def load_layer(self, spans, layer, stream=None, done=None):
        kvio_load_layer(self.handle, spans, layer, stream, done)

    def check(self):
        kvio_check(self.handle)

    def close(self):
        if self.handle:
            kvio_pool_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
