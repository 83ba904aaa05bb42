"""kvio: GPU-assisted paged-KV transfers between pinned host memory and an
MI355X paged KV pool (Strata, Sec. 4.2 and Sec. 4.2.1).

The transfer kernels and the C ABI live in ``libkvio.so`` (built from
``csrc/`` by ``_build.py``); ``kvio`` is its ctypes binding.
"""
from .kvio import (  # noqa: F401
    EXPORTS, HostBuffer, KVPool, KvioError, LIB_PATH,
    KVIO_OK, KVIO_EINVAL, KVIO_ERANGE, KVIO_EALIGN, KVIO_ENOTMAPPED, KVIO_EHIP, KVIO_ENOMEM,
    KVIO_HOST_COHERENT, KVIO_HOST_NONCOHERENT, KVIO_LAUNCH_CACHED, KVIO_MAX_SPANS_PER_LAUNCH,
    KVIO_HOST_TOKEN_MAJOR, KVIO_HOST_PAGE_FIRST, KVIO_HOST_HEAD_MAJOR, KVIO_LAUNCH_NO_LDS, KVIO_LAUNCH_STAGED,
    kvio_check, kvio_host_alloc, kvio_host_free, kvio_last_error, kvio_load, kvio_load_layer,
    kvio_memcpy, kvio_kernel_memcpy, kvio_naive_load, kvio_naive_offload, kvio_offload, kvio_pool_create,
    kvio_pool_destroy, kvio_span, kvio_strerror, launch, make_spans, Stream,
    kvio_stream_create, kvio_stream_destroy, kvio_schedule_round, kvio_disk_prefetch, kvio_disk_store_pages, DiskPrefetch,
    KVIO_DISK_PAGE_FIRST, KVIO_DISK_LAYER_FIRST, KVIO_EIO,
    KVIO_NOALLOC_MAX_LAYERS, kvio_load_noalloc, pool_desc,
)
