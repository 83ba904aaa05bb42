"""Storage tier in libkvio (kvio_disk_prefetch / kvio_disk_store_pages)
against the storage oracle, on temporary files, for both disk layouts, both
host layouts, buffered and O_DIRECT descriptors.  Host code: no GPU."""
import os

import numpy as np
import pytest

import oracle
from oracle import disk as odisk


@pytest.fixture(scope="module")
def kv():
    import paper_2508_18572_amd as kv
    return kv


HOST = {0: oracle.TOKEN_MAJOR, 1: oracle.PAGE_FIRST}


def aligned(nbytes, align=4096):
    """A 4 KiB-aligned numpy uint8 buffer (for O_DIRECT)."""
    raw = np.zeros(nbytes + align, np.uint8)
    off = (-raw.ctypes.data) % align
    return raw[off:off + nbytes]


@pytest.mark.parametrize("disk_layout", [0, 1])
@pytest.mark.parametrize("host_layout", [0, 1])
@pytest.mark.parametrize("threads", [1, 7])
def test_prefetch_matches_oracle(kv, tmp_path, disk_layout, host_layout, threads):
    N, L, P, R = 40, 3, 4, 512
    path = str(tmp_path / "store.bin")
    np.random.default_rng(disk_layout * 2 + host_layout).integers(0, 256, N * L * 2 * P * R,
                                                                  dtype=np.uint8).tofile(path)
    pages = [17, 3, 4, 5, 39, 0, 22]                # includes a consecutive run (merged)
    T = len(pages) * P + (0 if host_layout else 3)  # token-major chunk with spare capacity
    exp = np.full(L * 2 * T * R, 0x77, np.uint8)
    odisk.prefetch(path, disk_layout, N, L, P, R, pages, exp, T, HOST[host_layout])
    got = np.full_like(exp, 0x77)
    fd = os.open(path, os.O_RDONLY)
    try:
        kv.kvio_disk_prefetch(fd, disk_layout, N, L, P, R, pages, got.ctypes.data, T, host_layout, threads)
    finally:
        os.close(fd)
    assert np.array_equal(got, exp)


@pytest.mark.parametrize("disk_layout", [0, 1])
def test_store_then_prefetch(kv, tmp_path, disk_layout):
    N, L, P, R = 16, 2, 8, 256
    path = str(tmp_path / "rt.bin")
    np.zeros(N * L * 2 * P * R, np.uint8).tofile(path)
    pages = [9, 1, 14]
    T = len(pages) * P
    chunk = np.random.default_rng(4).integers(0, 256, L * 2 * T * R, dtype=np.uint8)
    fd = os.open(path, os.O_RDWR)
    try:
        kv.kvio_disk_store_pages(fd, disk_layout, N, L, P, R, pages, chunk.ctypes.data, T, 0, 4)
        os.fsync(fd)
    finally:
        os.close(fd)
    back = np.zeros_like(chunk)
    odisk.prefetch(path, disk_layout, N, L, P, R, pages, back, T, oracle.TOKEN_MAJOR)
    assert np.array_equal(back, chunk)


def test_o_direct(kv, tmp_path):
    N, L, P, R = 32, 2, 16, 1024            # 16 KiB runs: 4 KiB aligned
    path = str(tmp_path / "direct.bin")
    np.random.default_rng(5).integers(0, 256, N * L * 2 * P * R, dtype=np.uint8).tofile(path)
    try:
        fd = os.open(path, os.O_RDONLY | os.O_DIRECT)
    except OSError:
        pytest.skip("O_DIRECT not supported on this filesystem")
    pages = [31, 2, 3, 11]
    T = len(pages) * P
    got = aligned(L * 2 * T * R)
    try:
        kv.kvio_disk_prefetch(fd, 1, N, L, P, R, pages, got.ctypes.data, T, 1, 4)
    except kv.KvioError as e:
        if "Invalid argument" in e.detail:
            pytest.skip("filesystem refuses O_DIRECT reads")
        raise
    finally:
        os.close(fd)
    exp = np.zeros_like(got)
    odisk.prefetch(path, 1, N, L, P, R, pages, exp, T, oracle.PAGE_FIRST)
    assert np.array_equal(got, exp)


def test_errors(kv, tmp_path):
    N, L, P, R = 4, 1, 2, 64
    path = str(tmp_path / "short.bin")
    np.zeros(N * L * 2 * P * R - 64, np.uint8).tofile(path)      # one row short
    buf = np.zeros(L * 2 * 4 * R, np.uint8)
    fd = os.open(path, os.O_RDONLY)
    try:
        with pytest.raises(kv.KvioError) as e:                     # disk page out of range
            kv.kvio_disk_prefetch(fd, 0, N, L, P, R, [4], buf.ctypes.data, 2)
        assert e.value.status == kv.KVIO_EINVAL
        with pytest.raises(kv.KvioError) as e:                     # chunk too small for whole pages
            kv.kvio_disk_prefetch(fd, 0, N, L, P, R, [0, 1], buf.ctypes.data, 3)
        assert e.value.status == kv.KVIO_EINVAL
        with pytest.raises(kv.KvioError) as e:                     # last page runs past end of file
            kv.kvio_disk_prefetch(fd, 0, N, L, P, R, [3], buf.ctypes.data, 2)
        assert e.value.status == kv.KVIO_EIO
    finally:
        os.close(fd)
    with pytest.raises(kv.KvioError) as e:                         # bad descriptor
        kv.kvio_disk_prefetch(-1, 0, N, L, P, R, [0], buf.ctypes.data, 2)
    assert e.value.status == kv.KVIO_EINVAL
