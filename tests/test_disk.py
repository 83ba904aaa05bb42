"""Storage tier in libkvio (kvio_disk_prefetch / kvio_disk_store_pages)
against the storage oracle, on temporary files, for both disk layouts, both
host layouts, buffered and O_DIRECT descriptors.  Host code: no GPU."""
import os
import subprocess
import time

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


def _page_rows(chunk, j, L, P, R, T, host_layout):
    """Bytes of context page j in a host chunk, as one array (oracle offsets)."""
    out = []
    for layer in range(L):
        for kvi in range(2):
            for o in range(P):
                if host_layout == 1:
                    h = oracle.host_row_offset_page_first(layer, kvi, L, P, j * P + o, R)
                else:
                    h = oracle.host_row_offset(layer, kvi, T, j * P + o, R)
                out.append(chunk[h:h + R])
    return np.concatenate(out)


@pytest.mark.parametrize("disk_layout", [0, 1])
@pytest.mark.parametrize("host_layout", [0, 1])
def test_background_prefetch_waits_for_every_page(kv, tmp_path, disk_layout, host_layout):
    N, L, P, R = 48, 2, 4, 256
    path = str(tmp_path / "bg.bin")
    np.random.default_rng(11).integers(0, 256, N * L * 2 * P * R, dtype=np.uint8).tofile(path)
    pages = [5, 6, 7, 40, 1, 0, 33]
    T = len(pages) * P
    exp = np.zeros(L * 2 * T * R, np.uint8)
    odisk.prefetch(path, disk_layout, N, L, P, R, pages, exp, T, HOST[host_layout])
    got = np.zeros_like(exp)
    fd = os.open(path, os.O_RDONLY)
    try:
        job = kv.DiskPrefetch(fd, disk_layout, N, L, P, R, pages, got.ctypes.data, T, host_layout, 3)
        assert 0 <= job.progress() <= len(pages)
        done = job.finish(cancel=False)
    finally:
        os.close(fd)
    assert done.all()
    assert np.array_equal(got, exp)


@pytest.mark.parametrize("threads", [1, 4])
def test_cancelled_prefetch_reports_complete_pages(kv, tmp_path, threads):
    # large enough that a cancellation right after the start usually stops it early;
    # whatever the timing, every page reported complete must hold its bytes
    N, L, P, R = 256, 4, 16, 2048
    path = str(tmp_path / "cancel.bin")
    np.random.default_rng(12).integers(0, 256, N * L * 2 * P * R, dtype=np.uint8).tofile(path)
    pages = list(np.random.default_rng(13).permutation(N)[:128])
    T = len(pages) * P
    exp = np.zeros(L * 2 * T * R, np.uint8)
    odisk.prefetch(path, 1, N, L, P, R, pages, exp, T, oracle.TOKEN_MAJOR)
    for wait_pages in (0, 8):
        got = np.zeros_like(exp)
        fd = os.open(path, os.O_RDONLY)
        try:
            job = kv.DiskPrefetch(fd, 1, N, L, P, R, pages, got.ctypes.data, T, 0, threads)
            t0 = time.time()
            while job.progress() < wait_pages and time.time() - t0 < 60:
                time.sleep(0.0005)
            done = job.finish(cancel=True)
        finally:
            os.close(fd)
        assert done.sum() >= wait_pages
        for j in np.flatnonzero(done):
            assert np.array_equal(_page_rows(got, j, L, P, R, T, 0), _page_rows(exp, j, L, P, R, T, 0)), j


def test_prefetch_failure_names_complete_pages(kv, tmp_path):
    N, L, P, R = 8, 1, 2, 64
    path = str(tmp_path / "short2.bin")
    np.random.default_rng(14).integers(0, 256, N * L * 2 * P * R - 1, dtype=np.uint8).tofile(path)
    pages = [0, 1, 7]                      # page 7 runs past the end of the file
    T = len(pages) * P
    got = np.zeros(L * 2 * T * R, np.uint8)
    fd = os.open(path, os.O_RDONLY)
    try:
        job = kv.DiskPrefetch(fd, 0, N, L, P, R, pages, got.ctypes.data, T, 1, 1)
        with pytest.raises(kv.KvioError) as e:
            job.finish()
    finally:
        os.close(fd)
    assert e.value.status == kv.KVIO_EIO
    assert not e.value.page_done[2]
    with pytest.raises(kv.KvioError) as e:             # validation happens at the start
        kv.DiskPrefetch(-1, 0, N, L, P, R, [0], got.ctypes.data, T)
    assert e.value.status == kv.KVIO_EINVAL


@pytest.mark.parametrize("sanitizer", ["thread", "address"])
def test_thread_pool_under_sanitizers(tmp_path, sanitizer):
    """kvio_disk.cpp built alone with g++ and -fsanitize (host code only),
    driven by tests/c/disk_race.cpp: background jobs polled and cancelled from
    other threads, stores and prefetches on both layouts."""
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    exe = str(tmp_path / f"disk_race_{sanitizer}")
    cmd = ["g++", "-std=c++17", "-O1", "-g", f"-fsanitize={sanitizer}", "-pthread", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(root, "include"), "-I", "/opt/rocm/include",
           os.path.join(root, "tests", "c", "disk_race.cpp"),
           os.path.join(root, "paper_2508_18572_amd", "csrc", "kvio_disk.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0 and "sanitize" in r.stderr and "cannot find" in r.stderr:
        pytest.skip(f"no {sanitizer} sanitizer runtime: {r.stderr[-300:]}")
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1", ASAN_OPTIONS="detect_leaks=1")
    run = subprocess.run([exe, str(tmp_path / "race.bin")], capture_output=True, text=True, timeout=300, env=env)
    assert run.returncode == 0, run.stdout[-2000:] + run.stderr[-4000:]
    assert "disk race checks passed" in run.stdout
