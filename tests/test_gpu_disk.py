"""End to end through the storage tier on the GPU: disk store -> pinned host
chunk (kvio_disk_prefetch) -> paged pool (kvio_load), and back (kvio_offload
-> kvio_disk_store_pages), compared byte for byte with the same chain run by
the storage oracle and the copy oracle.  With O_DIRECT descriptors the pinned
chunks cannot take direct I/O, so these cases run the bounce-buffer staging."""
import os

import numpy as np
import pytest

import oracle
from oracle import disk as odisk

pytestmark = pytest.mark.gpu

HOST = {0: oracle.TOKEN_MAJOR, 1: oracle.PAGE_FIRST}


@pytest.fixture(scope="module")
def kv():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an AMD GPU"
    import paper_2508_18572_amd as kv
    return kv


@pytest.mark.parametrize("direct", [False, True], ids=["buffered", "o_direct"])
@pytest.mark.parametrize("disk_layout", [0, 1])
@pytest.mark.parametrize("host_layout", [0, 1])
def test_disk_to_pool_and_back(kv, tmp_path, disk_layout, host_layout, direct):
    import torch
    L, H, D, P, S, N = 4, 8, 128, 16, 2048, 64
    R = H * D * 2
    rng = np.random.default_rng(300 + disk_layout * 2 + host_layout)
    path = str(tmp_path / "store.bin")
    rng.integers(0, 256, N * L * 2 * P * R, dtype=np.uint8).tofile(path)
    disk_pages = rng.permutation(N)[:10]
    T = len(disk_pages) * P - 5                      # partial last page
    HT = len(disk_pages) * P
    pool_pages = rng.permutation(S // P)[:len(disk_pages)].astype(np.int32)
    pool_np = rng.integers(0, 256, size=(2, L, S, R), dtype=np.uint8)
    pool_t = torch.from_numpy(pool_np.view(np.uint16).reshape(2, L, S, H, D).copy()).cuda()
    nbytes = L * 2 * HT * R
    with kv.HostBuffer(nbytes) as hb, kv.HostBuffer(nbytes) as ob:
        try:
            fd = os.open(path, os.O_RDWR | (os.O_DIRECT if direct else 0))
        except OSError:
            pytest.skip("O_DIRECT not supported on this filesystem")
        try:
            kv.kvio_disk_prefetch(fd, disk_layout, N, L, P, R, disk_pages, hb.ptr, HT, host_layout, 4)
            pt = torch.from_numpy(pool_pages).cuda()
            pool = kv.KVPool(pool_t, P, host_layout=host_layout)
            pool.load([(hb.ptr, HT, T, pt.data_ptr())])
            torch.cuda.synchronize()
            pool.check()
            chunk = np.zeros(nbytes, np.uint8)
            odisk.prefetch(path, disk_layout, N, L, P, R, disk_pages, chunk, HT, HOST[host_layout])
            exp = pool_np.copy()
            oracle.load_layout(exp[0], exp[1], P, [(chunk, HT, T, pool_pages)], HOST[host_layout])
            got = pool_t.cpu().numpy().view(np.uint8).reshape(2, L, S, R)
            assert np.array_equal(got, exp), "pool differs after disk -> host -> pool"

            # back: offload the same pages to a fresh chunk and store it under other disk pages
            ob.array[:] = 0
            pool.offload([(ob.ptr, HT, HT, pt.data_ptr())])
            torch.cuda.synchronize()
            pool.check()
            pool.close()
            back_pages = rng.permutation(N)[:len(disk_pages)]
            kv.kvio_disk_store_pages(fd, disk_layout, N, L, P, R, back_pages, ob.ptr, HT, host_layout, 4)
            os.fsync(fd)
        finally:
            os.close(fd)
        ochunk = np.zeros(nbytes, np.uint8)
        oracle.offload_layout(exp[0], exp[1], P, [(ochunk, HT, HT, pool_pages)], HOST[host_layout])
        assert np.array_equal(ob.array, ochunk)
        again = np.zeros(nbytes, np.uint8)
        odisk.prefetch(path, disk_layout, N, L, P, R, back_pages, again, HT, HOST[host_layout])
        assert np.array_equal(again, ochunk), "disk pages differ after pool -> host -> disk"
