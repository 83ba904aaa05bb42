"""Pins of the storage-tier oracle: hand-worked offsets, numpy fancy indexing
of a page-first store (a library routine), agreement of page-first and
layer-first files holding the same content (built with numpy transposes), and
store -> prefetch round trips."""
import numpy as np
import pytest

import oracle
from oracle import disk


def test_hand_worked_offsets():
    # L = 2, P = 4, R = 16, N = 10 disk pages.  Page-first: page 3 starts after
    # 3 pages of 2*2*4 rows (48 rows); layer 1, V, offset 2 adds (1*2+1)*4 + 2 = 14 rows.
    assert disk.disk_row_offset(disk.DISK_PAGE_FIRST, 3, 1, 1, 2, 2, 4, 16, 10) == (48 + 14) * 16
    # Layer-first: layer 1 V is run 3 of 4, each run 10 pages of 4 rows; page 3 offset 2.
    assert disk.disk_row_offset(disk.DISK_LAYER_FIRST, 3, 1, 1, 2, 2, 4, 16, 10) == ((3 * 10 + 3) * 4 + 2) * 16


def store_file(tmp_path, arr_pf, layout):
    """arr_pf: (N, L, 2, P, R) page-first content; writes the file in `layout`."""
    path = str(tmp_path / f"store{layout}.bin")
    data = arr_pf if layout == disk.DISK_PAGE_FIRST else np.ascontiguousarray(arr_pf.transpose(1, 2, 0, 3, 4))
    data.tofile(path)
    return path


@pytest.mark.parametrize("host_layout", [oracle.TOKEN_MAJOR, oracle.PAGE_FIRST])
def test_prefetch_matches_fancy_indexing(tmp_path, host_layout):
    N, L, P, R = 12, 3, 4, 32
    arr = np.random.default_rng(1).integers(0, 256, size=(N, L, 2, P, R), dtype=np.uint8)
    pages = [7, 0, 11, 4, 5]
    T = len(pages) * P
    # expected chunk from numpy: page-first chunk = arr[pages]; token-major = its transpose
    pf = arr[pages]                                             # (n, L, 2, P, R)
    exp = pf.reshape(-1) if host_layout == oracle.PAGE_FIRST else \
        np.ascontiguousarray(pf.transpose(1, 2, 0, 3, 4)).reshape(-1)
    for layout in (disk.DISK_PAGE_FIRST, disk.DISK_LAYER_FIRST):
        path = store_file(tmp_path, arr, layout)
        chunk = np.zeros(L * 2 * T * R, np.uint8)
        disk.prefetch(path, layout, N, L, P, R, pages, chunk, T, host_layout)
        assert np.array_equal(chunk, exp), layout


@pytest.mark.parametrize("layout", [disk.DISK_PAGE_FIRST, disk.DISK_LAYER_FIRST])
def test_store_prefetch_round_trip(tmp_path, layout):
    N, L, P, R = 9, 2, 3, 16
    path = str(tmp_path / "rt.bin")
    np.zeros(N * L * 2 * P * R, np.uint8).tofile(path)
    pages = [8, 2, 5]
    T = len(pages) * P + 2                                      # chunk with spare room
    chunk = np.random.default_rng(2).integers(0, 256, L * 2 * T * R, dtype=np.uint8)
    disk.store(path, layout, N, L, P, R, pages, chunk, T, oracle.TOKEN_MAJOR)
    back = np.zeros_like(chunk)
    disk.prefetch(path, layout, N, L, P, R, pages, back, T, oracle.TOKEN_MAJOR)
    c = chunk.reshape(L, 2, T, R)
    b = back.reshape(L, 2, T, R)
    assert np.array_equal(b[:, :, :len(pages) * P], c[:, :, :len(pages) * P])
    assert not b[:, :, len(pages) * P:].any()
    # untouched disk pages stay zero
    raw = np.fromfile(path, np.uint8)
    if layout == disk.DISK_PAGE_FIRST:
        other = raw.reshape(N, -1)[[p for p in range(N) if p not in pages]]
    else:
        other = raw.reshape(L, 2, N, -1)[:, :, [p for p in range(N) if p not in pages]]
    assert not other.any()
