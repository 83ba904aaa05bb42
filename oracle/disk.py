"""Oracle for the storage tier (test infrastructure only).

Strata Sec. 4.2.1: cached contexts also live on disk, where the paper keeps
them page-first (all layers of a page together) so that loading a page is one
large transfer (Fig. 12 compares this with the layer-first order of the GPU
pool).  Plain Python: row by row, seek and read (or write) R bytes at the
offset the disk layout gives, and place them at the offset the host layout
gives (oracle.host_row_offset / host_row_offset_page_first).

Disk layouts of a store with N disk pages of P tokens, L layers, R-byte rows:
  page-first:  row (l, kv, o) of disk page p at ((p*L + l)*2 + kv)*P*R + o*R
  layer-first: row (l, kv, o) of disk page p at ((l*2 + kv)*N + p)*P*R + o*R
Context page j (tokens j*P .. j*P + P - 1) is disk page disk_pages[j].
"""
from __future__ import annotations

from typing import Sequence

import numpy as np

from . import PAGE_FIRST, TOKEN_MAJOR, host_row_offset, host_row_offset_page_first

DISK_PAGE_FIRST = 0
DISK_LAYER_FIRST = 1


def disk_row_offset(disk_layout: int, page: int, layer: int, kv: int, in_page: int, num_layers: int,
                    page_size: int, row_bytes: int, num_disk_pages: int) -> int:
    if disk_layout == DISK_PAGE_FIRST:
        return (((page * num_layers + layer) * 2 + kv) * page_size + in_page) * row_bytes
    return (((layer * 2 + kv) * num_disk_pages + page) * page_size + in_page) * row_bytes


def _host_off(host_layout, layer, kv, token, num_layers, page_size, host_tokens, row_bytes):
    if host_layout == PAGE_FIRST:
        return host_row_offset_page_first(layer, kv, num_layers, page_size, token, row_bytes)
    assert host_layout == TOKEN_MAJOR
    return host_row_offset(layer, kv, host_tokens, token, row_bytes)


def prefetch(path: str, disk_layout: int, num_disk_pages: int, num_layers: int, page_size: int,
             row_bytes: int, disk_pages: Sequence[int], chunk: np.ndarray, host_tokens: int,
             host_layout: int) -> None:
    """Fill `chunk` (flat uint8) with the context's pages, row by row."""
    with open(path, "rb") as f:
        for j, p in enumerate(disk_pages):
            assert 0 <= p < num_disk_pages
            for layer in range(num_layers):
                for kv in range(2):
                    for o in range(page_size):
                        f.seek(disk_row_offset(disk_layout, int(p), layer, kv, o, num_layers, page_size,
                                               row_bytes, num_disk_pages))
                        row = f.read(row_bytes)
                        assert len(row) == row_bytes
                        h = _host_off(host_layout, layer, kv, j * page_size + o, num_layers, page_size,
                                      host_tokens, row_bytes)
                        chunk[h:h + row_bytes] = np.frombuffer(row, np.uint8)


def store(path: str, disk_layout: int, num_disk_pages: int, num_layers: int, page_size: int,
          row_bytes: int, disk_pages: Sequence[int], chunk: np.ndarray, host_tokens: int,
          host_layout: int) -> None:
    """Write the context's pages from `chunk` into the file, row by row."""
    with open(path, "r+b") as f:
        for j, p in enumerate(disk_pages):
            for layer in range(num_layers):
                for kv in range(2):
                    for o in range(page_size):
                        h = _host_off(host_layout, layer, kv, j * page_size + o, num_layers, page_size,
                                      host_tokens, row_bytes)
                        f.seek(disk_row_offset(disk_layout, int(p), layer, kv, o, num_layers, page_size,
                                               row_bytes, num_disk_pages))
                        f.write(chunk[h:h + row_bytes].tobytes())
