"""Helpers for the full-size GPU workload tests: sampled oracle checks, sentinel
properties computed with plain torch ops, and a threaded byte comparison of
large pinned host buffers.  None of this touches the product's kernels."""
from __future__ import annotations

import ctypes
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle

SENTINEL = 0x5A5A          # int16 fill of untouched pool rows

_libc = ctypes.CDLL("libc.so.6")
_libc.memcmp.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t]
_libc.memcmp.restype = ctypes.c_int


def memequal(a_ptr: int, b_ptr: int, nbytes: int, threads: int = 16, chunk: int = 256 << 20) -> bool:
    """Byte equality of two host ranges (ctypes releases the GIL in memcmp)."""
    offs = range(0, nbytes, chunk)

    def one(o):
        n = min(chunk, nbytes - o)
        return _libc.memcmp(a_ptr + o, b_ptr + o, n) == 0

    with ThreadPoolExecutor(threads) as ex:
        return all(ex.map(one, offs))


def sampled_rows_match(pool_t, spans, page_size, num_slots, row_bytes, layers, n_samples, seed):
    """For n_samples random (span, layer, kv, token) rows, the oracle's slot and
    host offset must hold identical bytes in the GPU pool and the host chunk.
    spans: list of (host_uint8_array, host_tokens, num_tokens, page_idx)."""
    import torch
    rng = np.random.default_rng(seed)
    live = [i for i, s in enumerate(spans) if s[2] > 0]
    S = num_slots
    pool_b = pool_t.view(torch.uint8).view(2, layers, S, row_bytes)
    slots_cache = {}
    picks = []
    for _ in range(n_samples):
        i = live[int(rng.integers(0, len(live)))]
        host, ht, nt, pidx = spans[i]
        l = int(rng.integers(0, layers))
        kv = int(rng.integers(0, 2))
        t = int(rng.integers(0, nt))
        if i not in slots_cache:
            slots_cache[i] = oracle.expand_slots(pidx, page_size, nt, S)
        picks.append((i, l, kv, t, int(slots_cache[i][t])))
    idx_kv = torch.tensor([p[2] for p in picks], device=pool_t.device)
    idx_l = torch.tensor([p[1] for p in picks], device=pool_t.device)
    idx_s = torch.tensor([p[4] for p in picks], device=pool_t.device)
    got = pool_b[idx_kv, idx_l, idx_s].cpu().numpy()
    for (i, l, kv, t, slot), row in zip(picks, got):
        host, ht, nt, _ = spans[i]
        off = oracle.host_row_offset(l, kv, ht, t, row_bytes)
        if not np.array_equal(row, host[off:off + row_bytes]):
            raise AssertionError(f"span {i} layer {l} kv {kv} token {t} slot {slot}: pool row differs")
    return len(picks)


def touched_mask(spans, page_size, num_slots):
    """Bool[S] of slots the oracle's page-offset expansion assigns to any span."""
    m = np.zeros(num_slots, bool)
    for host, ht, nt, pidx in spans:
        if nt:
            m[oracle.expand_slots(pidx, page_size, nt, num_slots)] = True
    return m


def untouched_rows_hold_sentinel(pool_t, touched: np.ndarray, layers, layer_range=None):
    """Every slot outside `touched` still holds the sentinel in every (kv, layer)
    of the range, and every touched slot no longer does (random payload)."""
    import torch
    t_dev = torch.from_numpy(touched).to(pool_t.device)
    lo, hi = layer_range or (0, layers)
    for kv in range(2):
        for l in range(layers):
            rows = pool_t[kv, l].view(torch.int16).reshape(pool_t.shape[2], -1)
            is_sent = (rows == SENTINEL).all(dim=1)
            if lo <= l < hi:
                bad_untouched = (~is_sent & ~t_dev).sum().item()
                bad_touched = (is_sent & t_dev).sum().item()
                if bad_untouched or bad_touched:
                    raise AssertionError(f"kv {kv} layer {l}: {bad_untouched} untouched rows changed, "
                                         f"{bad_touched} touched rows still sentinel")
            elif not bool(is_sent.all()):
                raise AssertionError(f"kv {kv} layer {l} outside the layer range was written")
