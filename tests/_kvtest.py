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


_libc.memset.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t]
_libc.memset.restype = ctypes.c_void_p


def _for_each_slab(pool_t, check, workers):
    """Copy every (K|V, layer) slab of the GPU pool into pinned host memory and
    run check(kv, layer, image) on it, `workers` slabs at a time (the copies
    and the oracle's C calls run without the interpreter lock).  `image` is an
    (S, R) uint8 view valid during the call.  Returns the failure messages."""
    import torch

    import paper_2508_18572_amd as kvmod
    _, L, S = pool_t.shape[:3]
    R = pool_t[0, 0, 0].numel() * pool_t.element_size()
    pool_b = pool_t.view(torch.uint8).view(2, L, S, R)
    planes = [(kv, l) for l in range(L) for kv in range(2)]
    torch.cuda.synchronize()

    def work(w):
        errors = []
        with kvmod.HostBuffer(S * R) as img:
            dst = torch.from_numpy(img.array).view(S, R)
            stream = torch.cuda.Stream()
            with torch.cuda.stream(stream):
                for kv, l in planes[w::workers]:
                    dst.copy_(pool_b[kv, l])
                    stream.synchronize()
                    msg = check(kv, l, img.array.reshape(S, R))
                    if msg:
                        errors.append(msg)
        return errors

    with ThreadPoolExecutor(workers) as ex:
        return [m for errs in ex.map(work, range(workers)) for m in errs]


def _first_bad_row(a: np.ndarray, b: np.ndarray) -> int:
    rows = np.nonzero(np.any(a != b, axis=1))[0]
    return int(rows[0]) if rows.size else -1


def pool_matches_oracle(pool_t, spans, page_size, layer_range=None, workers=3):
    """Whole-image parity of a load.  Every (K|V, layer) slab of the GPU pool
    equals, byte for byte, the oracle's load of `spans` into a slab image that
    holds the sentinel everywhere (the pool was sentinel-filled before the
    load); layers outside layer_range equal the untouched sentinel image.
    spans: (host uint8 array of a token-major chunk, host_tokens, num_tokens,
    page_idx).  Returns the number of slabs compared."""
    _, L, S = pool_t.shape[:3]
    R = pool_t[0, 0, 0].numel() * pool_t.element_size()
    lo, hi = layer_range or (0, L)
    live = [(h, ht, nt, np.ascontiguousarray(p, np.int32)) for h, ht, nt, p in spans if nt > 0]
    expected = {}

    def check(kv, l, image):
        import threading
        exp = expected.get(threading.get_ident())
        if exp is None:
            exp = expected[threading.get_ident()] = np.empty((S, R), np.uint8)
        _libc.memset(exp.ctypes.data, SENTINEL & 0xFF, S * R)
        if lo <= l < hi:
            for host, ht, nt, pidx in live:
                a = oracle.host_row_offset(l, kv, ht, 0, R)
                oracle.load_slab(exp, page_size, host[a:a + nt * R], nt, pidx)
        if _libc.memcmp(image.ctypes.data, exp.ctypes.data, S * R) != 0:
            return f"kv {kv} layer {l}: pool slab differs from the oracle (first row {_first_bad_row(image, exp)})"
        return None

    assert (SENTINEL >> 8) == (SENTINEL & 0xFF)
    errors = _for_each_slab(pool_t, check, workers)
    if errors:
        raise AssertionError(f"{len(errors)} slab(s) differ: " + "; ".join(errors[:4]))
    return 2 * L


def offload_matches_oracle(pool_t, spans, page_size, before_byte, layer_range=None, workers=3):
    """Whole-chunk parity of an offload.  For every span, every (layer, K|V)
    slab region of its host chunk equals the oracle's offload of the GPU pool
    image into a region that held `before_byte` everywhere (the chunk was
    filled with it before the offload); the pool image itself is checked
    separately.  spans as for pool_matches_oracle; host arrays are the
    offload's destinations.  Returns the number of regions compared."""
    _, L, S = pool_t.shape[:3]
    R = pool_t[0, 0, 0].numel() * pool_t.element_size()
    lo, hi = layer_range or (0, L)
    live = [(h, ht, nt, np.ascontiguousarray(p, np.int32)) for h, ht, nt, p in spans if nt > 0]
    biggest = max([ht for _, ht, _, _ in live], default=0) * R
    expected = {}

    def check(kv, l, image):
        import threading
        exp = expected.get(threading.get_ident())
        if exp is None:
            exp = expected[threading.get_ident()] = np.empty(max(biggest, 1), np.uint8)
        for i, (host, ht, nt, pidx) in enumerate(live):
            a = oracle.host_row_offset(l, kv, ht, 0, R)
            region = exp[:ht * R]
            _libc.memset(region.ctypes.data, before_byte, ht * R)
            if lo <= l < hi:
                oracle.offload_slab(image, page_size, region, nt, pidx)
            if _libc.memcmp(host[a:a + ht * R].ctypes.data, region.ctypes.data, ht * R) != 0:
                got = host[a:a + ht * R].reshape(ht, R)
                return (f"span {i} kv {kv} layer {l}: host chunk differs from the oracle's offload "
                        f"(first row {_first_bad_row(got, region.reshape(ht, R))})")
        return None

    errors = _for_each_slab(pool_t, check, workers)
    if errors:
        raise AssertionError(f"{len(errors)} region(s) differ: " + "; ".join(errors[:4]))
    return 2 * L * len(live)


def threaded_memset(ptr: int, byte: int, nbytes: int, threads: int = 16, chunk: int = 256 << 20) -> None:
    """memset of a large host range from several threads."""
    def one(o):
        _libc.memset(ptr + o, byte, min(chunk, nbytes - o))

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(one, range(0, nbytes, chunk)))


def pool_matches_oracle_layout(pool_t, spans, page_size, layout, num_heads, workers=3):
    """Whole-image parity of a load from chunks in any host layout (oracle
    TOKEN_MAJOR / PAGE_FIRST / HEAD_MAJOR): layer by layer, the GPU pool's K and
    V slabs equal, byte for byte, the oracle's load of that layer of `spans`
    into slab images that hold the sentinel everywhere.  Returns the number of
    slabs compared."""
    import threading

    import torch

    import paper_2508_18572_amd as kvmod
    _, L, S = pool_t.shape[:3]
    R = pool_t[0, 0, 0].numel() * pool_t.element_size()
    pool_b = pool_t.view(torch.uint8).view(2, L, S, R)
    live = [(h, ht, nt, np.ascontiguousarray(p, np.int32)) for h, ht, nt, p in spans if nt > 0]
    torch.cuda.synchronize()

    def work(w):
        errors = []
        exp = [np.empty((S, R), np.uint8), np.empty((S, R), np.uint8)]
        with kvmod.HostBuffer(S * R) as ik, kvmod.HostBuffer(S * R) as iv:
            imgs = [ik, iv]
            stream = torch.cuda.Stream()
            with torch.cuda.stream(stream):
                for l in range(w, L, workers):
                    for kv in range(2):
                        torch.from_numpy(imgs[kv].array).view(S, R).copy_(pool_b[kv, l])
                        _libc.memset(exp[kv].ctypes.data, SENTINEL & 0xFF, S * R)
                    stream.synchronize()
                    oracle.load_layout_layer(exp[0], exp[1], page_size, live, layout, L, l, num_heads=num_heads)
                    for kv in range(2):
                        if _libc.memcmp(imgs[kv].ptr, exp[kv].ctypes.data, S * R) != 0:
                            got = imgs[kv].array.reshape(S, R)
                            errors.append(f"kv {kv} layer {l}: pool slab differs from the oracle "
                                          f"(first row {_first_bad_row(got, exp[kv])})")
        return errors

    with ThreadPoolExecutor(workers) as ex:
        errors = [m for errs in ex.map(work, range(workers)) for m in errs]
    if errors:
        raise AssertionError(f"{len(errors)} slab(s) differ: " + "; ".join(errors[:4]))
    return 2 * L
