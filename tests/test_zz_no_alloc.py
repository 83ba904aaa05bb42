"""kvio_load_noalloc (the load for callers that cannot allocate) against
kvio_load with a pool handle, through the C ABI: two calls in a row, the
second with a smaller input, on pools that start identical; both pools must
be byte for byte equal after each call, and equal to the CPU oracle's load
of the same host chunks.  Covers every host layout, a partial last page,
several spans, a layer sub-range, the largest layer count the static table
holds, and out-of-range page indices (skipped on both paths)."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kv():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an AMD GPU"
    import paper_2508_18572_amd as kv
    return kv


ORACLE_LAYOUT = {0: oracle.TOKEN_MAJOR, 1: oracle.PAGE_FIRST, 2: oracle.HEAD_MAJOR}


def _twin_pools(L, S, H, D, seed):
    import torch
    R = H * D * 2
    img = np.random.default_rng(seed).integers(0, 256, size=(2, L, S, R), dtype=np.uint8)
    a = torch.from_numpy(img.view(np.uint16).reshape(2, L, S, H, D).copy()).cuda()
    b = a.clone()
    return img, a, b


def _bytes(pool_t):
    L, S = pool_t.shape[1], pool_t.shape[2]
    return pool_t.cpu().numpy().view(np.uint8).reshape(2, L, S, -1)


def _one_call(kv, layout, H, D, P, img, pa, pb, handle, desc, calls, rng, bad_page=False):
    """calls: list of (num_tokens, host_tokens) spans of one call; returns
    after both paths ran and their pools were compared."""
    import torch
    _, L, S, R = img.shape
    keep, spans_dev, spans_ora = [], [], []
    free = rng.permutation(S // P).astype(np.int32)
    pos = 0
    for i, (T, HT) in enumerate(calls):
        pages = free[pos:pos + -(-T // P)].copy()
        pos += len(pages)
        nbytes = max(oracle.host_chunk_bytes(ORACLE_LAYOUT[layout], L, HT, R, P), 16)
        hb = kv.HostBuffer(nbytes)
        W.fill_np(hb.array, int(rng.integers(1 << 30)), W.LLAMA8B)
        dev_pages = pages.copy()
        if bad_page and i == 0 and len(pages) > 1:
            dev_pages[1] = S // P + 7                # outside [0, S / P): skipped on both paths
        pt = torch.from_numpy(dev_pages).cuda()
        keep += [hb, pt]
        spans_dev.append((hb.ptr, HT, T, pt.data_ptr()))
        spans_ora.append((hb.array, HT, T, pages, dev_pages))
    return keep, spans_dev, spans_ora


@pytest.mark.parametrize("layout", [0, 1, 2], ids=["token_major", "page_first", "head_major"])
def test_noalloc_load_matches_pool_handle_twice(kv, layout):
    import torch
    L, H, D, P, S = 4, 4, 64, 16, 8192                  # R = 512 B: narrow rows
    rng = np.random.default_rng(70 + layout)
    img, pa, pb = _twin_pools(L, S, H, D, seed=layout)
    R = H * D * 2
    handle = kv.KVPool(pa, P, host_layout=layout)
    desc, keep_desc = kv.pool_desc(L, H, D, 2, P, S, [pb[0, l].data_ptr() for l in range(L)],
                                   [pb[1, l].data_ptr() for l in range(L)], host_layout=layout)
    exp = img.copy()
    # first call: three contexts, partial last pages, chunks longer than the contexts (page-first
    # chunks hold whole pages)
    first = [(1000, 1024), (333, 352), (2048, 2048)]
    # second call: a smaller input -- one context, layers [1, 3)
    second = [(200, 208)]
    for calls, (l0, l1) in ((first, (0, L)), (second, (1, 3))):
        print(f"[no_alloc] layout {layout} spans {calls} layers [{l0}, {l1})", flush=True)
        keep, spans_dev, spans_ora = _one_call(kv, layout, H, D, P, img, pa, pb, handle, desc, calls, rng)
        handle.load(spans_dev, l0, l1)
        kv.kvio_load_noalloc(desc, spans_dev, l0, l1)
        torch.cuda.synchronize()
        handle.check()
        got_a, got_b = _bytes(pa), _bytes(pb)
        assert np.array_equal(got_a, got_b), "kvio_load_noalloc differs from kvio_load"
        oracle.load_layout(exp[0], exp[1], P, [(h, ht, t, pg) for h, ht, t, pg, _ in spans_ora],
                           ORACLE_LAYOUT[layout], num_heads=H, layer_begin=l0, layer_end=l1)
        assert np.array_equal(got_b, exp), "kvio_load_noalloc differs from the oracle"
        for x in keep:
            if hasattr(x, "free"):
                x.free()
    handle.close()
    del keep_desc


def test_noalloc_largest_layer_count_and_skipped_pages(kv):
    """128 layers (the static table's limit), then a smaller call whose first
    span names an out-of-range page: both paths skip those rows; the handle
    path reports it, the no-alloc path moves the rest identically."""
    import torch
    L, H, D, P, S = kv.KVIO_NOALLOC_MAX_LAYERS, 8, 128, 4, 512      # R = 2 KiB: wide rows
    rng = np.random.default_rng(90)
    img, pa, pb = _twin_pools(L, S, H, D, seed=9)
    handle = kv.KVPool(pa, P)
    desc, keep_desc = kv.pool_desc(L, H, D, 2, P, S, [pb[0, l].data_ptr() for l in range(L)],
                                   [pb[1, l].data_ptr() for l in range(L)])
    exp = img.copy()
    for calls, bad in (([(250, 250), (101, 128)], False), ([(37, 40)], True)):
        print(f"[no_alloc] L={L} spans {calls} bad page {bad}", flush=True)
        keep, spans_dev, spans_ora = _one_call(kv, 0, H, D, P, img, pa, pb, handle, desc, calls, rng,
                                               bad_page=bad)
        handle.load(spans_dev)
        kv.kvio_load_noalloc(desc, spans_dev, 0, L)
        torch.cuda.synchronize()
        if bad:
            with pytest.raises(kv.KvioError) as e:
                handle.check()
            assert e.value.status == kv.KVIO_ERANGE
        else:
            handle.check()
        got_a, got_b = _bytes(pa), _bytes(pb)
        assert np.array_equal(got_a, got_b), "kvio_load_noalloc differs from kvio_load"
        for h, ht, t, pages, dev_pages in spans_ora:
            if bad and not np.array_equal(pages, dev_pages):
                # the oracle moves every page but the skipped one
                for j in range(len(pages)):
                    if dev_pages[j] == pages[j]:
                        a, b = j * P, min(t, (j + 1) * P)
                        for l in range(L):
                            for kvi in range(2):
                                o = oracle.host_row_offset(l, kvi, ht, a, H * D * 2)
                                oracle.load_slab(exp[kvi, l], P, h[o:o + (b - a) * H * D * 2], b - a,
                                                 np.array([pages[j]], np.int32))
            else:
                oracle.load(exp[0], exp[1], P, [(h, ht, t, pages)])
        assert np.array_equal(got_b, exp), "kvio_load_noalloc differs from the oracle"
        for x in keep:
            if hasattr(x, "free"):
                x.free()
    handle.close()
    del keep_desc


def test_noalloc_rejects_what_it_cannot_hold(kv):
    import torch
    L, H, D, P, S = 2, 4, 64, 16, 1024
    pool = torch.zeros((2, L, S, H, D), dtype=torch.bfloat16, device="cuda")
    k = [pool[0, l].data_ptr() for l in range(L)]
    v = [pool[1, l].data_ptr() for l in range(L)]
    desc, keep = kv.pool_desc(L, H, D, 2, P, S, k, v, load_launch=kv.launch(flags=kv.KVIO_LAUNCH_STAGED))
    with pytest.raises(kv.KvioError) as e:
        kv.kvio_load_noalloc(desc, [], 0, L)
    assert e.value.status == kv.KVIO_EINVAL and "staged" in e.value.detail
    desc, keep = kv.pool_desc(L, H, D, 2, P, S, k, v)
    with pytest.raises(kv.KvioError) as e:
        kv.kvio_load_noalloc(desc, [(0, 0, 0, 0)] * (kv.KVIO_MAX_SPANS_PER_LAUNCH + 1), 0, L)
    assert e.value.status == kv.KVIO_EINVAL
    kv.kvio_load_noalloc(desc, [(0, 0, 0, 0)] * 3, 0, L)           # nothing to move: no error
    big, keep2 = kv.pool_desc(kv.KVIO_NOALLOC_MAX_LAYERS + 1, H, D, 2, P, S, k * 65, v * 65)
    with pytest.raises(kv.KvioError) as e:
        kv.kvio_load_noalloc(big, [], 0, 1)
    assert e.value.status == kv.KVIO_EINVAL and "layers exceed" in e.value.detail
    torch.cuda.synchronize()


def test_noalloc_load_replays_in_a_hip_graph(kv):
    """The callers the entry point exists for capture it: a load captured into
    a HIP graph (torch.cuda.CUDAGraph), replayed three times with new host
    bytes and eager work between replays; every replay equals the oracle."""
    import torch
    L, H, D, P, S, T = 3, 8, 128, 16, 4096, 1000
    R = H * D * 2
    rng = np.random.default_rng(88)
    pages = rng.permutation(S // P)[:-(-T // P)].astype(np.int32)
    img = rng.integers(0, 256, size=(2, L, S, R), dtype=np.uint8)
    pool_t = torch.from_numpy(img.view(np.uint16).reshape(2, L, S, H, D).copy()).cuda()
    desc, keep_desc = kv.pool_desc(L, H, D, 2, P, S, [pool_t[0, l].data_ptr() for l in range(L)],
                                   [pool_t[1, l].data_ptr() for l in range(L)])
    pt = torch.from_numpy(pages).cuda()
    with kv.HostBuffer(L * 2 * T * R) as hb:
        hb.array[:] = 0
        span = [(hb.ptr, T, T, pt.data_ptr())]
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        kv.kvio_load_noalloc(desc, span, 0, L, stream=s)          # warm-up outside the capture
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            kv.kvio_load_noalloc(desc, span, 0, L, stream=s)
        exp = img.copy()
        for rep in range(3):
            print(f"[no_alloc] graph replay {rep}", flush=True)
            W.fill_np(hb.array, 600 + rep, W.LLAMA8B)             # new bytes before each replay
            g.replay()
            torch.cuda.synchronize()
            oracle.load(exp[0], exp[1], P, [(hb.array, T, T, pages)])
            assert np.array_equal(_bytes(pool_t), exp), f"replay {rep}: pool differs from the oracle"
            pool_t.view(torch.int16).add_(0)                      # eager work between replays
            torch.cuda.synchronize()
        del g
    del keep_desc
