"""GPU parity: libkvio.so's kernels against the CPU oracle, byte for byte.

Every case runs the HIP path through the C ABI (via the ctypes binding) on
seeded inputs and compares the whole pool image (load) or the whole host chunk
(offload, starting from a sentinel fill) with what the oracle computes from
the same bytes.  Shapes cover both kernel paths (rows that are a multiple of
1 KiB and narrower or odd rows), partial last pages, chunks longer than the
context, layer sub-ranges, many spans (more than one launch), every tile size
and several launch shapes.
"""
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


def _pool(L, S, H, D, seed):
    import torch
    R = H * D * 2
    pool_np = np.random.default_rng(seed).integers(0, 256, size=(2, L, S, R), dtype=np.uint8)
    pool_t = torch.from_numpy(pool_np.view(np.uint16).reshape(2, L, S, H, D).copy()).cuda()
    return pool_np, pool_t


def _pool_bytes(pool_t):
    L, S = pool_t.shape[1], pool_t.shape[2]
    return pool_t.cpu().numpy().view(np.uint8).reshape(2, L, S, -1)


def run_case(kv, L, H, D, P, S, spans, l0=0, l1=None, launch=None, seed=0, shape=W.LLAMA8B, staging_bytes=0):
    """spans: list of (num_tokens, host_tokens).  Loads, checks, offloads, checks."""
    import torch
    l1 = L if l1 is None else l1
    R = H * D * 2
    rng = np.random.default_rng(1000 + seed)
    pool_np, pool_t = _pool(L, S, H, D, seed)
    need = sum(-(-T // P) for T, _ in spans)
    perm = rng.permutation(S // P)[:need].astype(np.int32)
    bufs, outs, pts, ora_spans, ora_out, dev_spans, dev_out = [], [], [], [], [], [], []
    pos = 0
    try:
        for i, (T, HT) in enumerate(spans):
            pages = perm[pos:pos + -(-T // P)]
            pos += len(pages)
            hb = kv.HostBuffer(max(L * 2 * HT * R, 16))
            ob = kv.HostBuffer(max(L * 2 * HT * R, 16))
            bufs.append(hb)
            outs.append(ob)
            W.fill_np(hb.array, seed * 100 + i, shape)
            ob.array[:] = 0xA5
            pt = torch.from_numpy(pages.copy() if len(pages) else np.zeros(1, np.int32)).cuda()
            pts.append(pt)
            ora_spans.append((hb.array, HT, T, pages))
            eo = np.full(ob.array.size, 0xA5, np.uint8)
            ora_out.append(eo)
            dev_spans.append((hb.ptr, HT, T, pt.data_ptr()))
            dev_out.append((ob.ptr, HT, T, pt.data_ptr()))
        pool = kv.KVPool(pool_t, P, load_launch=launch, offload_launch=launch, staging_bytes=staging_bytes)
        # load
        pool.load(dev_spans, l0, l1)
        torch.cuda.synchronize()
        pool.check()
        exp = pool_np.copy()
        oracle.load(exp[0], exp[1], P, ora_spans, l0, l1)
        got = _pool_bytes(pool_t)
        if not np.array_equal(got, exp):
            bad = np.argwhere(got != exp)
            raise AssertionError(f"load mismatch at {len(bad)} bytes, first (kv, l, slot, b) = {bad[:4].tolist()}")
        # offload into sentinel-filled chunks
        pool.offload(dev_out, l0, l1)
        torch.cuda.synchronize()
        pool.check()
        oracle.offload(exp[0], exp[1], P, [(eo, HT, T, pg) for eo, (_, HT, T, pg) in zip(ora_out, ora_spans)],
                       l0, l1)
        for i, (ob, eo) in enumerate(zip(outs, ora_out)):
            if not np.array_equal(ob.array, eo):
                bad = np.flatnonzero(ob.array != eo)
                raise AssertionError(f"offload mismatch in span {i} at {len(bad)} bytes, first {bad[:4]}")
        pool.close()
    finally:
        for b in bufs + outs:
            b.free()


@pytest.mark.parametrize("L,H,D,P,S,spans", [
    (2, 4, 64, 16, 4096, [(1024, 1024)]),                 # tiny-pool shape, R = 512 B
    (2, 4, 64, 16, 4096, [(1000, 1024)]),                 # partial last page
    (1, 1, 8, 3, 30, [(7, 9), (0, 2), (5, 5)]),           # R = 16 B, P = 3, empty span
    (3, 8, 128, 1, 5000, [(1000, 1200)]),                 # R = 2 KiB, page size 1
    (2, 4, 128, 16, 2048, [(333, 400), (17, 17), (1, 3)]),  # R = 1 KiB
    (2, 6, 128, 2, 600, [(201, 250)]),                    # R = 1536 B (odd vector count)
    (2, 12, 128, 4, 400, [(77, 80)]),                     # R = 3 KiB (wide, odd)
    (2, 128, 128, 1, 64, [(10, 12), (5, 5)]),             # R = 32 KiB > one step
    (2, 8, 128, 32, 4096, [(500, 512), (64, 64)]),        # P = 32
    (2, 8, 128, 64, 4096, [(1000, 1000)]),                # P = 64
    (2, 2, 64, 5, 1000, [(123, 130), (44, 50)]),          # R = 256 B, P = 5
    (2, 8, 128, 1, 1, [(1, 1)]),                          # a one-slot pool
    (1, 1, 8, 128, 128, [(100, 128)]),                    # a one-page pool, page > one tile
    (2, 8, 128, 256, 1024, [(700, 768)]),                 # P = 256: pages span several tiles
    (1, 4, 64, 100, 1000, [(250, 300), (100, 100)]),      # P = 100 (no shift), > one tile
    (40, 1, 8, 4, 64, [(30, 33), (9, 9)]),                # 80 layer pointers: more than one per lane
])
def test_parity_shapes(kv, L, H, D, P, S, spans):
    run_case(kv, L, H, D, P, S, spans, seed=L * 31 + P)


def test_parity_layer_subrange(kv):
    run_case(kv, 4, 8, 128, 16, 2048, [(300, 320), (50, 64)], l0=1, l1=3, seed=5)


def test_parity_many_spans(kv):
    # 70 contexts: more than one launch's worth of spans, some empty, some partial
    rng = np.random.default_rng(9)
    spans = [(int(t), int(t) + int(e)) for t, e in zip(rng.integers(0, 40, 70), rng.integers(0, 3, 70))]
    run_case(kv, 2, 8, 128, 16, 4096, spans, seed=9)


@pytest.mark.parametrize("wg,threads,tile,flags", [
    (1, 64, 4, 0), (7, 256, 8, 0), (128, 1024, 16, 0), (3, 512, 16, 1), (256, 256, 4, 1),
])
def test_parity_launch_shapes(kv, wg, threads, tile, flags):
    launch = kv.launch(wg, threads, tile, flags)
    run_case(kv, 2, 8, 128, 1, 3000, [(777, 800), (3, 3)], launch=launch, seed=wg)
    run_case(kv, 2, 4, 64, 16, 4096, [(1000, 1024)], launch=launch, seed=wg + 1)
    run_case(kv, 1, 1, 8, 3, 300, [(70, 80)], launch=launch, seed=wg + 2)
    # Rows of 24 and 96 vectors (384 B and 1536 B, narrow): a lane's vectors 64
    # apart advance by 2 rows + 16 columns and by 0 rows + 64 columns, so the
    # column carries into the row on some vectors and not on others.
    run_case(kv, 2, 3, 64, 5, 2000, [(403, 410), (64, 64)], launch=launch, seed=wg + 3)
    run_case(kv, 2, 12, 64, 2, 1200, [(301, 301), (5, 9)], launch=launch, seed=wg + 4)


@pytest.mark.parametrize("wg,threads,why", [
    (1, 256, "4 waves: the next tile is in the same plane"),
    (2, 1024, "32 waves: the next tile is in the next plane (wrap)"),
    (4, 1024, "64 waves: the next tile is planes further on (division)"),
    (16, 64, "16 waves over many small spans: the span search"),
])
def test_tile_cursor_paths(kv, wg, threads, why):
    """Each way a wave's tile cursor moves to its next tile, with planes of
    20 tiles (40 tokens of 2 KiB rows in 4 KiB steps) over 12 planes, and a
    run of one- to three-tile spans for the span search."""
    launch = kv.launch(wg, threads, 4, 0)
    run_case(kv, 6, 8, 128, 16, 2048, [(40, 40)], launch=launch, seed=wg)
    run_case(kv, 6, 8, 128, 16, 4096, [(2 * (i % 3) + 1, 6) for i in range(30)] + [(0, 4), (5, 5)],
             launch=launch, seed=wg + 50)


def _staging(slot_pages, P, R):
    """staging_bytes whose 4 slots hold slot_pages pages of K and V rows each
    (0 = the library default), plus a few bytes the library rounds away."""
    return 0 if slot_pages == 0 else 4 * slot_pages * 2 * P * R + 48


@pytest.mark.parametrize("slot_pages", [1, 3, 10])
def test_parity_staged(kv, slot_pages):
    """KVIO_LAUNCH_STAGED: copy-engine copies through HBM staging slots and a
    scatter / gather kernel.  Small slots split spans into units of whole
    pages and cycle the four slots many times per call.  Every call here
    moves at least one slot's worth of rows, so it takes the staged path
    (a staged call smaller than min(64 MiB, one slot) runs on the kernel
    path; test_small_staged_calls_take_the_kernel_path)."""
    for flags in (kv.KVIO_LAUNCH_STAGED, kv.KVIO_LAUNCH_STAGED | kv.KVIO_LAUNCH_CACHED):
        launch = kv.launch(flags=flags)
        run_case(kv, 2, 8, 128, 16, 4096, [(1000, 1024), (333, 400), (0, 5), (17, 17)], launch=launch,
                 seed=40 + flags, staging_bytes=_staging(slot_pages, 16, 2048))
        run_case(kv, 3, 8, 128, 1, 5000, [(1000, 1200), (1, 1)], l0=1, l1=3, launch=launch, seed=41,
                 staging_bytes=_staging(slot_pages, 1, 2048))
        run_case(kv, 1, 1, 8, 3, 300, [(70, 80), (5, 9)], launch=launch, seed=42,
                 staging_bytes=_staging(slot_pages, 3, 16))
        run_case(kv, 2, 6, 128, 2, 600, [(201, 250)], launch=launch, seed=43,
                 staging_bytes=_staging(slot_pages, 2, 1536))
    # small scatter launches and every tile size
    for wg, th, tile in ((1, 64, 4), (7, 256, 8), (64, 512, 16)):
        run_case(kv, 2, 4, 64, 16, 4096, [(1000, 1024)], launch=kv.launch(wg, th, tile, kv.KVIO_LAUNCH_STAGED),
                 seed=44 + wg, staging_bytes=_staging(slot_pages, 16, 512))


def test_parity_staged_many_spans(kv):
    # 70 contexts: more units than one scatter launch carries (2-page slots, so the call is staged)
    rng = np.random.default_rng(19)
    spans = [(int(t), int(t) + int(e)) for t, e in zip(rng.integers(0, 40, 70), rng.integers(0, 3, 70))]
    run_case(kv, 2, 8, 128, 16, 4096, spans, launch=kv.launch(flags=kv.KVIO_LAUNCH_STAGED), seed=20,
             staging_bytes=_staging(2, 16, 2048))


def test_small_staged_calls_take_the_kernel_path(kv):
    """With the default 4 GiB of staging (1 GiB slots), calls that move less
    than 64 MiB run on the kernel path in the default shape; the results are
    the same.  These cases check that fallback, not the staged path."""
    staged = kv.launch(flags=kv.KVIO_LAUNCH_STAGED)
    rng = np.random.default_rng(19)
    spans = [(int(t), int(t) + int(e)) for t, e in zip(rng.integers(0, 40, 70), rng.integers(0, 3, 70))]
    run_case(kv, 2, 8, 128, 16, 4096, spans, launch=staged, seed=19)
    run_case(kv, 2, 8, 128, 16, 4096, [(1000, 1024), (333, 400), (0, 5), (17, 17)], launch=staged, seed=40)
    run_case(kv, 3, 8, 128, 1, 5000, [(1000, 1200), (1, 1)], l0=1, l1=3, launch=staged, seed=41)
    run_case(kv, 1, 1, 8, 3, 300, [(70, 80), (5, 9)], launch=staged, seed=42)


def test_staged_calls_keep_stream_order(kv):
    """Staged offload, then staged load of the same host chunk into other
    pages, then an offload of those pages, all queued on one stream with no
    host synchronisation: each call must see the previous one's results (the
    copies of one run on the pool's own copy streams)."""
    import torch
    L, H, D, P, S, T = 4, 8, 128, 16, 4096, 1000
    R = H * D * 2
    pool_np, pool_t = _pool(L, S, H, D, 23)
    rng = np.random.default_rng(23)
    need = -(-T // P)
    perm = rng.permutation(S // P)[:2 * need].astype(np.int32)
    pa, pb = torch.from_numpy(perm[:need].copy()).cuda(), torch.from_numpy(perm[need:].copy()).cuda()
    staged = kv.launch(flags=kv.KVIO_LAUNCH_STAGED)
    with kv.HostBuffer(L * 2 * T * R) as mid, kv.HostBuffer(L * 2 * T * R) as out:
        mid.array[:] = 0
        out.array[:] = 0
        pool = kv.KVPool(pool_t, P, load_launch=staged, offload_launch=staged, staging_bytes=_staging(3, P, R))
        s = torch.cuda.Stream()
        for _ in range(2):
            pool.offload([(mid.ptr, T, T, pa.data_ptr())], stream=s)     # pages A -> mid
            pool.load([(mid.ptr, T, T, pb.data_ptr())], stream=s)        # mid -> pages B
            pool.offload([(out.ptr, T, T, pb.data_ptr())], stream=s)     # pages B -> out
        s.synchronize()
        pool.check()
        exp = pool_np.copy()
        e_mid = np.zeros(L * 2 * T * R, np.uint8)
        oracle.offload(exp[0], exp[1], P, [(e_mid, T, T, perm[:need])])
        oracle.load(exp[0], exp[1], P, [(e_mid, T, T, perm[need:])])
        assert np.array_equal(mid.array, e_mid)
        assert np.array_equal(out.array, e_mid)
        assert np.array_equal(_pool_bytes(pool_t), exp)
        pool.close()


def test_staged_layer_call_and_errors(kv):
    """kvio_load_layer in staged mode, its event, and an out-of-range page
    reported with the caller's span and context page although the span was
    split into staging units."""
    import torch
    L, H, D, P, S = 3, 8, 128, 16, 2048
    R = H * D * 2
    pool_np, pool_t = _pool(L, S, H, D, 21)
    T = 200
    pages = np.random.default_rng(21).permutation(S // P)[:-(-T // P)].astype(np.int32)
    pt = torch.from_numpy(pages.copy()).cuda()
    staged = kv.launch(flags=kv.KVIO_LAUNCH_STAGED)
    with kv.HostBuffer(L * 2 * T * R) as hb:
        W.fill_np(hb.array, 21, W.LLAMA8B)
        pool = kv.KVPool(pool_t, P, load_launch=staged, offload_launch=staged, staging_bytes=_staging(2, P, R))
        s = torch.cuda.Stream()
        ev = torch.cuda.Event()
        for l in range(L):
            pool.load_layer([(hb.ptr, T, T, pt.data_ptr())], l, stream=s, done=ev)
        ev.synchronize()
        torch.cuda.synchronize()
        pool.check()
        exp = pool_np.copy()
        oracle.load(exp[0], exp[1], P, [(hb.array, T, T, pages)])
        assert np.array_equal(_pool_bytes(pool_t), exp)
        bad = pages.copy()
        bad[9] = S // P + 5                                  # context page 9 of span 1 is out of range
        pb = torch.from_numpy(bad).cuda()
        pool.load([(hb.ptr, T, 0, pt.data_ptr()), (hb.ptr, T, T, pb.data_ptr())])
        torch.cuda.synchronize()
        with pytest.raises(kv.KvioError) as e:
            pool.check()
        assert e.value.status == kv.KVIO_ERANGE
        assert "span 1" in e.value.detail and "context page 9" in e.value.detail, e.value.detail
        pool.close()
    with pytest.raises(kv.KvioError) as e:                  # slots smaller than one page of K and V
        kv.KVPool(pool_t, P, load_launch=staged, staging_bytes=4 * 2 * P * R - 16)
    assert e.value.status == kv.KVIO_EINVAL
    with pytest.raises(kv.KvioError) as e:                  # staged transfers do not take page-first chunks
        kv.KVPool(pool_t, P, offload_launch=staged, host_layout=kv.KVIO_HOST_PAGE_FIRST)
    assert e.value.status == kv.KVIO_EINVAL


@pytest.mark.parametrize("flags", [0, 0x4])
def test_empty_batches_are_no_ops(kv, flags):
    """No spans, or spans with no tokens, in every call: nothing moves and
    nothing is reported (plain and staged launches)."""
    import torch
    L, H, D, P, S = 2, 8, 128, 16, 1024
    R = H * D * 2
    pool_np, pool_t = _pool(L, S, H, D, 30)
    launch = kv.launch(flags=flags)
    pool = kv.KVPool(pool_t, P, load_launch=launch, offload_launch=launch)
    pt = torch.zeros(1, dtype=torch.int32, device="cuda")
    with kv.HostBuffer(L * 2 * 16 * R) as hb:
        hb.array[:] = 0x77
        for spans in ([], [(hb.ptr, 16, 0, pt.data_ptr())], [(hb.ptr, 0, 0, pt.data_ptr())] * 3):
            pool.load(spans)
            pool.offload(spans)
            pool.load_layer(spans, L - 1)
        torch.cuda.synchronize()
        pool.check()
        assert np.array_equal(_pool_bytes(pool_t), pool_np)
        assert (hb.array == 0x77).all()
    pool.close()


def test_torch_pinned_host_memory(kv):
    """Host chunks from torch's pinned allocator work like kvio_host_alloc ones."""
    import torch
    L, H, D, P, S, T = 2, 8, 128, 1, 2000, 300
    R = H * D * 2
    pool_np, pool_t = _pool(L, S, H, D, 3)
    host = torch.empty(L * 2 * T * R, dtype=torch.uint8, pin_memory=True)
    W.fill_np(host.numpy(), 3, W.LLAMA8B)
    pages = W.random_slots(np.random.default_rng(3), S, T)
    pt = torch.from_numpy(pages).cuda()
    pool = kv.KVPool(pool_t, P)
    pool.load([(host.data_ptr(), T, T, pt.data_ptr())])
    torch.cuda.synchronize()
    exp = pool_np.copy()
    oracle.load(exp[0], exp[1], P, [(host.numpy(), T, T, pages)])
    assert np.array_equal(_pool_bytes(pool_t), exp)
    pool.close()


def test_load_layer_event_and_naive(kv):
    """kvio_load_layer per layer on a side stream (waited on through its event),
    and the naive per-page DMA baseline, both equal the whole-range oracle load."""
    import torch
    L, H, D, P, S, T = 4, 8, 128, 16, 2048, 500
    R = H * D * 2
    pool_np, pool_a = _pool(L, S, H, D, 4)
    pool_b = pool_a.clone()
    pages = W.random_pages(np.random.default_rng(4), S // P, -(-T // P))
    pt = torch.from_numpy(pages).cuda()
    with kv.HostBuffer(L * 2 * T * R) as hb:
        W.fill_np(hb.array, 4, W.LLAMA8B)
        span = [(hb.ptr, T, T, pt.data_ptr())]
        pa, pb = kv.KVPool(pool_a, P), kv.KVPool(pool_b, P)
        side = torch.cuda.Stream()
        compute = torch.cuda.current_stream()
        sums = []
        for l in range(L):
            ev = torch.cuda.Event()
            ev.record(side)                       # materialise the event handle
            pa.load_layer(span, l, stream=side, done=ev)
            compute.wait_event(ev)
            sums.append(pool_a[:, l].float().sum())   # compute-stream consumer of layer l
        kv.kvio_naive_load(pb.handle, span, 0, L, stream=side)
        torch.cuda.synchronize()
        exp = pool_np.copy()
        oracle.load(exp[0], exp[1], P, [(hb.array, T, T, pages)])
        assert np.array_equal(_pool_bytes(pool_a), exp)
        assert np.array_equal(_pool_bytes(pool_b), exp)
        # naive offload equals the oracle offload
        with kv.HostBuffer(L * 2 * T * R) as ob:
            ob.array[:] = 0x5A
            kv.kvio_naive_offload(pb.handle, [(ob.ptr, T, T, pt.data_ptr())], 0, L)
            torch.cuda.synchronize()
            eo = np.full(ob.array.size, 0x5A, np.uint8)
            oracle.offload(exp[0], exp[1], P, [(eo, T, T, pages)])
            assert np.array_equal(ob.array, eo)
        pa.close()
        pb.close()


def test_out_of_range_page_is_skipped_and_reported(kv):
    """A page index past the pool is caught by the kernel's own range check:
    the row is skipped (never dereferenced) and kvio_check reports it."""
    import torch
    L, H, D, P, S, T = 2, 8, 128, 16, 1024, 64
    R = H * D * 2
    pool_np, pool_t = _pool(L, S, H, D, 6)
    pages = np.array([3, S // P, 7, 1], np.int32)         # context page 1 is out of range
    pt = torch.from_numpy(pages).cuda()
    with kv.HostBuffer(L * 2 * T * R) as hb:
        W.fill_np(hb.array, 6, W.LLAMA8B)
        pool = kv.KVPool(pool_t, P)
        pool.load([(hb.ptr, T, T, pt.data_ptr())])
        torch.cuda.synchronize()
        with pytest.raises(kv.KvioError) as e:
            pool.check()
        assert e.value.status == kv.KVIO_ERANGE and "context page 1" in e.value.detail
        pool.check()                                     # the record was cleared
        # every other row moved exactly as the oracle moves the valid pages
        exp = pool_np.copy()
        h = hb.array.reshape(L, 2, T, R)
        for kvi in range(2):
            for l in range(L):
                for j in (0, 2, 3):
                    exp[kvi, l, pages[j] * P:(pages[j] + 1) * P] = h[l, kvi, j * P:(j + 1) * P]
        assert np.array_equal(_pool_bytes(pool_t), exp)
        pool.close()


@pytest.mark.parametrize("layout", [oracle.TOKEN_MAJOR, oracle.PAGE_FIRST, oracle.HEAD_MAJOR])
@pytest.mark.parametrize("tile", [4, 8, 16])
def test_out_of_range_page_every_layout_and_step(kv, layout, tile):
    """The range check on every host layout and step size, both directions
    (head-major loads with steps of 8 KiB or more check the page after their
    host reads are issued).  Expected images come from the oracle run on a
    pool one page larger, where the bad index is a valid page: its first S
    slots are the GPU pool after the load, and the offload leaves untouched
    exactly the host bytes that page would supply (found by running the
    oracle with that page all zeros and all ones)."""
    import torch
    L, H, D, P, S, T = 2, 8, 128, 16, 1024, 64
    R = H * D * 2
    pool_np, pool_t = _pool(L, S, H, D, 60 + tile + 7 * layout)
    pages = np.array([3, S // P, 7, 1], np.int32)         # context page 1 is out of range
    pt = torch.from_numpy(pages).cuda()
    nbytes = oracle.host_chunk_bytes(layout, L, T, R, P)
    shape = kv.launch(0, 0, tile, 0)
    with kv.HostBuffer(nbytes) as hb, kv.HostBuffer(nbytes) as ob:
        W.fill_np(hb.array, 60 + tile, W.LLAMA8B)
        ob.array[:] = 0x5A
        pool = kv.KVPool(pool_t, P, load_launch=shape, offload_launch=shape, host_layout=layout)
        try:
            pool.load([(hb.ptr, T, T, pt.data_ptr())])
            torch.cuda.synchronize()
            with pytest.raises(kv.KvioError) as e:
                pool.check()
            assert e.value.status == kv.KVIO_ERANGE and "context page 1" in e.value.detail
            big = np.zeros((2, L, S + P, R), np.uint8)
            big[:, :, :S] = pool_np
            oracle.load_layout(big[0], big[1], P, [(hb.array, T, T, pages)], layout, num_heads=H)
            assert np.array_equal(_pool_bytes(pool_t), big[:, :, :S])
            pool.offload([(ob.ptr, T, T, pt.data_ptr())])
            torch.cuda.synchronize()
            with pytest.raises(kv.KvioError) as e:
                pool.check()
            assert e.value.status == kv.KVIO_ERANGE and "context page 1" in e.value.detail
            outs = []
            for extra in (0x00, 0xFF):
                b2 = big.copy()
                b2[:, :, S:] = extra
                eo = np.full(nbytes, 0x5A, np.uint8)
                oracle.offload_layout(b2[0], b2[1], P, [(eo, T, T, pages)], layout, num_heads=H)
                outs.append(eo)
            exp = outs[0].copy()
            skipped = outs[0] != outs[1]
            assert skipped.sum() == L * 2 * P * R            # exactly that page's rows
            exp[skipped] = 0x5A
            assert np.array_equal(ob.array, exp)
        finally:
            pool.close()


def test_validation_errors(kv):
    """Synchronous validation: nothing is enqueued, the pool is untouched."""
    import torch
    L, H, D, P, S, T = 2, 8, 128, 16, 1024, 64
    R = H * D * 2
    pool_np, pool_t = _pool(L, S, H, D, 8)
    pt = torch.arange(4, dtype=torch.int32, device="cuda")
    pool = kv.KVPool(pool_t, P)
    with kv.HostBuffer(L * 2 * T * R + 64) as hb:
        cases = [
            ([(hb.ptr, T - 1, T, pt.data_ptr())], 0, L, kv.KVIO_EINVAL),     # num_tokens > host_tokens
            ([(hb.ptr, T, T, pt.data_ptr())], 0, L + 1, kv.KVIO_EINVAL),     # layer range past L
            ([(hb.ptr, T, T, pt.data_ptr())], 1, 1, kv.KVIO_EINVAL),         # empty layer range
            ([(hb.ptr + 8, T, T, pt.data_ptr())], 0, L, kv.KVIO_EALIGN),     # misaligned host chunk
            ([(0, T, T, pt.data_ptr())], 0, L, kv.KVIO_EINVAL),              # null host chunk
            ([(hb.ptr, T, T, 0)], 0, L, kv.KVIO_EINVAL),                     # null page table
        ]
        plain = np.zeros(L * 2 * T * R, np.uint8)                            # plain malloc memory
        cases.append(([(plain.ctypes.data, T, T, pt.data_ptr())], 0, L, kv.KVIO_ENOTMAPPED))
        for spans, l0, l1, code in cases:
            for call in (pool.load, pool.offload):
                with pytest.raises(kv.KvioError) as e:
                    call(spans, l0, l1)
                assert e.value.status == code, (call, spans, e.value)
                assert e.value.detail and kv.kvio_last_error() == e.value.detail
        torch.cuda.synchronize()
        assert np.array_equal(_pool_bytes(pool_t), pool_np)
    with pytest.raises(kv.KvioError) as e:
        kv.KVPool(pool_t, 3)                                  # S % P != 0
    assert e.value.status == kv.KVIO_EINVAL
    with pytest.raises(kv.KvioError) as e:
        kv.KVPool(pool_t, P, load_launch=kv.launch(threads=100))
    assert e.value.status == kv.KVIO_EINVAL
    pool.close()


def test_undersized_buffers_rejected(kv):
    """The runtime's allocation extent bounds every transfer: a host chunk, page
    table or pool layer shorter than the transfer reaches is refused."""
    import torch
    L, H, D, P, S, T = 2, 8, 128, 16, 1024, 64
    R = H * D * 2
    pool_np, pool_t = _pool(L, S, H, D, 10)
    pool = kv.KVPool(pool_t, P)
    pt = torch.arange(4, dtype=torch.int32, device="cuda")
    with kv.HostBuffer(L * 2 * T * R - 16) as hb:            # 16 B short of the last V row
        with pytest.raises(kv.KvioError) as e:
            pool.load([(hb.ptr, T, T, pt.data_ptr())])
        assert e.value.status == kv.KVIO_EINVAL and "allocation holds" in e.value.detail
        pool.load([(hb.ptr, T, T - 1, pt.data_ptr())], 0, L)  # one row fewer stays inside: accepted
    # A page table whose allocation ends after 3 entries (T = 64 needs 4).
    # (A torch tensor would sit inside a larger caching-allocator segment, so
    # the runtime extent is taken from a buffer of its own.)
    with kv.HostBuffer(L * 2 * T * R) as hb, kv.HostBuffer(4096) as tb:
        tb.array.view(np.int32)[-3:] = [0, 1, 2]
        with pytest.raises(kv.KvioError) as e:
            pool.load([(hb.ptr, T, T, tb.ptr + 4096 - 12)])
        assert e.value.status == kv.KVIO_EINVAL
    torch.cuda.synchronize()
    pool.close()
    # Pool layers in one raw device allocation 16 B short of 2 * L layers.
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so.7")
    dev = ctypes.c_void_p()
    nbytes = 2 * L * S * R - 16
    assert hip.hipMalloc(ctypes.byref(dev), ctypes.c_size_t(nbytes)) == 0
    try:
        layers = [dev.value + i * S * R for i in range(2 * L)]
        with pytest.raises(kv.KvioError) as e:
            kv.kvio_pool_create(L, H, D, 2, P, S, layers[:L], layers[L:])
        assert e.value.status == kv.KVIO_EINVAL and "allocation holds" in e.value.detail
        h = kv.kvio_pool_create(L, H, D, 2, P, S - P, layers[:L], layers[L:])   # one page fewer fits
        kv.kvio_pool_destroy(h)
    finally:
        torch.cuda.synchronize()
        hip.hipFree(dev)


@pytest.mark.parametrize("staged", [False, True])
def test_offload_reads_shared_and_repeated_pages(kv, staged):
    """Offload may name a pool page any number of times: contexts that share a
    prefix page, a page repeated inside one table.  Every host row receives its
    page's row, as the oracle's offload gives."""
    import torch
    L, H, D, P, S = 2, 4, 64, 16, 1024
    R = H * D * 2
    pool_np, pool_t = _pool(L, S, H, D, 55)
    pages = np.random.default_rng(55).permutation(S // P)[:6].astype(np.int32)
    tables = [pages[:6],                                        # context A
              np.concatenate([pages[:4], pages[[0, 0, 5]]]),    # B shares A's first pages, repeats one
              pages[[3, 3, 3]]]                                 # one page three times
    lens = [6 * P - 5, 7 * P, 2 * P + 1]
    launch = kv.launch(flags=kv.KVIO_LAUNCH_STAGED) if staged else None
    pool = kv.KVPool(pool_t, P, offload_launch=launch, staging_bytes=4 * 2 * 2 * P * R if staged else 0)
    outs, pts, ora = [], [], []
    try:
        for tab, T in zip(tables, lens):
            ob = kv.HostBuffer(L * 2 * T * R)
            ob.array[:] = 0x3C
            outs.append(ob)
            pts.append(torch.from_numpy(tab.copy()).cuda())
            ora.append((np.full(ob.array.size, 0x3C, np.uint8), T, T, tab))
        pool.offload([(ob.ptr, T, T, pt.data_ptr()) for ob, pt, (_, T, _, _) in zip(outs, pts, ora)])
        torch.cuda.synchronize()
        pool.check()
        exp = pool_np.copy()
        oracle.offload(exp[0], exp[1], P, ora)
        for i, ((eo, _, _, _), ob) in enumerate(zip(ora, outs)):
            assert np.array_equal(ob.array, eo), f"offload span {i} differs from the oracle"
        assert np.array_equal(_pool_bytes(pool_t), pool_np), "an offload changed the pool"
    finally:
        pool.close()
        for ob in outs:
            ob.free()


def test_load_naming_a_slot_twice_fills_it_from_its_rows(kv):
    """A load whose table names a page twice is the caller's mistake (the
    oracle rejects it); the library promises only that each 16-byte piece of
    such a slot holds that piece of one of the rows named for it.  Every other
    slot gets exactly what the oracle gives for the same load without the
    repeat."""
    import torch
    L, H, D, P, S = 2, 8, 128, 4, 256               # R = 2 KiB: rows span several 16-byte pieces
    R = H * D * 2
    pool_np, pool_t = _pool(L, S, H, D, 66)
    pages = np.random.default_rng(66).permutation(S // P)[:3].astype(np.int32)
    table = np.array([pages[0], pages[1], pages[0], pages[2]], np.int32)   # context pages 0 and 2 collide
    T = 4 * P - 1
    pool = kv.KVPool(pool_t, P)
    with kv.HostBuffer(L * 2 * T * R) as hb:
        W.fill_np(hb.array, 66, W.LLAMA8B)
        pt = torch.from_numpy(table).cuda()
        pool.load([(hb.ptr, T, T, pt.data_ptr())])
        torch.cuda.synchronize()
        pool.check()
        got = _pool_bytes(pool_t)
        # the oracle's load of context pages 1 and 3 only (no repeat)
        exp = pool_np.copy()
        host = hb.array.reshape(L, 2, T, R)
        for j in (1, 3):
            n = min(P, T - j * P)
            sub = np.ascontiguousarray(host[:, :, j * P:j * P + n]).reshape(-1)
            oracle.load(exp[0], exp[1], P, [(sub, n, n, table[j:j + 1])])
        dup = set(range(int(pages[0]) * P, int(pages[0]) * P + P))
        other = np.array([s not in dup for s in range(S)])
        assert np.array_equal(got[:, :, other], exp[:, :, other]), "a slot outside the repeated page differs"
        for o in range(P):
            slot = int(pages[0]) * P + o
            cands = [host[:, :, j * P + o] for j in (0, 2) if j * P + o < T]
            pieces_got = got[:, :, slot].transpose(1, 0, 2).reshape(L, 2, R // 16, 16)   # (layer, kv, ...)
            ok = np.zeros((L, 2, R // 16), bool)
            for c in cands:
                ok |= (pieces_got == c.reshape(L, 2, R // 16, 16)).all(axis=-1)
            assert ok.all(), f"slot {slot}: a 16-byte piece matches none of its rows"
    pool.close()


def test_one_pool_from_several_host_threads(kv):
    """One pool handle used by four host threads at once, each on its own
    stream with its own context in pages no other thread touches (ctypes
    releases the interpreter lock during the calls).  Each thread also makes an
    invalid call and must read its own error text (the text is per thread)."""
    import threading
    import torch
    L, H, D, P, S = 2, 8, 128, 16, 8192
    R = H * D * 2
    n_threads, T = 4, 300
    need = -(-T // P)
    pool_np, pool_t = _pool(L, S, H, D, 88)
    perm = np.random.default_rng(88).permutation(S // P)[:n_threads * need].astype(np.int32)
    tables = [perm[i * need:(i + 1) * need] for i in range(n_threads)]
    pts = [torch.from_numpy(t.copy()).cuda() for t in tables]
    streams = [torch.cuda.Stream() for _ in range(n_threads)]
    hbs = [kv.HostBuffer(L * 2 * T * R) for _ in range(n_threads)]
    obs = [kv.HostBuffer(L * 2 * T * R) for _ in range(n_threads)]
    pool = kv.KVPool(pool_t, P)
    failures = [None] * n_threads
    try:
        for i in range(n_threads):
            W.fill_np(hbs[i].array, 880 + i, W.LLAMA8B)
            obs[i].array[:] = 0
        torch.cuda.synchronize()

        def work(i):
            try:
                span_in = [(hbs[i].ptr, T, T, pts[i].data_ptr())]
                span_out = [(obs[i].ptr, T, T, pts[i].data_ptr())]
                for _ in range(10):
                    pool.load(span_in, stream=streams[i])
                    pool.offload(span_out, stream=streams[i])
                    with pytest.raises(kv.KvioError) as e:
                        pool.load(span_in, 0, L + 1 + i, stream=streams[i])
                    assert f"[0, {L + 1 + i})" in e.value.detail, e.value.detail
                streams[i].synchronize()
            except BaseException as exc:          # reported by the main thread
                failures[i] = exc

        threads = [threading.Thread(target=work, args=(i,)) for i in range(n_threads)]
        for t in threads:
            t.start()
        for t in threads:
            t.join()
        assert failures == [None] * n_threads, failures
        torch.cuda.synchronize()
        pool.check()
        exp = pool_np.copy()
        oracle.load(exp[0], exp[1], P, [(hbs[i].array, T, T, tables[i]) for i in range(n_threads)])
        assert np.array_equal(_pool_bytes(pool_t), exp), "pool differs from the oracle"
        for i in range(n_threads):
            assert np.array_equal(obs[i].array, hbs[i].array), f"thread {i}: round trip differs"
    finally:
        pool.close()
        for b in hbs + obs:
            b.free()


def test_transfers_on_a_stream_masked_to_16_cus(kv):
    """kvio_stream_create with a CU mask of 16 compute units (the load's default
    quota): a load and an offload on that stream match the oracle.  The runtime
    allows few masked streams per process; if it refuses one more, the test is
    skipped."""
    import torch
    try:
        st = kv.Stream(list(range(16)))
    except kv.KvioError as e:
        pytest.skip(f"the runtime refused another CU-masked stream: {e.detail}")
    try:
        L, H, D, P, S = 2, 8, 128, 16, 4096
        R = H * D * 2
        pool_np, pool_t = _pool(L, S, H, D, 99)
        T = 1500
        pages = np.random.default_rng(99).permutation(S // P)[:-(-T // P)].astype(np.int32)
        pt = torch.from_numpy(pages).cuda()
        pool = kv.KVPool(pool_t, P)
        with kv.HostBuffer(L * 2 * T * R) as hb, kv.HostBuffer(L * 2 * T * R) as ob:
            W.fill_np(hb.array, 99, W.LLAMA8B)
            ob.array[:] = 0
            torch.cuda.synchronize()
            pool.load([(hb.ptr, T, T, pt.data_ptr())], stream=st)
            pool.offload([(ob.ptr, T, T, pt.data_ptr())], stream=st)
            torch.cuda.synchronize()
            pool.check()
            exp = pool_np.copy()
            oracle.load(exp[0], exp[1], P, [(hb.array, T, T, pages)])
            assert np.array_equal(_pool_bytes(pool_t), exp)
            assert np.array_equal(ob.array, hb.array)
        pool.close()
    finally:
        st.close()


@pytest.mark.parametrize("layout,staged", [(0, False), (0, True), (2, False), (2, True)])
def test_noncoherent_host_chunks(kv, layout, staged):
    """Coarse-grained (non-coherent) pinned host chunks: the offload's host
    writes are visible to the CPU after synchronisation and both directions
    match the oracle, on the kernel path and staged."""
    import torch
    L, H, D, P, S = 2, 8, 128, 16, 4096
    R = H * D * 2
    T, HT = 1000, 1010
    pool_np, pool_t = _pool(L, S, H, D, 101 + layout)
    pages = np.random.default_rng(101).permutation(S // P)[:-(-T // P)].astype(np.int32)
    pt = torch.from_numpy(pages).cuda()
    launch = kv.launch(flags=kv.KVIO_LAUNCH_STAGED) if staged else None
    pool = kv.KVPool(pool_t, P, load_launch=launch, offload_launch=launch, host_layout=layout,
                     staging_bytes=4 * 4 * 2 * P * R if staged else 0)
    ora_layout = {0: oracle.TOKEN_MAJOR, 2: oracle.HEAD_MAJOR}[layout]
    nbytes = oracle.host_chunk_bytes(ora_layout, L, HT, R, P)
    with kv.HostBuffer(nbytes, kv.KVIO_HOST_NONCOHERENT) as hb, \
            kv.HostBuffer(nbytes, kv.KVIO_HOST_NONCOHERENT) as ob:
        W.fill_np(hb.array, 101, W.LLAMA8B)
        ob.array[:] = 0x77
        pool.load([(hb.ptr, HT, T, pt.data_ptr())])
        pool.offload([(ob.ptr, HT, T, pt.data_ptr())])
        torch.cuda.synchronize()
        pool.check()
        exp = pool_np.copy()
        oracle.load_layout(exp[0], exp[1], P, [(hb.array, HT, T, pages)], ora_layout, num_heads=H)
        assert np.array_equal(_pool_bytes(pool_t), exp), "load differs from the oracle"
        exp_out = np.full(nbytes, 0x77, np.uint8)
        oracle.offload_layout(exp[0], exp[1], P, [(exp_out, HT, T, pages)], ora_layout, num_heads=H)
        assert np.array_equal(ob.array, exp_out), "offload differs from the oracle"
    pool.close()


@pytest.mark.parametrize("layout", [0, 1, 2])
def test_chunks_in_device_memory(kv, layout):
    """A span's chunk may be device memory (a contiguous copy of the context
    kept in HBM): the same layout conversion, HBM to HBM, matches the oracle."""
    import torch
    L, H, D, P, S = 2, 8, 128, 16, 4096
    R = H * D * 2
    T, HT = 777, 784                               # HT: whole pages, valid for every layout
    pool_np, pool_t = _pool(L, S, H, D, 111 + layout)
    pages = np.random.default_rng(111).permutation(S // P)[:-(-T // P)].astype(np.int32)
    pt = torch.from_numpy(pages).cuda()
    ora_layout = {0: oracle.TOKEN_MAJOR, 1: oracle.PAGE_FIRST, 2: oracle.HEAD_MAJOR}[layout]
    nbytes = oracle.host_chunk_bytes(ora_layout, L, HT, R, P)
    src = np.zeros(nbytes, np.uint8)
    W.fill_np(src, 111, W.LLAMA8B)
    d_src = torch.from_numpy(src).cuda()
    d_out = torch.full((nbytes,), 0x55, dtype=torch.uint8, device="cuda")
    pool = kv.KVPool(pool_t, P, host_layout=layout)
    pool.load([(d_src.data_ptr(), HT, T, pt.data_ptr())])
    pool.offload([(d_out.data_ptr(), HT, T, pt.data_ptr())])
    torch.cuda.synchronize()
    pool.check()
    exp = pool_np.copy()
    oracle.load_layout(exp[0], exp[1], P, [(src, HT, T, pages)], ora_layout, num_heads=H)
    assert np.array_equal(_pool_bytes(pool_t), exp), "load differs from the oracle"
    exp_out = np.full(nbytes, 0x55, np.uint8)
    oracle.offload_layout(exp[0], exp[1], P, [(exp_out, HT, T, pages)], ora_layout, num_heads=H)
    assert np.array_equal(d_out.cpu().numpy(), exp_out), "offload differs from the oracle"
    pool.close()


def test_staged_load_and_offload_concurrently_on_one_handle(kv):
    """Both directions staged on one pool handle, a load of context X on one
    stream while an offload of context Y (other pages) runs on another, several
    times over without host synchronisation: each direction has its own staging
    slots and side stream, so the two may overlap."""
    import torch
    L, H, D, P, S, T = 4, 8, 128, 16, 4096, 1000
    R = H * D * 2
    pool_np, pool_t = _pool(L, S, H, D, 121)
    need = -(-T // P)
    perm = np.random.default_rng(121).permutation(S // P)[:2 * need].astype(np.int32)
    px, py = perm[:need].copy(), perm[need:].copy()
    tx, ty = torch.from_numpy(px).cuda(), torch.from_numpy(py).cuda()
    staged = kv.launch(flags=kv.KVIO_LAUNCH_STAGED)
    pool = kv.KVPool(pool_t, P, load_launch=staged, offload_launch=staged, staging_bytes=_staging(2, P, R))
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    with kv.HostBuffer(L * 2 * T * R) as hx, kv.HostBuffer(L * 2 * T * R) as oy:
        W.fill_np(hx.array, 121, W.LLAMA8B)
        oy.array[:] = 0
        torch.cuda.synchronize()
        for _ in range(3):
            pool.load([(hx.ptr, T, T, tx.data_ptr())], stream=sa)
            pool.offload([(oy.ptr, T, T, ty.data_ptr())], stream=sb)
        sa.synchronize()
        sb.synchronize()
        pool.check()
        exp = pool_np.copy()
        oracle.load(exp[0], exp[1], P, [(hx.array, T, T, px)])
        e_y = np.zeros(L * 2 * T * R, np.uint8)
        oracle.offload(pool_np[0].copy(), pool_np[1].copy(), P, [(e_y, T, T, py)])
        assert np.array_equal(_pool_bytes(pool_t), exp), "load differs from the oracle"
        assert np.array_equal(oy.array, e_y), "offload differs from the oracle"
    pool.close()


@pytest.mark.parametrize("layout,staged", [(0, False), (0, True), (1, False), (2, False)])
def test_one_byte_elements(kv, layout, staged):
    """An 8-bit KV cache (e.g. fp8 elements; the copy never looks at values):
    rows of H * D bytes, against the oracle."""
    import torch
    L, H, D, P, S = 2, 8, 128, 16, 4096            # R = 1 KiB; head segments of 128 B
    R = H * D
    T, HT = 900, 912
    rng = np.random.default_rng(131 + layout)
    pool_np = rng.integers(0, 256, size=(2, L, S, R), dtype=np.uint8)
    pool_t = torch.from_numpy(pool_np.reshape(2, L, S, H, D).copy()).cuda()
    pages = rng.permutation(S // P)[:-(-T // P)].astype(np.int32)
    pt = torch.from_numpy(pages).cuda()
    launch = kv.launch(flags=kv.KVIO_LAUNCH_STAGED) if staged else None
    pool = kv.KVPool(pool_t, P, load_launch=launch, offload_launch=launch, host_layout=layout,
                     staging_bytes=4 * 4 * 2 * P * R if staged else 0)
    assert pool.row_bytes == R
    ora_layout = {0: oracle.TOKEN_MAJOR, 1: oracle.PAGE_FIRST, 2: oracle.HEAD_MAJOR}[layout]
    nbytes = oracle.host_chunk_bytes(ora_layout, L, HT, R, P)
    with kv.HostBuffer(nbytes) as hb, kv.HostBuffer(nbytes) as ob:
        hb.array[:] = rng.integers(0, 256, nbytes, dtype=np.uint8)
        ob.array[:] = 0x2D
        pool.load([(hb.ptr, HT, T, pt.data_ptr())])
        pool.offload([(ob.ptr, HT, T, pt.data_ptr())])
        torch.cuda.synchronize()
        pool.check()
        exp = pool_np.copy()
        oracle.load_layout(exp[0], exp[1], P, [(hb.array, HT, T, pages)], ora_layout, num_heads=H)
        got = pool_t.cpu().numpy().reshape(2, L, S, R)
        assert np.array_equal(got, exp), "load differs from the oracle"
        exp_out = np.full(nbytes, 0x2D, np.uint8)
        oracle.offload_layout(exp[0], exp[1], P, [(exp_out, HT, T, pages)], ora_layout, num_heads=H)
        assert np.array_equal(ob.array, exp_out), "offload differs from the oracle"
    pool.close()


def test_load_layer_records_a_fresh_torch_event(kv):
    """`done` may be a torch event that was never recorded (torch creates its
    HIP event lazily): the binding materialises it and the library records it
    after the launch, so waiting on it alone (no device-wide synchronisation)
    leaves the layer fully loaded.  The layer is 64 MiB, about a millisecond
    of transfer, so an event recorded before the launch would expose rows
    still in flight."""
    import torch
    L, H, D, P, S, T = 2, 8, 128, 16, 32768, 16384
    R = H * D * 2
    pool_np, pool_t = _pool(L, S, H, D, 141)
    pages = np.random.default_rng(141).permutation(S // P)[:T // P].astype(np.int32)
    pt = torch.from_numpy(pages).cuda()
    pool = kv.KVPool(pool_t, P)
    s = torch.cuda.Stream()
    with kv.HostBuffer(L * 2 * T * R) as hb:
        W.fill_np(hb.array, 141, W.LLAMA8B)
        torch.cuda.synchronize()
        ev = torch.cuda.Event()
        assert ev.cuda_event == 0
        pool.load_layer([(hb.ptr, T, T, pt.data_ptr())], 1, stream=s, done=ev)
        assert ev.cuda_event != 0
        ev.synchronize()
        got = pool_t[:, 1].cpu().numpy().view(np.uint8).reshape(2, S, R)   # current stream: idle
        exp = pool_np.copy()
        oracle.load(exp[0], exp[1], P, [(hb.array, T, T, pages)], 1, 2)
        assert np.array_equal(got, exp[:, 1]), "layer 1 incomplete after waiting on its event"
    torch.cuda.synchronize()
    pool.close()


def test_a_failed_runtime_call_does_not_leak_into_the_callers_next_call(kv):
    """A HIP failure inside the library is reported by its status only: the
    runtime's per-thread last error is cleared, so torch's next kernel launch
    (which checks it) still succeeds.  Forced from the host: pinned memory far
    beyond what the machine holds."""
    import torch
    pool_t = torch.zeros((2, 2, 1024, 8, 128), dtype=torch.bfloat16, device="cuda")
    staged = kv.launch(flags=kv.KVIO_LAUNCH_STAGED)
    with pytest.raises(kv.KvioError) as e:          # 1 PiB of HBM staging: the device allocation fails
        kv.KVPool(pool_t, 16, load_launch=staged, staging_bytes=1 << 50)
    assert e.value.status == kv.KVIO_ENOMEM
    x = torch.ones(1 << 20, device="cuda")          # torch checks the last error after its launch
    assert float(x.sum().item()) == float(1 << 20)
    with pytest.raises(kv.KvioError) as e:
        kv.kvio_host_alloc(1 << 52)                 # 4 PiB of pinned host memory
    assert e.value.status in (kv.KVIO_ENOMEM, kv.KVIO_EHIP)
    assert float(torch.ones(1 << 10, device="cuda").sum().item()) == float(1 << 10)


@pytest.mark.parametrize("nbytes", [16, 1008, 16 * 1024 + 16, (5 << 20) + 48, (64 << 20) + 4096])
def test_kernel_memcpy_both_directions(kv, nbytes):
    """kvio_kernel_memcpy (the plain-kernel link ceiling) copies host -> device
    and device -> host byte for byte, partial last steps and several grid
    rounds included, and writes nothing past the end (sentinel tails)."""
    import torch
    src = kv.HostBuffer(nbytes)
    src.array[:] = np.random.default_rng(nbytes).integers(0, 256, nbytes, dtype=np.uint8)
    dev = torch.full((nbytes + 4096,), 0xA5, dtype=torch.uint8, device="cuda")
    kv.kvio_kernel_memcpy(dev.data_ptr(), src.ptr, nbytes)
    torch.cuda.synchronize()
    got = dev.cpu().numpy()
    assert np.array_equal(got[:nbytes], src.array)
    assert (got[nbytes:] == 0xA5).all()
    dst = kv.HostBuffer(nbytes + 4096)
    dst.array[:] = 0x5A
    kv.kvio_kernel_memcpy(dst.ptr, dev.data_ptr(), nbytes)
    torch.cuda.synchronize()
    assert np.array_equal(dst.array[:nbytes], src.array)
    assert (dst.array[nbytes:] == 0x5A).all()
    dev2 = torch.full((nbytes + 4096,), 0x3C, dtype=torch.uint8, device="cuda")   # device -> device
    kv.kvio_kernel_memcpy(dev2.data_ptr(), dev.data_ptr(), nbytes)
    torch.cuda.synchronize()
    assert torch.equal(dev2[:nbytes], dev[:nbytes])
    assert bool((dev2[nbytes:] == 0x3C).all())
    with pytest.raises(kv.KvioError) as e:                      # past the end of the destination
        kv.kvio_kernel_memcpy(dev2.data_ptr(), src.ptr, nbytes + 8192)
    assert e.value.status == kv.KVIO_EINVAL and "allocation holds only" in e.value.detail
    pageable = np.zeros(nbytes, np.uint8)                        # memory the runtime does not know
    with pytest.raises(kv.KvioError) as e:
        kv.kvio_kernel_memcpy(pageable.ctypes.data, dev.data_ptr(), nbytes)
    assert e.value.status == kv.KVIO_ENOTMAPPED
    src.free()
    dst.free()
