"""The five evaluation workloads at full size, through the C ABI, in the launch
configuration bench.py times (library defaults), checked against the CPU
oracle element by element:

  * whole pool image: every (K|V, layer) slab of the pool is copied back and
    compared byte for byte with the oracle's load of the same host chunks into
    a sentinel-filled slab image (so every moved row is in its slot and every
    other byte -- untouched slots, partial-page tails, the pages a churn left
    allocated -- still holds the sentinel);
  * whole host chunk after an offload: every (layer, K|V) region of the
    destination chunk equals the oracle's offload of the (checked) pool image
    into a chunk that held a fill byte before;
  * round trips and, for the staged path, sampled rows plus sentinel
    properties.

Inputs are seeded (workloads module): data seed k, placement seed 100 + k,
churn seed 200 + k for workload k.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from _kvtest import (SENTINEL, memequal, offload_matches_oracle, pool_matches_oracle, pool_matches_oracle_layout,
                     sampled_rows_match, threaded_memset, touched_mask, untouched_rows_hold_sentinel)

pytestmark = pytest.mark.gpu

GiB = 1 << 30


@pytest.fixture(scope="module")
def kv():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an AMD GPU"
    import paper_2508_18572_amd as kv
    return kv


def new_pool(L, S, H, D, dtype):
    import torch
    pool = torch.empty((2, L, S, H, D), dtype=dtype, device="cuda")
    pool.view(torch.int16).fill_(SENTINEL)
    return pool


def test_workload1_tiny_pool_exact(kv):
    """Tiny pool: the whole pool image and the round trip are compared byte for byte."""
    import torch
    wl = W.WORKLOADS[1]
    shp = wl.shape
    L, H, D, P, S, T = shp.num_layers, shp.num_kv_heads, shp.head_dim, wl.page_size, wl.num_slots, wl.tokens
    R = shp.row_bytes
    pages = W.random_pages(np.random.default_rng(W.placement_seed(1)), S // P, T // P)
    pool_t = new_pool(L, S, H, D, torch.float16)
    pool_np = pool_t.cpu().numpy().view(np.uint8).reshape(2, L, S, R).copy()
    with kv.HostBuffer(L * 2 * T * R) as hb, kv.HostBuffer(L * 2 * T * R) as ob:
        W.fill_np(hb.array, W.data_seed(1), shp)
        pt = torch.from_numpy(pages).cuda()
        pool = kv.KVPool(pool_t, P)
        pool.load([(hb.ptr, T, T, pt.data_ptr())])
        ob.array[:] = 0
        pool.offload([(ob.ptr, T, T, pt.data_ptr())])
        torch.cuda.synchronize()
        pool.check()
        exp = pool_np.copy()
        oracle.load(exp[0], exp[1], P, [(hb.array, T, T, pages)])
        assert np.array_equal(pool_t.cpu().numpy().view(np.uint8).reshape(2, L, S, R), exp)
        assert np.array_equal(ob.array, hb.array)
        # 1000 back-to-back loads leave the same image (steady-state path)
        for _ in range(1000):
            pool.load([(hb.ptr, T, T, pt.data_ptr())])
        torch.cuda.synchronize()
        assert np.array_equal(pool_t.cpu().numpy().view(np.uint8).reshape(2, L, S, R), exp)
        pool.close()


FILL = 0xA5       # host bytes an offload must overwrite


def single_context_workload(kv, k, io_stream, layerwise=False, staged=False):
    import torch
    wl = W.WORKLOADS[k]
    shp = wl.shape
    L, H, D, P, S, T = shp.num_layers, shp.num_kv_heads, shp.head_dim, wl.page_size, wl.num_slots, wl.tokens
    R = shp.row_bytes
    nbytes = L * 2 * T * R
    rng = np.random.default_rng(W.placement_seed(k))
    pages = W.random_slots(rng, S, T) if P == 1 else W.random_pages(rng, S // P, -(-T // P))
    print(f"[workload{k}] layerwise {layerwise} staged {staged}: L={L} S={S} T={T} R={R}", flush=True)
    pool_t = new_pool(L, S, H, D, torch.bfloat16)
    pt = torch.from_numpy(pages).cuda()
    with kv.HostBuffer(nbytes) as hb, kv.HostBuffer(nbytes) as ob:
        W.fill_cuda(hb.ptr, nbytes, W.data_seed(k), shp)
        launch = kv.launch(flags=kv.KVIO_LAUNCH_STAGED) if staged else None
        pool = kv.KVPool(pool_t, P, load_launch=launch, offload_launch=launch)
        span = [(hb.ptr, T, T, pt.data_ptr())]
        if layerwise:
            side = io_stream
            compute = torch.cuda.current_stream()
            for l in range(L):
                ev = torch.cuda.Event()
                ev.record(side)
                pool.load_layer(span, l, stream=side, done=ev)
                compute.wait_event(ev)
                pool_t[:, l, :1].float().sum()   # a compute-stream consumer of layer l
        else:
            pool.load(span, stream=io_stream)
        torch.cuda.synchronize()
        pool.check()
        spans_np = [(hb.array, T, T, pages)]
        assert pool_matches_oracle(pool_t, spans_np, P, workers=4) == 2 * L
        threaded_memset(ob.ptr, FILL, nbytes)
        pool.offload([(ob.ptr, T, T, pt.data_ptr())], stream=io_stream)
        torch.cuda.synchronize()
        pool.check()
        assert offload_matches_oracle(pool_t, [(ob.array, T, T, pages)], P, FILL, workers=4) == 2 * L
        assert memequal(ob.ptr, hb.ptr, nbytes), "offload round trip differs from the host chunk"
        pool.close()


def test_workload2_llama8b_page1(kv, io_stream):
    single_context_workload(kv, 2, io_stream)


def test_workload3_70b_layerwise(kv, io_stream):
    single_context_workload(kv, 3, io_stream, layerwise=True)


def test_workload2_staged(kv, io_stream):
    """Staged transfers at full size: a 4 GiB context, whole layers per slot."""
    single_context_workload(kv, 2, io_stream, staged=True)


def test_workload3_staged_layerwise(kv, io_stream):
    """Staged layer-wise loads of the 70B context (one slot per layer)."""
    single_context_workload(kv, 3, io_stream, layerwise=True, staged=True)


@pytest.mark.parametrize("k,layout,layerwise", [(2, "head", False), (3, "page", True)],
                         ids=["workload2_head_major", "workload3_page_first_layerwise"])
def test_other_host_layouts_at_full_size(kv, io_stream, k, layout, layerwise):
    """The head/token transpose (head-major chunks, through LDS) on workload 2
    and the paper's page-first chunks on workload 3 loaded layer by layer, at
    full size in the default launch shapes: the whole pool image against the
    oracle's load of the same chunks, layer by layer, and the offload's round
    trip back into a refilled chunk."""
    import torch
    wl = W.WORKLOADS[k]
    shp = wl.shape
    L, H, D, P, S, T = shp.num_layers, shp.num_kv_heads, shp.head_dim, wl.page_size, wl.num_slots, wl.tokens
    R = shp.row_bytes
    nbytes = L * 2 * T * R
    hl = {"head": kv.KVIO_HOST_HEAD_MAJOR, "page": kv.KVIO_HOST_PAGE_FIRST}[layout]
    ol = {"head": oracle.HEAD_MAJOR, "page": oracle.PAGE_FIRST}[layout]
    rng = np.random.default_rng(W.placement_seed(k))
    pages = W.random_slots(rng, S, T) if P == 1 else W.random_pages(rng, S // P, -(-T // P))
    print(f"[workload{k} {layout}] L={L} S={S} T={T} R={R} layerwise {layerwise}", flush=True)
    torch.cuda.empty_cache()
    pool_t = new_pool(L, S, H, D, torch.bfloat16)
    pt = torch.from_numpy(pages).cuda()
    with kv.HostBuffer(nbytes) as hb, kv.HostBuffer(nbytes) as ob:
        W.fill_cuda(hb.ptr, nbytes, W.data_seed(k) + 50, shp)
        pool = kv.KVPool(pool_t, P, host_layout=hl)
        span = [(hb.ptr, T, T, pt.data_ptr())]
        if layerwise:
            compute = torch.cuda.current_stream()
            for l in range(L):
                ev = torch.cuda.Event()
                ev.record(io_stream)
                pool.load_layer(span, l, stream=io_stream, done=ev)
                compute.wait_event(ev)
        else:
            pool.load(span, stream=io_stream)
        torch.cuda.synchronize()
        pool.check()
        assert pool_matches_oracle_layout(pool_t, [(hb.array, T, T, pages)], P, ol, H) == 2 * L
        threaded_memset(ob.ptr, FILL, nbytes)
        pool.offload([(ob.ptr, T, T, pt.data_ptr())], stream=io_stream)
        torch.cuda.synchronize()
        pool.check()
        assert memequal(ob.ptr, hb.ptr, nbytes), "offload round trip differs from the host chunk"
        pool.close()
    del pool_t
    torch.cuda.empty_cache()


def batched_setup():
    k = 4
    shp = W.LLAMA8B
    req = W.batched_requests(k)
    hit = [int(h) for h in req.hit_tokens]
    sizes = [shp.num_layers * 2 * h * shp.row_bytes for h in hit]
    return k, shp, req, hit, sizes, W.batch_waves(sizes, 40 * GiB)


N_WAVES = len(batched_setup()[5])


@pytest.mark.parametrize("wave", range(N_WAVES))
def test_workload4_batched_churned_wave(kv, io_stream, wave):
    """64 partial-hit contexts of the 8B shape at page size 16 into a churned
    pool, one batched kvio_load per wave, as the benchmark times them.  Each
    wave is loaded into a sentinel-filled pool and the whole pool image is
    compared with the oracle's load of that wave's spans (the slots the churn
    left allocated and every other untouched slot included); then the wave is
    offloaded with one batched kvio_offload into its own chunks, refilled
    first, and every chunk is compared with the oracle's offload."""
    import torch
    k, shp, req, hit, sizes, waves = batched_setup()
    L, H, D, P = shp.num_layers, shp.num_kv_heads, shp.head_dim, 16
    R = shp.row_bytes
    S = req.pool_pages * P
    w = waves[wave]
    nb = sum(sizes[i] for i in w)
    print(f"[workload4] wave {wave}/{len(waves)}: spans {w[0]}..{w[-1]}, {nb / GiB:.1f} GiB, pool {S} slots, "
          f"mean run length {req.mean_run_length:.2f}", flush=True)
    torch.cuda.empty_cache()                 # the pool takes most of HBM
    pool_t = new_pool(L, S, H, D, torch.bfloat16)
    pool = kv.KVPool(pool_t, P)
    pts = {i: torch.from_numpy(req.page_lists[i]).cuda() for i in w}
    with kv.HostBuffer(nb) as hb:
        offs, o = {}, 0
        for i in w:
            offs[i] = o
            W.fill_cuda(hb.ptr + o, sizes[i], W.data_seed(k) * 1000 + i, shp)
            o += sizes[i]
        spans = [(hb.ptr + offs[i], hit[i], hit[i], pts[i].data_ptr()) for i in w]
        pool.load(spans, stream=io_stream)
        torch.cuda.synchronize()
        pool.check()
        spans_np = [(hb.array[offs[i]:offs[i] + sizes[i]], hit[i], hit[i], req.page_lists[i]) for i in w]
        assert pool_matches_oracle(pool_t, spans_np, P, workers=3) == 2 * L
        threaded_memset(hb.ptr, FILL, nb)
        pool.offload(spans, stream=io_stream)
        torch.cuda.synchronize()
        pool.check()
        assert offload_matches_oracle(pool_t, spans_np, P, FILL, workers=3) == 2 * L * len(w)
    pool.close()
    del pool_t
    torch.cuda.empty_cache()


def test_workload4_batched_churned_staged(kv):
    """The batched workload through the staged path (both directions through
    the default 4 GiB of HBM staging each): every wave loaded into one pool,
    sampled rows against the oracle, per-span round trips, and the sentinel of
    every slot no request names (the churn's live pages among them)."""
    import torch
    k, shp, req, hit, sizes, waves = batched_setup()
    L, H, D, P = shp.num_layers, shp.num_kv_heads, shp.head_dim, 16
    R = shp.row_bytes
    S = req.pool_pages * P
    print(f"[workload4 staged] {sum(hit)} tokens, {sum(sizes) / GiB:.1f} GiB, pool {S} slots, "
          f"{len(waves)} wave(s)", flush=True)
    torch.cuda.empty_cache()
    pool_t = new_pool(L, S, H, D, torch.bfloat16)
    launch = kv.launch(flags=kv.KVIO_LAUNCH_STAGED)
    pool = kv.KVPool(pool_t, P, load_launch=launch, offload_launch=launch)
    pts = [torch.from_numpy(pl).cuda() for pl in req.page_lists]
    all_spans_np = []
    for w in waves:
        nb = sum(sizes[i] for i in w)
        with kv.HostBuffer(nb) as hb:
            offs, o = {}, 0
            for i in w:
                offs[i] = o
                W.fill_cuda(hb.ptr + o, sizes[i], W.data_seed(k) * 1000 + i, shp)
                o += sizes[i]
            spans = [(hb.ptr + offs[i], hit[i], hit[i], pts[i].data_ptr()) for i in w]
            pool.load(spans)
            torch.cuda.synchronize()
            pool.check()
            spans_np = [(hb.array[offs[i]:offs[i] + sizes[i]], hit[i], hit[i], req.page_lists[i]) for i in w]
            sampled_rows_match(pool_t, spans_np, P, S, R, L, 4096, seed=k + len(all_spans_np))
            # round trip of every span through one scratch chunk
            big = max(sizes[i] for i in w)
            with kv.HostBuffer(big) as sb:
                for i in w:
                    pool.offload([(sb.ptr, hit[i], hit[i], pts[i].data_ptr())])
                    torch.cuda.synchronize()
                    assert memequal(sb.ptr, hb.ptr + offs[i], sizes[i]), f"span {i} round trip differs"
            pool.check()
            all_spans_np += [(None, hit[i], hit[i], req.page_lists[i]) for i in w]
    # churn-resident pages and every slot of no request keep the sentinel
    untouched_rows_hold_sentinel(pool_t, touched_mask(all_spans_np, P, S), L)
    pool.close()
    del pool_t
    torch.cuda.empty_cache()


@pytest.mark.parametrize("staged", [False, True], ids=["kernel", "staged_load"])
def test_workload5_1m_with_concurrent_offload(kv, io_stream, staged):
    """1M-token load at page size 1 on one stream while 16K other slots are
    offloaded repeatedly to a separate host chunk on a second stream (the
    load through the kernels, or staged through HBM slots: 2 GiB per layer,
    so spans split across slots)."""
    import torch
    k = 5
    wl = W.WORKLOADS[k]
    shp = wl.shape
    L, H, D, P, S, T = shp.num_layers, shp.num_kv_heads, shp.head_dim, wl.page_size, wl.num_slots, wl.tokens
    R = shp.row_bytes
    TO = 16384
    rng = np.random.default_rng(W.placement_seed(k))
    both = W.random_slots(rng, S, T + TO)
    load_slots, off_slots = both[:T].copy(), both[T:].copy()
    nb, nbo = L * 2 * T * R, L * 2 * TO * R
    pool_t = new_pool(L, S, H, D, torch.bfloat16)
    pool = kv.KVPool(pool_t, P, load_launch=kv.launch(flags=kv.KVIO_LAUNCH_STAGED) if staged else None)
    pl, po = torch.from_numpy(load_slots).cuda(), torch.from_numpy(off_slots).cuda()
    with kv.HostBuffer(nb) as hb, kv.HostBuffer(nbo) as src_o, kv.HostBuffer(nbo) as dst_o:
        W.fill_cuda(hb.ptr, nb, W.data_seed(k), shp)
        W.fill_cuda(src_o.ptr, nbo, W.data_seed(k) * 1000 + 1, shp)
        pool.load([(src_o.ptr, TO, TO, po.data_ptr())])          # set-up: resident data to offload
        torch.cuda.synchronize()
        sa, sb = io_stream, torch.cuda.Stream()
        done = torch.cuda.Event()
        pool.load([(hb.ptr, T, T, pl.data_ptr())], stream=sa)
        done.record(sa)
        runs = 0
        while True:
            pool.offload([(dst_o.ptr, TO, TO, po.data_ptr())], stream=sb)
            runs += 1
            sb.synchronize()
            if done.query() or runs >= 200:
                break
        torch.cuda.synchronize()
        pool.check()
        print(f"[workload5] {runs} concurrent offload runs during the 1M-token load", flush=True)
        assert memequal(dst_o.ptr, src_o.ptr, nbo), "concurrent offload differs from its source"
        spans_np = [(hb.array, T, T, load_slots), (src_o.array, TO, TO, off_slots)]
        if staged:
            sampled_rows_match(pool_t, spans_np, P, S, R, L, 4096, seed=k)
            untouched_rows_hold_sentinel(pool_t, touched_mask(spans_np, P, S), L)
        else:
            # two workers: the host chunks here already hold 57.75 GiB of pinned memory
            assert pool_matches_oracle(pool_t, spans_np, P, workers=2) == 2 * L
        # Round trip in token ranges through a 4 GiB chunk (pinned memory per
        # process may be capped at 64 GiB): offloading tokens
        # [a, b) uses the page table from entry a and a chunk of b - a tokens.
        piece = (4 * GiB) // (L * 2 * R)
        with kv.HostBuffer(L * 2 * piece * R) as ob:
            for a in range(0, T, piece):
                n = min(piece, T - a)
                pool.offload([(ob.ptr, n, n, pl.data_ptr() + 4 * a)])
                torch.cuda.synchronize()
                for plane in range(2 * L):
                    assert memequal(ob.ptr + plane * n * R, hb.ptr + (plane * T + a) * R, n * R), \
                        f"1M-token round trip differs in tokens [{a}, {a + n}) plane {plane}"
    pool.check()
    pool.close()
