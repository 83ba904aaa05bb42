"""GPU parity of the page-first and head-major host layouts against the CPU
oracle, byte for byte: whole pool images after a load and whole host chunks
(from a sentinel fill) after an offload.  Head-major runs through both the LDS
transpose and the direct gather; rows wider than one step take the direct
gather automatically."""
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


ORACLE_LAYOUT = {1: oracle.PAGE_FIRST, 2: oracle.HEAD_MAJOR}


def run_layout_case(kv, layout, L, H, D, P, S, spans, l0=0, l1=None, launch=None, seed=0):
    import torch
    l1 = L if l1 is None else l1
    R = H * D * 2
    rng = np.random.default_rng(2000 + seed)
    pool_np = rng.integers(0, 256, size=(2, L, S, R), dtype=np.uint8)
    pool_t = torch.from_numpy(pool_np.view(np.uint16).reshape(2, L, S, H, D).copy()).cuda()
    need = sum(-(-T // P) for T, _ in spans)
    perm = rng.permutation(S // P)[:need].astype(np.int32)
    bufs, pts, ora_in, ora_out, dev_in, dev_out = [], [], [], [], [], []
    pos = 0
    try:
        for i, (T, HT) in enumerate(spans):
            pages = perm[pos:pos + -(-T // P)]
            pos += len(pages)
            nbytes = max(oracle.host_chunk_bytes(ORACLE_LAYOUT[layout], L, HT, R, P), 16)
            hb, ob = kv.HostBuffer(nbytes), kv.HostBuffer(nbytes)
            bufs += [hb, ob]
            W.fill_np(hb.array, seed * 100 + i, W.LLAMA8B)
            ob.array[:] = 0x6B
            pt = torch.from_numpy(pages.copy() if len(pages) else np.zeros(1, np.int32)).cuda()
            pts.append(pt)
            ora_in.append((hb.array, HT, T, pages))
            ora_out.append((np.full(nbytes, 0x6B, np.uint8), HT, T, pages))
            dev_in.append((hb.ptr, HT, T, pt.data_ptr()))
            dev_out.append((ob.ptr, HT, T, pt.data_ptr()))
        pool = kv.KVPool(pool_t, P, load_launch=launch, offload_launch=launch, host_layout=layout)
        pool.load(dev_in, l0, l1)
        torch.cuda.synchronize()
        pool.check()
        exp = pool_np.copy()
        oracle.load_layout(exp[0], exp[1], P, ora_in, ORACLE_LAYOUT[layout], num_heads=H,
                           layer_begin=l0, layer_end=l1)
        got = pool_t.cpu().numpy().view(np.uint8).reshape(2, L, S, R)
        if not np.array_equal(got, exp):
            bad = np.argwhere(got != exp)
            raise AssertionError(f"load mismatch at {len(bad)} bytes, first {bad[:4].tolist()}")
        pool.offload(dev_out, l0, l1)
        torch.cuda.synchronize()
        pool.check()
        oracle.offload_layout(exp[0], exp[1], P, ora_out, ORACLE_LAYOUT[layout], num_heads=H,
                              layer_begin=l0, layer_end=l1)
        for i, ((eo, _, _, _), ob) in enumerate(zip(ora_out, bufs[1::2])):
            if not np.array_equal(ob.array, eo):
                bad = np.flatnonzero(ob.array != eo)
                raise AssertionError(f"offload mismatch in span {i} at {len(bad)} bytes, first {bad[:4]}")
        pool.close()
    finally:
        for b in bufs:
            b.free()


SHAPES = [
    (2, 8, 128, 1, 3000, [(700, 700), (3, 3)]),         # R = 2 KiB, page size 1
    (2, 4, 64, 16, 4096, [(1000, 1008)]),               # R = 512 B, partial last page
    (3, 8, 128, 16, 2048, [(333, 336), (17, 32)]),      # R = 2 KiB, P = 16
    (2, 6, 128, 4, 600, [(201, 204)]),                  # R = 1536 B (odd vectors)
    (2, 2, 64, 5, 1000, [(123, 125), (0, 5)]),          # R = 256 B, P = 5, empty span
    (2, 128, 128, 1, 64, [(10, 12)]),                   # R = 32 KiB: wider than a step
    (1, 4, 64, 100, 1000, [(250, 300), (100, 100)]),    # P = 100 (no shift), page > one tile
    (1, 1, 8, 128, 128, [(100, 128)]),                  # a one-page pool, R = 16 B
    (40, 2, 8, 4, 64, [(30, 32)]),                      # 80 layer pointers: more than one per lane
]


@pytest.mark.parametrize("L,H,D,P,S,spans", SHAPES)
def test_page_first_parity(kv, L, H, D, P, S, spans):
    run_layout_case(kv, 1, L, H, D, P, S, spans, seed=L * 7 + P)


@pytest.mark.parametrize("L,H,D,P,S,spans", SHAPES)
@pytest.mark.parametrize("lds", [True, False])
def test_head_major_parity(kv, L, H, D, P, S, spans, lds):
    launch = None if lds else kv.launch(flags=kv.KVIO_LAUNCH_NO_LDS)
    run_layout_case(kv, 2, L, H, D, P, S, spans, launch=launch, seed=L * 5 + P + lds)


@pytest.mark.parametrize("wg,threads,tile", [(1, 64, 4), (5, 1024, 16), (64, 256, 8)])
@pytest.mark.parametrize("layout", [1, 2])
def test_layout_launch_shapes_and_subrange(kv, layout, wg, threads, tile):
    launch = kv.launch(wg, threads, tile, 0)
    run_layout_case(kv, layout, 4, 8, 128, 16, 4096, [(500, 512), (40, 48)], l0=1, l1=3, launch=launch,
                    seed=wg)
    run_layout_case(kv, layout, 2, 4, 64, 1, 3000, [(900, 900)], launch=launch, seed=wg + 1)


def test_layout_many_spans(kv):
    rng = np.random.default_rng(21)
    spans = [(int(t), int(t) + 16 - int(t) % 16) for t in rng.integers(0, 60, 70)]
    run_layout_case(kv, 1, 2, 8, 128, 16, 8192, spans, seed=21)
    run_layout_case(kv, 2, 2, 8, 128, 16, 8192, spans, seed=22)


def test_layout_validation(kv):
    import torch
    L, H, D, P, S = 2, 8, 128, 16, 1024
    pool_t = torch.zeros((2, L, S, H, D), dtype=torch.bfloat16, device="cuda")
    pool = kv.KVPool(pool_t, P, host_layout=kv.KVIO_HOST_PAGE_FIRST)
    pt = torch.arange(4, dtype=torch.int32, device="cuda")
    with kv.HostBuffer(L * 2 * 64 * H * D * 2) as hb:
        with pytest.raises(kv.KvioError) as e:                  # host_tokens not whole pages
            pool.load([(hb.ptr, 60, 60, pt.data_ptr())])
        assert e.value.status == kv.KVIO_EINVAL
        with pytest.raises(kv.KvioError) as e:                  # 64 tokens = 4 pages > 3 pages' room
            pool.load([(hb.ptr + L * 2 * 16 * H * D * 2, 64, 64, pt.data_ptr())])
        assert e.value.status == kv.KVIO_EINVAL
    pool.close()
    with pytest.raises(kv.KvioError) as e:                      # head_dim * 2 = 8 B: not 16-aligned
        kv.kvio_pool_create(L, 256, 4, 2, P, S, [pool_t[0, l].data_ptr() for l in range(L)],
                            [pool_t[1, l].data_ptr() for l in range(L)], host_layout=kv.KVIO_HOST_HEAD_MAJOR)
    assert e.value.status == kv.KVIO_EALIGN
    hm = kv.KVPool(pool_t, P, host_layout=kv.KVIO_HOST_HEAD_MAJOR)
    with pytest.raises(kv.KvioError) as e:                      # no per-page baseline for head-major
        kv.kvio_naive_load(hm.handle, [], 0, L)
    assert e.value.status == kv.KVIO_EINVAL
    hm.close()
