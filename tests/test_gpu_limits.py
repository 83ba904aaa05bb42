"""GPU parity at the size limits of the pool: per-layer K and V pools whose byte
offsets pass 2^32, up to the largest slot count the pool accepts (2^31 - 16
slots of 16-byte rows, a 34 GB pool per layer and K|V).  The pools are far too
large for a whole-image comparison on the CPU, so each case moves one context
into pages drawn from the top of the pool (the last page included, once as the
partial last page) and checks:

  * the rows of the touched pages against the CPU oracle, which loads the same
    chunk into a compact pool of just those pages (pages 0..n-1);
  * the offloaded host chunk, byte for byte, against the oracle's offload of
    that compact pool into a sentinel-filled chunk;
  * that every other byte of the pool still holds its sentinel (on the GPU).

Every host layout runs through the kernel path, and token-major and
head-major through the staged path."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

SENTINEL = 0x5A5A                      # int16 fill of the pool; bytes 0x5A
ORACLE_LAYOUT = {0: oracle.TOKEN_MAJOR, 1: oracle.PAGE_FIRST, 2: oracle.HEAD_MAJOR}

# (L, H, D, P, S, T, first page of the high region)
SHAPES = {
    # 4 KiB rows, S = 1.25 * 2^20: 5.4 GB per layer pool, pages past 2^32 bytes
    "4k_rows_5gb_layer_pools": (2, 16, 128, 16, 1_310_720, 1000, 65_536),
    # 16-byte rows at the largest slot count: slots up to 2^31 - 17
    "16b_rows_max_slots": (1, 1, 8, 16, 2**31 - 16, 1000, 2**27 - 2**20),
}
MODES = [  # (host layout, staged)
    (0, False), (1, False), (2, False), (0, True), (2, True),
]


@pytest.fixture(scope="module")
def kv():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an AMD GPU"
    import paper_2508_18572_amd as kv
    return kv


def pool_all_sentinel(torch, pool_t) -> bool:
    flat = pool_t.view(-1)
    step = 1 << 30
    for i in range(0, flat.numel(), step):
        if bool((flat[i:i + step] != SENTINEL).any()):
            return False
    return True


def draw_pages(rng, num_pages, need, high_from, last_at_end):
    """`need` distinct pages: page 0, the last page of the pool and the rest from
    [high_from, num_pages - 1), in random order; the last page goes to the
    context's final (partial) page when `last_at_end`."""
    top = num_pages - 1
    rest = rng.choice(top - high_from, size=need - 2, replace=False) + high_from
    pages = np.concatenate([[0], rest]).astype(np.int32)
    rng.shuffle(pages)
    if last_at_end:
        return np.append(pages, np.int32(top))
    return np.insert(pages, int(rng.integers(0, need)), np.int32(top))


@pytest.mark.parametrize("name", list(SHAPES))
def test_pool_limits(kv, name):
    import torch
    L, H, D, P, S, T, high_from = SHAPES[name]
    R = H * D * 2
    need = -(-T // P)
    HT = need * P                                   # whole pages: valid for every layout
    assert T % P != 0                               # the last context page is partial
    pool_t = torch.full((2, L, S, H, D), SENTINEL, dtype=torch.int16, device="cuda")
    try:
        for m, (layout, staged) in enumerate(MODES):
            rng = np.random.default_rng(4100 + m + 10 * len(name))
            pages = draw_pages(rng, S // P, need, high_from, last_at_end=(m == 0))
            nbytes = oracle.host_chunk_bytes(ORACLE_LAYOUT[layout], L, HT, R, P)
            print(f"[limits] {name} layout {layout} staged {staged}: pages {pages.min()}..{pages.max()}",
                  flush=True)
            launch = kv.launch(flags=kv.KVIO_LAUNCH_STAGED) if staged else None
            # Four slots of 4 pages' K and V rows: the chunk spans several slots.
            staging = 4 * 4 * 2 * P * R if staged else 0
            pool = kv.KVPool(pool_t, P, load_launch=launch, offload_launch=launch, host_layout=layout,
                             staging_bytes=staging)
            pt = torch.from_numpy(pages).cuda()
            with kv.HostBuffer(nbytes) as src, kv.HostBuffer(nbytes) as out:
                W.fill_np(src.array, 77 + m, W.LLAMA8B)
                out.array[:] = 0x6B
                pool.load([(src.ptr, HT, T, pt.data_ptr())])
                torch.cuda.synchronize()
                pool.check()

                # The oracle's pool: the same chunk loaded into pages 0..need-1.
                compact = np.full((2, L, need * P, R), 0x5A, np.uint8)
                dense = np.arange(need, dtype=np.int32)
                oracle.load_layout(compact[0], compact[1], P, [(src.array, HT, T, dense)],
                                   ORACLE_LAYOUT[layout], num_heads=H)
                slots = oracle.expand_slots(pages, P, need * P, S)
                idx = torch.from_numpy(slots).cuda()
                for kvi in range(2):
                    for layer in range(L):
                        got = pool_t[kvi, layer].index_select(0, idx).cpu().numpy()
                        got = got.view(np.uint8).reshape(need * P, R)
                        if not np.array_equal(got, compact[kvi, layer]):
                            bad = np.argwhere(got != compact[kvi, layer])
                            raise AssertionError(f"{name} layout {layout} staged {staged}: load mismatch "
                                                 f"(kv {kvi}, layer {layer}) at {len(bad)} bytes, "
                                                 f"first rows {np.unique(bad[:, 0])[:4].tolist()}")

                pool.offload([(out.ptr, HT, T, pt.data_ptr())])
                torch.cuda.synchronize()
                pool.check()
                expect = np.full(nbytes, 0x6B, np.uint8)
                oracle.offload_layout(compact[0], compact[1], P, [(expect, HT, T, dense)],
                                      ORACLE_LAYOUT[layout], num_heads=H)
                if not np.array_equal(out.array, expect):
                    bad = np.flatnonzero(out.array != expect)
                    raise AssertionError(f"{name} layout {layout} staged {staged}: offload mismatch at "
                                         f"{len(bad)} bytes, first {bad[:4].tolist()}")

            # Nothing outside the touched pages changed; reset them for the next mode.
            for kvi in range(2):
                for layer in range(L):
                    pool_t[kvi, layer].index_fill_(0, idx, SENTINEL)
            torch.cuda.synchronize()
            assert pool_all_sentinel(torch, pool_t), f"{name} layout {layout} staged {staged}: " \
                                                     "a byte outside the moved pages changed"
            pool.close()
    finally:
        del pool_t
        torch.cuda.empty_cache()
