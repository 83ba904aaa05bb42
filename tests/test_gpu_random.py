"""Seeded random parity sweep on the GPU: random shapes (rows from 16 B to
6 KiB, page sizes 1..64), spans (empty, partial pages, spare chunk capacity),
layer sub-ranges, host layouts, launch shapes, tile sizes and modes (plain,
non-temporal, staged, head-major with and without LDS), each case loaded and
offloaded through the C ABI and compared byte for byte with the CPU oracle
(whole pool image; whole host chunks from a sentinel fill)."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

LAYOUTS = {0: oracle.TOKEN_MAJOR, 1: oracle.PAGE_FIRST, 2: oracle.HEAD_MAJOR}
N_CASES = 1000


@pytest.fixture(scope="module")
def kv():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an AMD GPU"
    import paper_2508_18572_amd as kv
    return kv


def draw_case(seed):
    """A random case; every draw satisfies the library's preconditions."""
    rng = np.random.default_rng(9000 + seed)
    layout = int(rng.choice([0, 0, 1, 2]))
    D = int(rng.choice([8, 16, 64, 128]))
    if layout == 2:
        D = max(D, 8)                                  # head segment D * 2 bytes, a multiple of 16
    H = int(rng.choice([1, 2, 3, 4, 8, 12]))
    L = int(rng.integers(1, 5))
    P = int(rng.choice([1, 2, 3, 4, 5, 16, 32, 64]))
    n_spans = int(rng.integers(1, 6))
    spans = []
    for _ in range(n_spans):
        T = int(rng.choice([0, 1, int(rng.integers(1, 300))]))
        spare = int(rng.integers(0, 3 * P + 1))
        HT = T + spare
        if layout == 1:
            HT = -(-max(HT, 1) // P) * P               # whole pages
        spans.append((T, HT))
    pages_needed = sum(-(-T // P) for T, _ in spans)
    S = P * (pages_needed + int(rng.integers(1, 40)))
    l0 = int(rng.integers(0, L))
    l1 = int(rng.integers(l0 + 1, L + 1))
    flags = 0
    if rng.random() < 0.3:
        flags |= 0x1                                   # cached instead of non-temporal
    staged = layout in (0, 2) and rng.random() < 0.3
    if staged:
        flags |= 0x4
    if layout == 2 and rng.random() < 0.5:
        flags |= 0x2                                   # head-major without LDS
    wg = int(rng.choice([0, 1, 3, 16, 100]))
    threads = int(rng.choice([0, 64, 256, 512, 1024]))
    tile = int(rng.choice([0, 4, 8, 16]))
    slot_pages = int(rng.integers(1, 5))
    R = H * D * 2
    staging = 4 * slot_pages * 2 * P * R + 16 * int(rng.integers(0, 8)) if staged and rng.random() < 0.7 else 0
    return dict(layout=layout, L=L, H=H, D=D, P=P, S=S, spans=spans, l0=l0, l1=l1, flags=flags, wg=wg,
                threads=threads, tile=tile, staging=staging)


def test_draws_are_varied():
    cases = [draw_case(i) for i in range(N_CASES)]
    assert {c["layout"] for c in cases} == {0, 1, 2}
    assert any(c["flags"] & 0x4 for c in cases) and any(c["flags"] & 0x2 for c in cases)
    assert any(T == 0 for c in cases for T, _ in c["spans"])


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_parity(kv, seed):
    import torch
    c = draw_case(seed)
    L, H, D, P, S, l0, l1 = c["L"], c["H"], c["D"], c["P"], c["S"], c["l0"], c["l1"]
    R = H * D * 2
    layout = c["layout"]
    rng = np.random.default_rng(seed)
    pool_np = rng.integers(0, 256, size=(2, L, S, R), dtype=np.uint8)
    pool_t = torch.from_numpy(pool_np.view(np.uint16).reshape(2, L, S, H, D).copy()).cuda()
    perm = rng.permutation(S // P).astype(np.int32)
    bufs, pts, ora_in, ora_out, dev_in, dev_out = [], [], [], [], [], []
    pos = 0
    try:
        for i, (T, HT) in enumerate(c["spans"]):
            pages = perm[pos:pos + -(-T // P)]
            pos += len(pages)
            nbytes = max(oracle.host_chunk_bytes(LAYOUTS[layout], L, HT, R, P), 16)
            hb, ob = kv.HostBuffer(nbytes), kv.HostBuffer(nbytes)
            bufs += [hb, ob]
            W.fill_np(hb.array, seed * 10 + i, W.LLAMA8B)
            ob.array[:] = 0x3C
            pt = torch.from_numpy(pages.copy() if len(pages) else np.zeros(1, np.int32)).cuda()
            pts.append(pt)
            ora_in.append((hb.array, HT, T, pages))
            ora_out.append((np.full(nbytes, 0x3C, np.uint8), HT, T, pages))
            dev_in.append((hb.ptr, HT, T, pt.data_ptr()))
            dev_out.append((ob.ptr, HT, T, pt.data_ptr()))
        launch = kv.launch(c["wg"], c["threads"], c["tile"], c["flags"])
        pool = kv.KVPool(pool_t, P, load_launch=launch, offload_launch=launch, host_layout=layout,
                         staging_bytes=c["staging"])
        pool.load(dev_in, l0, l1)
        torch.cuda.synchronize()
        pool.check()
        exp = pool_np.copy()
        oracle.load_layout(exp[0], exp[1], P, ora_in, LAYOUTS[layout], num_heads=H, layer_begin=l0, layer_end=l1)
        got = pool_t.cpu().numpy().view(np.uint8).reshape(2, L, S, R)
        assert np.array_equal(got, exp), f"load mismatch for {c}"
        pool.offload(dev_out, l0, l1)
        torch.cuda.synchronize()
        pool.check()
        oracle.offload_layout(exp[0], exp[1], P, ora_out, LAYOUTS[layout], num_heads=H, layer_begin=l0,
                              layer_end=l1)
        for i, ((eo, _, _, _), ob) in enumerate(zip(ora_out, bufs[1::2])):
            assert np.array_equal(ob.array, eo), f"offload mismatch in span {i} for {c}"
        pool.close()
    finally:
        for b in bufs:
            b.free()
