"""Transfers captured in a HIP graph (torch.cuda.CUDAGraph) and replayed:
each replay must move the host chunk's current bytes, checked against the
CPU oracle after every replay, with host writes and eager work in between.
The library enqueues no memset, so its calls are capturable as they are."""
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


@pytest.mark.parametrize("staged", [False, True], ids=["kernel", "staged"])
def test_graph_replays(kv, staged):
    import torch
    L, H, D, P, S, T = 3, 8, 128, 16, 4096, 1000
    R = H * D * 2
    rng = np.random.default_rng(77)
    pages = rng.permutation(S // P)[:-(-T // P)].astype(np.int32)
    pool_np = rng.integers(0, 256, size=(2, L, S, R), dtype=np.uint8)
    pool_t = torch.from_numpy(pool_np.view(np.uint16).reshape(2, L, S, H, D).copy()).cuda()
    pt = torch.from_numpy(pages).cuda()
    launch = kv.launch(flags=kv.KVIO_LAUNCH_STAGED) if staged else None
    # staged: slots of 4 pages of K and V rows, so the call cycles the slots
    pool = kv.KVPool(pool_t, P, load_launch=launch, offload_launch=launch,
                     staging_bytes=4 * 4 * 2 * P * R if staged else 0)
    with kv.HostBuffer(L * 2 * T * R) as hb, kv.HostBuffer(L * 2 * T * R) as ob:
        hb.array[:] = 0
        ob.array[:] = 0
        span_in = [(hb.ptr, T, T, pt.data_ptr())]
        span_out = [(ob.ptr, T, T, pt.data_ptr())]
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):                      # warm-up outside the capture
            pool.load(span_in, stream=s)
            pool.offload(span_out, stream=s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            pool.load(span_in, stream=s)
            pool.offload(span_out, stream=s)
        exp = pool_np.copy()
        for rep in range(4):
            W.fill_np(hb.array, 500 + rep, W.LLAMA8B)   # new bytes in the chunk before each replay
            ob.array[:] = 0
            g.replay()
            torch.cuda.synchronize()
            pool.check()
            oracle.load(exp[0], exp[1], P, [(hb.array, T, T, pages)])
            got = pool_t.cpu().numpy().view(np.uint8).reshape(2, L, S, R)
            assert np.array_equal(got, exp), f"replay {rep}: pool differs"
            assert np.array_equal(ob.array, hb.array), f"replay {rep}: offload differs"
            pool_t.view(torch.int16).add_(0)            # eager work between replays
            torch.cuda.synchronize()
        del g
        pool.close()
