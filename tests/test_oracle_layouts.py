"""Pins of the oracle's other host layouts: page-first (Strata Sec. 4.2.1,
Fig. 6: the layers of one page stored together) and head-major (one run per
(layer, K|V, head), the layout that needs a head/token transpose).

Every layout holds the same rows, so numpy's transpose of a token-major chunk
(a library routine) gives the page-first and head-major chunks of the same
content, and loading any of them must give the same pool; offloading must give
back the transposed chunk.  Brute force by the inverse mapping and hand-worked
offsets pin the formulas themselves.
"""
import numpy as np
import pytest

import oracle


def pool_of(L, S, R, seed=0):
    return np.random.default_rng(seed).integers(0, 256, size=(2, L, S, R), dtype=np.uint8)


def chunks(L, T, H, De, P, seed=1):
    """A token-major chunk and the page-first and head-major chunks of the same
    content, built with numpy reshapes and transposes."""
    R = H * De
    tm = np.random.default_rng(seed).integers(0, 256, size=(L, 2, T, R), dtype=np.uint8)
    pf = np.ascontiguousarray(tm.reshape(L, 2, T // P, P, R).transpose(2, 0, 1, 3, 4))
    hm = np.ascontiguousarray(tm.reshape(L, 2, T, H, De).transpose(0, 1, 3, 2, 4))
    return tm.reshape(-1), pf.reshape(-1), hm.reshape(-1)


def test_hand_worked_offsets():
    # page-first, L = 2, P = 2, R = 16: token 3 is page 1 offset 1; row (1, V, 3) sits after
    # page 0 (2 layers x 2 x 2 rows = 8 rows) + layer 1 of page 1 K (2 rows) + ... :
    # (((1*2 + 1)*2 + 1)*2 + 1) = 15 rows -> byte 240
    assert oracle.host_row_offset_page_first(1, 1, 2, 2, 3, 16) == 240
    assert oracle.host_row_offset_page_first(0, 0, 2, 2, 1, 16) == 16
    assert oracle.host_row_offset_page_first(0, 0, 2, 2, 2, 16) == 128
    # head-major, H = 2, host_tokens = 4, De = 8: segment (l=1, K, h=1, t=3) is run
    # (1*2 + 0)*2 + 1 = 5, token 3 of it -> (5*4 + 3)*8 = 184
    assert oracle.host_seg_offset_head_major(1, 0, 1, 2, 4, 3, 8) == 184
    assert oracle.host_seg_offset_head_major(0, 1, 0, 2, 4, 0, 8) == 64


@pytest.mark.parametrize("L,H,De,P,S,T,N", [
    (2, 2, 16, 1, 64, 24, 24),
    (3, 4, 32, 4, 128, 32, 29),      # partial last page
    (2, 8, 16, 16, 256, 64, 50),
    (1, 1, 16, 3, 30, 9, 7),
])
def test_layouts_agree_by_transpose(L, H, De, P, S, T, N):
    R = H * De
    tm, pf, hm = chunks(L, T, H, De, P, seed=L + P)
    pidx = np.random.default_rng(P).permutation(S // P)[:-(-N // P)].astype(np.int32)
    base = pool_of(L, S, R, seed=3)
    results = []
    for layout, chunk in ((oracle.TOKEN_MAJOR, tm), (oracle.PAGE_FIRST, pf), (oracle.HEAD_MAJOR, hm)):
        pool = base.copy()
        oracle.load_layout(pool[0], pool[1], P, [(chunk, T, N, pidx)], layout, num_heads=H)
        results.append(pool)
    assert np.array_equal(results[0], results[1]) and np.array_equal(results[0], results[2])
    # token-major through the layout entry equals the original entry point
    pool = base.copy()
    oracle.load(pool[0], pool[1], P, [(tm, T, N, pidx)])
    assert np.array_equal(pool, results[0])
    # offload in each layout returns the transposed chunk on the moved rows
    outs = []
    for layout, chunk in ((oracle.TOKEN_MAJOR, tm), (oracle.PAGE_FIRST, pf), (oracle.HEAD_MAJOR, hm)):
        out = np.full_like(chunk, 0xC3)
        oracle.offload_layout(results[0][0], results[0][1], P, [(out, T, N, pidx)], layout, num_heads=H)
        outs.append(out)
    t_tm = outs[0].reshape(L, 2, T, R)
    assert np.array_equal(t_tm[:, :, :N], tm.reshape(L, 2, T, R)[:, :, :N])
    assert np.all(t_tm[:, :, N:] == 0xC3)
    back_pf = outs[1].reshape(T // P, L, 2, P, R).transpose(1, 2, 0, 3, 4).reshape(L, 2, T, R)
    back_hm = outs[2].reshape(L, 2, H, T, De).transpose(0, 1, 3, 2, 4).reshape(L, 2, T, R)
    assert np.array_equal(back_pf[:, :, :N], t_tm[:, :, :N]) and np.all(back_pf[:, :, N:] == 0xC3)
    assert np.array_equal(back_hm[:, :, :N], t_tm[:, :, :N]) and np.all(back_hm[:, :, N:] == 0xC3)


def owner(pidx, P, N, slot):
    page, off = divmod(slot, P)
    for j, p in enumerate(pidx):
        if p == page:
            t = j * P + off
            return t if t < N else None
    return None


@pytest.mark.parametrize("layout", [oracle.PAGE_FIRST, oracle.HEAD_MAJOR])
def test_brute_force_inverse_layouts(layout):
    L, H, De, P, S, T, N = 2, 3, 4, 2, 16, 6, 5
    R = H * De
    rng = np.random.default_rng(layout)
    pidx = rng.permutation(S // P)[:3].astype(np.int32)
    n = L * 2 * T * R
    host = rng.integers(0, 256, n, dtype=np.uint8)
    pool = pool_of(L, S, R, seed=11)
    before = pool.copy()
    oracle.load_layout(pool[0], pool[1], P, [(host, T, N, pidx)], layout, num_heads=H)
    for kv in range(2):
        for l in range(L):
            for s in range(S):
                t = owner(pidx, P, N, s)
                for b in range(R):
                    if t is None:
                        exp = before[kv, l, s, b]
                    elif layout == oracle.PAGE_FIRST:
                        # element (l, kv, t, b): page t // P holds layers, K/V, P rows each
                        exp = host[((((t // P) * L + l) * 2 + kv) * P + t % P) * R + b]
                    else:
                        h, d = divmod(b, De)
                        exp = host[(((l * 2 + kv) * H + h) * T + t) * De + d]
                    assert pool[kv, l, s, b] == exp, (kv, l, s, b)


def test_page_first_requires_whole_pages():
    L, H, De, P, S = 2, 2, 8, 4, 64
    host = np.zeros(L * 2 * 12 * H * De, np.uint8)
    pool = pool_of(L, S, H * De)
    with pytest.raises(oracle.OracleError) as e:
        oracle.load_layout(pool[0], pool[1], P, [(host, 10, 10, np.arange(3, dtype=np.int32))],
                           oracle.PAGE_FIRST, num_heads=H)
    assert e.value.code == oracle.EINVAL
    with pytest.raises(oracle.OracleError):
        oracle.load_layout(pool[0], pool[1], P, [(host, 12, 12, np.arange(3, dtype=np.int32))], 7, num_heads=H)


@pytest.mark.parametrize("L,H,De,P,S,T,N", [
    (3, 4, 32, 4, 128, 32, 29),
    (2, 8, 16, 16, 256, 64, 50),
    (4, 1, 16, 1, 64, 24, 24),
])
def test_one_layer_at_a_time_equals_the_whole_load(L, H, De, P, S, T, N):
    """load_layout_layer builds the expected pool one layer at a time; layer by
    layer it must give exactly the slabs of load_layout (the numpy transpose of
    the token-major chunk gives the other layouts' chunks, as above)."""
    R = H * De
    tm, pf, hm = chunks(L, T, H, De, P, seed=L * 7 + P)
    pidx = np.random.default_rng(P + 1).permutation(S // P)[:-(-N // P)].astype(np.int32)
    base = pool_of(L, S, R, seed=5)
    for layout, chunk in ((oracle.TOKEN_MAJOR, tm), (oracle.PAGE_FIRST, pf), (oracle.HEAD_MAJOR, hm)):
        whole = base.copy()
        oracle.load_layout(whole[0], whole[1], P, [(chunk, T, N, pidx)], layout, num_heads=H)
        for l in range(L):
            k, v = base[0, l].copy(), base[1, l].copy()
            oracle.load_layout_layer(k, v, P, [(chunk, T, N, pidx)], layout, L, l, num_heads=H)
            assert np.array_equal(k, whole[0, l]) and np.array_equal(v, whole[1, l]), (layout, l)
