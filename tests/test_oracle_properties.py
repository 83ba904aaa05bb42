"""Hypothesis-drawn shapes for the transfer oracle (Strata Sec. 4.2 / 4.2.1):
random layer counts, row widths, page sizes, span counts, partial last pages,
spare chunk capacity, layer sub-ranges and host layouts.  Each draw checks the
oracle against formulations that share none of its index arithmetic:

  * token-major loads equal numpy fancy indexing of the pool reshaped into
    pages (full pages by page index, then the partial last page);
  * page-first and head-major chunks built from the token-major chunk by numpy
    reshapes and transposes load to the same pool;
  * offload of a loaded context returns its rows and leaves the rest of the
    chunk alone;
  * a load split into two layer ranges equals the whole-range load;
  * the page-offset expansion equals the pool's slot grid indexed by page.
"""
import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle

SETTINGS = settings(max_examples=200, deadline=None, suppress_health_check=[HealthCheck.too_slow])


@st.composite
def cases(draw):
    L = draw(st.integers(1, 3))
    H = draw(st.integers(1, 3))
    De = 16 * draw(st.integers(1, 2))                 # head segment bytes (multiple of 16)
    P = draw(st.integers(1, 6))
    n = draw(st.integers(1, 3))
    spans = []
    for _ in range(n):
        T = draw(st.integers(0, 4 * P + 3))
        spans.append(T)
    spare_pages = draw(st.integers(1, 5))
    need = sum(-(-T // P) for T in spans)
    S = P * (need + spare_pages)
    l0 = draw(st.integers(0, L - 1))
    l1 = draw(st.integers(l0 + 1, L))
    seed = draw(st.integers(0, 2**31 - 1))
    return L, H, De, P, S, spans, l0, l1, seed


def setup(L, H, De, P, S, spans, seed):
    R = H * De
    rng = np.random.default_rng(seed)
    perm = rng.permutation(S // P).astype(np.int32)
    tables, chunks, pos = [], [], 0
    for T in spans:
        k = -(-T // P)
        tables.append(perm[pos:pos + k])
        pos += k
        HT = -(-max(T, 1) // P) * P                   # whole pages: valid for every layout
        chunks.append((rng.integers(0, 256, size=L * 2 * HT * R, dtype=np.uint8), HT, T))
    pool = rng.integers(0, 256, size=(2, L, S, R), dtype=np.uint8)
    return R, tables, chunks, pool


def fancy_load(pool, P, R, chunks, tables, l0, l1):
    """The load written with numpy indexing over pages (no slot arithmetic)."""
    S = pool.shape[2]
    out = pool.copy()
    for (host, HT, T), pidx in zip(chunks, tables):
        L = host.size // (2 * HT * R)
        h = host.reshape(L, 2, HT, R)
        full = T // P
        for kv in range(2):
            for layer in range(l0, l1):
                pages = out[kv, layer].reshape(S // P, P, R)
                pages[pidx[:full]] = h[layer, kv, :full * P].reshape(full, P, R)
                if T > full * P:
                    pages[pidx[full], :T - full * P] = h[layer, kv, full * P:T]
    return out


@SETTINGS
@given(cases())
def test_token_major_load_equals_fancy_indexing(c):
    L, H, De, P, S, spans, l0, l1, seed = c
    R, tables, chunks, pool = setup(L, H, De, P, S, spans, seed)
    exp = fancy_load(pool, P, R, chunks, tables, l0, l1)
    got = pool.copy()
    oracle.load(got[0], got[1], P, [(h, HT, T, t) for (h, HT, T), t in zip(chunks, tables)], l0, l1)
    assert np.array_equal(got, exp)


@SETTINGS
@given(cases())
def test_other_layouts_equal_the_transposed_chunk(c):
    L, H, De, P, S, spans, l0, l1, seed = c
    R, tables, chunks, pool = setup(L, H, De, P, S, spans, seed)
    exp = fancy_load(pool, P, R, chunks, tables, l0, l1)
    pf_spans, hm_spans = [], []
    for (host, HT, T), t in zip(chunks, tables):
        tm = host.reshape(L, 2, HT, R)
        pf = np.ascontiguousarray(tm.reshape(L, 2, HT // P, P, R).transpose(2, 0, 1, 3, 4)).reshape(-1)
        hm = np.ascontiguousarray(tm.reshape(L, 2, HT, H, De).transpose(0, 1, 3, 2, 4)).reshape(-1)
        pf_spans.append((pf, HT, T, t))
        hm_spans.append((hm, HT, T, t))
    for layout, sp in ((oracle.PAGE_FIRST, pf_spans), (oracle.HEAD_MAJOR, hm_spans)):
        got = pool.copy()
        oracle.load_layout(got[0], got[1], P, sp, layout, num_heads=H, layer_begin=l0, layer_end=l1)
        assert np.array_equal(got, exp), layout


@SETTINGS
@given(cases())
def test_offload_returns_the_loaded_rows(c):
    L, H, De, P, S, spans, l0, l1, seed = c
    R, tables, chunks, pool = setup(L, H, De, P, S, spans, seed)
    oracle.load(pool[0], pool[1], P, [(h, HT, T, t) for (h, HT, T), t in zip(chunks, tables)], l0, l1)
    for (host, HT, T), t in zip(chunks, tables):
        out = np.full_like(host, 0xC3)
        oracle.offload(pool[0], pool[1], P, [(out, HT, T, t)], l0, l1)
        o, h = out.reshape(L, 2, HT, R), host.reshape(L, 2, HT, R)
        assert np.array_equal(o[l0:l1, :, :T], h[l0:l1, :, :T])
        assert np.all(o[l0:l1, :, T:] == 0xC3)
        assert np.all(o[:l0] == 0xC3) and np.all(o[l1:] == 0xC3)


@SETTINGS
@given(cases())
def test_split_layer_range_equals_whole(c):
    L, H, De, P, S, spans, l0, l1, seed = c
    R, tables, chunks, pool = setup(L, H, De, P, S, spans, seed)
    sp = [(h, HT, T, t) for (h, HT, T), t in zip(chunks, tables)]
    whole = pool.copy()
    oracle.load(whole[0], whole[1], P, sp, 0, L)
    split = pool.copy()
    cut = (l0 + l1) // 2 if l1 - l0 > 1 else l0
    if cut > 0:
        oracle.load(split[0], split[1], P, sp, 0, cut)
    oracle.load(split[0], split[1], P, sp, cut, L)
    assert np.array_equal(split, whole)


@SETTINGS
@given(cases())
def test_expand_slots_equals_the_slot_grid_by_page(c):
    L, H, De, P, S, spans, l0, l1, seed = c
    R, tables, chunks, pool = setup(L, H, De, P, S, spans, seed)
    grid = np.arange(S, dtype=np.int64).reshape(S // P, P)        # slot ids, one row per page
    for (host, HT, T), t in zip(chunks, tables):
        exp = grid[t].reshape(-1)[:T]
        assert np.array_equal(oracle.expand_slots(t, P, T, S), exp)
