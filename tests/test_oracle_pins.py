"""Pins of the CPU oracle against what the definition of the transfer fixes.

The paper prints no worked example and its figures carry no values, so the
oracle is pinned by (Strata, Sec. 4.2 / Sec. 4.2.1 / Sec. 2.2):
  * a hand-worked tiny example (values derived by hand from the definition),
  * the identity page table, where a load must equal a plain memcpy,
  * numpy fancy indexing of the pool reshaped into pages (a library routine),
  * brute force by the INVERSE mapping: for every pool element, search the
    page table for the context token that owns it (pool-centric, the opposite
    direction of the oracle's token loop),
  * round-trip identities, sentinel invariants for untouched bytes,
  * rejection of invalid inputs.
A plausible mistake in the oracle (dropped term, swapped K/V, wrong stride,
div/mod swapped, dropped row) fails at least one of these; see
test_oracle_mutants.py.
"""
import numpy as np
import pytest

import oracle
from workloads import tagged_payload

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def make_pool(L, S, R, seed=0):
    """Pool images filled with a per-(kv, layer, slot) sentinel byte pattern."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, 256, size=(2, L, S, R), dtype=np.uint8)


def rand_host(L, host_tokens, R, seed=1):
    return np.random.default_rng(seed).integers(0, 256, size=L * 2 * host_tokens * R, dtype=np.uint8)


# ---------------------------------------------------------------------------
# Hand-worked example
# ---------------------------------------------------------------------------

def test_hand_worked_example():
    # L = 2 layers, R = 16 B (1 head x 8 dims x 2 B), P = 2, S = 8 slots (4 pages).
    # Context of 3 tokens in a chunk of host_tokens = 4; page table [3, 1]:
    #   token 0 -> page 3 offset 0 -> slot 6
    #   token 1 -> page 3 offset 1 -> slot 7
    #   token 2 -> page 1 offset 0 -> slot 2     (slot 3 = tail of the partial page)
    # Host row (l, kv, t) starts at ((l*2 + kv)*4 + t)*16, e.g. (1, V, 2) -> (3*4 + 2)*16 = 224.
    assert list(oracle.expand_slots(np.array([3, 1]), 2, 3, 8)) == [6, 7, 2]
    assert oracle.host_row_offset(1, 1, 4, 2, 16) == 224
    assert oracle.host_row_offset(0, 1, 4, 0, 16) == 64
    assert oracle.host_row_offset(1, 0, 4, 3, 16) == 176

    L, S, R, T, HT = 2, 8, 16, 3, 4
    host = np.zeros(L * 2 * HT * R, dtype=np.uint8)
    for l in range(L):
        for kv in range(2):
            for t in range(HT):
                off = ((l * 2 + kv) * HT + t) * R
                host[off:off + R] = 100 + l * 40 + kv * 20 + t   # row id byte
    pool = np.full((2, L, S, R), 0xEE, dtype=np.uint8)
    oracle.load(pool[0], pool[1], 2, [(host, HT, T, np.array([3, 1], np.int32))])
    for kv in range(2):
        for l in range(L):
            got = [int(pool[kv, l, s, 0]) for s in range(S)]
            exp = [0xEE] * S
            exp[6] = 100 + l * 40 + kv * 20 + 0
            exp[7] = 100 + l * 40 + kv * 20 + 1
            exp[2] = 100 + l * 40 + kv * 20 + 2
            assert got == exp, (kv, l, got)
            assert np.all(pool[kv, l] == pool[kv, l, :, :1])   # rows are uniform bytes


# ---------------------------------------------------------------------------
# Identity table == memcpy
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("P", [1, 2, 4, 16])
def test_identity_table_is_memcpy(P):
    L, R, S = 3, 48, 64
    host = rand_host(L, S, R)
    pool = make_pool(L, S, R)
    pidx = np.arange(S // P, dtype=np.int32)
    oracle.load(pool[0], pool[1], P, [(host, S, S, pidx)])
    h = host.reshape(L, 2, S, R)
    for l in range(L):
        assert pool[0, l].tobytes() == h[l, 0].tobytes()
        assert pool[1, l].tobytes() == h[l, 1].tobytes()
    out = np.zeros_like(host)
    oracle.offload(pool[0], pool[1], P, [(out, S, S, pidx)])
    assert out.tobytes() == host.tobytes()


# ---------------------------------------------------------------------------
# numpy fancy indexing (library routine)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("P,T,HT", [(1, 37, 40), (3, 37, 37), (4, 13, 20), (16, 50, 64), (5, 1, 1)])
def test_fancy_index_load_offload(P, T, HT):
    L, R, S = 2, 32, 240
    rng = np.random.default_rng(P * 100 + T)
    n_pages = -(-T // P)
    pidx = rng.permutation(S // P)[:n_pages].astype(np.int32)
    host = rand_host(L, HT, R, seed=T)
    pool = make_pool(L, S, R, seed=P)
    exp = pool.copy()
    h = host.reshape(L, 2, HT, R)
    full = T // P
    for kv in range(2):
        for l in range(L):
            pages = exp[kv, l].reshape(S // P, P, R)
            pages[pidx[:full]] = h[l, kv, :full * P].reshape(full, P, R)
            rem = T - full * P
            if rem:
                pages[pidx[full], :rem] = h[l, kv, full * P:T]
    oracle.load(pool[0], pool[1], P, [(host, HT, T, pidx)])
    assert np.array_equal(pool, exp)

    # offload = np.take of pages, into a sentinel-filled chunk
    out = np.full_like(host, 0x5A)
    oracle.offload(pool[0], pool[1], P, [(out, HT, T, pidx)])
    o = out.reshape(L, 2, HT, R)
    for kv in range(2):
        for l in range(L):
            pages = pool[kv, l].reshape(S // P, P, R)
            got = np.take(pages, pidx, axis=0).reshape(-1, R)[:T]
            assert np.array_equal(o[l, kv, :T], got)
            assert np.all(o[l, kv, T:] == 0x5A)


# ---------------------------------------------------------------------------
# Brute force by the inverse mapping, element by element
# ---------------------------------------------------------------------------

def inverse_owner(pidx, P, T, slot):
    """Context token stored in `slot`, found by scanning the page table; None if unowned."""
    page, off = divmod(slot, P)
    for j, p in enumerate(pidx):
        if p == page:
            t = j * P + off
            return t if t < T else None
    return None


@pytest.mark.parametrize("L,H,D,P,S,T,HT", [
    (1, 1, 8, 1, 6, 4, 5),
    (2, 3, 8, 2, 12, 5, 7),
    (3, 2, 8, 3, 18, 7, 7),
    (2, 1, 16, 4, 16, 9, 12),
    (2, 3, 8, 16, 64, 33, 40),
])
def test_brute_force_inverse(L, H, D, P, S, T, HT):
    R = H * D * 2
    rng = np.random.default_rng(L * 7 + P)
    pidx = rng.permutation(S // P)[:-(-T // P)].astype(np.int32)
    host = tagged_payload(L, HT, H, D)
    pool = make_pool(L, S, R, seed=3)
    before = pool.copy()
    oracle.load(pool[0], pool[1], P, [(host, HT, T, pidx)])
    pool16 = pool.view(np.uint16).reshape(2, L, S, H, D)
    before16 = before.view(np.uint16).reshape(2, L, S, H, D)
    host16 = host.view(np.uint16)
    for kv in range(2):
        for l in range(L):
            for s in range(S):
                t = inverse_owner(pidx, P, T, s)
                for h in range(H):
                    for d in range(D):
                        if t is None:
                            exp = before16[kv, l, s, h, d]
                        else:
                            flat = (((l * 2 + kv) * HT + t) * H + h) * D + d
                            exp = host16[flat]
                        assert pool16[kv, l, s, h, d] == exp, (kv, l, s, h, d)

    # offload, brute force per host element: owner slot by scanning all slots
    out = np.full_like(host, 0x33)
    oracle.offload(pool[0], pool[1], P, [(out, HT, T, pidx)])
    out16 = out.view(np.uint16).reshape(L, 2, HT, H, D)
    owner = {}
    for s in range(S):
        t = inverse_owner(pidx, P, T, s)
        if t is not None:
            owner[t] = s
    assert sorted(owner) == list(range(T))
    for l in range(L):
        for kv in range(2):
            for t in range(HT):
                for h in range(H):
                    for d in range(D):
                        exp = pool16[kv, l, owner[t], h, d] if t < T else np.uint16(0x3333)
                        assert out16[l, kv, t, h, d] == exp


# ---------------------------------------------------------------------------
# Round trip, layer ranges, batches, sentinels
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("P", [1, 2, 16])
def test_round_trip_and_untouched(P):
    L, R, S, T, HT = 4, 64, 256, 100, 120
    rng = np.random.default_rng(P)
    pidx = rng.permutation(S // P)[:-(-T // P)].astype(np.int32)
    host = rand_host(L, HT, R, seed=P)
    pool = make_pool(L, S, R)
    before = pool.copy()
    oracle.load(pool[0], pool[1], P, [(host, HT, T, pidx)])
    slots = oracle.expand_slots(pidx, P, T, S)
    untouched = np.setdiff1d(np.arange(S), slots)
    assert np.array_equal(pool[:, :, untouched], before[:, :, untouched])
    out = np.full_like(host, 0x77)
    oracle.offload(pool[0], pool[1], P, [(out, HT, T, pidx)])
    h = host.reshape(L, 2, HT, R)
    o = out.reshape(L, 2, HT, R)
    assert np.array_equal(o[:, :, :T], h[:, :, :T])
    assert np.all(o[:, :, T:] == 0x77)
    # load(offload(pool)) restores the touched rows of a scrambled pool
    scrambled = make_pool(L, S, R, seed=9)
    scr_before = scrambled.copy()
    oracle.load(scrambled[0], scrambled[1], P, [(out, HT, T, pidx)])
    assert np.array_equal(scrambled[:, :, slots], pool[:, :, slots])
    assert np.array_equal(scrambled[:, :, untouched], scr_before[:, :, untouched])


def test_layer_range_partition():
    L, R, S, T, P = 5, 32, 64, 30, 2
    pidx = np.random.default_rng(5).permutation(S // P)[:15].astype(np.int32)
    host = rand_host(L, T, R)
    a = make_pool(L, S, R)
    b = a.copy()
    oracle.load(a[0], a[1], P, [(host, T, T, pidx)])
    for lo, hi in [(0, 2), (2, 3), (3, 5)]:
        oracle.load(b[0], b[1], P, [(host, T, T, pidx)], lo, hi)
    assert np.array_equal(a, b)
    c = make_pool(L, S, R)
    c_before = c.copy()
    oracle.load(c[0], c[1], P, [(host, T, T, pidx)], 1, 3)
    assert np.array_equal(c[:, [0, 3, 4]], c_before[:, [0, 3, 4]])
    assert np.array_equal(c[:, 1:3], a[:, 1:3])


def test_batch_equals_sequential():
    L, R, S, P = 2, 32, 512, 4
    rng = np.random.default_rng(11)
    perm = rng.permutation(S // P).astype(np.int32)
    spans, pos = [], 0
    for i, (T, HT) in enumerate([(10, 12), (1, 1), (33, 40), (0, 5), (16, 16)]):
        n = -(-T // P)
        spans.append((rand_host(L, HT, R, seed=20 + i), HT, T, perm[pos:pos + n]))
        pos += n
    a = make_pool(L, S, R)
    b = a.copy()
    oracle.load(a[0], a[1], P, spans)
    for sp in spans:
        oracle.load(b[0], b[1], P, [sp])
    assert np.array_equal(a, b)


def test_slab_matches_batch():
    L, R, S, T, P = 2, 32, 64, 21, 4
    pidx = np.random.default_rng(2).permutation(S // P)[:6].astype(np.int32)
    host = rand_host(L, 24, R)
    a = make_pool(L, S, R)
    b = a.copy()
    oracle.load(a[0], a[1], P, [(host, 24, T, pidx)])
    h = host.reshape(L, 2, 24 * R)
    for l in range(L):
        for kv in range(2):
            oracle.load_slab(b[kv, l], P, np.ascontiguousarray(h[l, kv]), T, pidx)
    assert np.array_equal(a, b)


# ---------------------------------------------------------------------------
# Invalid inputs
# ---------------------------------------------------------------------------

def test_rejects_invalid():
    L, R, S, P = 2, 32, 64, 4
    host = rand_host(L, 8, R)
    pool = make_pool(L, S, R)
    before = pool.copy()
    with pytest.raises(oracle.OracleError) as e:        # duplicate page
        oracle.load(pool[0], pool[1], P, [(host, 8, 8, np.array([3, 3], np.int32))])
    assert e.value.code == oracle.EDUP
    with pytest.raises(oracle.OracleError) as e:        # two contexts sharing a page
        oracle.load(pool[0], pool[1], P, [(host, 8, 2, np.array([5], np.int32)),
                                          (host, 8, 1, np.array([5], np.int32))])
    assert e.value.code == oracle.EDUP
    with pytest.raises(oracle.OracleError) as e:        # page out of range
        oracle.load(pool[0], pool[1], P, [(host, 8, 8, np.array([1, 16], np.int32))])
    assert e.value.code == oracle.ERANGE
    with pytest.raises(oracle.OracleError) as e:        # negative page
        oracle.load(pool[0], pool[1], P, [(host, 8, 8, np.array([-1, 2], np.int32))])
    assert e.value.code == oracle.ERANGE
    with pytest.raises(oracle.OracleError) as e:        # num_tokens > host_tokens
        oracle.load(pool[0], pool[1], P, [(host, 4, 8, np.array([1, 2], np.int32))])
    assert e.value.code == oracle.EINVAL
    with pytest.raises(oracle.OracleError):             # empty layer range
        oracle.load(pool[0], pool[1], P, [(host, 8, 8, np.array([1, 2], np.int32))], 1, 1)
    with pytest.raises(oracle.OracleError):             # layer range past L
        oracle.load(pool[0], pool[1], P, [(host, 8, 8, np.array([1, 2], np.int32))], 0, 3)
    assert np.array_equal(pool, before)                 # nothing moved on any error
    # duplicate reads are legal for offload
    out = np.zeros_like(host)
    oracle.offload(pool[0], pool[1], P, [(out, 8, 8, np.array([3, 3], np.int32))])
    o = out.reshape(L, 2, 8, R)
    assert np.array_equal(o[:, :, :4], o[:, :, 4:])
    with pytest.raises(oracle.OracleError):
        oracle.expand_slots(np.array([0]), 3, 2, 64)    # S % P != 0


def test_empty_transfers_do_nothing():
    L, R, S, P = 2, 32, 64, 4
    pool = make_pool(L, S, R)
    before = pool.copy()
    host = rand_host(L, 4, R)
    oracle.load(pool[0], pool[1], P, [])
    oracle.load(pool[0], pool[1], P, [(host, 4, 0, np.zeros(0, np.int32))])
    assert np.array_equal(pool, before)
    assert oracle.expand_slots(np.zeros(0, np.int32), P, 0, S).size == 0
