"""Seeded input generators: determinism and structural invariants."""
import numpy as np

import workloads as W


def test_shapes_match_stated_bytes_per_token():
    assert W.TINY.bytes_per_token == 2 * 1024
    assert W.LLAMA8B.bytes_per_token == 128 * 1024
    assert W.GQA70B.bytes_per_token == 320 * 1024
    assert W.QWEN7B1M.bytes_per_token == 56 * 1024
    assert W.LLAMA8B.row_bytes == 2048 and W.TINY.row_bytes == 512


def test_placements_distinct_and_deterministic():
    a = W.random_slots(np.random.default_rng(102), 500_000, 32768)
    b = W.random_slots(np.random.default_rng(102), 500_000, 32768)
    assert np.array_equal(a, b)
    assert len(np.unique(a)) == a.size and a.min() >= 0 and a.max() < 500_000
    p = W.random_pages(np.random.default_rng(101), 256, 64)
    assert len(np.unique(p)) == 64 and p.max() < 256


def test_churn_never_double_allocates():
    free, live = W.churned_pool(np.random.default_rng(204), 5000, ops=10_000)
    allp = np.concatenate([np.asarray(free, np.int64)] + [b.astype(np.int64) for b in live])
    assert np.array_equal(np.sort(allp), np.arange(5000))


def test_batched_requests_scaled():
    r = W.batched_requests(k=4, scale=1 / 64, churn_ops=1000, max_block=8)
    assert len(r.page_lists) == 64
    allp = np.concatenate(r.page_lists + [r.live_pages])
    assert len(np.unique(allp)) == allp.size
    assert allp.max() < r.pool_pages
    for h, pl in zip(r.hit_tokens, r.page_lists):
        assert len(pl) == -(-int(h) // 16)
    assert np.all(r.hit_tokens >= 1) and np.all(r.hit_tokens <= r.prefix_tokens)
    assert r.mean_run_length >= 1.0
    r2 = W.batched_requests(k=4, scale=1 / 64, churn_ops=1000, max_block=8)
    assert all(np.array_equal(x, y) for x, y in zip(r.page_lists, r2.page_lists))


def test_full_size_batched_workload():
    r = W.batched_requests(k=4)
    assert len(r.page_lists) == 64
    allp = np.concatenate(r.page_lists + [r.live_pages])
    assert len(np.unique(allp)) == allp.size and allp.max() < r.pool_pages
    assert int(r.hit_tokens.sum()) == 1_476_853     # 180.3 GiB at 128 KiB per token


def test_full_size_batched_lengths():
    rng = np.random.default_rng(W.placement_seed(4))
    prefix, hit = W.batched_lengths(rng)
    assert prefix.min() >= 2048 and prefix.max() < 131072
    assert np.all(hit >= prefix // 2 - 1) and np.all(hit <= prefix)


def test_payload_determinism_and_distribution():
    x = np.empty(1 << 16, np.uint8)
    y = np.empty(1 << 16, np.uint8)
    W.fill_np(x, 2, W.LLAMA8B)
    W.fill_np(y, 2, W.LLAMA8B)
    assert np.array_equal(x, y)
    v = (x.view(np.uint16).astype(np.uint32) << 16).view(np.float32)
    assert abs(float(v.mean())) < 0.05 and abs(float(v.std()) - 1.0) < 0.05
    W.fill_np(x, 1, W.TINY)
    f = x.view(np.float16).astype(np.float32)
    assert f.min() >= -1.0 and f.max() <= 1.0 and abs(float(f.mean())) < 0.05


def test_bf16_rounding_nearest_even():
    vals = np.array([1.0, 1.00390625, 1.01171875, -2.5, 3.0e38], np.float32)
    bits = W._f32_to_bf16_bits(vals)
    back = (bits.astype(np.uint32) << 16).view(np.float32)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: rounds to the even mantissa (1.0)
    assert back[0] == 1.0 and back[1] == 1.0 and back[2] == 1.015625 and back[3] == -2.5


def test_tagged_payload_unique_enough():
    t = W.tagged_payload(2, 64, 2, 8).view(np.uint16)
    assert t.size == 2 * 2 * 64 * 2 * 8
    assert len(np.unique(t)) > 0.9 * min(t.size, 65536) * 0.5


def test_batch_waves_split_in_order_within_the_budget():
    assert W.batch_waves([], 10) == []
    assert W.batch_waves([4, 4, 4, 4], 8) == [[0, 1], [2, 3]]
    assert W.batch_waves([9, 1, 1], 8) == [[0], [1, 2]]          # an oversized request goes alone
    req = W.batched_requests(4)
    sizes = [32 * 2 * int(h) * 2048 for h in req.hit_tokens]
    waves = W.batch_waves(sizes, 40 << 30)
    assert [i for w in waves for i in w] == list(range(64))
    assert all(sum(sizes[i] for i in w) <= 40 << 30 for w in waves)
    # fewest waves: no wave could have taken the next wave's first request
    assert all(sum(sizes[i] for i in a) + sizes[b[0]] > 40 << 30 for a, b in zip(waves, waves[1:]))
