"""Pins of the batch-formation oracle (Strata Sec. 4.3.1 and Sec. 4.3.2).

The paper's Figure 7 narrative gives the worked example: with C and D0 both
needing large context loads, FIFO would batch (C, D0) and stall on loading;
balanced batch formation forms (C, F) so C's load overlaps F's compute, and D0 with D1 —
which share one context — form a bundle-hit batch next.  The numbers below
are chosen so that exactly those decisions follow from a ratio of 100.
"""
import json
import math
import os

from oracle.sched import Request, batch_formation, schedule_round

INF = math.inf


def ids(rs):
    return [r.rid for r in rs]


def fig7():
    # C: 80K cached tokens to load, 1K new tokens       (load/compute 80  <= 100)
    # D0, D1: share context 7, 60K to load, 200 new each
    # F: nothing cached, 2K new tokens
    C = Request(0, 80_000, 1_000, context=3)
    D0 = Request(1, 60_000, 200, context=7)
    D1 = Request(2, 60_000, 200, context=7)
    F = Request(3, 0, 2_000)
    return [C, D0, D1, F]


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "fig7_batch_formation.json")


def golden_fig7():
    g = json.load(open(GOLDEN))
    reqs = [Request(i, r["load_tokens"], r["compute_tokens"], r["context"]) for i, r in enumerate(g["requests"])]
    names = [r["name"] for r in g["requests"]]
    return g, reqs, names


def test_figure7_golden_rounds():
    """The stored Figure 7 fixture, round by round, through schedule_round."""
    g, reqs, names = golden_fig7()
    pol = g["policy"]
    by_name = dict(zip(names, reqs))
    queue = reqs
    for rnd in g["rounds"]:
        batch, nxt = schedule_round(queue, pol["max_tokens"], pol["max_requests"], pol["loading_bound_ratio"],
                                    pol["delay_hit_threshold"])
        assert [names[i] for i in batch] == rnd["batch"]
        assert [names[i] for i in nxt] == rnd["next_queue"]
        queue = [by_name[n] for n in rnd["next_queue"]]
    fifo, _ = batch_formation(reqs, pol["max_tokens"], pol["max_requests"], ratio=INF)
    assert [names[i] for i in fifo] == g["fifo_first_batch"]


def test_figure7_worked_example():
    q = fig7()
    # C alone: 80K / 1K = 80.  C + D0: 140K / 1.2K = 116.7 > 100 -> D0 deprioritized;
    # D1 is no bundle hit yet (D0 is not in the batch): same ratio -> deprioritized;
    # C + F: 80K / 3K = 26.7 -> F joins.  The queue is empty, the batch is not full
    # (budget 8K tokens, cap 2 requests reached) -> nothing more.
    batch, rest = batch_formation(q, max_tokens=8_000, max_requests=2)
    assert batch == [0, 3] and rest == [1, 2]
    # next round: D0 heads the batch and pulls in its bundle hit D1 (context loaded once)
    batch2, rest2 = batch_formation([q[1], q[2]], max_tokens=8_000, max_requests=2)
    assert batch2 == [1, 2] and rest2 == []


def test_fifo_would_have_batched_c_and_d0():
    # with no loading-bound limit the same queue is plain FIFO
    batch, rest = batch_formation(fig7(), max_tokens=8_000, max_requests=2, ratio=INF)
    # D0 enters second and D1, its bundle hit, follows it regardless of the cap
    assert batch == [0, 1, 2] and rest == [3]


def test_deprioritized_fill_room_in_order():
    q = [Request(0, 0, 100), Request(1, 10**9, 10), Request(2, 10**9, 10), Request(3, 0, 100)]
    batch, rest = batch_formation(q, max_tokens=10**6, max_requests=10)
    # 1 and 2 are loading-bound and wait; 3 joins; then 1 and 2 fill the room in order
    assert batch == [0, 3, 1, 2] and rest == []
    batch, rest = batch_formation(q, max_tokens=10**6, max_requests=3)
    assert batch == [0, 3, 1] and rest == [2]


def test_head_always_taken_even_if_loading_bound():
    q = [Request(0, 10**9, 1), Request(1, 0, 50)]
    batch, rest = batch_formation(q, max_tokens=10, max_requests=8)
    # the head alone exceeds the ratio but always enters; request 1 would keep the batch
    # loading-bound, so it waits in the deprioritized list and then fills the room left
    assert batch == [0, 1] and rest == []


def test_token_budget_stops_the_scan():
    q = [Request(i, 0, 400) for i in range(6)]
    batch, rest = batch_formation(q, max_tokens=1_000, max_requests=64)
    # 400, 800 (< 1000, not full), 1200 (full): three requests, the last overshoots
    assert batch == [0, 1, 2] and rest == [3, 4, 5]


def test_bundle_hits_jump_the_queue():
    q = [Request(0, 1_000, 100, context=1), Request(1, 0, 100), Request(2, 0, 100),
         Request(3, 1_000, 100, context=1)]
    batch, rest = batch_formation(q, max_tokens=250, max_requests=64)
    # the head pulls its bundle hit (3) in before anything else; then 1 fills the budget
    assert batch == [0, 3, 1] and rest == [2]


def test_delay_hit_deferral():
    q = [Request(0, 0, 100, transient_matches=101), Request(1, 0, 100, transient_matches=100),
         Request(2, 0, 100), Request(3, 0, 100, transient_matches=5000)]
    batch, nxt = schedule_round(q, max_tokens=10**6, max_requests=64)
    # > 100 matched tokens defers; exactly 100 does not; deferred go first next round
    assert batch == [1, 2] and nxt == [0, 3]


def test_rounds_drain_any_queue():
    import random
    rnd = random.Random(5)
    q = [Request(i, rnd.choice([0, 10, 10**5, 10**7]), rnd.randint(1, 3000), context=rnd.choice([None, 1, 2, 3]))
         for i in range(40)]
    seen = []
    by_id = {r.rid: r for r in q}
    cur = q
    for _ in range(100):
        if not cur:
            break
        batch, rest = batch_formation(cur, max_tokens=4096, max_requests=8)
        assert batch and batch[0] == cur[0].rid          # progress, head first
        seen += batch
        cur = [by_id[i] for i in rest]
        # the rest keeps queue order
        assert [r.rid for r in cur] == sorted(rest, key=lambda i: [x.rid for x in q].index(i))
    assert sorted(seen) == list(range(40))


def test_deferred_requests_go_to_the_front():
    # Sec. 4.3.1: a deferred request waits for the next round at the FRONT of the queue,
    # ahead of eligible requests this round could not take
    q = [Request(0, 0, 100, transient_matches=500), Request(1, 0, 100), Request(2, 0, 100)]
    batch, nxt = schedule_round(q, max_tokens=10**6, max_requests=1)
    assert batch == [1] and nxt == [0, 2]


def test_budget_reached_exactly_is_full():
    # a batch whose compute tokens reach the budget exactly is full (reading of is_full)
    q = [Request(0, 0, 400), Request(1, 0, 600), Request(2, 0, 100)]
    batch, rest = batch_formation(q, max_tokens=1_000, max_requests=64)
    assert batch == [0, 1] and rest == [2]


def test_shared_context_loads_once():
    # A and its bundle hit B share context 1: the batch loads 1000 tokens, not 2000.
    # C then keeps the batch at 2000 / 25 = 80 <= 100 and joins (full at 3 requests);
    # counting the shared context twice would give 3000 / 25 = 120 and let D in instead.
    q = [Request(0, 1000, 10, context=1), Request(1, 1000, 10, context=1), Request(2, 1000, 5),
         Request(3, 0, 5)]
    batch, rest = batch_formation(q, max_tokens=10**6, max_requests=3)
    assert batch == [0, 1, 2] and rest == [3]


def test_ratio_test_is_exact_past_double_precision():
    # Sec. 4.3.2: loading-bound when load / compute exceeds the ratio.  With
    # compute 2^60 and load 2^60 + 1 the ratio is above 1 by 2^-60, which a
    # double cannot see (2^60 + 1 rounds to 2^60): request 1 is set aside and
    # fills the room only after request 2.
    big = 2**60
    q = [Request(0, 0, big), Request(1, big + 1, 0), Request(2, 0, 1)]
    assert batch_formation(q, max_tokens=2**62, max_requests=8, ratio=1.0) == ([0, 2, 1], [])
    # exactly at the ratio is not above it: request 1 joins in queue order
    q = [Request(0, 0, big), Request(1, big, 0), Request(2, 0, 1)]
    assert batch_formation(q, max_tokens=2**62, max_requests=8, ratio=1.0) == ([0, 1, 2], [])


def test_no_compute_is_loading_bound_once_anything_loads():
    # load / 0 exceeds any finite ratio; 0 / 0 does not (nothing to load)
    q = [Request(0, 0, 0), Request(1, 5, 0), Request(2, 0, 0)]
    assert batch_formation(q, max_tokens=10, max_requests=8, ratio=10**9) == ([0, 2, 1], [])
    # an infinite ratio is plain FIFO
    assert batch_formation(q, max_tokens=10, max_requests=8, ratio=INF) == ([0, 1, 2], [])
