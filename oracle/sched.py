"""Oracle for cache-aware batch formation (test infrastructure only).

Strata Sec. 4.3.1 (deferral on delay hit) and Sec. 4.3.2 (Balanced Batch
Formation), restated from the paper's description in plain Python.  Only the
tests may use it; it shares nothing with the library's implementation.

What the paper fixes (Sec. 4.3.1, Sec. 4.3.2):
  * A request that matches transient (in-queue / in-flight) cache entries by
    more than a threshold number of tokens (default 100) is deferred to the
    next scheduling round and placed at the front of the waiting queue.
  * Every batch formation begins with the first request of the queue.
  * Whenever a request enters the batch, the rest of the queue is searched
    for requests that reuse a context already in the batch (bundle hits);
    they enter too, ahead of anything else.
  * The queue is walked in order while the batch is not full.  A request
    whose entry would push the batch's aggregated load over aggregated
    compute above a ratio (default 100) is set aside in a deprioritized list;
    any other request enters (and pulls in its bundle hits).
  * If the batch still has room once the walk is over, the set-aside requests
    fill it, in their original order (this also prevents starvation).

Readings where the paper is silent (also listed in the design notes):
  * load = tokens of cached context to bring in from host memory, compute =
    new tokens to prefill.  A context shared by several requests of a batch is
    loaded once, so a bundle hit adds no load.
  * "Full": the batch's compute tokens reached the token budget, or its
    request count reached the request cap.  Entry is not checked against the
    room left (the request that fills the batch may overshoot it), and bundle
    hits enter regardless of room.
  * The loading-bound test is the real-valued ratio test of the paper:
    load / compute > ratio, i.e. load > ratio * compute, evaluated exactly
    (rational arithmetic on the integer token sums and on the ratio's exact
    binary value).  A batch with no compute is loading-bound as soon as it has
    any load; an infinite ratio never is (plain FIFO).
  * Requests the round does not take keep their relative order; the next
    round's queue is the deferred delay hits (in order), then the rest.
"""
from __future__ import annotations

import dataclasses
import math
from fractions import Fraction
from typing import List, Optional, Sequence, Tuple

DEFAULT_RATIO = 100.0
DEFAULT_DELAY_HIT_THRESHOLD = 100


@dataclasses.dataclass(frozen=True)
class Request:
    rid: int
    load_tokens: int            # cached tokens to load from host memory
    compute_tokens: int         # new tokens to prefill
    context: Optional[int] = None   # id of the cached context it reuses
    transient_matches: int = 0      # tokens matched on in-queue / in-flight nodes


def exceeds_ratio(load: int, compute: int, ratio: float) -> bool:
    """Sec. 4.3.2: the ratio of aggregated load to aggregated compute exceeds
    the threshold, as exact rational arithmetic."""
    if math.isinf(ratio):
        return False
    return Fraction(load) > Fraction(ratio) * compute


# States of a queue position during one batch formation.
_WAITING, _IN_BATCH, _SET_ASIDE = 0, 1, 2


def batch_formation(queue: Sequence[Request], max_tokens: int, max_requests: int,
                    ratio: float = DEFAULT_RATIO) -> Tuple[List[int], List[int]]:
    """Balanced batch formation (Sec. 4.3.2).  Returns (batch ids in the order
    they entered, ids left for later rounds in queue order)."""
    n = len(queue)
    if n == 0:
        return [], []
    state = [_WAITING] * n
    entered: List[int] = []          # queue positions, in the order they entered
    contexts_in_batch = set()
    totals = {"load": 0, "compute": 0}

    def load_if_entered(pos: int) -> int:
        r = queue[pos]
        shared = r.context is not None and r.context in contexts_in_batch
        return totals["load"] + (0 if shared else r.load_tokens)

    def enter(pos: int) -> None:
        r = queue[pos]
        totals["load"] = load_if_entered(pos)
        totals["compute"] += r.compute_tokens
        state[pos] = _IN_BATCH
        entered.append(pos)
        if r.context is not None:
            contexts_in_batch.add(r.context)

    def enter_bundle_hits() -> None:
        # every request still in the queue that reuses a context of the batch
        for pos in range(n):
            c = queue[pos].context
            if state[pos] == _WAITING and c is not None and c in contexts_in_batch:
                enter(pos)

    def has_room() -> bool:
        return totals["compute"] < max_tokens and len(entered) < max_requests

    enter(0)                         # the head of the queue always starts the batch
    enter_bundle_hits()
    for pos in range(1, n):
        if not has_room():
            break
        if state[pos] != _WAITING:   # already pulled in as a bundle hit
            continue
        r = queue[pos]
        if exceeds_ratio(load_if_entered(pos), totals["compute"] + r.compute_tokens, ratio):
            state[pos] = _SET_ASIDE
        else:
            enter(pos)
            enter_bundle_hits()
    for pos in range(n):             # set-aside requests fill the room left, in queue order
        if state[pos] == _SET_ASIDE:
            if not has_room():
                break
            enter(pos)
    batch = [queue[p].rid for p in entered]
    rest = [queue[p].rid for p in range(n) if state[p] != _IN_BATCH]
    return batch, rest


def schedule_round(queue: Sequence[Request], max_tokens: int, max_requests: int,
                   ratio: float = DEFAULT_RATIO,
                   delay_hit_threshold: int = DEFAULT_DELAY_HIT_THRESHOLD) -> Tuple[List[int], List[int]]:
    """One scheduling round: defer delay hits (Sec. 4.3.1), form a batch from
    the others (Sec. 4.3.2).  Returns (batch ids, next round's queue ids)."""
    deferred = [r.rid for r in queue if r.transient_matches > delay_hit_threshold]
    eligible = [r for r in queue if r.transient_matches <= delay_hit_threshold]
    batch, rest = batch_formation(eligible, max_tokens, max_requests, ratio)
    return batch, deferred + rest
