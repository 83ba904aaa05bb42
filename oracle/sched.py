"""Oracle for cache-aware batch formation (test infrastructure only).

Strata Sec. 4.3.1 (deferral on delay hit) and Sec. 4.3.2 (Balanced Batch
Formation, Algorithm 1), written out step by step in plain Python.  Only the
tests may use it; it shares nothing with the library's implementation.

What the paper fixes:
  * A request whose tokens match transient (in-queue / in-flight) nodes beyond
    a threshold (default 100 tokens) is deferred to the next scheduling round
    and placed at the front of the waiting queue (Sec. 4.3.1).
  * Batch formation (Algorithm 1): the head of the queue always enters the
    batch, followed by every queued request that bundle-hits the batch (shares
    a cached context with a request already in it).  Then requests are taken
    in queue order while the batch is not full: one that would make the batch
    loading-bound -- aggregated load over aggregated compute above a ratio
    (default 100) -- goes to a deprioritized list, otherwise it joins the
    batch, again followed by its bundle hits.  Finally, deprioritized requests
    fill any room left, in their original order (Sec. 4.3.2).

Readings where the paper is silent (also listed in the design notes):
  * load = tokens of cached context to bring in from host memory, compute =
    new tokens to prefill; a context shared by several batched requests is
    loaded once, so a bundle hit adds no load.
  * is_full: the batch's compute tokens reached the token budget, or its
    request count reached the request cap.  Like Algorithm 1, adding a request
    does not check the remaining room (the last one may overshoot).
  * loading_bound(r): load(B + r) > ratio * compute(B + r), compared in
    double precision; a batch with no compute is loading-bound as soon as it
    has any load.
  * Requests not placed in the batch keep their relative order; the next
    round's queue is: deferred delay hits (in order), then the rest.
"""
from __future__ import annotations

import dataclasses
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


class Batch:
    def __init__(self, max_tokens: int, max_requests: int, ratio: float):
        self.max_tokens = max_tokens
        self.max_requests = max_requests
        self.ratio = ratio
        self.requests: List[Request] = []
        self.contexts = set()
        self.load = 0
        self.compute = 0

    def is_full(self) -> bool:
        return self.compute >= self.max_tokens or len(self.requests) >= self.max_requests

    def is_bundle_hit(self, r: Request) -> bool:
        return r.context is not None and r.context in self.contexts

    def added_load(self, r: Request) -> int:
        return 0 if self.is_bundle_hit(r) else r.load_tokens

    def loading_bound(self, r: Request) -> bool:
        load = self.load + self.added_load(r)
        compute = self.compute + r.compute_tokens
        # the decision is taken in double precision, as the library takes it
        return float(load) > float(self.ratio) * float(compute)

    def add(self, r: Request) -> None:
        self.load += self.added_load(r)
        self.compute += r.compute_tokens
        self.requests.append(r)
        if r.context is not None:
            self.contexts.add(r.context)


def add_bundle_hit(queue: List[Request], batch: Batch) -> None:
    """Move every queued request that bundle-hits the batch into it."""
    i = 0
    while i < len(queue):
        if batch.is_bundle_hit(queue[i]):
            batch.add(queue.pop(i))
        else:
            i += 1


def batch_formation(queue: Sequence[Request], max_tokens: int, max_requests: int,
                    ratio: float = DEFAULT_RATIO) -> Tuple[List[int], List[int]]:
    """Algorithm 1.  Returns (batch ids in the order they joined, ids left
    for later rounds in queue order)."""
    q = list(queue)
    if not q:
        return [], []
    order = {r.rid: i for i, r in enumerate(queue)}
    batch = Batch(max_tokens, max_requests, ratio)
    deprioritized: List[Request] = []
    batch.add(q.pop(0))
    add_bundle_hit(q, batch)
    while q and not batch.is_full():
        r = q.pop(0)
        if batch.loading_bound(r):
            deprioritized.append(r)
        else:
            batch.add(r)
            add_bundle_hit(q, batch)
    for r in deprioritized:
        if batch.is_full():
            break
        batch.add(r)
    taken = {r.rid for r in batch.requests}
    rest = sorted((r for r in queue if r.rid not in taken), key=lambda r: order[r.rid])
    return [r.rid for r in batch.requests], [r.rid for r in rest]


def schedule_round(queue: Sequence[Request], max_tokens: int, max_requests: int,
                   ratio: float = DEFAULT_RATIO,
                   delay_hit_threshold: int = DEFAULT_DELAY_HIT_THRESHOLD) -> Tuple[List[int], List[int]]:
    """One scheduling round: defer delay hits (Sec. 4.3.1), form a batch from
    the others (Algorithm 1).  Returns (batch ids, next round's queue ids)."""
    deferred = [r for r in queue if r.transient_matches > delay_hit_threshold]
    eligible = [r for r in queue if r.transient_matches <= delay_hit_threshold]
    batch, rest = batch_formation(eligible, max_tokens, max_requests, ratio)
    return batch, [r.rid for r in deferred] + rest
