"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module generates inputs only: KV pool shapes, page placements, the
allocate/free churn that fragments a pool, and host payload bytes.  It holds
none of the transfer's arithmetic (no slot or offset computation) and imports
neither the oracle nor the product library, so both sides can consume the same
bytes without sharing code.

Shapes follow the workloads of Strata's evaluation (Sec. 5.1: Llama-3.1-8B,
Llama-3.1-70B, Qwen2.5 1M-context models; Table 1 context lengths up to the 1M
window).  The datasets themselves are not used: every payload is synthetic.

Seeds: workload k uses data seed k, placement seed 100 + k and churn seed
200 + k (numpy ``default_rng``).
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
from typing import List, Sequence, Tuple

import numpy as np

KiB = 1024
MiB = 1024 * KiB
GiB = 1024 * MiB


@dataclasses.dataclass(frozen=True)
class KVShape:
    """Per-layer K/V geometry of one model's paged KV pool."""
    name: str
    num_layers: int
    num_kv_heads: int
    head_dim: int
    dtype: str            # "fp16" | "bf16"
    dist: str             # "uniform" (U[-1, 1)) | "normal" (N(0, 1))

    @property
    def elem_bytes(self) -> int:
        return 2

    @property
    def row_bytes(self) -> int:
        """Bytes of one token of one layer's K (or V)."""
        return self.num_kv_heads * self.head_dim * self.elem_bytes

    @property
    def bytes_per_token(self) -> int:
        return self.num_layers * 2 * self.row_bytes


TINY = KVShape("tiny-2L-4H-64D", 2, 4, 64, "fp16", "uniform")
LLAMA8B = KVShape("llama-3.1-8b", 32, 8, 128, "bf16", "normal")
GQA70B = KVShape("llama-3.1-70b", 80, 8, 128, "bf16", "normal")
QWEN7B1M = KVShape("qwen2.5-7b-1m", 28, 4, 128, "bf16", "normal")


@dataclasses.dataclass(frozen=True)
class Workload:
    """One of the five evaluation workloads (full size)."""
    index: int
    shape: KVShape
    page_size: int
    num_slots: int
    tokens: int            # tokens of the (single) cached context; 0 for the batched workload
    description: str


WORKLOADS = {
    1: Workload(1, TINY, 16, 4096, 1024,
                "tiny pool (2 layers, 4 KV heads x 64 dims, fp16, 4096 slots), page size 16, "
                "1024-token context into 64 random pages, round trip"),
    2: Workload(2, LLAMA8B, 1, 500_000, 32 * KiB,
                "Llama-3.1-8B KV, page size 1, 32K-token prefix into random free slots"),
    3: Workload(3, GQA70B, 16, 131_072, 64 * KiB,
                "70B GQA KV, page size 16, 64K-token context loaded layer by layer"),
    4: Workload(4, LLAMA8B, 16, 0, 0,
                "Llama-3.1-8B KV, page size 16, 64 partial-hit requests into a churned pool"),
    5: Workload(5, QWEN7B1M, 1, 1_310_720, 1 << 20,
                "Qwen2.5-7B-1M KV, page size 1, 1M-token load with concurrent 16K offloads"),
}


def data_seed(k: int) -> int:
    return k


def placement_seed(k: int) -> int:
    return 100 + k


def churn_seed(k: int) -> int:
    return 200 + k


# ----------------------------------------------------------------------------
# Page placement
# ----------------------------------------------------------------------------

def random_pages(rng: np.random.Generator, pool_pages: int, count: int) -> np.ndarray:
    """`count` distinct pool pages in random order (a random sample of free pages)."""
    if count > pool_pages:
        raise ValueError("more pages requested than the pool holds")
    return rng.permutation(pool_pages)[:count].astype(np.int32)


def random_slots(rng: np.random.Generator, num_slots: int, count: int) -> np.ndarray:
    """`count` distinct slots drawn uniformly without replacement, in random order
    (page size 1: worst-case fragmentation)."""
    return rng.choice(num_slots, count, replace=False).astype(np.int32)


@dataclasses.dataclass
class BatchedRequests:
    """The batched partial-hit workload: per-request hit lengths and page lists."""
    prefix_tokens: np.ndarray       # int64[n], full cached-prefix lengths
    hit_tokens: np.ndarray          # int64[n], tokens actually loaded (host chunk size)
    page_lists: List[np.ndarray]    # int32 pages per request
    pool_pages: int
    live_pages: np.ndarray          # pages left allocated by the churn (must stay untouched)
    mean_run_length: float          # mean contiguous-run length of the page lists


def batched_lengths(rng: np.random.Generator, n: int = 64, lo: int = 2 * KiB, hi: int = 128 * KiB,
                    hit_lo: float = 0.5, hit_hi: float = 1.0) -> Tuple[np.ndarray, np.ndarray]:
    """Cached-prefix lengths log-uniform in [lo, hi) and partial hits of 50-100%."""
    prefix = np.floor(np.exp(rng.uniform(math.log(lo), math.log(hi), n))).astype(np.int64)
    frac = rng.uniform(hit_lo, hit_hi, n)
    hit = np.maximum(1, np.floor(frac * prefix)).astype(np.int64)
    return prefix, hit


def churned_pool(rng: np.random.Generator, pool_pages: int, ops: int = 10_000,
                 max_block: int = 64) -> Tuple[List[int], List[np.ndarray]]:
    """Fragment a pool with a seeded allocate/free churn.

    The free list starts as the FIFO [0, pool_pages).  Each op allocates with
    probability 1/2 (k ~ U{1..max_block} pages popped from the head, kept as a
    live block) when the free list has room for k, and otherwise frees a
    uniformly chosen live block, appending its pages to the tail.  An op that
    can do neither does nothing.  Returns (free list, live blocks).
    """
    from collections import deque
    free = deque(range(pool_pages))
    live: List[np.ndarray] = []
    for _ in range(ops):
        alloc = rng.random() < 0.5
        k = int(rng.integers(1, max_block + 1))
        if alloc and k <= len(free):
            live.append(np.array([free.popleft() for _ in range(k)], dtype=np.int32))
        elif live:
            j = int(rng.integers(0, len(live)))
            blk = live.pop(j)
            free.extend(int(p) for p in blk)
    return list(free), live


def mean_run_length(page_lists: Sequence[np.ndarray]) -> float:
    """Mean length of maximal runs of consecutive pages (p, p+1, ...) in the lists."""
    runs = 0
    pages = 0
    for pl in page_lists:
        if len(pl) == 0:
            continue
        d = np.diff(pl.astype(np.int64))
        runs += 1 + int(np.count_nonzero(d != 1))
        pages += len(pl)
    return pages / runs if runs else 0.0


def batched_requests(k: int = 4, n: int = 64, page_size: int = 16, headroom: float = 1.15,
                     churn_ops: int = 10_000, max_block: int = 64,
                     scale: float = 1.0) -> BatchedRequests:
    """The batched mixed-hit workload (lengths from the placement seed, churn from
    the churn seed).  `scale` < 1 shrinks the lengths for CPU-sized tests (pass a
    smaller churn too, or the churn can fill a small pool)."""
    rng = np.random.default_rng(placement_seed(k))
    lo, hi = max(1, int(2 * KiB * scale)), max(2, int(128 * KiB * scale))
    prefix, hit = batched_lengths(rng, n, lo, hi)
    need = int(sum(-(-int(h) // page_size) for h in hit))
    pool_pages = int(math.ceil(headroom * need))
    free, live = churned_pool(np.random.default_rng(churn_seed(k)), pool_pages, churn_ops, max_block)
    if need > len(free):
        raise RuntimeError("churn left too few free pages for the batch")
    lists = []
    pos = 0
    for h in hit:
        c = -(-int(h) // page_size)
        lists.append(np.asarray(free[pos:pos + c], dtype=np.int32))
        pos += c
    live_pages = np.concatenate(live).astype(np.int32) if live else np.zeros(0, np.int32)
    return BatchedRequests(prefix, hit, lists, pool_pages, live_pages, mean_run_length(lists))


def batch_waves(sizes: Sequence[int], budget: int = 40 * GiB) -> List[List[int]]:
    """Split requests, in order, into the fewest consecutive waves whose host
    chunks total at most `budget` bytes each (a request larger than the budget
    forms a wave alone).  Pinned host memory per process may be capped (64 GiB
    on some machines), so the batched workload moves its ~180 GiB in waves,
    one batched call each."""
    waves: List[List[int]] = []
    cur: List[int] = []
    acc = 0
    for i, b in enumerate(sizes):
        if cur and acc + b > budget:
            waves.append(cur)
            cur, acc = [], 0
        cur.append(i)
        acc += b
    if cur:
        waves.append(cur)
    return waves


# ----------------------------------------------------------------------------
# Payload bytes
# ----------------------------------------------------------------------------

def _f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest even) and return the uint16 bit patterns."""
    u = x.astype(np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def payload_np(rng: np.random.Generator, n_elems: int, shape: KVShape) -> np.ndarray:
    """`n_elems` 16-bit KV elements as uint16 bit patterns (CPU generator)."""
    if shape.dist == "uniform":
        return rng.uniform(-1.0, 1.0, n_elems).astype(np.float16).view(np.uint16)
    return _f32_to_bf16_bits(rng.standard_normal(n_elems, dtype=np.float32))


def fill_np(dst: np.ndarray, seed: int, shape: KVShape, chunk_elems: int = 1 << 24) -> None:
    """Fill a flat uint8 array (even length) with seeded payload elements."""
    rng = np.random.default_rng(seed)
    view = dst.view(np.uint16)
    for a in range(0, view.size, chunk_elems):
        b = min(view.size, a + chunk_elems)
        view[a:b] = payload_np(rng, b - a, shape)


def fill_cuda(dst_ptr: int, nbytes: int, seed: int, shape: KVShape,
              chunk_bytes: int = 512 * MiB) -> None:
    """Fill host memory (pinned) or device memory at `dst_ptr` with seeded payload
    elements drawn on the GPU (torch's Philox generator, one fresh seed per
    chunk) and copied over.  Used for buffers too large to draw on the CPU in
    seconds.  Deterministic for a given seed and chunk size."""
    import torch
    assert nbytes % 2 == 0
    dst = torch.frombuffer((ctypes.c_uint8 * nbytes).from_address(dst_ptr), dtype=torch.uint8) \
        if nbytes else None
    gen = torch.Generator(device="cuda")
    for i, a in enumerate(range(0, nbytes, chunk_bytes)):
        b = min(nbytes, a + chunk_bytes)
        gen.manual_seed(seed * 1_000_003 + i)
        n = (b - a) // 2
        if shape.dist == "uniform":
            x = torch.rand(n, device="cuda", generator=gen, dtype=torch.float32).mul_(2.0).sub_(1.0)
            x = x.to(torch.float16)
        else:
            x = torch.randn(n, device="cuda", generator=gen, dtype=torch.float32).to(torch.bfloat16)
        dst[a:b].copy_(x.view(torch.uint8))
    torch.cuda.synchronize()


def tagged_payload(num_layers: int, host_tokens: int, heads: int, head_dim: int,
                   ctx: int = 0) -> np.ndarray:
    """Self-describing payload: every 16-bit element is a hash of its own
    (context, layer, kv, token, head, dim) coordinates, laid out layer-major and
    token-major, so a misplaced element names where it came from."""
    l, kv, t, h, d = np.meshgrid(np.arange(num_layers), np.arange(2), np.arange(host_tokens),
                                 np.arange(heads), np.arange(head_dim), indexing="ij")
    key = ((((ctx * 1009 + l) * 3 + kv) * 1_000_003 + t) * 257 + h) * 131 + d
    key = key.astype(np.uint64)
    key ^= key >> np.uint64(29)
    key *= np.uint64(0xBF58476D1CE4E5B9)
    key ^= key >> np.uint64(32)
    return (key & np.uint64(0xFFFF)).astype(np.uint16).reshape(-1).view(np.uint8)
