"""Benchmark of the paged-KV host<->HBM transfer path on one MI355X.

Default run (the headline): the batched workload 4 -- 64 cached contexts of
the Llama-3.1-8B KV shape (32 layers, K and V, 8 KV heads x 128 dims, bf16,
128 KiB per token) with prefixes log-uniform in [2K, 128K) tokens and 50-100%
hits, 1.48 M tokens = 180 GiB per direction, in a pool of 1.7 M slots at page
size 16 fragmented by a seeded 10,000-op allocate/free churn.  Pinned host
memory per process may be capped (64 GiB on some machines), so the contexts
move in 6 waves of at most 40 GiB through one host buffer.  Set-up (untimed)
fills every wave's chunk and loads it, so the pool holds all contexts.  One
step = for every wave, one batched kvio_offload (pool -> host) and one batched
kvio_load (host -> pool) of the wave's contexts.  Workloads 1, 2, 3 and 5 are
measured afterwards (--other-reps repetitions each) and summarised in the same
line under "other_workloads".

Reported (one JSON line):
  value       effective GB/s (1e9 B/s) of the whole step: load + offload
              payload bytes / mean step time (HIP events on the transfer
              stream); inputs are resident (host chunks pinned, pool in HBM)
              before the timed region.
  load/offload per-direction GB/s and tokens/s, each against the measured
              contiguous hipMemcpyAsync peak of the same direction, measured in the
              same run.
  roofline    the load kernel (the critical-path direction): algorithmic
              bytes per launch / mean launch time from HIP events on its
              stream, against the published PCIe Gen5 x16 rate (64 GB/s),
              with the ratio to the measured contiguous memcpy peak beside
              it; HBM side too; traffic from the committed rocprofv3 counters
              while the kernel sources match them.
  cpu_baseline the CPU oracle on the contexts of one wave, one core and all
              cores.

Other workloads alone: --config 1 (tiny pool, P = 16), --config 2 (Llama-3.1-8B
KV, P = 1, one 32K-token context), --config 3 (70B KV, P = 16, layer-wise load
on a side stream against a per-layer bf16 GEMM), --config 4 (the headline
without the others), --config 5 (1M-token load with concurrent offloads);
--staged (copy engine + HBM scatter), --interference, --page-sweep,
--row-sweep, --schedule, --disk.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

GB = 1e9
HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, vendor figure
PCIE_SPEC_GBPS = 64.0           # PCIe Gen5 x16 per direction (raw)
BIDIR_OVERLAP = 1.3             # H2D || D2H counts as overlapped above this x the faster direction


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=0, choices=[0, 1, 2, 3, 4, 5],
                    help="0 (default): the batched workload 4 is the headline and workloads 1, 2, 3 and 5 "
                         "are measured after it, in the same JSON line; 1-5: that workload alone")
    ap.add_argument("--other-reps", type=int, default=5,
                    help="timed repetitions of each other workload in the default run (reported as reps)")
    ap.add_argument("--no-other-workloads", action="store_true")
    ap.add_argument("--swap", action="store_true",
                    help="the batched workload swapped in both directions at once through two host buffers")
    ap.add_argument("--swap-wave-gib", type=int, default=30, help="host bytes per wave of the swap (two buffers)")
    ap.add_argument("--workgroups", type=int, default=0)
    ap.add_argument("--threads", type=int, default=0)
    ap.add_argument("--tile-kib", type=int, default=0)
    ap.add_argument("--cached", action="store_true", help="plain instead of non-temporal loads/stores")
    ap.add_argument("--bg-offload", type=str, default="16,64,4",
                    help="workgroups,threads,tile_kib of the background offload that runs beside a load "
                         "(the bidirectional workload); a small quota, as the paper gives backups")
    ap.add_argument("--noncoherent-host", action="store_true", help="coarse-grained pinned host chunks")
    ap.add_argument("--host-layout", choices=["token", "page", "head"], default="token",
                    help="host chunk layout: token-major (default), page-first, or head-major")
    ap.add_argument("--no-lds", action="store_true", help="head-major chunks: direct gather, no LDS staging")
    ap.add_argument("--staged", action="store_true",
                    help="copy engine through an HBM staging buffer + scatter/gather kernel (KVIO_LAUNCH_STAGED)")
    ap.add_argument("--staging-mib", type=int, default=0, help="staging per direction (4 slots); 0 = default")
    ap.add_argument("--cu-partition", type=int, default=0,
                    help="--config 3: load on a stream masked to the first N CUs, GEMMs on a stream masked to "
                         "the rest (0 = both streams over every CU)")
    ap.add_argument("--gemm-m", type=int, default=4096,
                    help="layer-wise workload: rows of the per-layer GEMM (4096 = load-bound; 65536 = compute-bound)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-naive", action="store_true")
    ap.add_argument("--no-peak", action="store_true")
    ap.add_argument("--peak-only", action="store_true",
                    help="measure the contiguous hipMemcpyAsync peaks only and print them as JSON")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--interference", action="store_true",
                    help="resource-quota sweep (Strata Fig. 5 analogue): load GB/s and the slowdown of a "
                         "co-running Llama-3.1-8B prefill pass (2 x 4K tokens) or decoding step (16 x 4K) vs. "
                         "the load's quota and CU placement, on the Llama-3.1-8B page-size-1 workload")
    ap.add_argument("--quotas", type=str, default="",
                    help="--interference: unmasked load quotas as WGxTHREADS,... (default: the full sweep)")
    ap.add_argument("--masked", type=str, default="",
                    help="--interference: CU partitions as NCUS:WGxTHREADS,... ('none' for no partition rows)")
    ap.add_argument("--page-sweep", action="store_true",
                    help="Llama-3.1-8B KV: kvio vs one hipMemcpyAsync per page segment over page sizes "
                         "1..256 (32K tokens), plus 8192 tokens at page size 32")
    ap.add_argument("--row-sweep", action="store_true",
                    help="GB/s against the token row size (KV heads x 128 dims x bf16 from 256 B to 8 KiB), "
                         "page size 1 and 16: the per-rank shapes of tensor-parallel serving")
    ap.add_argument("--schedule", action="store_true",
                    help="cache-aware batch formation: scheduling cost per round, and FIFO vs Algorithm 1 "
                         "on a synthetic queue under a cost model built from measured load and GEMM rates")
    ap.add_argument("--disk", action="store_true",
                    help="storage tier: 8192 tokens at page size 32 from a local disk store into pinned "
                         "host memory, page-first vs layer-first, then into the paged pool")
    ap.add_argument("--disk-dir", type=str, default=os.environ.get("TMPDIR", "/tmp"))
    ap.add_argument("--disk-threads", type=str, default="1,8")
    ap.add_argument("--calibrate-copy", type=int, default=0,
                    help="only run a plain device-to-device elementwise copy of this many bytes, three "
                         "times (the known-size kernel that scales the HBM byte counters), then exit")
    ap.add_argument("--naive-tokens", type=int, default=2048,
                    help="tokens of the context the naive per-page baseline copies (all layers)")
    return ap.parse_args()


COUNTER_FILES = {2: "kvio_copy_kernel__llama8b_p1_32k.counters.txt",
                 4: "kvio_copy_kernel__llama8b_p16_batched.counters.txt"}


def measured_traffic(config, default_launch):
    """HBM/link bytes per load launch from the committed rocprofv3 counter
    summary of a workload, if it was taken on the current kernels: the kernel
    source and the header that holds the kernel arguments and default launch
    shapes (else None).  A summary over several launches (load_launches) gives
    their mean."""
    import hashlib
    name = COUNTER_FILES.get(config)
    path = os.path.join(ROOT, "profiles", name) if name else None
    if not path or not default_launch or not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if line.strip() and not line.startswith("#"):
            key, val = line.split(":", 1)
            kv[key.strip()] = val.strip()
    csrc = os.path.join(ROOT, "paper_2508_18572_amd", "csrc")
    cur = " ".join(hashlib.sha256(open(os.path.join(csrc, f), "rb").read()).hexdigest()
                   for f in ("kvio_kernels.hip", "kvio_internal.h"))
    if cur != kv.get("kernel_sources_sha256"):
        return None
    launches = float(kv.get("load_launches", 1))
    fetch = float(kv["load_fetch_kib"]) * float(kv["fetch_scale"]) * 1024 / launches
    write = float(kv["load_write_kib"]) * float(kv["write_scale"]) * 1024 / launches
    return {"bytes": round(fetch + write), "fetch_bytes": round(fetch), "write_bytes": round(write),
            "source": os.path.relpath(path, ROOT)}


_IO = {}


def io_stream(torch, kv):
    """The transfer stream: a stream over every compute unit created through
    kvio_stream_create with a CU mask, which gives it a hardware queue of its
    own (ordinary streams share the few hardware queues round-robin, so two of
    them can serialise).  Created once per process; a plain torch stream if the
    runtime refuses."""
    if "s" not in _IO:
        try:
            n = torch.cuda.get_device_properties(0).multi_processor_count
            st = kv.Stream(list(range(n)))
            _IO["s"], _IO["kind"] = st.torch, f"dedicated queue (CU mask of all {n} CUs)"
            _IO["keep"] = st
        except kv.KvioError as e:
            _IO["s"], _IO["kind"] = torch.cuda.Stream(), f"torch stream ({e.detail})"
    return _IO["s"]


def close_io_stream(torch, kv):
    if "keep" in _IO:
        torch.cuda.synchronize()
        _IO.pop("keep").close()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class Timer:
    """HIP events on one stream."""

    def __init__(self, torch, stream):
        self.torch, self.stream = torch, stream
        self.pairs = []

    def start(self):
        e = self.torch.cuda.Event(enable_timing=True)
        e.record(self.stream)
        return e

    def stop(self, e0):
        e1 = self.torch.cuda.Event(enable_timing=True)
        e1.record(self.stream)
        self.pairs.append((e0, e1))

    def ms(self):
        return [a.elapsed_time(b) for a, b in self.pairs]


def memcpy_peak(torch, kv, src_ptr, dst_ptr, dev_ptr, nbytes, reps=5):
    """Median GB/s of one contiguous pinned hipMemcpyAsync per direction (H2D from
    src_ptr, D2H into dst_ptr), of the same copies by a plain kernel
    (kvio_kernel_memcpy: the kernel path's own ceiling, keys kernel_h2d and
    kernel_d2h), and of H2D and D2H memcpys running concurrently on two
    streams (each half the size)."""
    s1, s2 = io_stream(torch, kv), torch.cuda.Stream()
    half = nbytes // 2
    res = {}
    def one_direction(name, fn):
        fn(s1)
        torch.cuda.synchronize()
        t = Timer(torch, s1)
        for _ in range(reps):
            e = t.start()
            fn(s1)
            t.stop(e)
        torch.cuda.synchronize()
        res[name] = nbytes / (statistics.median(t.ms()) * 1e-3) / GB

    one_direction("h2d", lambda s: kv.kvio_memcpy(dev_ptr, src_ptr, nbytes, s))
    one_direction("d2h", lambda s: kv.kvio_memcpy(dst_ptr, dev_ptr, nbytes, s))
    # bidirectional: H2D of one half while D2H of the other half.  Copies on
    # two ordinary streams can serialise (they may share a hardware queue);
    # a pair of the transfer stream (or the null stream) with a stream made
    # before the transfer stream runs concurrently, later-made streams do so
    # only on some runs.  Several pairs are tried and the best (the link's
    # real bidirectional capacity) is kept.
    best = 0.0
    null = torch.cuda.default_stream()
    early = _PEAK.get("early_streams", [])
    pairs = [(s1, e) for e in early] + [(null, e) for e in early] + [(s1, s2)] + \
            [(s1, torch.cuda.Stream()) for _ in range(2)] + [(null, torch.cuda.Stream()) for _ in range(2)]
    for a, b in pairs:
        ts = []
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            kv.kvio_memcpy(dev_ptr, src_ptr, half, a)
            kv.kvio_memcpy(dst_ptr + half, dev_ptr + half, half, b)
            torch.cuda.synchronize()
            ts.append(time.perf_counter() - t0)
        best = max(best, 2 * half / statistics.median(ts) / GB)
    # In a few processes every pair above serialises; fresh HIP streams (new
    # runtime queues) are tried next, and if the two directions still never
    # overlap the bidirectional peak is reported as unmeasured, not as the
    # one-direction rate.
    overlap = BIDIR_OVERLAP * max(res["h2d"], res["d2h"])
    fresh = []
    try:
        while best < overlap and len(fresh) < 6:
            fresh.append(kv.Stream())
            for a, b in ((s1, fresh[-1].torch), (null, fresh[-1].torch)):
                ts = []
                for _ in range(reps):
                    torch.cuda.synchronize()
                    t0 = time.perf_counter()
                    kv.kvio_memcpy(dev_ptr, src_ptr, half, a)
                    kv.kvio_memcpy(dst_ptr + half, dev_ptr + half, half, b)
                    torch.cuda.synchronize()
                    ts.append(time.perf_counter() - t0)
                best = max(best, 2 * half / statistics.median(ts) / GB)
    finally:
        for f in fresh:
            f.close()
    if best >= overlap:
        res["bidir"] = best
    else:
        res["bidir"] = None
        res["bidir_note"] = (f"unmeasured: the runtime serialised H2D and D2H copies on every stream pair "
                             f"tried in this process (best {best:.2f} GB/s)")
    one_direction("kernel_h2d", lambda s: kv.kvio_kernel_memcpy(dev_ptr, src_ptr, nbytes, s))
    one_direction("kernel_d2h", lambda s: kv.kvio_kernel_memcpy(dst_ptr, dev_ptr, nbytes, s))
    res["bytes"] = nbytes
    return res


def peak_report(peak):
    """The measured memcpy peaks for the JSON line (GB/s rounded)."""
    if not peak:
        return None
    return {k: round(v, 3) if isinstance(v, float) else v for k, v in peak.items()}


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo), else the machine type."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.machine() or "host CPU"


def cpu_baseline(pool_rows, row_bytes, host, host_tokens, num_tokens, pages, page_size, L, seconds):
    """The CPU oracle (single thread) loading then offloading the same context,
    one (layer, K|V) slab at a time into a host image of one pool slab, until
    `seconds` have passed (whole context passes only)."""
    import oracle
    slab = np.zeros((pool_rows, row_bytes), np.uint8)
    out = np.zeros(num_tokens * row_bytes, np.uint8)
    h = host.reshape(L, 2, host_tokens * row_bytes)
    t0 = time.perf_counter()
    passes = 0
    while True:
        for l in range(L):
            for kvi in range(2):
                src = h[l, kvi]
                oracle.load_slab(slab, page_size, src, num_tokens, pages)
                oracle.offload_slab(slab, page_size, out, num_tokens, pages)
        passes += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    nbytes = passes * 2 * L * 2 * num_tokens * row_bytes
    return nbytes, el, passes


def cpu_baseline_all_cores(pool_rows, row_bytes, host, host_tokens, num_tokens, pages, page_size, L, seconds,
                           threads):
    """The same CPU oracle, unchanged, on `threads` host threads at once: each
    thread loads then offloads its own share of the (layer, K|V) slabs into a
    slab image of its own (the oracle's C calls run without the interpreter
    lock), until `seconds` have passed."""
    import threading

    import oracle
    h = host.reshape(L, 2, host_tokens * row_bytes)
    planes = [(l, kvi) for l in range(L) for kvi in range(2)]
    done = [0] * threads
    stop = threading.Event()

    def work(w):
        slab = np.zeros((pool_rows, row_bytes), np.uint8)
        out = np.zeros(num_tokens * row_bytes, np.uint8)
        i = w
        while not stop.is_set():
            l, kvi = planes[i % len(planes)]
            oracle.load_slab(slab, page_size, h[l, kvi], num_tokens, pages)
            oracle.offload_slab(slab, page_size, out, num_tokens, pages)
            done[w] += 1
            i += threads

    workers = [threading.Thread(target=work, args=(w,)) for w in range(threads)]
    t0 = time.perf_counter()
    for t in workers:
        t.start()
    time.sleep(seconds)
    stop.set()
    for t in workers:
        t.join()
    el = time.perf_counter() - t0
    return sum(done) * 2 * num_tokens * row_bytes, el, sum(done)


def steady_state(torch, kv, pool, span, host, stream, payload, reps):
    """Small-context latency: one load alone (host launch to completion, and
    GPU time), then `reps` back-to-back loads; the same for a contiguous
    hipMemcpyAsync of the same size into device memory."""
    dev = torch.empty(payload, dtype=torch.uint8, device="cuda")
    out = {}
    for name, fn in (("load", lambda: pool.load(span, stream=stream)),
                     ("memcpy", lambda: kv.kvio_memcpy(dev.data_ptr(), host.ptr, payload, stream))):
        fn()
        torch.cuda.synchronize()
        shots = []
        gpu = []
        for _ in range(20):
            t = Timer(torch, stream)
            c0 = time.perf_counter()
            e = t.start()
            fn()
            t.stop(e)
            stream.synchronize()
            shots.append((time.perf_counter() - c0) * 1e6)
            gpu.append(t.ms()[0] * 1e3)
        t = Timer(torch, stream)
        e = t.start()
        for _ in range(reps):
            fn()
        t.stop(e)
        torch.cuda.synchronize()
        ms = t.ms()[0]
        out[f"{name}_gbps"] = round(reps * payload / (ms * 1e-3) / GB, 3)
        out[f"{name}_us_per_transfer"] = round(ms * 1e3 / reps, 3)
        out[f"{name}_single_shot_wall_us"] = round(statistics.median(shots), 2)
        out[f"{name}_single_shot_gpu_us"] = round(statistics.median(gpu), 2)
    out["single_shot_us"] = out["load_single_shot_wall_us"]
    out["reps"] = reps
    del dev
    return out


def launch_breakdown(torch, kv, pool, span, page_span, page_bytes, payload, h2d_peak, n=200):
    """Where the time of a small load goes.  Three chains of n launches are
    captured in HIP graphs (torch.cuda.CUDAGraph) and replayed, so the host
    never gates the GPU: the whole small context, a single page of it, and a
    one-element torch kernel.  Per launch: the empty kernel gives the GPU's
    launch-to-launch cost, the one-page load adds the host link's first-byte
    latency, and the rest of the small context's time is streaming, compared
    with its bytes at the measured H2D peak."""
    s = torch.cuda.Stream()
    x = torch.zeros(1, device="cuda")
    chains = {"context": lambda: pool.load(span, stream=s), "page": lambda: pool.load(page_span, stream=s),
              "empty_kernel": lambda: x.add_(1.0)}
    out = {}
    for name, fn in chains.items():
        with torch.cuda.stream(s):
            for _ in range(3):
                fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for _ in range(n):
                fn()
        ts = []
        with torch.cuda.stream(s):                      # replay() launches on the current stream
            g.replay()
            torch.cuda.synchronize()
            for _ in range(5):
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(s)
                g.replay()
                b.record(s)
                torch.cuda.synchronize()
                ts.append(a.elapsed_time(b) * 1e3 / n)
        out[f"{name}_us_per_launch"] = round(statistics.median(ts), 3)
        del g
    pool.check()
    if h2d_peak:
        stream_us = payload / (h2d_peak * GB) * 1e6
        out["context_at_h2d_peak_us"] = round(stream_us, 3)
        out["page_bytes"] = page_bytes
        out["first_byte_us"] = round(out["page_us_per_launch"] - out["empty_kernel_us_per_launch"]
                                     - page_bytes / (h2d_peak * GB) * 1e6, 3)
        out["context_minus_streaming_us"] = round(out["context_us_per_launch"] - stream_us, 3)
    return out


def small_context_pipelines(torch, kv, pool, host, T, P, S, used_pages, stream, payload, reps=1000):
    """Independent small contexts as a server meets them, beside the one-stream
    steady state: (a) alternating over two streams (the transfer stream and one
    made before it), each stream loading into its own pages, so one launch's
    ramp-up overlaps the other's drain; (b) four contexts per batched call.
    Every context has a host chunk of its own (a repeated chunk would let the
    GPU serve repeated reads without crossing the link), and the page sets are
    disjoint, so loads that may run at once never write the same slot."""
    need = -(-T // P)
    free = np.setdiff1d(np.arange(S // P, dtype=np.int32), np.asarray(used_pages, np.int32))
    free = np.random.default_rng(400).permutation(free).astype(np.int32)
    sets = [np.asarray(used_pages, np.int32)] + [free[i * need:(i + 1) * need] for i in range(len(free) // need)]
    if len(sets) < 4:
        return {}
    tabs = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in sets[:4]]
    chunks = [kv.HostBuffer(payload) for _ in range(4)]
    early = _PEAK.get("early_streams") or [torch.cuda.Stream()]
    streams = [stream, early[0]]
    out = {}

    def timed(issue, n):
        for _ in range(10):
            issue(0)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        streams[1].wait_event(e0)
        for i in range(n):
            issue(i)
        joined = torch.cuda.Event()
        joined.record(streams[1])
        stream.wait_event(joined)
        e1 = torch.cuda.Event(enable_timing=True)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    try:
        for c in chunks:
            c.array[:] = host.array[:payload]
        ms = timed(lambda i: pool.load([(chunks[i % 2].ptr, T, T, tabs[i % 2].data_ptr())], stream=streams[i % 2]),
                   reps)
        out["two_streams_load_gbps"] = round(reps * payload / (ms * 1e-3) / GB, 3)
        batch = [(c.ptr, T, T, t.data_ptr()) for c, t in zip(chunks, tabs)]
        calls = reps // 4
        ms = timed(lambda i: pool.load(batch, stream=stream), calls)
        out["batched4_load_gbps"] = round(calls * 4 * payload / (ms * 1e-3) / GB, 3)
        pool.check()
    finally:
        for c in chunks:
            c.free()
    return out


def base_result(args, value, ms_per_step, workload, extra_config):
    cfg = {"workload": workload}
    cfg.update(extra_config)
    cfg["io_stream"] = _IO.get("kind")
    return {
        "metric": "effective KV load/offload GB/s and tokens/s; % of measured host-link peak",
        "value": round(value, 3), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u8", "data": "synthetic", "config": cfg,
    }


_PEAK = {}


def h2d_d2h_peak(torch, kv, nbytes=2 << 30):
    """The contiguous hipMemcpyAsync peak on buffers of its own (2 GiB pinned
    host, 2 GiB device).  Measured once per process, first thing after the
    transfer stream exists: later in a run, after other streams and large
    allocations, the runtime has been seen to serialise the two directions
    of the bidirectional measurement."""
    if "peak" in _PEAK:
        return _PEAK["peak"]
    scratch = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    with kv.HostBuffer(nbytes) as hb:
        hb.array[::4096] = 1                      # touch every page once
        peak = memcpy_peak(torch, kv, hb.ptr, hb.ptr, scratch.data_ptr(), nbytes)
    del scratch
    if peak["bidir"] is None and not _PEAK.get("child"):
        child = peak_in_child()
        if child and child.get("bidir"):
            peak["bidir"] = child["bidir"]
            peak["bidir_note"] = ("measured in a fresh child process: this process's runtime serialised "
                                  "H2D and D2H copies on every stream pair tried")
    bidir = f"{peak['bidir']:.2f} GB/s" if peak["bidir"] else peak["bidir_note"]
    log(f"memcpy peak: h2d {peak['h2d']:.2f} GB/s, d2h {peak['d2h']:.2f} GB/s, bidir {bidir}; plain copy kernel: "
        f"h2d {peak['kernel_h2d']:.2f} GB/s, d2h {peak['kernel_d2h']:.2f} GB/s")
    _PEAK["peak"] = peak
    return peak


def peak_in_child():
    """The contiguous memcpy peaks measured by a fresh Python process running
    this script with --peak-only (a new HIP runtime, whose streams get new
    hardware queues); None if it fails."""
    import subprocess
    try:
        r = subprocess.run([sys.executable, os.path.abspath(__file__), "--peak-only"], capture_output=True,
                           text=True, timeout=180)
        if r.returncode != 0:
            log(f"peak child failed (rc {r.returncode}): {r.stderr[-300:]}")
            return None
        return json.loads(r.stdout.strip().splitlines()[-1])
    except (subprocess.TimeoutExpired, ValueError, IndexError) as e:
        log(f"peak child failed: {e}")
        return None


def roofline(kernel, achieved, measured_peak, directions=1, traffic=None, **extra):
    """Roofline block of a host-link-bound kernel.  `peak` is the published
    PCIe Gen5 x16 rate (64 GB/s per direction, 128 both ways); the measured
    contiguous hipMemcpyAsync peak of the same run -- the achievable ceiling
    the targets are set against -- is reported beside it.  HBM (8 TB/s) is
    reported too; the path uses under 1% of it."""
    spec = PCIE_SPEC_GBPS * directions
    out = {"bound": "host_link" + (" (both directions)" if directions == 2 else ""), "kernel": kernel,
           "achieved": round(achieved, 3), "peak": spec, "unit": "GB/s", "frac": round(achieved / spec, 4),
           "peak_source": f"PCIe Gen5 x16, {spec:.0f} GB/s" + (" both directions" if directions == 2 else
                                                               " per direction") + " (published)",
           "measured_memcpy_peak": round(measured_peak, 3) if measured_peak else None,
           "frac_of_measured_peak": round(achieved / measured_peak, 4) if measured_peak else None,
           "traffic": traffic["bytes"] if traffic else None, "traffic_detail": traffic,
           "hbm": {"achieved": round(achieved, 3), "peak": HBM_PEAK_GBPS, "frac": round(achieved / HBM_PEAK_GBPS, 5)}}
    out.update(extra)
    return out


def launch_from(args, kv):
    flags = (kv.KVIO_LAUNCH_CACHED if args.cached else 0) | (kv.KVIO_LAUNCH_NO_LDS if args.no_lds else 0) | \
        (kv.KVIO_LAUNCH_STAGED if args.staged else 0)
    return kv.launch(args.workgroups, args.threads, args.tile_kib, flags)


def layout_from(args, kv):
    return {"token": kv.KVIO_HOST_TOKEN_MAJOR, "page": kv.KVIO_HOST_PAGE_FIRST,
            "head": kv.KVIO_HOST_HEAD_MAJOR}[args.host_layout]


def run_layerwise(args, torch, kv, W):
    """70B GQA KV at page size 16: a 64K-token context loaded layer by layer on a
    side stream (kvio_load_layer, one event per layer) while a compute stream
    runs one bf16 GEMM (M x 8192 x 8192, M = 4096 by default: load-bound) per
    layer, each GEMM waiting on its layer's event (layer-wise overlap, Strata
    Sec. 4.1 / Sec. 4.2.1)."""
    k = 3
    wl = W.WORKLOADS[k]
    shp = wl.shape
    L, H, D, P, S, T = shp.num_layers, shp.num_kv_heads, shp.head_dim, wl.page_size, wl.num_slots, wl.tokens
    R = shp.row_bytes
    log(f"{wl.description}; L={L} P={P} S={S} T={T}")
    pool_t = torch.empty((2, L, S, H, D), dtype=torch.bfloat16, device="cuda")
    pages = W.random_pages(np.random.default_rng(W.placement_seed(k)), S // P, -(-T // P))
    pidx = torch.from_numpy(pages).cuda()
    nbytes = L * 2 * T * R
    host = kv.HostBuffer(nbytes)
    peak = None if args.no_peak else h2d_d2h_peak(torch, kv)
    W.fill_cuda(host.ptr, nbytes, W.data_seed(k), shp)
    pool = kv.KVPool(pool_t, P, load_launch=launch_from(args, kv), host_layout=layout_from(args, kv),
                     staging_bytes=args.staging_mib << 20)
    span = [(host.ptr, T, T, pidx.data_ptr())]
    side, comp = io_stream(torch, kv), torch.cuda.Stream()
    masked = []
    if args.cu_partition:
        # The load on its own CUs, the GEMMs on the others: neither waits for
        # CUs the other holds (Sec. 4.2: confine the I/O kernel to few CUs).
        n_cu = torch.cuda.get_device_properties(0).multi_processor_count
        masked = [kv.Stream(list(range(args.cu_partition))), kv.Stream(list(range(args.cu_partition, n_cu)))]
        side, comp = masked[0].torch, masked[1].torch
    M, N, K = args.gemm_m, 8192, 8192
    g = torch.Generator(device="cuda").manual_seed(W.data_seed(k))
    A = torch.randn(M, K, device="cuda", dtype=torch.bfloat16, generator=g)
    B = torch.randn(K, N, device="cuda", dtype=torch.bfloat16, generator=g)
    C = torch.empty(M, N, device="cuda", dtype=torch.bfloat16)
    per_layer = 2 * T * R

    def loads_alone():
        t = Timer(torch, side)
        e = t.start()
        for l in range(L):
            pool.load_layer(span, l, stream=side)
        t.stop(e)
        torch.cuda.synchronize()
        return t.ms()[0]

    def gemms_alone():
        t = Timer(torch, comp)
        e = t.start()
        with torch.cuda.stream(comp):
            for l in range(L):
                torch.matmul(A, B, out=C)
        t.stop(e)
        torch.cuda.synchronize()
        return t.ms()[0]

    def both():
        # Event handles exist before the timed region (torch creates one at its
        # first record), so the side stream carries only the library's record.
        evs_all = [torch.cuda.Event(enable_timing=True) for _ in range(L)]
        for ev in evs_all:
            ev.record(comp)
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        start.record(comp)
        side.wait_event(start)
        g0, g1, evs = [], [], []
        for l in range(L):
            ev = evs_all[l]
            pool.load_layer(span, l, stream=side, done=ev)
            evs.append(ev)
            comp.wait_event(ev)
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(comp)
            with torch.cuda.stream(comp):
                torch.matmul(A, B, out=C)
            b.record(comp)
            g0.append(a)
            g1.append(b)
        torch.cuda.synchronize()
        t_both = start.elapsed_time(g1[-1])
        t_load = start.elapsed_time(evs[-1])
        gemm_ms = sum(x.elapsed_time(y) for x, y in zip(g0, g1))
        return t_both, t_load, gemm_ms

    for _ in range(max(1, args.warmup)):
        loads_alone()
        gemms_alone()
        both()
    reps = max(1, args.steps)
    tl = statistics.median(loads_alone() for _ in range(reps))
    tg = statistics.median(gemms_alone() for _ in range(reps))
    runs = [both() for _ in range(reps)]
    tb = statistics.median(r[0] for r in runs)
    tl_co = statistics.median(r[1] for r in runs)
    tg_co = statistics.median(r[2] for r in runs)
    pool.check()
    overlap = (tl + tg - tb) / min(tl, tg)
    load_gbps = nbytes / (tl * 1e-3) / GB
    load_gbps_co = nbytes / (tl_co * 1e-3) / GB
    gemm_tflops = L * 2 * M * N * K / (tg * 1e-3) / 1e12
    log(f"load alone {tl:.2f} ms ({load_gbps:.2f} GB/s), GEMMs alone {tg:.2f} ms ({gemm_tflops:.0f} TFLOP/s), "
        f"both {tb:.2f} ms; load co-run {load_gbps_co:.2f} GB/s; GEMM time co-run {tg_co:.2f} ms; "
        f"overlap efficiency {overlap:.3f}")
    res = base_result(args, load_gbps_co, tb, wl.description,
                      {"kv_shape": shp.name, "layers": L, "page_size": P, "pool_slots": S, "tokens": T,
                       "payload_bytes": nbytes, "bytes_per_layer_launch": per_layer,
                       "gemm_per_layer": [M, N, K], "step": "80 x (kvio_load_layer on a side stream; "
                       "event; bf16 GEMM on the compute stream)",
                       "cu_partition": (f"load on CUs 0-{args.cu_partition - 1}, GEMMs on the others"
                                        if args.cu_partition else "none: both streams over every CU")})
    res.update({
        "tokens_per_s": round(T / (tl_co * 1e-3), 1),
        "layerwise": {"t_load_alone_ms": round(tl, 3), "t_gemm_alone_ms": round(tg, 3), "t_both_ms": round(tb, 3),
                      "t_load_in_corun_ms": round(tl_co, 3), "gemm_ms_in_corun": round(tg_co, 3),
                      "overlap_efficiency": round(overlap, 4), "load_gbps_alone": round(load_gbps, 3),
                      "load_gbps_corun": round(load_gbps_co, 3), "gemm_slowdown": round(tg_co / tg, 4),
                      "gemm_tflops_alone": round(gemm_tflops, 1)},
        "load": {"gbps": round(load_gbps_co, 3), "frac_of_h2d_peak": round(load_gbps_co / peak["h2d"], 4) if peak else None},
        "host_link_peak": peak_report(peak),
        "roofline": roofline("kvio_copy_kernel<load> (per layer)", load_gbps, peak["h2d"] if peak else None,
                             algorithmic_bytes_per_launch=per_layer),
        "reps": reps,
    })
    pool.close()
    for st in masked:
        st.close()
    del pool_t
    host.free()
    torch.cuda.empty_cache()
    return res


def cpu_baseline_batched(slab_rows, row_bytes, chunk, spans, page_size, L, seconds, threads):
    """The CPU oracle, unchanged, on the spans of one wave of the batched
    workload: load then offload of every span, one (layer, K|V) slab at a
    time, into one host image of a pool slab (S rows), plane after plane until
    `seconds` have passed.  With threads > 1 the spans are cut into pieces of
    whole pages (at most 8192 tokens) that the threads share out; pieces write
    disjoint rows of the one slab image and offload into buffers of their
    own.  spans: (byte offset of the chunk in `chunk`, host_tokens,
    num_tokens, page_idx).  Returns (bytes moved, seconds, planes done)."""
    import threading

    import oracle
    R = row_bytes
    piece = 8192 - 8192 % page_size if page_size <= 8192 else page_size
    items = []
    for off, ht, nt, pages in spans:
        for a in range(0, nt, piece):
            items.append((off, ht, a, min(piece, nt - a), pages[a // page_size:]))
    slab = np.zeros((slab_rows, R), np.uint8)
    slab.fill(1)                     # touch every page before the clock starts
    planes = [(l, kvi) for l in range(L) for kvi in range(2)]
    done = [0] * threads
    moved = [0] * threads
    stop = threading.Event()

    def work(w):
        mine = items[w::threads]
        out = np.ones(max([n for _, _, _, n, _ in mine], default=1) * R, np.uint8)
        i = 0
        while not stop.is_set():
            l, kvi = planes[i % len(planes)]
            for off, ht, a, n, pages in mine:
                base = off + ((l * 2 + kvi) * ht + a) * R
                oracle.load_slab(slab, page_size, chunk[base:base + n * R], n, pages)
                oracle.offload_slab(slab, page_size, out, n, pages)
                moved[w] += 2 * n * R
            done[w] += 1
            i += 1
            if threads == 1 and time.perf_counter() - t0 >= seconds:
                break

    if threads == 1:
        t0 = time.perf_counter()
        work(0)
    else:
        workers = [threading.Thread(target=work, args=(w,)) for w in range(threads)]
        t0 = time.perf_counter()
        for t in workers:
            t.start()
        time.sleep(seconds)
        stop.set()
        for t in workers:
            t.join()
    el = time.perf_counter() - t0
    return sum(moved), el, min(done)


def run_batched(args, torch, kv, W):
    """The batched workload: 64 partial-hit contexts of the Llama-3.1-8B KV
    shape at page size 16, placed in a pool fragmented by a seeded 10,000-op
    allocate/free churn.  Pinned host memory per process may be capped (64 GiB
    on some machines), so the ~180 GiB of host chunks move in waves of at most
    40 GiB through one host buffer, one batched call per wave and direction.

    Set-up (untimed): every wave's chunk is filled with its seeded payload and
    loaded, so the pool holds all 64 contexts.  One step = for every wave, a
    batched kvio_offload of the wave's contexts from the pool into the host
    buffer, then a batched kvio_load of them back into their pages: every
    context crosses the host link once in each direction, and the data a load
    moves is the data its offload wrote.  Every step is timed with HIP events
    on the transfer stream, each launch with its own pair."""
    k = 4
    shp = W.LLAMA8B
    L, H, D, P = shp.num_layers, shp.num_kv_heads, shp.head_dim, 16
    R = shp.row_bytes
    req = W.batched_requests(k)
    S = req.pool_pages * P
    hit = [int(h) for h in req.hit_tokens]
    sizes = [L * 2 * h * R for h in hit]
    waves = W.batch_waves(sizes, 40 << 30)
    total = sum(sizes)
    wave_bytes = [sum(sizes[i] for i in w) for w in waves]
    log(f"batched partial hits: {sum(hit)} tokens, {total / 2**30:.1f} GiB per direction, pool {S} slots, "
        f"{len(waves)} waves, mean page-run length {req.mean_run_length:.2f}")
    peak = None if args.no_peak else h2d_d2h_peak(torch, kv)
    torch.cuda.empty_cache()
    pool_t = torch.empty((2, L, S, H, D), dtype=torch.bfloat16, device="cuda")
    lc = launch_from(args, kv)
    pool = kv.KVPool(pool_t, P, load_launch=lc, offload_launch=lc, staging_bytes=args.staging_mib << 20)
    pts = [torch.from_numpy(pl).cuda() for pl in req.page_lists]
    host = kv.HostBuffer(max(wave_bytes))
    stream = io_stream(torch, kv)
    wave_spans, offs_of = [], []
    for w in waves:
        offs, o = {}, 0
        for i in w:
            offs[i] = o
            o += sizes[i]
        offs_of.append(offs)
        wave_spans.append([(host.ptr + offs[i], hit[i], hit[i], pts[i].data_ptr()) for i in w])
    t0 = time.perf_counter()
    for j, (w, spans) in enumerate(zip(waves, wave_spans)):
        for i in w:
            W.fill_cuda(host.ptr + offs_of[j][i], sizes[i], W.data_seed(k) * 1000 + i, shp)
        pool.load(spans, stream=stream)
        torch.cuda.synchronize()
    pool.check()
    log(f"set-up: {len(waves)} waves filled and loaded in {time.perf_counter() - t0:.1f} s")

    def step(tl, to):
        for spans in wave_spans:
            e = to.start()
            pool.offload(spans, stream=stream)
            to.stop(e)
            e = tl.start()
            pool.load(spans, stream=stream)
            tl.stop(e)

    for _ in range(args.warmup):
        step(Timer(torch, stream), Timer(torch, stream))
    torch.cuda.synchronize()
    tl, to, tstep = Timer(torch, stream), Timer(torch, stream), Timer(torch, stream)
    w0 = time.perf_counter()
    for _ in range(args.steps):
        e = tstep.start()
        step(tl, to)
        tstep.stop(e)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    pool.check()
    load_ms, off_ms, step_ms = tl.ms(), to.ms(), tstep.ms()
    n_w = len(waves)
    # per-step totals (every step moves every wave once in each direction)
    t_load = sum(load_ms) / args.steps
    t_off = sum(off_ms) / args.steps
    t_step = statistics.mean(step_ms)
    load_gbps, off_gbps = total / (t_load * 1e-3) / GB, total / (t_off * 1e-3) / GB
    value = 2 * total / (t_step * 1e-3) / GB
    wave_load_ms = [statistics.mean(load_ms[j::n_w]) for j in range(n_w)]
    log(f"step {t_step:.1f} ms ({value:.2f} GB/s both directions), wall {wall / args.steps * 1e3:.1f} ms/step; "
        f"load {load_gbps:.2f} GB/s, offload {off_gbps:.2f} GB/s over {n_w} waves")

    # the data survived every round trip: the last wave's first context against its seed
    i0 = waves[-1][0]
    with kv.HostBuffer(sizes[i0]) as ref:
        W.fill_cuda(ref.ptr, sizes[i0], W.data_seed(k) * 1000 + i0, shp)
        ok = memequal_ptr(host.ptr + offs_of[-1][i0], ref.ptr, sizes[i0])
    assert ok, "the batched round trips changed a context's bytes"

    cpu = cpu_all = None
    if not args.no_cpu_baseline:
        # the first (largest) wave's contexts, brought back into the host buffer untimed
        pool.offload(wave_spans[0], stream=stream)
        torch.cuda.synchronize()
        first = [(offs_of[0][i], hit[i], hit[i], req.page_lists[i]) for i in waves[0]]
        desc = (f"the {len(first)} contexts of the first wave ({wave_bytes[0] / 2**30:.1f} GiB per direction), "
                f"load + offload one (layer, K|V) slab at a time through a {S}-row host slab image")
        nb, el, planes = cpu_baseline_batched(S, R, host.array, first, P, L, args.cpu_seconds, 1)
        cpu = {"value": round(nb / el / GB, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
               "sample": f"{desc}: {planes} plane(s) in {el:.1f} s on {cpu_model()} "
                         f"({len(os.sched_getaffinity(0))} cores available, 1 used)"}
        nthreads = min(len(os.sched_getaffinity(0)), 16)
        nb, el, planes = cpu_baseline_batched(S, R, host.array, first, P, L, args.cpu_seconds, nthreads)
        cpu_all = {"value": round(nb / el / GB, 3), "unit": "GB/s", "cores": nthreads, "kind": "oracle",
                   "sample": f"{desc}, pieces of <= 8192 tokens shared by {nthreads} threads: "
                             f"{planes}+ plane(s) in {el:.1f} s on {cpu_model()}"}
        log(f"cpu oracle: {cpu['value']:.2f} GB/s on 1 core, {cpu_all['value']:.2f} GB/s on {nthreads} threads")

    default_launch = not (args.workgroups or args.threads or args.tile_kib or args.cached or args.staged)
    traffic = measured_traffic(4, default_launch)
    res = base_result(args, value, t_step, "batched partial hits (workload 4): 64 Llama-3.1-8B KV contexts, "
                      "page size 16, prefixes log-uniform in [2K, 128K) tokens with 50-100% hits, in a pool "
                      "fragmented by a 10,000-op allocate/free churn",
                      {"kv_shape": shp.name, "layers": L, "page_size": P, "pool_slots": S, "requests": len(hit),
                       "tokens": sum(hit), "payload_bytes_per_direction": total, "waves": n_w,
                       "wave_payload_bytes": wave_bytes, "mean_page_run_length": round(req.mean_run_length, 3),
                       "step": "for each wave: batched kvio_offload (pool -> host) then batched kvio_load "
                               "(host -> pool) of the wave's contexts"})
    res.update({
        "tokens_per_s": round(2 * sum(hit) / (t_step * 1e-3), 1),
        "load": {"gbps": round(load_gbps, 3), "ms_per_step": round(t_load, 3),
                 "tokens_per_s": round(sum(hit) / (t_load * 1e-3), 1),
                 "frac_of_h2d_peak": round(load_gbps / peak["h2d"], 4) if peak else None,
                 "frac_of_kernel_h2d_peak": round(load_gbps / peak["kernel_h2d"], 4) if peak else None},
        "offload": {"gbps": round(off_gbps, 3), "ms_per_step": round(t_off, 3),
                    "tokens_per_s": round(sum(hit) / (t_off * 1e-3), 1),
                    "frac_of_d2h_peak": round(off_gbps / peak["d2h"], 4) if peak else None,
                    "frac_of_kernel_d2h_peak": round(off_gbps / peak["kernel_d2h"], 4) if peak else None},
        "frac_of_host_link_peak": round((total / (peak["h2d"] * GB) + total / (peak["d2h"] * GB)) * 1e3 / t_step, 4)
        if peak else None,
        "wave_load_ms": [round(x, 3) for x in wave_load_ms],
        "host_link_peak": peak_report(peak),
        "roofline": roofline("kvio_copy_kernel<load> (batched spans, one launch per wave)", load_gbps,
                             peak["h2d"] if peak else None, traffic=traffic,
                             algorithmic_bytes_per_launch=round(total / n_w),
                             algorithmic_traffic_per_launch=round(2 * total / n_w),
                             launches_per_step=n_w,
                             plain_kernel_copy_peak=round(peak["kernel_h2d"], 3) if peak else None,
                             frac_of_plain_kernel_copy_peak=round(load_gbps / peak["kernel_h2d"], 4)
                             if peak else None),
        "cpu_baseline": cpu,
        "cpu_baseline_all_cores": cpu_all,
    })
    pool.close()
    del pool_t
    host.free()
    torch.cuda.empty_cache()
    return res


def run_swap(args, torch, kv, W):
    """The batched workload swapped through the link in both directions at
    once: the 64 contexts of workload 4 move in waves of at most
    --swap-wave-gib GiB (30 by default) through two host buffers, so wave w's offload (pool -> buffer w % 2, on its own
    stream, with the background quota of --bg-offload) runs while wave w - 1
    loads back (buffer (w - 1) % 2 -> pool, on the transfer stream).  A wave's
    load waits for its offload; an offload into a buffer waits for the load
    that last read it.  One step moves every context once in each direction;
    set-up loads every wave first, as in the headline."""
    k = 4
    shp = W.LLAMA8B
    L, H, D, P = shp.num_layers, shp.num_kv_heads, shp.head_dim, 16
    R = shp.row_bytes
    req = W.batched_requests(k)
    S = req.pool_pages * P
    hit = [int(h) for h in req.hit_tokens]
    sizes = [L * 2 * h * R for h in hit]
    waves = W.batch_waves(sizes, args.swap_wave_gib << 30)
    total = sum(sizes)
    wave_bytes = [sum(sizes[i] for i in w) for w in waves]
    log(f"swap: {total / 2**30:.1f} GiB per direction in {len(waves)} waves through two host buffers")
    peak = None if args.no_peak else h2d_d2h_peak(torch, kv)
    torch.cuda.empty_cache()
    pool_t = torch.empty((2, L, S, H, D), dtype=torch.bfloat16, device="cuda")
    bg = [int(x) for x in args.bg_offload.split(",")]
    pool = kv.KVPool(pool_t, P)
    pool_off = kv.KVPool(pool_t, P, offload_launch=kv.launch(bg[0], bg[1], bg[2], 0))
    pts = [torch.from_numpy(pl).cuda() for pl in req.page_lists]
    bufs = [kv.HostBuffer(max(wave_bytes)), kv.HostBuffer(max(wave_bytes))]
    sl, so = io_stream(torch, kv), torch.cuda.Stream()
    spans = []
    for j, w in enumerate(waves):
        o, sp = 0, []
        for i in w:
            sp.append((bufs[j % 2].ptr + o, hit[i], hit[i], pts[i].data_ptr()))
            o += sizes[i]
        spans.append(sp)
    for j, w in enumerate(waves):                          # set-up: every wave loaded once
        o = 0
        for i in w:
            W.fill_cuda(bufs[j % 2].ptr + o, sizes[i], W.data_seed(k) * 1000 + i, shp)
            o += sizes[i]
        pool.load(spans[j], stream=sl)
        torch.cuda.synchronize()
    pool.check()

    def step():
        """Returns the events bracketing the step on the transfer stream."""
        e0 = torch.cuda.Event(enable_timing=True)
        e0.record(sl)
        so.wait_event(e0)
        loaded = [None, None]                             # last load that read each buffer
        for j in range(len(waves)):
            if loaded[j % 2] is not None:
                so.wait_event(loaded[j % 2])
            pool_off.offload(spans[j], stream=so)
            off_done = torch.cuda.Event()
            off_done.record(so)
            sl.wait_event(off_done)
            pool.load(spans[j], stream=sl)
            ld = torch.cuda.Event()
            ld.record(sl)
            loaded[j % 2] = ld
        e1 = torch.cuda.Event(enable_timing=True)
        e1.record(sl)
        return e0, e1

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    marks = [step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    pool.check()
    t_step = statistics.mean(a.elapsed_time(b) for a, b in marks)
    value = 2 * total / (t_step * 1e-3) / GB
    log(f"swap step {t_step:.1f} ms: {value:.2f} GB/s both directions")
    res = base_result(args, value, t_step, "batched partial hits (workload 4) swapped in both directions at "
                      "once: each wave's offload beside the previous wave's load, through two host buffers",
                      {"kv_shape": shp.name, "layers": L, "page_size": P, "pool_slots": S, "requests": len(hit),
                       "tokens": sum(hit), "payload_bytes_per_direction": total, "waves": len(waves),
                       "wave_payload_bytes": wave_bytes,
                       "offload_launch": {"workgroups": bg[0], "threads": bg[1], "tile_kib": bg[2]}})
    res.update({
        "tokens_per_s": round(2 * sum(hit) / (t_step * 1e-3), 1),
        "frac_of_bidir_peak": round(value / peak["bidir"], 4) if peak and peak["bidir"] else None,
        "host_link_peak": peak_report(peak),
    })
    pool.close()
    pool_off.close()
    del pool_t
    for b in bufs:
        b.free()
    torch.cuda.empty_cache()
    return res


def run_bidirectional(args, torch, kv, W):
    """Qwen2.5-7B-1M KV at page size 1: a 1M-token load on one stream while a
    second stream offloads 16K other resident slots back to back into a
    separate host chunk; reports load, offload and combined GB/s over the load
    window against the measured bidirectional memcpy peak."""
    k = 5
    wl = W.WORKLOADS[k]
    shp = wl.shape
    L, H, D, P, S, T = shp.num_layers, shp.num_kv_heads, shp.head_dim, wl.page_size, wl.num_slots, wl.tokens
    R = shp.row_bytes
    TO = 16384
    both = W.random_slots(np.random.default_rng(W.placement_seed(k)), S, T + TO)
    pl = torch.from_numpy(both[:T].copy()).cuda()
    po = torch.from_numpy(both[T:].copy()).cuda()
    nb, nbo = L * 2 * T * R, L * 2 * TO * R
    pool_t = torch.empty((2, L, S, H, D), dtype=torch.bfloat16, device="cuda")
    lc = launch_from(args, kv)
    pool = kv.KVPool(pool_t, P, load_launch=lc, offload_launch=lc, staging_bytes=args.staging_mib << 20)
    bg = [int(x) for x in args.bg_offload.split(",")]
    # a second handle on the same pool whose offloads run with the background quota
    pool_bg = kv.KVPool(pool_t, P, offload_launch=kv.launch(bg[0], bg[1], bg[2], 0))
    hflags = kv.KVIO_HOST_NONCOHERENT if args.noncoherent_host else kv.KVIO_HOST_COHERENT
    host = kv.HostBuffer(nb, hflags)
    src_o, dst_o = kv.HostBuffer(nbo, hflags), kv.HostBuffer(nbo, hflags)
    peak = None if args.no_peak else h2d_d2h_peak(torch, kv)
    W.fill_cuda(host.ptr, nb, W.data_seed(k), shp)
    W.fill_cuda(src_o.ptr, nbo, W.data_seed(k) * 1000 + 1, shp)
    pool.load([(src_o.ptr, TO, TO, po.data_ptr())])
    sa, sb = io_stream(torch, kv), torch.cuda.Stream()
    span_l = [(host.ptr, T, T, pl.data_ptr())]
    span_o = [(dst_o.ptr, TO, TO, po.data_ptr())]
    # each direction alone
    tla, toa = Timer(torch, sa), Timer(torch, sb)
    pool.load(span_l, stream=sa)
    pool_bg.offload(span_o, stream=sb)
    torch.cuda.synchronize()
    e = tla.start()
    pool.load(span_l, stream=sa)
    tla.stop(e)
    torch.cuda.synchronize()
    for _ in range(5):
        e = toa.start()
        pool_bg.offload(span_o, stream=sb)
        toa.stop(e)
    torch.cuda.synchronize()
    t_load_alone = tla.ms()[0]
    t_off_alone = statistics.median(toa.ms())
    n_off = int(t_load_alone / t_off_alone * 1.5) + 4
    # concurrent
    reps = max(1, args.steps)
    rows = []
    for _ in range(reps):
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        start.record(sa)
        sb.wait_event(start)
        pool.load(span_l, stream=sa)
        lend = torch.cuda.Event(enable_timing=True)
        lend.record(sa)
        ends = []
        for _ in range(n_off):
            pool_bg.offload(span_o, stream=sb)
            ev = torch.cuda.Event(enable_timing=True)
            ev.record(sb)
            ends.append(ev)
        torch.cuda.synchronize()
        t_load = start.elapsed_time(lend)
        done = [start.elapsed_time(ev) for ev in ends]
        inside = [t for t in done if t <= t_load]
        rows.append((t_load, len(inside), inside[-1] if inside else None))
    pool.check()
    t_load = statistics.median(r[0] for r in rows)
    n_in = min(r[1] for r in rows)
    off_bytes = n_in * nbo
    t_off_window = statistics.median(r[2] for r in rows if r[2] is not None) if n_in else None
    load_gbps = nb / (t_load * 1e-3) / GB
    off_gbps = off_bytes / (t_off_window * 1e-3) / GB if n_in else 0.0
    bidir = (nb + off_bytes) / (t_load * 1e-3) / GB
    log(f"load alone {nb / (t_load_alone * 1e-3) / GB:.2f} GB/s, offload alone {nbo / (t_off_alone * 1e-3) / GB:.2f} "
        f"GB/s; concurrent: load {load_gbps:.2f} GB/s, offload {off_gbps:.2f} GB/s ({n_in} runs), "
        f"combined {bidir:.2f} GB/s")
    res = base_result(args, bidir, t_load, wl.description,
                      {"kv_shape": shp.name, "layers": L, "page_size": P, "pool_slots": S, "tokens": T,
                       "offload_tokens_per_run": TO, "payload_bytes_load": nb, "payload_bytes_per_offload": nbo,
                       "background_offload_launch": {"workgroups": bg[0], "threads": bg[1], "tile_kib": bg[2]},
                       "step": "kvio_load of 1M tokens on stream A || back-to-back 16K-token kvio_offload "
                               "runs on stream B"})
    res.update({
        "tokens_per_s": round((T + n_in * TO) / (t_load * 1e-3), 1),
        "load": {"gbps_concurrent": round(load_gbps, 3), "gbps_alone": round(nb / (t_load_alone * 1e-3) / GB, 3),
                 "frac_of_h2d_peak_concurrent": round(load_gbps / peak["h2d"], 4) if peak else None,
                 "frac_of_h2d_peak_alone": round(nb / (t_load_alone * 1e-3) / GB / peak["h2d"], 4) if peak else None},
        "offload": {"gbps_concurrent": round(off_gbps, 3), "runs_in_window": n_in,
                    "frac_of_d2h_peak_concurrent": round(off_gbps / peak["d2h"], 4) if peak else None,
                    "gbps_alone": round(nbo / (t_off_alone * 1e-3) / GB, 3),
                    "frac_of_d2h_peak_alone": round(nbo / (t_off_alone * 1e-3) / GB / peak["d2h"], 4) if peak else None},
        "bidirectional_gbps": round(bidir, 3),
        "frac_of_bidir_peak": round(bidir / peak["bidir"], 4) if peak and peak["bidir"] else None,
        "host_link_peak": peak_report(peak),
        "roofline": roofline("kvio_copy_kernel<load> || <offload>", bidir, peak["bidir"] if peak else None,
                             directions=2, algorithmic_bytes_per_launch=nb),
    })
    res["reps"] = reps
    pool.close()
    pool_bg.close()
    del pool_t
    host.free()
    src_o.free()
    dst_o.free()
    torch.cuda.empty_cache()
    return res


class Fig5Corunners:
    """The co-runners of the paper's interference experiment (Fig. 5), on the
    Llama-3.1-8B shape (32 layers, hidden 4096, 32 query / 8 KV heads of 128,
    MLP 14336), bf16, random weights, one set per layer:

      prefill: one forward pass over 2 requests x 4K tokens (8192 rows): per
               layer the QKV projection (8192 x 4096 x 6144), the output
               projection (8192 x 4096 x 4096), gate and up together
               (8192 x 4096 x 28672) and down (8192 x 14336 x 4096), in order;
      decode:  one decoding step of 16 requests with 4K-token contexts: per
               layer the same four projections at 16 rows, and attention
               reading the layer's K and V of the 16 x 4096 tokens (128 MiB
               each) as two batched products.

    Attention inside the prefill pass (about 8% of its FLOPs at 4K) is left
    out; every product has contiguous operands."""

    def __init__(self, torch):
        self.torch = torch
        L, Hd, I, KVd = 32, 4096, 14336, 1024
        g = torch.Generator(device="cuda").manual_seed(55)
        bf = torch.bfloat16

        def r(*shape):
            return torch.randn(*shape, device="cuda", dtype=bf, generator=g).mul_(0.02)

        self.layers = [(r(Hd, Hd + 2 * KVd), r(Hd, Hd), r(Hd, 2 * I), r(I, Hd)) for _ in range(L)]
        self.x = r(8192, Hd)
        self.qkv = torch.empty(8192, Hd + 2 * KVd, device="cuda", dtype=bf)
        self.o = r(8192, Hd)
        self.gu = torch.empty(8192, 2 * I, device="cuda", dtype=bf)
        self.h = r(8192, I)
        self.y = torch.empty(8192, Hd, device="cuda", dtype=bf)
        self.xd = r(16, Hd)
        self.dq = torch.empty(16, Hd + 2 * KVd, device="cuda", dtype=bf)
        self.do = r(16, Hd)
        self.dgu = torch.empty(16, 2 * I, device="cuda", dtype=bf)
        self.dh = r(16, I)
        self.dy = torch.empty(16, Hd, device="cuda", dtype=bf)
        self.kcache = [r(16, 4096, KVd) for _ in range(L)]
        self.vcache = [r(16, 4096, KVd) for _ in range(L)]
        self.q = r(16, KVd, 4)
        self.p = r(16, 4, 4096)
        self.s = torch.empty(16, 4096, 4, device="cuda", dtype=bf)
        self.a = torch.empty(16, 4, KVd, device="cuda", dtype=bf)
        self.flop = {"prefill": 2.0 * 8192 * L * (Hd * (Hd + 2 * KVd) + Hd * Hd + Hd * 2 * I + I * Hd)}

    def prefill(self):
        mm = self.torch.matmul
        for wqkv, wo, wgu, wd in self.layers:
            mm(self.x, wqkv, out=self.qkv)
            mm(self.o, wo, out=self.y)
            mm(self.x, wgu, out=self.gu)
            mm(self.h, wd, out=self.y)

    def decode(self):
        mm, bmm = self.torch.matmul, self.torch.bmm
        for (wqkv, wo, wgu, wd), kc, vc in zip(self.layers, self.kcache, self.vcache):
            mm(self.xd, wqkv, out=self.dq)
            bmm(kc, self.q, out=self.s)
            bmm(self.p, vc, out=self.a)
            mm(self.do, wo, out=self.dy)
            mm(self.xd, wgu, out=self.dgu)
            mm(self.dh, wd, out=self.dy)


def run_interference(args, torch, kv, W):
    """Load bandwidth and co-runner slowdown against the load's quota and
    placement (the paper's Fig. 5 on the kernel path).  The co-runners are a
    prefill pass and a decoding step of the Llama-3.1-8B shape
    (Fig5Corunners).  A co-runner repeats its pass on its own stream while
    4 GiB loads of the Llama-3.1-8B KV (page size 1, 32K tokens into random
    slots) run back to back on the transfer stream; the passes that lie wholly
    inside the loads' window give the co-run time per pass, against the
    faster of its median alone before and after the sweep.

    Placements: every quota runs unmasked (the dispatcher places the load's
    workgroups); the masked rows put the load on a stream limited to the
    first n CUs and the co-runner on a stream limited to the others.

    Residency rows: one idle wave (torch's one-thread spin kernel, no memory
    traffic) in place of the load, and the load with one one-wave workgroup
    per CU (256 x 64), which leaves no CU without a resident wave.

    --quotas and --masked replace the default unmasked quotas and CU
    partitions with the ones listed."""
    k = 2
    wl = W.WORKLOADS[k]
    shp = wl.shape
    L, H, D, P, S, T = shp.num_layers, shp.num_kv_heads, shp.head_dim, wl.page_size, wl.num_slots, wl.tokens
    R = shp.row_bytes
    pool_t = torch.empty((2, L, S, H, D), dtype=torch.bfloat16, device="cuda")
    pages = W.random_slots(np.random.default_rng(W.placement_seed(k)), S, T)
    pidx = torch.from_numpy(pages).cuda()
    nb = L * 2 * T * R
    host = kv.HostBuffer(nb)
    W.fill_cuda(host.ptr, nb, W.data_seed(k), shp)
    io, comp = io_stream(torch, kv), torch.cuda.Stream()
    span = [(host.ptr, T, T, pidx.data_ptr())]
    co = Fig5Corunners(torch)
    corunners = {"prefill": co.prefill, "decode": co.decode}
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count

    def alone(fn, n, stream):
        ts = []
        for _ in range(n):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            with torch.cuda.stream(stream):
                fn()
            b.record(stream)
            ts.append((a, b))
        torch.cuda.synchronize()
        return statistics.median(x.elapsed_time(y) for x, y in ts)

    def load_alone(pool, stream):
        pool.load(span, stream=stream)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        pool.load(span, stream=stream)
        b.record(stream)
        torch.cuda.synchronize()
        return nb / (a.elapsed_time(b) * 1e-3) / GB

    def corun(pool, fn, t_alone, io_s, comp_s):
        """Passes of fn on comp_s beside back-to-back loads on io_s covering
        at least 3 passes (and 150 ms): load GB/s over the loads' window and
        the median pass inside it (None if no pass lies inside)."""
        n_loads = max(2, int(max(3 * t_alone, 150.0) / 75.0) + 1)

        def issue():
            for _ in range(n_loads):
                pool.load(span, stream=io_s)
            return n_loads * nb

        return corun_with(issue, n_loads * 75.0, fn, t_alone, io_s, comp_s)

    def corun_with(issue, window_ms, fn, t_alone, io_s, comp_s):
        """Passes of fn on comp_s while issue() runs on io_s (about window_ms
        long): GB/s of the bytes issue() moved over its window, the median
        pass inside the window, the number of such passes and the number of
        passes that ended inside it (0 when the co-runner made no progress)."""
        n_pass = int(window_ms / t_alone) + 4
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        start.record(comp_s)
        marks = []
        with torch.cuda.stream(comp_s):
            for _ in range(n_pass):
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(comp_s)
                fn()
                b.record(comp_s)
                marks.append((a, b))
        io_s.wait_event(marks[1][0])                        # the co-runner is already running
        l0, l1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        l0.record(io_s)
        moved = issue()
        l1.record(io_s)
        torch.cuda.synchronize()
        t0, t1 = start.elapsed_time(l0), start.elapsed_time(l1)
        inside = [x.elapsed_time(y) for x, y in marks
                  if start.elapsed_time(x) >= t0 and start.elapsed_time(y) <= t1]
        ended = sum(1 for _, y in marks if t0 < start.elapsed_time(y) <= t1)
        return (round(moved / ((t1 - t0) * 1e-3) / GB, 3),
                round(statistics.median(inside), 4) if inside else None, len(inside), ended)

    for fn in corunners.values():                       # warm the clocks and the GEMM heuristics
        alone(fn, 5, comp)
    base = {name: alone(fn, 10, comp) for name, fn in corunners.items()}
    log("co-runners alone: " + ", ".join(f"{n} {t:.3f} ms" for n, t in base.items()) +
        f" (prefill {co.flop['prefill'] / (base['prefill'] * 1e-3) / 1e12:.0f} TFLOP/s)")
    rows = []
    quotas = [(1, 1024), (2, 1024), (4, 1024), (8, 256), (8, 512), (8, 1024), (16, 192), (16, 256), (32, 64),
              (64, 64), (256, 64)]
    if args.quotas:
        quotas = [tuple(int(x) for x in q.split("x")) for q in args.quotas.split(",")]
    partitions = [(16, (16, 192)), (12, (12, 256)), (8, (8, 384)), (8, (8, 256)), (8, (8, 192)), (32, (32, 128))]
    if args.masked == "none":
        partitions = []
    elif args.masked:
        partitions = [(int(n), tuple(int(x) for x in q.split("x")))
                      for n, q in (m.split(":") for m in args.masked.split(","))]
    for wg, th in quotas:
        pool = kv.KVPool(pool_t, P, load_launch=kv.launch(wg, th, 4, 0))
        row = {"placement": "unmasked", "workgroups": wg, "threads": th, "waves": wg * th // 64,
               "load_gbps_alone": round(load_alone(pool, io), 3)}
        for name, fn in corunners.items():
            (row[f"load_gbps_with_{name}"], row[f"{name}_ms_corun"], row[f"{name}_passes"],
             row[f"{name}_passes_ended_in_window"]) = corun(pool, fn, base[name], io, comp)
        pool.close()
        rows.append(row)
        log(f"quota {wg} x {th}: " + ", ".join(f"{k2} {v}" for k2, v in row.items() if k2 not in ("workgroups",
                                                                                                   "threads")))
    # One idle wave in place of the load: torch's spin kernel (one thread, no
    # memory traffic) on the transfer stream, long enough for 5 passes alone
    # (2 or more at the slowdown a resident load causes).
    spin = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    spin[0].record(io)
    with torch.cuda.stream(io):
        torch.cuda._sleep(10_000_000)
    spin[1].record(io)
    torch.cuda.synchronize()
    cycles_per_ms = 10_000_000 / spin[0].elapsed_time(spin[1])
    row = {"placement": "one idle wave (spin kernel, no memory traffic) instead of the load", "workgroups": 1,
           "threads": 1, "waves": 1, "load_gbps_alone": 0.0}
    for name, fn in corunners.items():
        window = max(5 * base[name], 150.0)

        def idle(ms=window):
            with torch.cuda.stream(io):
                torch.cuda._sleep(int(ms * cycles_per_ms))
            return 0

        _, row[f"{name}_ms_corun"], row[f"{name}_passes"], row[f"{name}_passes_ended_in_window"] = corun_with(
            idle, window, fn, base[name], io, comp)
    rows.append(row)
    log("idle wave: " + ", ".join(f"{k2} {v}" for k2, v in row.items() if k2 != "placement"))
    # CU partitions: the load on a stream masked to the first n CUs (one workgroup
    # per CU; 24 to 64 waves), the co-runner on a stream masked to the rest.
    for n_io, (wg, th) in partitions:
        try:
            io_m = kv.Stream(list(range(n_io)))
        except kv.KvioError as e:
            log(f"{n_io} CUs: masked stream refused ({e.detail})")
            continue
        try:
            comp_m = kv.Stream(list(range(n_io, n_cu)))
        except kv.KvioError as e:
            log(f"{n_io} CUs: masked stream refused ({e.detail})")
            io_m.close()
            continue
        pool = kv.KVPool(pool_t, P, load_launch=kv.launch(wg, th, 4, 0))
        row = {"placement": f"load on CUs 0-{n_io - 1}, co-runner on the other {n_cu - n_io}", "workgroups": wg,
               "threads": th, "waves": wg * th // 64, "load_gbps_alone": round(load_alone(pool, io_m.torch), 3)}
        for name, fn in corunners.items():
            row[f"{name}_ms_alone_on_{n_cu - n_io}_cus"] = round(alone(fn, 10, comp_m.torch), 4)
            (row[f"load_gbps_with_{name}"], row[f"{name}_ms_corun"], row[f"{name}_passes"],
             row[f"{name}_passes_ended_in_window"]) = corun(pool, fn, base[name], io_m.torch, comp_m.torch)
        pool.close()
        comp_m.close()
        io_m.close()
        rows.append(row)
        log(f"masked {n_io}: " + ", ".join(f"{k2} {v}" for k2, v in row.items() if k2 != "placement"))
    after = {name: alone(fn, 10, comp) for name, fn in corunners.items()}
    base = {n: min(base[n], after[n]) for n in base}
    log("co-runners alone (best of before / after the sweep): " +
        ", ".join(f"{n} {t:.3f} ms" for n, t in base.items()))
    for row in rows:
        for name in corunners:
            t = row[f"{name}_ms_corun"]
            row[f"{name}_slowdown"] = round(t / base[name], 4) if t else None
    res = base_result(args, max(r["load_gbps_alone"] for r in rows), 0.0,
                      "interference sweep (the paper's Fig. 5): 4 GiB Llama-3.1-8B KV loads beside a prefill "
                      "pass (2 x 4K tokens) or a decoding step (16 x 4K) of the Llama-3.1-8B shape",
                      {"corunners": {"prefill": "32 x [8192x4096x6144, 8192x4096x4096, 8192x4096x28672, "
                                                "8192x14336x4096] bf16 GEMMs",
                                     "decode": "32 x [16-row projections + K, V reads of 16 x 4096 tokens]"},
                       "corunner_ms_alone": {n: round(t, 4) for n, t in base.items()}})
    res["sweep"] = rows
    host.free()
    return res


def run_row_sweep(args, torch, kv, W):
    """GB/s against the token row size R = H x 128 x 2 bytes for H = 1 .. 32 KV
    heads (256 B .. 8 KiB; a 70B model's 8 KV heads split over 4 or 8
    tensor-parallel ranks gives R = 512 B or 256 B per rank), 80 layers, 2 GiB
    per direction per case, at page size 1 (random slots) and 16 (random
    pages); default launch shapes, HIP events on the transfer stream, median
    of 5 after a warm-up, round trip checked."""
    L, D = 80, 128
    nb = 2 << 30
    stream = io_stream(torch, kv)
    peak = None if args.no_peak else h2d_d2h_peak(torch, kv)
    host, out = kv.HostBuffer(nb), kv.HostBuffer(nb)
    W.fill_cuda(host.ptr, nb, W.data_seed(3), W.GQA70B)
    rows = []
    try:
        for H in (1, 2, 4, 8, 16, 32):
            R = H * D * 2
            T = nb // (L * 2 * R)
            for P in (1, 16):
                S = -(-2 * T // P) * P
                pool_t = torch.empty((2, L, S, H, D), dtype=torch.bfloat16, device="cuda")
                rng = np.random.default_rng(600 + H * 7 + P)
                pages = W.random_slots(rng, S, T) if P == 1 else W.random_pages(rng, S // P, -(-T // P))
                pidx = torch.from_numpy(pages).cuda()
                pool = kv.KVPool(pool_t, P)
                span_in, span_out = [(host.ptr, T, T, pidx.data_ptr())], [(out.ptr, T, T, pidx.data_ptr())]
                row = {"kv_heads": H, "row_bytes": R, "page_size": P, "tokens": T, "bytes": L * 2 * T * R}
                for name, fn in (("load", lambda: pool.load(span_in, stream=stream)),
                                 ("offload", lambda: pool.offload(span_out, stream=stream))):
                    fn()
                    torch.cuda.synchronize()
                    t = Timer(torch, stream)
                    for _ in range(5):
                        e = t.start()
                        fn()
                        t.stop(e)
                    torch.cuda.synchronize()
                    row[f"{name}_gbps"] = round(row["bytes"] / (statistics.median(t.ms()) * 1e-3) / GB, 3)
                pool.check()
                if not memequal_np(out.array, host.array, row["bytes"]):
                    raise SystemExit(f"round trip differs at H={H}, P={P}")
                if peak:
                    row["load_frac_of_h2d_peak"] = round(row["load_gbps"] / peak["h2d"], 4)
                    row["offload_frac_of_d2h_peak"] = round(row["offload_gbps"] / peak["d2h"], 4)
                log(", ".join(f"{k2} {v}" for k2, v in row.items()))
                rows.append(row)
                pool.close()
                del pool_t
    finally:
        host.free()
        out.free()
    res = base_result(args, min(r["load_gbps"] for r in rows), 0.0,
                      "row-size sweep: 80 layers, 1..32 KV heads x 128 dims bf16, 2 GiB per direction, "
                      "page sizes 1 and 16", {})
    res["metric"] = "kvio load / offload GB/s against the token row size"
    res["host_link_peak"] = peak_report(peak)
    res["sweep"] = rows
    print(json.dumps(res), flush=True)


def memequal_ptr(a_ptr, b_ptr, n):
    """Bytes [a_ptr, a_ptr + n) == [b_ptr, b_ptr + n) of host memory (libc memcmp)."""
    import ctypes
    libc = ctypes.CDLL("libc.so.6")
    libc.memcmp.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t]
    libc.memcmp.restype = ctypes.c_int
    return libc.memcmp(a_ptr, b_ptr, n) == 0


def memequal_np(a, b, n):
    """a[:n] == b[:n] for two large uint8 arrays, compared in 256 MiB pieces."""
    step = 256 << 20
    return all(np.array_equal(a[i:min(i + step, n)], b[i:min(i + step, n)]) for i in range(0, n, step))


def run_page_sweep(args, torch, kv, W):
    """GB/s against page size (the synthetic analogue of Fig. 10's page-size
    axis) and the paper's own microbenchmark of Fig. 3 (8192 tokens at page
    size 32), Llama-3.1-8B KV.  For every page size: kvio_load and
    kvio_offload of the context (median of 5 after a warm-up, HIP events on
    the transfer stream) and the naive path -- one hipMemcpyAsync per
    (page, layer, K|V) segment of P*R bytes -- timed over at most 2^17 calls
    (a prefix of the context's pages when there are more).  The pool holds
    2^19 slots, so every page size divides it; pages are a random sample of
    the pool's pages in random order."""
    shp = W.LLAMA8B
    L, H, D, R = shp.num_layers, shp.num_kv_heads, shp.head_dim, shp.row_bytes
    S = 1 << 19
    cases = [(32768, P) for P in (1, 2, 4, 16, 32, 64, 256)] + [(8192, 32)]
    pool_t = torch.empty((2, L, S, H, D), dtype=torch.bfloat16, device="cuda")
    pool_t.view(torch.int16).fill_(0x5A5A)
    Tmax = max(T for T, _ in cases)
    nb_max = L * 2 * Tmax * R
    host, out = kv.HostBuffer(nb_max), kv.HostBuffer(nb_max)
    W.fill_cuda(host.ptr, nb_max, W.data_seed(2), shp)
    stream = io_stream(torch, kv)
    peak = None if args.no_peak else h2d_d2h_peak(torch, kv)
    rows = []
    try:
        for T, P in cases:
            rng = np.random.default_rng(500 + P + T)
            pages = W.random_pages(rng, S // P, -(-T // P)) if P > 1 else W.random_slots(rng, S, T)
            pidx = torch.from_numpy(pages).cuda()
            nb = L * 2 * T * R
            pool = kv.KVPool(pool_t, P)
            span_in, span_out = [(host.ptr, T, T, pidx.data_ptr())], [(out.ptr, T, T, pidx.data_ptr())]
            row = {"tokens": T, "page_size": P, "bytes": nb, "segment_bytes": P * R}
            for name, fn in (("load", lambda: pool.load(span_in, stream=stream)),
                             ("offload", lambda: pool.offload(span_out, stream=stream))):
                fn()
                torch.cuda.synchronize()
                t = Timer(torch, stream)
                for _ in range(5):
                    e = t.start()
                    fn()
                    t.stop(e)
                torch.cuda.synchronize()
                ms = statistics.median(t.ms())
                row[f"kvio_{name}_gbps"] = round(nb / (ms * 1e-3) / GB, 3)
            pool.check()
            if not np.array_equal(out.array[:nb], host.array[:nb]):
                raise SystemExit(f"round trip differs at page size {P}")
            max_calls = 1 << 17
            n_pages = min(len(pages), max(1, max_calls // (L * 2)))
            nt = min(T, n_pages * P)
            kv.kvio_naive_load(pool.handle, [(host.ptr, T, min(nt, P * 4), pidx.data_ptr())], 0, 1, stream)
            torch.cuda.synchronize()
            t = Timer(torch, stream)
            c0 = time.perf_counter()
            e = t.start()
            kv.kvio_naive_load(pool.handle, [(host.ptr, T, nt, pidx.data_ptr())], 0, L, stream)
            t.stop(e)
            torch.cuda.synchronize()
            wall = time.perf_counter() - c0
            nbn = L * 2 * nt * R
            row["naive_calls"] = L * 2 * (-(-nt // P))
            row["naive_prefix_of_calls"] = round(row["naive_calls"] / (L * 2 * (-(-T // P))), 4)
            row["naive_load_gbps"] = round(nbn / max(wall, t.ms()[0] * 1e-3) / GB, 3)
            row["speedup_vs_naive"] = round(row["kvio_load_gbps"] / row["naive_load_gbps"], 1)
            if peak:
                row["load_frac_of_h2d_peak"] = round(row["kvio_load_gbps"] / peak["h2d"], 4)
            pool.close()
            log(", ".join(f"{k2} {v}" for k2, v in row.items()))
            rows.append(row)
    finally:
        host.free()
        out.free()
    res = base_result(args, min(r["kvio_load_gbps"] for r in rows), 0.0,
                      "page-size sweep: Llama-3.1-8B KV, 32K tokens at page sizes 1..256 and 8192 tokens at "
                      "page size 32, pool of 2^19 slots", {"pool_slots": S})
    res["metric"] = "kvio vs per-page hipMemcpyAsync load GB/s against page size"
    res["host_link_peak"] = peak_report(peak)
    res["sweep"] = rows
    print(json.dumps(res), flush=True)


def synthetic_queue(n, seed, bursty=False):
    """n requests (load_tokens, compute_tokens, context or None, 0): half reuse
    a cached 8K-128K-token context (log-uniform) with 64-512 new tokens, a
    third of those sharing the previous request's context (a bundle hit);
    half are fresh 1K-8K-token prompts.  Shuffled: kinds drawn independently;
    bursty: runs of 1-8 requests of one kind (sessions arriving together)."""
    rng = np.random.default_rng(seed)
    if bursty:
        kinds = []
        while len(kinds) < n:
            kinds += [bool(rng.random() < 0.5)] * int(rng.integers(1, 9))
        kinds = kinds[:n]
    else:
        kinds = [bool(x) for x in rng.random(n) < 0.5]
    q, ctx = [], 0
    for cached in kinds:
        if cached:
            if q and q[-1][2] is not None and rng.random() < 1 / 3:
                q.append((q[-1][0], int(rng.integers(64, 512)), q[-1][2], 0))
            else:
                ctx += 1
                q.append((int(np.exp(rng.uniform(np.log(8192), np.log(131072)))), int(rng.integers(64, 512)),
                          ctx, 0))
        else:
            q.append((0, int(rng.integers(1024, 8192)), None, 0))
    return q


def drain_queue(kv, q, ratio, load_tok_s, prefill_tok_s, max_tokens=8192, max_requests=16):
    """Schedule rounds until the queue is empty (every request present at
    time 0); each batch costs max(load time, compute time) (layer-wise
    overlap), a shared context loading once per batch.  Returns the drain
    time, the mean completion time of a request, and batch counts."""
    cur = list(range(len(q)))
    total, batches, loading_bound = 0.0, 0, 0
    done = []
    while cur:
        batch, rest = kv.kvio_schedule_round([q[i] for i in cur], max_tokens, max_requests, ratio)
        loaded, load_tok, comp_tok = set(), 0, 0
        for j in batch:
            ld, cp, cx, _ = q[cur[j]]
            if cx is None or cx not in loaded:
                load_tok += ld
            if cx is not None:
                loaded.add(cx)
            comp_tok += cp
        t_load, t_comp = load_tok / load_tok_s, comp_tok / prefill_tok_s
        total += max(t_load, t_comp)
        done += [total] * len(batch)
        loading_bound += t_load > t_comp
        batches += 1
        cur = [cur[j] for j in rest]
    return {"drain_s": round(total, 4), "mean_completion_s": round(float(np.mean(done)), 4), "batches": batches,
            "loading_bound_batches": loading_bound}


def run_schedule(args, torch, kv, W):
    """Cache-aware batch formation measured two ways.

    (1) Host cost of kvio_schedule_round on queues of 64 .. 16,384 requests.
    (2) FIFO (no loading-bound test) against Algorithm 1 draining the same
    synthetic queue, with every batch timed by a cost model whose rates are
    measured in this run: load time = cached tokens x 128 KiB / kvio_load GB/s
    (Llama-3.1-8B KV, page size 16), compute time = new tokens / prefill
    tokens/s, where prefill tokens/s = the measured bf16 GEMM rate / (2 x 8.03e9
    FLOP per token, the 8B model's dense work).  Loads overlap compute layer
    by layer, so a batch takes max(load, compute).  The queue mixes the
    paper's two request kinds (see synthetic_queue), all present at time 0."""
    shp = W.LLAMA8B
    L, H, D, R = shp.num_layers, shp.num_kv_heads, shp.head_dim, shp.row_bytes
    tok_bytes = L * 2 * R
    # ---- measured rates ------------------------------------------------------------------
    P, T, S = 16, 16384, 1 << 17
    pool_t = torch.empty((2, L, S, H, D), dtype=torch.bfloat16, device="cuda")
    pidx = torch.from_numpy(W.random_pages(np.random.default_rng(600), S // P, T // P)).cuda()
    stream = io_stream(torch, kv)
    with kv.HostBuffer(T * tok_bytes) as hb:
        hb.array[::4096] = 1
        pool = kv.KVPool(pool_t, P)
        span = [(hb.ptr, T, T, pidx.data_ptr())]
        pool.load(span, stream=stream)
        torch.cuda.synchronize()
        t = Timer(torch, stream)
        for _ in range(5):
            e = t.start()
            pool.load(span, stream=stream)
            t.stop(e)
        torch.cuda.synchronize()
        pool.check()
        pool.close()
    load_gbps = T * tok_bytes / (statistics.median(t.ms()) * 1e-3) / GB
    del pool_t
    g = torch.Generator(device="cuda").manual_seed(8)
    A = torch.randn(8192, 4096, device="cuda", dtype=torch.bfloat16, generator=g)
    B = torch.randn(4096, 14336, device="cuda", dtype=torch.bfloat16, generator=g)
    C = torch.empty(8192, 14336, device="cuda", dtype=torch.bfloat16)
    for _ in range(3):
        torch.matmul(A, B, out=C)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(20):
        torch.matmul(A, B, out=C)
    b.record()
    torch.cuda.synchronize()
    gemm_tflops = 20 * 2 * 8192 * 4096 * 14336 / (a.elapsed_time(b) * 1e-3) / 1e12
    del A, B, C
    load_tok_s = load_gbps * GB / tok_bytes
    prefill_tok_s = gemm_tflops * 1e12 / (2 * 8.03e9)
    cost_ratio = load_tok_s / prefill_tok_s
    log(f"kvio load {load_gbps:.2f} GB/s = {load_tok_s:.0f} tokens/s; bf16 GEMM {gemm_tflops:.0f} TFLOP/s = "
        f"{prefill_tok_s:.0f} prefill tokens/s; loading-bound when load tokens > {cost_ratio:.2f} x compute tokens")

    # ---- (1) host cost of one scheduling round ---------------------------------------------
    import ctypes
    from paper_2508_18572_amd import kvio as kvmod
    cost = {}
    for n in (64, 1024, 16384):
        q = synthetic_queue(n, 700 + n)
        arr = (kvmod.kvio_request * n)()
        for i, (ld, cp, cx, m) in enumerate(q):
            arr[i] = kvmod.kvio_request(ld, cp, -1 if cx is None else cx, m)
        pol = kvmod.kvio_batch_policy(8192, 16, 0, 0.0, -1)
        bout, qout = (ctypes.c_int32 * n)(), (ctypes.c_int32 * n)()
        nb_, nq_ = ctypes.c_int32(), ctypes.c_int32()
        reps = max(5, 20000 // n)
        c0 = time.perf_counter()
        for _ in range(reps):                    # the C call alone, arrays already built
            kvmod._lib.kvio_schedule_round(arr, n, ctypes.byref(pol), bout, ctypes.byref(nb_), qout,
                                           ctypes.byref(nq_))
        raw = (time.perf_counter() - c0) / reps * 1e6
        c0 = time.perf_counter()
        for _ in range(reps):                    # through the Python binding (marshalling included)
            kv.kvio_schedule_round(q, 8192, 16)
        cost[n] = {"c_call_us": round(raw, 2), "with_python_marshalling_us": round((time.perf_counter() - c0) / reps * 1e6, 2)}
    log("scheduling round: " + ", ".join(f"{n} requests {c['c_call_us']:.1f} us in C "
                                         f"({c['with_python_marshalling_us']:.1f} us through Python)"
                                         for n, c in cost.items()))

    # ---- (2) FIFO vs Algorithm 1 under the measured cost model -------------------------------
    sim = {}
    for order in ("shuffled", "bursty"):
        q = synthetic_queue(512, 800, bursty=order == "bursty")
        r = {"fifo": drain_queue(kv, q, float("inf"), load_tok_s, prefill_tok_s),
             "algorithm1_ratio_100": drain_queue(kv, q, 100.0, load_tok_s, prefill_tok_s),
             "algorithm1_ratio_cost_model": drain_queue(kv, q, cost_ratio, load_tok_s, prefill_tok_s)}
        for k2 in ("algorithm1_ratio_100", "algorithm1_ratio_cost_model"):
            r[k2]["drain_speedup_vs_fifo"] = round(r["fifo"]["drain_s"] / r[k2]["drain_s"], 3)
            r[k2]["completion_speedup_vs_fifo"] = round(r["fifo"]["mean_completion_s"] / r[k2]["mean_completion_s"], 3)
        r["aggregate_load_s"] = round(sum(x[0] for x in q) / load_tok_s, 3)
        r["aggregate_compute_s"] = round(sum(x[1] for x in q) / prefill_tok_s, 3)
        sim[order] = r
        log(f"drain 512 requests ({order}): " + "; ".join(f"{k2} {v}" for k2, v in r.items()))
    res = base_result(args, load_gbps, 0.0,
                      "batch formation: 512 synthetic requests (half cached 8K-128K-token contexts with 64-512 new "
                      "tokens, half fresh 1K-8K-token prompts; shuffled and bursty orders), token budget 8192, "
                      "at most 16 requests per batch",
                      {"kv_shape": shp.name, "page_size": P})
    res["metric"] = "batch formation: queue drain time under measured load/compute rates, FIFO vs Algorithm 1"
    res["rates"] = {"kvio_load_gbps": round(load_gbps, 3), "load_tokens_per_s": round(load_tok_s, 1),
                    "gemm_tflops": round(gemm_tflops, 1), "prefill_tokens_per_s": round(prefill_tok_s, 1),
                    "cost_model_ratio": round(cost_ratio, 3)}
    res["schedule_round"] = {str(n): c for n, c in cost.items()}
    res["simulation"] = sim
    print(json.dumps(res), flush=True)


def _open_store(path, direct):
    """O_DIRECT when the filesystem takes it; otherwise a buffered descriptor
    whose cached pages are dropped before every timed read."""
    if direct:
        try:
            return os.open(path, os.O_RDONLY | os.O_DIRECT), True
        except OSError:
            pass
    return os.open(path, os.O_RDONLY), False


def run_disk(args, torch, kv, W):
    """Fig. 12 analogue: latency of bringing 8192 cached tokens (page size 32)
    of three models' KV from a local disk store into pinned host memory, with
    the store and the host chunk page-first (one read of L*2*P*R bytes per
    page) or layer-first (L*2 reads of P*R bytes per page), through O_DIRECT
    descriptors (pinned chunks are then staged through bounce buffers) and
    through buffered ones with the file's cached pages dropped before every
    read.  The context's 256
    pages sit at random disk pages of a 1024-page store (other contexts fill
    the rest), so reads rarely merge and read-ahead rarely helps by accident.  Both stores hold the same logical KV; after timing, the
    layer-first store is also read into a page-first chunk (pieces of P*R) and
    must equal the page-first result, and the two chunks loaded into the
    layer-first paged pool (kvio_load, host layout to match) must give equal
    pools."""
    P, T = 32, 8192
    n_ctx = T // P
    N = 4 * n_ctx
    threads = [int(x) for x in args.disk_threads.split(",")]
    reps = 3
    rows = []
    os.makedirs(args.disk_dir, exist_ok=True)
    for si, shp in enumerate([W.LLAMA8B, W.GQA70B, W.QWEN7B1M]):
        L, H, D, R = shp.num_layers, shp.num_kv_heads, shp.head_dim, shp.row_bytes
        piece = P * R
        page_bytes = L * 2 * piece
        rng = np.random.default_rng(400 + si)
        t0 = time.perf_counter()
        logical = np.frombuffer(rng.bytes(N * page_bytes), np.uint8).reshape(N, L * 2, piece)
        paths = {0: os.path.join(args.disk_dir, f"kv_store_page_first_{si}.bin"),
                 1: os.path.join(args.disk_dir, f"kv_store_layer_first_{si}.bin")}
        for lay, arr in ((0, logical), (1, np.ascontiguousarray(logical.transpose(1, 0, 2)))):
            with open(paths[lay], "wb") as f:
                arr.tofile(f)
                f.flush()
                os.fsync(f.fileno())
        del logical
        log(f"{shp.name}: two {N * page_bytes / 2**30:.2f} GiB stores written in {time.perf_counter() - t0:.1f}s")
        disk_pages = rng.permutation(N)[:n_ctx]
        nb = L * 2 * T * R
        host_layout = {0: kv.KVIO_HOST_PAGE_FIRST, 1: kv.KVIO_HOST_TOKEN_MAJOR}
        bufs = {0: kv.HostBuffer(nb), 1: kv.HostBuffer(nb)}
        row = {"model": shp.name, "L": L, "R": R, "context_bytes": nb,
               "reads_per_page": {"page_first": 1, "layer_first": L * 2},
               "read_bytes": {"page_first": page_bytes, "layer_first": piece}}
        try:
            for lay, name in ((0, "page_first"), (1, "layer_first")):
                for want_direct in (True, False):
                    fd, direct = _open_store(paths[lay], want_direct)
                    if want_direct and not direct:
                        os.close(fd)
                        continue
                    mode = "direct" if direct else "buffered"
                    try:
                        for th in threads:
                            ts = []
                            for _ in range(reps):
                                if not direct:
                                    os.posix_fadvise(fd, 0, 0, os.POSIX_FADV_DONTNEED)
                                t0 = time.perf_counter()
                                kv.kvio_disk_prefetch(fd, lay, N, L, P, R, disk_pages, bufs[lay].ptr, T,
                                                      host_layout[lay], th)
                                ts.append(time.perf_counter() - t0)
                            ms = statistics.median(ts) * 1e3
                            row[f"{name}_{mode}_ms_t{th}"] = round(ms, 2)
                            row[f"{name}_{mode}_gbps_t{th}"] = round(nb / (ms * 1e-3) / GB, 3)
                    finally:
                        os.close(fd)
            for mode in ("direct", "buffered"):
                for th in threads:
                    if f"page_first_{mode}_ms_t{th}" in row:
                        row[f"speedup_{mode}_t{th}"] = round(row[f"layer_first_{mode}_ms_t{th}"]
                                                             / row[f"page_first_{mode}_ms_t{th}"], 2)
            # same logical KV: the layer-first store read into a page-first chunk equals the page-first read
            with kv.HostBuffer(nb) as chk:
                fd, _ = _open_store(paths[1], True)
                try:
                    kv.kvio_disk_prefetch(fd, 1, N, L, P, R, disk_pages, chk.ptr, T, kv.KVIO_HOST_PAGE_FIRST, 8)
                finally:
                    os.close(fd)
                row["cross_layout_equal"] = bool(np.array_equal(chk.array, bufs[0].array))
            # on to the GPU: both chunks into the same layer-first pool layout
            S = 2 * T
            pidx = torch.from_numpy(W.random_pages(rng, S // P, n_ctx)).cuda()
            pools = []
            for lay in (0, 1):
                pool_t = torch.zeros((2, L, S, H, D), dtype=torch.bfloat16, device="cuda")
                pool = kv.KVPool(pool_t, P, host_layout=host_layout[lay])
                span = [(bufs[lay].ptr, T, T, pidx.data_ptr())]
                pool.load(span)
                torch.cuda.synchronize()
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                pool.load(span)
                b.record()
                torch.cuda.synchronize()
                pool.check()
                row[f"{('page_first', 'layer_first')[lay]}_gpu_load_ms"] = round(a.elapsed_time(b), 3)
                pool.close()
                pools.append(pool_t)
            row["pools_equal"] = bool(torch.equal(pools[0].view(torch.int16), pools[1].view(torch.int16)))
            del pools
        finally:
            for b in bufs.values():
                b.free()
            for pth in paths.values():
                os.remove(pth)
        log(", ".join(f"{k2} {v}" for k2, v in row.items()))
        rows.append(row)
        if not (row["cross_layout_equal"] and row["pools_equal"]):
            raise SystemExit(f"storage tier check failed for {shp.name}")
    best = max(v for r in rows for k2, v in r.items() if k2.startswith("page_first_") and "_gbps_" in k2)
    res = base_result(args, best, 0.0,
                      "storage tier: 8192 tokens, page size 32, disk -> pinned host (page-first vs layer-first) "
                      "-> paged pool", {"disk_threads": threads, "store_pages": N, "context_pages": n_ctx})
    res["metric"] = "disk -> host GB/s of a cached context, page-first vs layer-first store"
    res["sweep"] = rows
    print(json.dumps(res), flush=True)


EXTRA_MODES = {3: run_layerwise, 4: run_batched, 5: run_bidirectional}


def run_other_workloads(args, torch, kv, W):
    """Workloads 1, 2, 3 and 5 after the headline, each with --other-reps
    timed repetitions (2 warm-ups), summarised for the same JSON line."""
    sub = argparse.Namespace(**vars(args))
    sub.steps, sub.warmup, sub.no_cpu_baseline = max(1, args.other_reps), min(args.warmup, 2), True
    out = {}
    r = run_single(sub, torch, kv, W, 1)
    st = r.get("steady_state", {})
    out["workload_1"] = {
        "workload": r["config"]["workload"], "reps": sub.steps,
        "steady_state_load_gbps": st.get("load_gbps"), "frac_of_h2d_peak": st.get("load_frac_of_h2d_peak"),
        "steady_state_loads": st.get("reps"), "single_shot_us": st.get("single_shot_us"),
        "batched4_load_gbps": st.get("batched4_load_gbps"), "two_streams_load_gbps": st.get("two_streams_load_gbps")}
    r = run_single(sub, torch, kv, W, 2)
    out["workload_2"] = {
        "workload": r["config"]["workload"], "reps": sub.steps, "step_gbps": r["value"],
        "ms_per_step": r["ms_per_step"], "load_gbps": r["load"]["gbps"],
        "load_frac_of_h2d_peak": r["load"]["frac_of_h2d_peak"], "offload_gbps": r["offload"]["gbps"],
        "offload_frac_of_d2h_peak": r["offload"]["frac_of_d2h_peak"],
        "offload_frac_of_kernel_d2h_peak": r["offload"]["frac_of_kernel_d2h_peak"], "tokens_per_s": r["tokens_per_s"],
        "naive_per_page_memcpy_gbps": round(r["naive"]["gbps"], 3) if r.get("naive") else None}
    r = run_layerwise(sub, torch, kv, W)
    lw = r["layerwise"]
    out["workload_3"] = {
        "workload": r["config"]["workload"], "reps": r["reps"], "load_gbps_alone": lw["load_gbps_alone"],
        "load_gbps_beside_gemms": lw["load_gbps_corun"], "load_frac_of_h2d_peak": r["load"]["frac_of_h2d_peak"],
        "overlap_efficiency": lw["overlap_efficiency"], "gemm_slowdown": lw["gemm_slowdown"],
        "t_both_ms": lw["t_both_ms"]}
    r = run_bidirectional(sub, torch, kv, W)
    out["workload_5"] = {
        "workload": r["config"]["workload"], "reps": r["reps"], "bidirectional_gbps": r["bidirectional_gbps"],
        "frac_of_bidir_peak": r["frac_of_bidir_peak"], "load_gbps_concurrent": r["load"]["gbps_concurrent"],
        "offload_gbps_concurrent": r["offload"]["gbps_concurrent"],
        "load_frac_of_h2d_peak_concurrent": r["load"]["frac_of_h2d_peak_concurrent"],
        "offload_frac_of_d2h_peak_concurrent": r["offload"]["frac_of_d2h_peak_concurrent"],
        "load_gbps_alone": r["load"]["gbps_alone"],
        "offload_gbps_alone": r["offload"]["gbps_alone"]}
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "kvio moves one GPU's KV over its own host link and has no "
                                   "cross-GPU step; run with --gpus 1"}))
        sys.exit(2)
    import torch
    import paper_2508_18572_amd as kv
    import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.calibrate_copy:
        n = args.calibrate_copy
        src = torch.ones(n // 4, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.bitwise_not(src, out=dst)      # reads n bytes, writes n bytes
        torch.cuda.synchronize()
        print(json.dumps({"calibration_copy_bytes_read": n, "calibration_copy_bytes_written": n,
                          "launches": 3}), flush=True)
        return
    k = args.config
    if args.peak_only:
        _PEAK["child"] = True
        try:
            _PEAK["early_streams"] = [torch.cuda.Stream() for _ in range(3)]
            io_stream(torch, kv)
            print(json.dumps(peak_report(h2d_d2h_peak(torch, kv))), flush=True)
        finally:
            close_io_stream(torch, kv)
        return
    try:
        # a few plain streams for the bidirectional peak, then the transfer stream
        _PEAK["early_streams"] = [torch.cuda.Stream() for _ in range(3)]
        io_stream(torch, kv)
        if not args.no_peak and not args.disk and not args.schedule:
            h2d_d2h_peak(torch, kv)
        if args.interference:
            print(json.dumps(run_interference(args, torch, kv, W)), flush=True)
        elif args.disk:
            run_disk(args, torch, kv, W)
        elif args.swap:
            print(json.dumps(run_swap(args, torch, kv, W)), flush=True)
        elif args.page_sweep:
            run_page_sweep(args, torch, kv, W)
        elif args.row_sweep:
            run_row_sweep(args, torch, kv, W)
        elif args.schedule:
            run_schedule(args, torch, kv, W)
        elif k == 0:
            res = run_batched(args, torch, kv, W)
            if not args.no_other_workloads:
                res["other_workloads"] = run_other_workloads(args, torch, kv, W)
            print(json.dumps(res), flush=True)
        elif k in EXTRA_MODES:
            print(json.dumps(EXTRA_MODES[k](args, torch, kv, W)), flush=True)
        else:
            print(json.dumps(run_single(args, torch, kv, W, k)), flush=True)
    finally:
        close_io_stream(torch, kv)


def run_single(args, torch, kv, W, k):
    """Configs 1 and 2: one cached context, load + offload per step."""
    wl = W.WORKLOADS[k]
    shp = wl.shape
    L, H, D, P, S, T = shp.num_layers, shp.num_kv_heads, shp.head_dim, wl.page_size, wl.num_slots, wl.tokens
    R = shp.row_bytes
    dtype = torch.float16 if shp.dtype == "fp16" else torch.bfloat16
    log(f"{wl.description}; L={L} H={H} D={D} P={P} S={S} T={T} R={R}")

    # ---- inputs, resident before timing -------------------------------------------------
    pool_t = torch.empty((2, L, S, H, D), dtype=dtype, device="cuda")
    pool_t.view(torch.int16).fill_(0x5A5A)
    rng = np.random.default_rng(W.placement_seed(k))
    if P == 1:
        pages = W.random_slots(rng, S, T)
    else:
        pages = W.random_pages(rng, S // P, -(-T // P))
    pidx = torch.from_numpy(pages).cuda()
    host_bytes = L * 2 * T * R
    hflags = kv.KVIO_HOST_NONCOHERENT if args.noncoherent_host else kv.KVIO_HOST_COHERENT
    host = kv.HostBuffer(host_bytes, hflags)
    out = kv.HostBuffer(host_bytes, hflags)
    t0 = time.perf_counter()
    W.fill_cuda(host.ptr, host_bytes, W.data_seed(k), shp)
    log(f"host chunk {host_bytes / 2**30:.2f} GiB filled in {time.perf_counter() - t0:.1f}s")

    launch = launch_from(args, kv)
    pool = kv.KVPool(pool_t, P, load_launch=launch, offload_launch=launch, host_layout=layout_from(args, kv),
                     staging_bytes=args.staging_mib << 20)
    span_in = [(host.ptr, T, T, pidx.data_ptr())]
    span_out = [(out.ptr, T, T, pidx.data_ptr())]
    stream = io_stream(torch, kv)

    # ---- contiguous host-link peak (denominator) ----------------------------------------
    peak = None if args.no_peak else h2d_d2h_peak(torch, kv)

    # ---- timed steps ---------------------------------------------------------------------
    tl, to, tstep = Timer(torch, stream), Timer(torch, stream), Timer(torch, stream)
    for _ in range(args.warmup):
        pool.load(span_in, stream=stream)
        pool.offload(span_out, stream=stream)
    torch.cuda.synchronize()
    pool.check()
    w0 = time.perf_counter()
    for _ in range(args.steps):
        e = tstep.start()
        el = tl.start()
        pool.load(span_in, stream=stream)
        tl.stop(el)
        eo = to.start()
        pool.offload(span_out, stream=stream)
        to.stop(eo)
        tstep.stop(e)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    pool.check()
    load_ms, off_ms, step_ms = statistics.mean(tl.ms()), statistics.mean(to.ms()), statistics.mean(tstep.ms())
    payload = L * 2 * T * R
    load_gbps = payload / (load_ms * 1e-3) / GB
    off_gbps = payload / (off_ms * 1e-3) / GB
    value = 2 * payload / (step_ms * 1e-3) / GB
    log(f"load {load_ms:.3f} ms ({load_gbps:.2f} GB/s), offload {off_ms:.3f} ms ({off_gbps:.2f} GB/s), "
        f"step {step_ms:.3f} ms, wall {wall / args.steps * 1e3:.3f} ms/step")

    # round-trip property of the last step (full parity lives in the tests)
    assert np.array_equal(out.array, host.array), "offload round trip differs from the host chunk"

    # ---- naive per-page DMA baseline (prefix of the calls) -------------------------------
    naive = None
    if not args.no_naive and args.host_layout != "head":
        nt = min(T, args.naive_tokens)
        nt -= nt % P if nt > P else 0
        spn = [(host.ptr, T, nt, pidx.data_ptr())]
        kv.kvio_naive_load(pool.handle, [(host.ptr, T, min(nt, P * 4), pidx.data_ptr())], 0, 1, stream)
        torch.cuda.synchronize()
        t = Timer(torch, stream)
        c0 = time.perf_counter()
        e = t.start()
        kv.kvio_naive_load(pool.handle, spn, 0, L, stream)
        t.stop(e)
        torch.cuda.synchronize()
        wall_n = time.perf_counter() - c0
        nbytes = L * 2 * nt * R
        calls = L * 2 * (-(-nt // P))
        gpu_ms = t.ms()[0]
        naive = {"calls": calls, "tokens": nt, "bytes": nbytes, "gbps": nbytes / max(wall_n, gpu_ms * 1e-3) / GB,
                 "gpu_ms": gpu_ms, "wall_ms": wall_n * 1e3, "prefix_of_calls": calls / (L * 2 * (-(-T // P))),
                 "note": "one hipMemcpyAsync per (page, layer, K|V) segment; rate over a prefix of the calls"}
        log(f"naive per-page memcpy: {calls} calls, {naive['gbps']:.2f} GB/s")

    # ---- CPU oracle baseline --------------------------------------------------------------
    cpu = cpu_all = None
    if not args.no_cpu_baseline and args.host_layout == "token":
        nbytes, el, passes = cpu_baseline(S, R, host.array, T, T, pages, P, L, args.cpu_seconds)
        cpu = {"value": nbytes / el / GB, "unit": "GB/s", "cores": 1, "kind": "oracle",
               "sample": f"{passes} pass(es) of load+offload of the whole {T}-token context, one "
                         f"(layer, K|V) slab at a time into a {S}-row host slab image, "
                         f"{el:.1f} s on {cpu_model()} "
                         f"({len(os.sched_getaffinity(0))} cores available, 1 used)"}
        log(f"cpu oracle: {cpu['value']:.2f} GB/s on 1 core")
        nthreads = min(len(os.sched_getaffinity(0)), 16)
        nbytes, el, slabs = cpu_baseline_all_cores(S, R, host.array, T, T, pages, P, L, args.cpu_seconds, nthreads)
        cpu_all = {"value": nbytes / el / GB, "unit": "GB/s", "cores": nthreads, "kind": "oracle",
                   "sample": f"{slabs} (layer, K|V) slab load+offloads of the same context on {nthreads} threads, "
                             f"each into its own {S}-row slab image, {el:.1f} s on {cpu_model()}"}
        log(f"cpu oracle: {cpu_all['value']:.2f} GB/s on {nthreads} threads")

    steady = None
    if k == 1:
        steady = steady_state(torch, kv, pool, span_in, host, stream, payload, reps=1000)
        steady.update(small_context_pipelines(torch, kv, pool, host, T, P, S, pages, stream, payload))
        steady["breakdown"] = launch_breakdown(torch, kv, pool, span_in, [(host.ptr, T, P, pidx.data_ptr())],
                                               L * 2 * P * R, payload, peak["h2d"] if peak else None)
        if peak:   # the target is set against the steady state (a single 2 MiB shot is latency-bound)
            for key in ("load", "memcpy", "two_streams_load", "batched4_load"):
                if f"{key}_gbps" in steady:
                    steady[f"{key}_frac_of_h2d_peak"] = round(steady[f"{key}_gbps"] / peak["h2d"], 4)
        log(f"steady state over 1000 loads: {steady['load_gbps']:.2f} GB/s, single shot "
            f"{steady['single_shot_us']:.1f} us; same-size memcpy {steady['memcpy_gbps']:.2f} GB/s; "
            f"independent contexts on two streams {steady.get('two_streams_load_gbps')} GB/s, "
            f"four per batched call {steady.get('batched4_load_gbps')} GB/s")
        log(f"launch breakdown (HIP graphs): {steady['breakdown']}")

    default_launch = not (args.workgroups or args.threads or args.tile_kib or args.cached or args.noncoherent_host
                          or args.no_lds or args.staged or args.host_layout != "token")
    traffic = measured_traffic(k, default_launch)
    frac_h2d = load_gbps / peak["h2d"] if peak else None
    frac_d2h = off_gbps / peak["d2h"] if peak else None
    ideal_ms = (payload / (peak["h2d"] * GB) + payload / (peak["d2h"] * GB)) * 1e3 if peak else None
    result = {
        "metric": "effective KV load/offload GB/s and tokens/s; % of measured host-link peak",
        "value": round(value, 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": wl.description, "kv_shape": shp.name, "layers": L,
                   "kv_heads": H, "head_dim": D, "kv_dtype": shp.dtype, "page_size": P, "pool_slots": S,
                   "tokens": T, "payload_bytes_per_direction": payload,
                   "step": "kvio_load (all layers) + kvio_offload (all layers)",
                   "launch": {"workgroups": args.workgroups or "default", "threads": args.threads or "default",
                              "tile_kib": args.tile_kib or "default", "nontemporal": not args.cached,
                              "staged": args.staged},
                   "host_memory": "non-coherent" if args.noncoherent_host else "coherent",
                   "host_layout": args.host_layout + ("" if not args.no_lds else " (no LDS)"),
                   "io_stream": _IO.get("kind")},
        "tokens_per_s": round(2 * T / (step_ms * 1e-3), 1),
        "load": {"ms": round(load_ms, 4), "gbps": round(load_gbps, 3), "tokens_per_s": round(T / (load_ms * 1e-3), 1),
                 "frac_of_h2d_peak": round(frac_h2d, 4) if peak else None,
                 "frac_of_kernel_h2d_peak": round(load_gbps / peak["kernel_h2d"], 4) if peak else None},
        "offload": {"ms": round(off_ms, 4), "gbps": round(off_gbps, 3),
                    "tokens_per_s": round(T / (off_ms * 1e-3), 1),
                    "frac_of_d2h_peak": round(frac_d2h, 4) if peak else None,
                    "frac_of_kernel_d2h_peak": round(off_gbps / peak["kernel_d2h"], 4) if peak else None},
        "frac_of_host_link_peak": round(ideal_ms / step_ms, 4) if peak else None,
        "host_link_peak": peak_report(peak),
        "roofline": roofline(("kvio_head_major_kernel<load>" if args.host_layout == "head" else "kvio_copy_kernel<load>")
                             + (" (staged)" if args.staged else ""), load_gbps,
                             peak["h2d"] if peak else None, traffic=traffic,
                             algorithmic_bytes_per_launch=payload, algorithmic_traffic_per_launch=2 * payload),
        "naive": naive,
        "cpu_baseline": cpu,
        "cpu_baseline_all_cores": cpu_all,
    }
    if steady:
        result["steady_state"] = steady
    pool.close()
    del pool_t
    host.free()
    out.free()
    torch.cuda.empty_cache()
    return result


if __name__ == "__main__":
    main()
