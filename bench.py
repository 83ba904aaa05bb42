"""Benchmark of the paged-KV host<->HBM transfer path on one MI355X.

Default workload: Llama-3.1-8B KV (32 layers, K and V, 8 KV heads x 128 dims,
bf16, 128 KiB per token), a pool of 500,000 token slots at page size 1, and
one 32K-token cached prefix placed in slots drawn uniformly at random (worst
case fragmentation).  One step = one pass of the hot path over that context:
kvio_load of all layers (host chunk -> scattered pool slots) followed by
kvio_offload of all layers (pool slots -> a second host chunk), each one
kernel launch on the same stream.

Reported (one JSON line):
  value       effective GB/s (1e9 B/s) of the whole step: load + offload
              payload bytes / mean step time; inputs are resident (host chunk
              pinned, pool in HBM) before the timed region.
  load/offload per-direction GB/s and tokens/s, each against the measured
              contiguous hipMemcpyAsync peak of the same direction on this machine.
  roofline    the load kernel (the critical-path direction): algorithmic
              bytes per launch / mean launch time from HIP events on its
              stream, against the measured host-link peak; HBM side too.
  naive       the per-page hipMemcpyAsync baseline on a prefix of the calls.
  cpu_baseline the CPU oracle, single thread, on the same context.

Other workloads: --config 1 (tiny pool, P = 16), --config 3 (70B KV, P = 16,
layer-wise load on a side stream against a per-layer bf16 GEMM), --config 5
(1M-token load with concurrent offloads).
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


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 5])
    ap.add_argument("--workgroups", type=int, default=0)
    ap.add_argument("--threads", type=int, default=0)
    ap.add_argument("--tile-kib", type=int, default=0)
    ap.add_argument("--cached", action="store_true", help="plain instead of non-temporal loads/stores")
    ap.add_argument("--noncoherent-host", action="store_true", help="coarse-grained pinned host chunks")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-naive", action="store_true")
    ap.add_argument("--no-peak", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--calibrate-copy", type=int, default=0,
                    help="only run a plain device-to-device elementwise copy of this many bytes, three "
                         "times (the known-size kernel that scales the HBM byte counters), then exit")
    ap.add_argument("--naive-tokens", type=int, default=2048,
                    help="tokens of the context the naive per-page baseline copies (all layers)")
    return ap.parse_args()


def measured_traffic(config, default_launch):
    """HBM/link bytes per load launch from the committed rocprofv3 counter
    summary, if it was taken on the current kernel sources (else None)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "kvio_copy_kernel__llama8b_p1_32k.counters.txt")
    if config != 2 or not default_launch or not os.path.exists(path):
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
    fetch = float(kv["load_fetch_kib"]) * float(kv["fetch_scale"]) * 1024
    write = float(kv["load_write_kib"]) * float(kv["write_scale"]) * 1024
    return {"bytes": round(fetch + write), "fetch_bytes": round(fetch), "write_bytes": round(write),
            "source": os.path.relpath(path, ROOT)}


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
    src_ptr, D2H into dst_ptr), and of H2D and D2H running concurrently on two
    streams (each half the size)."""
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    half = nbytes // 2
    res = {}
    for name, fn in (("h2d", lambda s: kv.kvio_memcpy(dev_ptr, src_ptr, nbytes, s)),
                     ("d2h", lambda s: kv.kvio_memcpy(dst_ptr, dev_ptr, nbytes, s))):
        fn(s1)
        torch.cuda.synchronize()
        t = Timer(torch, s1)
        for _ in range(reps):
            e = t.start()
            fn(s1)
            t.stop(e)
        torch.cuda.synchronize()
        res[name] = nbytes / (statistics.median(t.ms()) * 1e-3) / GB
    # bidirectional: H2D of one half while D2H of the other half
    ts = []
    for _ in range(reps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        kv.kvio_memcpy(dev_ptr, src_ptr, half, s1)
        kv.kvio_memcpy(dst_ptr + half, dev_ptr + half, half, s2)
        torch.cuda.synchronize()
        ts.append(time.perf_counter() - t0)
    res["bidir"] = 2 * half / statistics.median(ts) / GB
    res["bytes"] = nbytes
    return res


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


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only: the transfer path has no "
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
    wl = W.WORKLOADS[k]
    shp = wl.shape
    L, H, D, P, S, T = shp.num_layers, shp.num_kv_heads, shp.head_dim, wl.page_size, wl.num_slots, wl.tokens
    R = shp.row_bytes
    dtype = torch.float16 if shp.dtype == "fp16" else torch.bfloat16
    log(f"config {k}: {wl.description}; L={L} H={H} D={D} P={P} S={S} T={T} R={R}")

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

    launch = kv.launch(args.workgroups, args.threads, args.tile_kib, kv.KVIO_LAUNCH_CACHED if args.cached else 0)
    pool = kv.KVPool(pool_t, P, load_launch=launch, offload_launch=launch)
    span_in = [(host.ptr, T, T, pidx.data_ptr())]
    span_out = [(out.ptr, T, T, pidx.data_ptr())]
    stream = torch.cuda.Stream()

    # ---- contiguous host-link peak (denominator) ----------------------------------------
    peak = None
    if not args.no_peak:
        scratch = torch.empty(min(host_bytes, 2 << 30), dtype=torch.uint8, device="cuda")
        peak = memcpy_peak(torch, kv, host.ptr, out.ptr, scratch.data_ptr(), scratch.numel())
        del scratch
        log(f"memcpy peak: h2d {peak['h2d']:.2f} GB/s, d2h {peak['d2h']:.2f} GB/s, bidir {peak['bidir']:.2f} GB/s")

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

    # quick sampled correctness check of the last step (full parity lives in the tests)
    h = host.array.reshape(L, 2, T, R)
    sample = np.random.default_rng(0).integers(0, T, 16)
    got = pool_t.view(torch.uint8).view(2, L, S, R)[:, :, torch.from_numpy(pages[sample].astype(np.int64)).cuda()]
    got = got.cpu().numpy()
    for i, t in enumerate(sample):
        assert np.array_equal(got[0, :, i], h[:, 0, t]) and np.array_equal(got[1, :, i], h[:, 1, t])
    assert np.array_equal(out.array, host.array), "offload round trip differs from the host chunk"

    # ---- naive per-page DMA baseline (prefix of the calls) -------------------------------
    naive = None
    if not args.no_naive:
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
    cpu = None
    if not args.no_cpu_baseline:
        nbytes, el, passes = cpu_baseline(S, R, host.array, T, T, pages, P, L, args.cpu_seconds)
        cpu = {"value": nbytes / el / GB, "unit": "GB/s", "cores": 1, "kind": "oracle",
               "sample": f"{passes} pass(es) of load+offload of the whole {T}-token context, one "
                         f"(layer, K|V) slab at a time into a {S}-row host slab image, "
                         f"{el:.1f} s on {platform.processor() or 'host CPU'} "
                         f"({len(os.sched_getaffinity(0))} cores available, 1 used)"}
        log(f"cpu oracle: {cpu['value']:.2f} GB/s on 1 core")

    default_launch = not (args.workgroups or args.threads or args.tile_kib or args.cached or args.noncoherent_host)
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
        "config": {"workload": f"config{k}: {wl.description}", "kv_shape": shp.name, "layers": L,
                   "kv_heads": H, "head_dim": D, "kv_dtype": shp.dtype, "page_size": P, "pool_slots": S,
                   "tokens": T, "payload_bytes_per_direction": payload,
                   "step": "kvio_load (all layers) + kvio_offload (all layers)",
                   "launch": {"workgroups": args.workgroups or "default", "threads": args.threads or "default",
                              "tile_kib": args.tile_kib or "default", "nontemporal": not args.cached},
                   "host_memory": "non-coherent" if args.noncoherent_host else "coherent"},
        "tokens_per_s": round(2 * T / (step_ms * 1e-3), 1),
        "load": {"ms": round(load_ms, 4), "gbps": round(load_gbps, 3), "tokens_per_s": round(T / (load_ms * 1e-3), 1),
                 "frac_of_h2d_peak": round(frac_h2d, 4) if peak else None},
        "offload": {"ms": round(off_ms, 4), "gbps": round(off_gbps, 3),
                    "tokens_per_s": round(T / (off_ms * 1e-3), 1),
                    "frac_of_d2h_peak": round(frac_d2h, 4) if peak else None},
        "frac_of_host_link_peak": round(ideal_ms / step_ms, 4) if peak else None,
        "host_link_peak": {k2: round(v, 3) for k2, v in peak.items()} if peak else None,
        "roofline": {"bound": "host_link", "kernel": "kvio_copy_kernel<load>",
                     "achieved": round(load_gbps, 3), "peak": round(peak["h2d"], 3) if peak else None,
                     "unit": "GB/s", "frac": round(frac_h2d, 4) if peak else None,
                     "traffic": traffic["bytes"] if traffic else None,
                     "traffic_detail": traffic,
                     "algorithmic_bytes_per_launch": payload,
                     "algorithmic_traffic_per_launch": 2 * payload,
                     "pcie_spec_peak": PCIE_SPEC_GBPS, "frac_of_spec": round(load_gbps / PCIE_SPEC_GBPS, 4),
                     "hbm": {"achieved": round(load_gbps, 3), "peak": HBM_PEAK_GBPS,
                             "frac": round(load_gbps / HBM_PEAK_GBPS, 5)}},
        "naive": naive,
        "cpu_baseline": cpu,
    }
    pool.close()
    host.free()
    out.free()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
