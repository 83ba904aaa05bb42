"""Host-side helpers of bench.py (no GPU): the roofline block, the counter
summary lookup keyed to the kernel sources, and the batch-formation drain
model's accounting."""
import hashlib
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_roofline_block():
    r = bench.roofline("k", 57.6, 57.3, traffic=None, algorithmic_bytes_per_launch=4 << 30)
    assert r["peak"] == 64.0 and r["unit"] == "GB/s" and r["bound"] == "host_link"
    assert r["frac"] == round(57.6 / 64.0, 4)
    assert r["frac_of_measured_peak"] == round(57.6 / 57.3, 4)
    assert r["hbm"]["peak"] == 8000.0 and r["algorithmic_bytes_per_launch"] == 4 << 30
    b = bench.roofline("k", 100.0, 97.3, directions=2)
    assert b["peak"] == 128.0 and "both directions" in b["bound"]
    assert bench.roofline("k", 50.0, None)["frac_of_measured_peak"] is None


def test_measured_traffic_follows_the_kernel_sources(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2508_18572_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "kvio_kernels.hip").write_bytes(b"kernel")
    (csrc / "kvio_internal.h").write_bytes(b"header")
    prof = tmp_path / "profiles"
    prof.mkdir()
    hashes = " ".join(hashlib.sha256(x).hexdigest() for x in (b"kernel", b"header"))
    (prof / "kvio_copy_kernel__llama8b_p1_32k.counters.txt").write_text(
        f"# c\nkernel_sources_sha256: {hashes}\nload_fetch_kib: 100.0\nload_write_kib: 200.0\n"
        "fetch_scale: 2.0\nwrite_scale: 1.0\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    t = bench.measured_traffic(2, True)
    assert t["fetch_bytes"] == 200 * 1024 and t["write_bytes"] == 200 * 1024 and t["bytes"] == 400 * 1024
    assert bench.measured_traffic(2, False) is None           # another launch shape
    assert bench.measured_traffic(1, True) is None            # another workload
    (csrc / "kvio_kernels.hip").write_bytes(b"changed")
    assert bench.measured_traffic(2, True) is None            # kernel changed since the counters


def test_committed_counters_match_the_kernel_sources():
    """Whether the committed counter summary names the current kernel sources
    (then the bench reports measured traffic; otherwise traffic is null until
    the counters are re-taken)."""
    stale = [k for k in bench.COUNTER_FILES if bench.measured_traffic(k, True) is None]
    if stale:
        pytest.skip(f"the committed counters of workload(s) {stale} were taken on other kernel sources: "
                    "re-take them")


class _FakeKv:
    """Algorithm 1 stand-in for the drain model: FIFO batches of two."""

    @staticmethod
    def kvio_schedule_round(q, max_tokens, max_requests, ratio):
        take = list(range(min(2, len(q))))
        return take, list(range(len(take), len(q)))


def test_drain_model_counts_a_shared_context_once():
    q = [(1000, 10, 7, 0), (1000, 10, 7, 0), (0, 50, None, 0)]
    r = bench.drain_queue(_FakeKv, q, 100.0, load_tok_s=1000.0, prefill_tok_s=10.0)
    # batch 1: context 7 once -> load 1 s, compute 2 s -> 2 s; batch 2: compute 5 s
    assert r["drain_s"] == pytest.approx(7.0) and r["batches"] == 2 and r["loading_bound_batches"] == 0
    assert r["mean_completion_s"] == pytest.approx((2 + 2 + 7) / 3, abs=1e-3)


def test_synthetic_queue_is_seeded():
    a, b = bench.synthetic_queue(200, 5), bench.synthetic_queue(200, 5, bursty=True)
    assert a == bench.synthetic_queue(200, 5) and len(a) == len(b) == 200
    cached = [r for r in a if r[2] is not None]
    assert cached and all(8192 <= r[0] < 131072 and 64 <= r[1] < 512 for r in cached)
    assert all(r[0] == 0 and 1024 <= r[1] < 8192 for r in a if r[2] is None)


def test_more_than_one_gpu_is_refused():
    import json
    import subprocess
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]


def test_memequal_np_stops_at_n():
    import numpy as np
    a = np.zeros(3 << 20, np.uint8)
    b = a.copy()
    b[(2 << 20) + 5:] = 1
    assert bench.memequal_np(a, b, (2 << 20) + 5)
    assert not bench.memequal_np(a, b, (2 << 20) + 6)


def test_peak_report_keeps_an_unmeasured_bidirectional_peak():
    assert bench.peak_report(None) is None
    ok = bench.peak_report({"h2d": 57.30512, "d2h": 57.0391, "bidir": 97.3049, "bytes": 2 << 30})
    assert ok == {"h2d": 57.305, "d2h": 57.039, "bidir": 97.305, "bytes": 2 << 30}
    note = "unmeasured: the runtime serialised H2D and D2H copies"
    r = bench.peak_report({"h2d": 57.3, "d2h": 57.0, "bidir": None, "bidir_note": note, "bytes": 2 << 30})
    assert r["bidir"] is None and r["bidir_note"] == note
    # the roofline of the bidirectional workload then has no measured ceiling
    assert bench.roofline("k", 88.0, r["bidir"], directions=2)["frac_of_measured_peak"] is None


def test_measured_traffic_averages_over_launches(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2508_18572_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "kvio_kernels.hip").write_bytes(b"kernel")
    (csrc / "kvio_internal.h").write_bytes(b"header")
    prof = tmp_path / "profiles"
    prof.mkdir()
    hashes = " ".join(hashlib.sha256(x).hexdigest() for x in (b"kernel", b"header"))
    (prof / bench.COUNTER_FILES[4]).write_text(
        f"kernel_sources_sha256: {hashes}\nload_launches: 4\nload_fetch_kib: 400.0\nload_write_kib: 800.0\n"
        "fetch_scale: 2.0\nwrite_scale: 1.0\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    t = bench.measured_traffic(4, True)
    assert t["fetch_bytes"] == 200 * 1024 and t["write_bytes"] == 200 * 1024


def test_cpu_baseline_batched_moves_what_it_counts():
    """The batched CPU baseline runs the oracle on pieces of whole pages and
    counts 2 x rows x R per piece and plane; its slab image ends up holding the
    last plane's rows where the oracle puts them."""
    import numpy as np

    import oracle
    L, R, P, S = 2, 64, 16, 32768
    rng = np.random.default_rng(3)
    hit = [1000, 20000, 37]
    sizes = [L * 2 * h * R for h in hit]
    chunk = rng.integers(0, 256, sum(sizes), dtype=np.uint8)
    pages = rng.permutation(S // P).astype(np.int32)
    spans, o, p0 = [], 0, 0
    for h, b in zip(hit, sizes):
        n = -(-h // P)
        spans.append((o, h, h, pages[p0:p0 + n]))
        o += b
        p0 += n
    for threads in (1, 3):
        nb, el, planes = bench.cpu_baseline_batched(S, R, chunk, spans, P, L, 0.2, threads)
        assert planes >= 1 and el > 0
        assert nb % (2 * R) == 0 and nb >= 2 * R * sum(hit) * planes
    # the same pieces through the oracle directly reproduce one plane's slab
    exp = np.zeros((S, R), np.uint8)
    for off, ht, nt, pg in spans:
        oracle.load_slab(exp, P, chunk[off:off + nt * R], nt, pg)
    slab = np.zeros((S, R), np.uint8)
    for off, ht, nt, pg in spans:
        for a in range(0, nt, 8192):
            n = min(8192, nt - a)
            oracle.load_slab(slab, P, chunk[off + a * R:off + (a + n) * R], n, pg[a // P:])
    assert np.array_equal(slab, exp)
