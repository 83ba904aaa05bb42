// kvio_staged.cpp -- KVIO_LAUNCH_STAGED transfers: copy-engine copies of
// contiguous token runs through HBM staging slots, with the layout
// conversion done by the transfer kernels on the pool's side stream.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <algorithm>
#include <vector>

#include "kvio.h"
#include "kvio_internal.h"
#include "kvio_pool.h"

namespace kvio {

// Staged transfer (KVIO_LAUNCH_STAGED).  Work is packed into staging slots as
// units: span s, tokens [t0, t0 + n), layers [lb, lb + g) (shared by every
// unit of a slot), laid out like a chunk of n tokens in the pool's host
// layout: token-major row (l, kv, t) at ((l - lb)*2 + kv)*n*R + (t - t0)*R
// from the unit; head-major segment (l, kv, h, t) at
// (((l - lb)*2 + kv)*H + h)*n*De + (t - t0)*De.  When one layer of every
// span fits a slot, units are whole spans over as many layers as fit, and a
// span whose planes are contiguous (num_tokens == host_tokens) moves with one
// copy; otherwise layer by layer, spans split into runs of whole pages.  The
// copy engine works on the caller's stream, the scatter / gather kernel on
// the pool's side stream for this direction; events hand each slot over:
//   load:    caller: [wait slot free] copies in -> filled
//            side:   wait filled -> scatter -> slot free
//   offload: side:   [wait slot free] gather -> filled
//            caller: wait filled -> copies out -> slot free
// An offload's side stream first waits for the work already on the caller's
// stream (the pool rows it reads may come from it); a load ends with the
// caller's stream waiting for the last scatter.  So the call keeps stream
// order.  The kernel sees a unit as a span whose chunk starts lb*2*n*R bytes
// before it, so its usual row address ((l*2 + kv)*n + t)*R lands inside.
kvio_status run_staged(kvio_pool_t p, const std::vector<Resolved> &rs, const kvio_span *spans, int32_t n,
                       int32_t l0, int32_t l1, hipStream_t stream, kvio::Direction dir, const kvio::Shape &shape,
                       const char *fn) {
    const int64_t R = p->g.row_bytes, P = p->g.page_size, cap = p->slot_bytes;
    if (p->stage[dir] == nullptr) return fail(KVIO_EINVAL, "%s: the pool has no staging buffer for this direction", fn);
    hipStream_t ks = p->side_stream[dir];
    struct Unit { int32_t span; int64_t t0, n, off; };
    std::vector<Unit> units;
    units.reserve(KVIO_MAX_SPANS_PER_LAUNCH);
    int64_t used = 0, chunk = 0;
    hipError_t e = hipSuccess;
    if (dir == kvio::kOffload) {
        e = hipEventRecord(p->ev_start[dir], stream);
        if (e == hipSuccess) e = hipStreamWaitEvent(ks, p->ev_start[dir], 0);
        if (e != hipSuccess) return fail_hip(e, fn);
    }
    // Host <-> slot copies of one unit over layers [lb, lb + g).
    auto copy_unit = [&](const Unit &u, uint8_t *slot, int32_t lb, int32_t g, bool to_stage) -> hipError_t {
        uint8_t *host = static_cast<uint8_t *>(spans[u.span].host);
        const int64_t ht = spans[u.span].host_tokens;
        auto one = [&](uint8_t *h, uint8_t *d, int64_t bytes) {
            return to_stage ? hipMemcpyAsync(d, h, size_t(bytes), hipMemcpyHostToDevice, stream)
                            : hipMemcpyAsync(h, d, size_t(bytes), hipMemcpyDeviceToHost, stream);
        };
        if (u.t0 == 0 && u.n == ht)           // whole planes: one contiguous run
            return one(host + int64_t(lb) * 2 * ht * R, slot + u.off, int64_t(g) * 2 * u.n * R);
        // Token runs of one plane: contiguous rows (token-major), or one run
        // of head segments per head (head-major: [H][host_tokens][De]).
        const bool hm = p->g.host_layout == KVIO_HOST_HEAD_MAJOR;
        const int64_t runs = hm ? p->g.num_heads : 1, run = hm ? p->g.seg_bytes : R;
        for (int32_t l = lb; l < lb + g; ++l)
            for (int kv = 0; kv < 2; ++kv)
                for (int64_t h = 0; h < runs; ++h) {
                    hipError_t err = one(host + (((int64_t(l) * 2 + kv) * runs + h) * ht + u.t0) * run,
                                         slot + u.off + (((int64_t(l - lb) * 2 + kv) * runs + h) * u.n) * run,
                                         u.n * run);
                    if (err != hipSuccess) return err;
                }
        return hipSuccess;
    };
    auto flush = [&](int32_t lb, int32_t g) -> kvio_status {
        if (units.empty()) return KVIO_OK;
        const int k = int(chunk % kStageSlots);
        uint8_t *slot = p->stage[dir] + int64_t(k) * cap;
        hipEvent_t filled = p->ev_filled[dir][k], freed = p->ev_free[dir][k];
        hipError_t err = hipSuccess;
        if (dir == kvio::kLoad) {
            if (chunk >= kStageSlots) err = hipStreamWaitEvent(stream, freed, 0);
            for (size_t i = 0; i < units.size() && err == hipSuccess; ++i) err = copy_unit(units[i], slot, lb, g, true);
            if (err == hipSuccess) err = hipEventRecord(filled, stream);
            if (err == hipSuccess) err = hipStreamWaitEvent(ks, filled, 0);
        } else if (chunk >= kStageSlots) {
            err = hipStreamWaitEvent(ks, freed, 0);
        }
        if (err != hipSuccess) return fail_hip(err, fn);
        kvio::CopyArgs a;
        common_args(p, shape, lb, &a);
        a.n_spans = static_cast<int32_t>(units.size());
        int64_t tiles = 0;
        for (size_t i = 0; i < units.size(); ++i) {
            const Unit &u = units[i];
            a.tile_prefix[i] = tiles;
            a.spans[i].host = reinterpret_cast<const uint8_t *>(reinterpret_cast<uintptr_t>(slot) + uintptr_t(u.off) -
                                                                uintptr_t(int64_t(lb) * 2 * u.n * R));
            a.spans[i].page_idx = rs[size_t(u.span)].page_idx + u.t0 / P;
            a.spans[i].host_tokens = u.n;
            a.spans[i].num_tokens = static_cast<int32_t>(u.n);
            a.spans[i].origin = u.span;
            a.spans[i].page_base = static_cast<int32_t>(u.t0 / P);
            tiles += (u.n + a.rows_per_tile - 1) / a.rows_per_tile;
        }
        a.tile_prefix[units.size()] = tiles;
        a.plane_tiles = tiles;
        a.total_tiles = tiles * 2 * g;
        if ((err = launch_capped(a, dir, shape, ks)) != hipSuccess) return fail_hip(err, fn);
        if (dir == kvio::kLoad) {
            err = hipEventRecord(freed, ks);
        } else {
            err = hipEventRecord(filled, ks);
            if (err == hipSuccess) err = hipStreamWaitEvent(stream, filled, 0);
            for (size_t i = 0; i < units.size() && err == hipSuccess; ++i)
                err = copy_unit(units[i], slot, lb, g, false);
            if (err == hipSuccess) err = hipEventRecord(freed, stream);
        }
        if (err != hipSuccess) return fail_hip(err, fn);
        units.clear();
        used = 0;
        ++chunk;
        return KVIO_OK;
    };
    int64_t layer_bytes = 0;                  // one layer of every span
    for (int32_t s = 0; s < n; ++s) layer_bytes += 2 * rs[size_t(s)].num_tokens * R;
    if (layer_bytes == 0) return KVIO_OK;
    auto plan = [&]() -> kvio_status {
        for (int32_t l = l0; l < l1;) {
            if (layer_bytes <= cap) {
                // whole spans over g layers per slot
                const int32_t g = int32_t(std::min<int64_t>(l1 - l, cap / layer_bytes));
                for (int32_t s = 0; s < n; ++s) {
                    const int64_t T = rs[size_t(s)].num_tokens;
                    if (T == 0) continue;
                    if (units.size() == size_t(KVIO_MAX_SPANS_PER_LAUNCH)) {
                        kvio_status st = flush(l, g);
                        if (st != KVIO_OK) return st;
                    }
                    units.push_back({s, 0, T, used});
                    used += int64_t(g) * 2 * T * R;
                }
                kvio_status st = flush(l, g);
                if (st != KVIO_OK) return st;
                l += g;
                continue;
            }
            // one layer per slot, spans split into runs of whole pages
            for (int32_t s = 0; s < n; ++s) {
                const int64_t T = rs[size_t(s)].num_tokens;
                int64_t t0 = 0;
                while (t0 < T) {
                    const int64_t room = (cap - used) / (2 * R);
                    const int64_t take = T - t0 <= room ? T - t0 : room / P * P;
                    if (take == 0 || units.size() == size_t(KVIO_MAX_SPANS_PER_LAUNCH)) {
                        if (units.empty()) return fail(KVIO_EINVAL, "%s: staging slot below one page", fn);
                        kvio_status st = flush(l, 1);
                        if (st != KVIO_OK) return st;
                        continue;
                    }
                    units.push_back({s, t0, take, used});
                    used += 2 * take * R;
                    t0 += take;
                }
            }
            kvio_status st = flush(l, 1);
            if (st != KVIO_OK) return st;
            ++l;
        }
        return KVIO_OK;
    };
    const kvio_status st = plan();
    // A load joins the side stream back even when a later slot failed, so the
    // next call's copies cannot refill a slot that a queued scatter still reads.
    if (dir == kvio::kLoad && chunk > 0) {
        e = hipEventRecord(p->ev_done[dir], ks);
        if (e == hipSuccess) e = hipStreamWaitEvent(stream, p->ev_done[dir], 0);
        if (e != hipSuccess && st == KVIO_OK) return fail_hip(e, fn);
    }
    return st;
}

}  // namespace kvio
