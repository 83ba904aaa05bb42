// kvio_api.cpp -- the C ABI of libkvio.so: validation, pool handles, launch
// shaping, staged transfers, the naive per-page DMA baseline and thread-local
// error text.  Every layout-converting step of kvio_load / kvio_offload runs
// in the kernels of kvio_kernels.hip; this file checks arguments and enqueues
// them (staged launches also enqueue copy-engine copies of contiguous runs).
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "kvio.h"
#include "kvio_internal.h"
#include "kvio_pool.h"

namespace {

// Thread-local error text of the last failure (a fixed buffer: recording an
// error allocates nothing).
thread_local char g_last_error[1024];

}  // namespace

namespace kvio {

kvio_status fail(kvio_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return st;
}

void clear_error() { g_last_error[0] = '\0'; }

kvio_status fail_hip(hipError_t e, const char *what) {
    // The status and the text carry the error; clear the runtime's per-thread
    // last error so the caller's next, unrelated HIP call does not report it.
    (void)hipGetLastError();
    return fail(KVIO_EHIP, "%s: %s (%s)", what, hipGetErrorString(e), hipGetErrorName(e));
}

}  // namespace kvio

using kvio::fail;
using kvio::fail_hip;
using kvio::kStageSlots;
using kvio::Resolved;

namespace {

int ilog2_exact(int64_t v) {
    if (v <= 0 || (v & (v - 1)) != 0) return -1;
    int s = 0;
    while ((int64_t(1) << s) < v) ++s;
    return s;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int64_t kDefaultStagingBytes = int64_t(4) << 30;
// A staged call that moves less than this (or less than one slot, if slots
// are smaller) runs on the kernel path instead: each slot hand-over and copy
// costs the staged path tens of microseconds, which a small transfer cannot
// amortise (a 2 MiB context: 13 GB/s staged, 52 GB/s through the kernels).
constexpr int64_t kStagedMinBytes = int64_t(64) << 20;

}  // namespace

namespace kvio {

Shape resolve(const kvio_launch &l, const Shape &def) {
    kvio::Shape s;
    s.workgroups = l.workgroups > 0 ? l.workgroups : def.workgroups;
    s.threads = l.threads > 0 ? l.threads : def.threads;
    s.tile_kib = l.tile_kib > 0 ? l.tile_kib : def.tile_kib;
    s.nontemporal = (l.flags & KVIO_LAUNCH_CACHED) == 0;
    s.head_major_lds = (l.flags & KVIO_LAUNCH_NO_LDS) == 0;
    return s;
}

kvio_status check_launch(const kvio_launch &l, const char *which) {
    if (l.workgroups < 0 || l.threads < 0 || l.tile_kib < 0)
        return fail(KVIO_EINVAL, "%s: negative launch field", which);
    if (l.threads != 0 && (l.threads % 64 != 0 || l.threads > 1024))
        return fail(KVIO_EINVAL, "%s: threads %d is not a multiple of 64 in [64, 1024]", which, l.threads);
    if (l.tile_kib != 0 && l.tile_kib != 4 && l.tile_kib != 8 && l.tile_kib != 16)
        return fail(KVIO_EINVAL, "%s: tile_kib %d is not 4, 8 or 16", which, l.tile_kib);
    if ((l.flags & ~(KVIO_LAUNCH_CACHED | KVIO_LAUNCH_NO_LDS | KVIO_LAUNCH_STAGED)) != 0)
        return fail(KVIO_EINVAL, "%s: unknown launch flags 0x%x", which, l.flags);
    return KVIO_OK;
}

// Device-visible address of [p, p + bytes), or an error if the device cannot
// reach it or the allocation that holds it is shorter than `bytes`.
kvio_status device_view(const void *p, uint64_t bytes, bool want_device_memory, const char *what,
                        const uint8_t **out) {
    hipPointerAttribute_t attr;
    memset(&attr, 0, sizeof attr);
    hipError_t e = hipPointerGetAttributes(&attr, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();   // clear the sticky error of the failed lookup
        return fail(want_device_memory ? KVIO_EINVAL : KVIO_ENOTMAPPED,
                    "%s %p is not memory known to the HIP runtime (%s)", what, p, hipGetErrorName(e));
    }
    if (want_device_memory && attr.type != hipMemoryTypeDevice)
        return fail(KVIO_EINVAL, "%s %p is not device memory", what, p);
    if (attr.devicePointer == nullptr)
        return fail(KVIO_ENOTMAPPED, "%s %p is not mapped into the device address space", what, p);
    // The runtime reports both addresses offset to the queried pointer; host
    // allocations are identity-mapped (device address == host address).
    // Anything else is refused rather than guessed.
    const uint8_t *dev = static_cast<const uint8_t *>(attr.devicePointer);
    if (attr.hostPointer != nullptr && attr.hostPointer != p) {
        if (attr.devicePointer == attr.hostPointer)
            dev = static_cast<const uint8_t *>(p);
        else
            return fail(KVIO_ENOTMAPPED, "%s %p: cannot resolve its device address", what, p);
    }
    // Extent: the allocation holding `dev` must reach dev + bytes.  A region
    // whose extent the runtime cannot report is refused, so a kernel never
    // reads or writes past an allocation.
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    e = hipMemGetAddressRange(&base, &size, const_cast<uint8_t *>(dev));
    if (e != hipSuccess || base == nullptr) {
        (void)hipGetLastError();
        return fail(KVIO_ENOTMAPPED, "%s %p: the runtime cannot report the allocation that holds it", what, p);
    }
    const uint8_t *b = static_cast<const uint8_t *>(base);
    if (dev < b || static_cast<uint64_t>(dev - b) + bytes > size)
        return fail(KVIO_EINVAL, "%s %p: the transfer reaches %llu bytes but the allocation holds "
                    "only %llu from there", what, p, (unsigned long long)bytes,
                    (unsigned long long)(dev >= b && static_cast<uint64_t>(dev - b) <= size ? size - (dev - b) : 0));
    *out = dev;
    return KVIO_OK;
}

kvio_status check_desc(const kvio_pool_desc *d, const char *fn, PoolGeom *g) {
    if (d->num_layers < 1 || d->num_kv_heads < 1 || d->head_dim < 1 || d->elem_bytes < 1 ||
        d->page_size < 1)
        return fail(KVIO_EINVAL, "%s: sizes must be >= 1", fn);
    if (d->host_layout != KVIO_HOST_TOKEN_MAJOR && d->host_layout != KVIO_HOST_PAGE_FIRST &&
        d->host_layout != KVIO_HOST_HEAD_MAJOR)
        return fail(KVIO_EINVAL, "%s: unknown host layout %d", fn, d->host_layout);
    if (d->host_layout == KVIO_HOST_HEAD_MAJOR && (int64_t(d->head_dim) * d->elem_bytes) % 16 != 0)
        return fail(KVIO_EALIGN, "%s: head-major chunks need head_dim * elem_bytes (%lld) to be "
                    "a multiple of 16", fn, (long long)(int64_t(d->head_dim) * d->elem_bytes));
    if (d->num_slots < 1 || d->num_slots > INT32_MAX || d->num_slots % d->page_size != 0)
        return fail(KVIO_EINVAL, "%s: num_slots %lld must be in [1, 2^31) and a multiple "
                    "of page_size %d", fn, (long long)d->num_slots, d->page_size);
    const int64_t R = int64_t(d->num_kv_heads) * d->head_dim * d->elem_bytes;
    if (R % 16 != 0) return fail(KVIO_EALIGN, "%s: row bytes %lld not a multiple of 16", fn, (long long)R);
    if (R > (int64_t(1) << 26)) return fail(KVIO_EINVAL, "%s: row bytes %lld too large", fn, (long long)R);
    if (d->k_layers == nullptr || d->v_layers == nullptr) return fail(KVIO_EINVAL, "%s: null layer table", fn);
    kvio_status st = check_launch(d->load_launch, "load_launch");
    if (st != KVIO_OK) return st;
    st = check_launch(d->offload_launch, "offload_launch");
    if (st != KVIO_OK) return st;
    g->num_layers = d->num_layers;
    g->num_heads = d->num_kv_heads;
    g->host_layout = d->host_layout;
    g->seg_bytes = int64_t(d->head_dim) * d->elem_bytes;
    g->page_size = d->page_size;
    g->num_slots = d->num_slots;
    g->row_bytes = R;
    return KVIO_OK;
}

kvio_status resolve_layers(const kvio_pool_desc *d, const PoolGeom &g, const char *fn, uint8_t **layers) {
    const uint64_t layer_bytes = uint64_t(g.num_slots) * uint64_t(g.row_bytes);
    for (int kv = 0; kv < 2; ++kv) {
        void *const *tab = kv == 0 ? d->k_layers : d->v_layers;
        for (int l = 0; l < g.num_layers; ++l) {
            void *ptr = tab[l];
            if (ptr == nullptr) return fail(KVIO_EINVAL, "%s: %c layer %d is null", fn, kv ? 'V' : 'K', l);
            if (!aligned16(ptr))
                return fail(KVIO_EALIGN, "%s: %c layer %d not 16-byte aligned", fn, kv ? 'V' : 'K', l);
            const uint8_t *dev = nullptr;
            kvio_status st = device_view(ptr, layer_bytes, true, kv ? "V layer" : "K layer", &dev);
            if (st != KVIO_OK) return st;
            layers[size_t(kv) * g.num_layers + l] = const_cast<uint8_t *>(dev);
        }
    }
    return KVIO_OK;
}

}  // namespace kvio

using kvio::check_launch;
using kvio::device_view;
using kvio::resolve;

// Error path shared with kvio_sched.cpp (same thread-local error text).
kvio_status kvio_sched_fail(kvio_status st, const char *msg) {
    kvio::clear_error();
    if (st == KVIO_OK) return KVIO_OK;
    return fail(st, "%s", msg);
}


namespace {

// Release what kvio_pool_create allocated (null members are skipped); waits
// for the side streams first.  Returns the first failure.
hipError_t release_pool(kvio_pool *p) {
    hipError_t first = hipSuccess;
    auto keep = [&](hipError_t e) { if (first == hipSuccess && e != hipSuccess) first = e; };
    for (int dir = 0; dir < 2; ++dir) {
        if (p->side_stream[dir] != nullptr) {
            keep(hipStreamSynchronize(p->side_stream[dir]));
            keep(hipStreamDestroy(p->side_stream[dir]));
        }
        for (int k = 0; k < kStageSlots; ++k) {
            if (p->ev_filled[dir][k] != nullptr) keep(hipEventDestroy(p->ev_filled[dir][k]));
            if (p->ev_free[dir][k] != nullptr) keep(hipEventDestroy(p->ev_free[dir][k]));
        }
        if (p->ev_start[dir] != nullptr) keep(hipEventDestroy(p->ev_start[dir]));
        if (p->ev_done[dir] != nullptr) keep(hipEventDestroy(p->ev_done[dir]));
        if (p->stage[dir] != nullptr) keep(hipFree(p->stage[dir]));
    }
    if (p->d_layers != nullptr) keep(hipFree(p->d_layers));
    if (p->d_err != nullptr) keep(hipFree(p->d_err));
    delete p;
    return first;
}

// Staging buffer, side stream and events of one staged direction.
hipError_t create_staging(kvio_pool *p, int dir, int64_t stage_bytes) {
    hipError_t e = hipMalloc(reinterpret_cast<void **>(&p->stage[dir]), size_t(stage_bytes));
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&p->side_stream[dir], hipStreamNonBlocking);
    for (int k = 0; k < kStageSlots && e == hipSuccess; ++k) {
        e = hipEventCreateWithFlags(&p->ev_filled[dir][k], hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&p->ev_free[dir][k], hipEventDisableTiming);
    }
    if (e == hipSuccess) e = hipEventCreateWithFlags(&p->ev_start[dir], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&p->ev_done[dir], hipEventDisableTiming);
    return e;
}

}  // namespace

extern "C" {

const char *kvio_strerror(kvio_status st) {
    switch (st) {
        case KVIO_OK: return "KVIO_OK: success";
        case KVIO_EINVAL: return "KVIO_EINVAL: invalid argument";
        case KVIO_ERANGE: return "KVIO_ERANGE: page index out of range";
        case KVIO_EALIGN: return "KVIO_EALIGN: row size or pointer not 16-byte aligned";
        case KVIO_ENOTMAPPED: return "KVIO_ENOTMAPPED: host memory not accessible from the device";
        case KVIO_EHIP: return "KVIO_EHIP: HIP runtime error";
        case KVIO_ENOMEM: return "KVIO_ENOMEM: out of memory";
        case KVIO_EIO: return "KVIO_EIO: disk read or write failed";
    }
    return "unknown kvio_status";
}

const char *kvio_last_error(void) { return g_last_error; }

kvio_status kvio_pool_create(const kvio_pool_desc *d, kvio_pool_t *out) {
    kvio::clear_error();
    if (d == nullptr || out == nullptr) return fail(KVIO_EINVAL, "kvio_pool_create: null argument");
    kvio::PoolGeom g;
    kvio_status st = kvio::check_desc(d, "kvio_pool_create", &g);
    if (st != KVIO_OK) return st;
    const int64_t R = g.row_bytes;
    const bool staged[2] = {(d->load_launch.flags & KVIO_LAUNCH_STAGED) != 0,
                            (d->offload_launch.flags & KVIO_LAUNCH_STAGED) != 0};
    const int64_t stage_bytes = d->staging_bytes > 0 ? d->staging_bytes : kDefaultStagingBytes;
    if ((staged[0] || staged[1]) && d->host_layout == KVIO_HOST_PAGE_FIRST)
        return fail(KVIO_EINVAL, "kvio_pool_create: staged transfers take token-major or head-major host chunks");
    const int64_t slot_bytes = stage_bytes / kStageSlots / 16 * 16;
    if ((staged[0] || staged[1]) && (d->staging_bytes < 0 || slot_bytes < 2 * int64_t(d->page_size) * R))
        return fail(KVIO_EINVAL, "kvio_pool_create: staging_bytes %lld must hold %d slots of at least one page "
                    "of K and V rows (%lld bytes each)", (long long)d->staging_bytes, kStageSlots,
                    (long long)(2 * int64_t(d->page_size) * R));

    kvio_pool *p = new (std::nothrow) kvio_pool();
    if (p == nullptr) return fail(KVIO_ENOMEM, "kvio_pool_create: host allocation failed");
    p->g = g;
    p->load_launch = d->load_launch;
    p->offload_launch = d->offload_launch;
    p->layers.resize(2 * size_t(d->num_layers));
    p->d_layers = nullptr;
    p->d_err = nullptr;
    p->slot_bytes = slot_bytes;
    st = kvio::resolve_layers(d, g, "kvio_pool_create", p->layers.data());
    if (st != KVIO_OK) {
        delete p;
        return st;
    }
    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) {
        delete p;
        return fail_hip(e, "kvio_pool_create: hipGetDevice");
    }
    e = hipMalloc(reinterpret_cast<void **>(&p->d_layers), p->layers.size() * sizeof(uint8_t *));
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&p->d_err), sizeof(unsigned long long));
    if (e == hipSuccess)
        e = hipMemcpy(p->d_layers, p->layers.data(), p->layers.size() * sizeof(uint8_t *),
                      hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemset(p->d_err, 0, sizeof(unsigned long long));
    for (int dir = 0; dir < 2 && e == hipSuccess; ++dir)
        if (staged[dir]) e = create_staging(p, dir, int64_t(kStageSlots) * slot_bytes);
    if (e != hipSuccess) {
        (void)release_pool(p);
        (void)hipGetLastError();
        return e == hipErrorOutOfMemory ? fail(KVIO_ENOMEM, "kvio_pool_create: device allocation failed")
                                        : fail_hip(e, "kvio_pool_create");
    }
    *out = p;
    return KVIO_OK;
}

kvio_status kvio_pool_destroy(kvio_pool_t p) {
    kvio::clear_error();
    if (p == nullptr) return KVIO_OK;
    const hipError_t e = release_pool(p);
    if (e != hipSuccess) return fail_hip(e, "kvio_pool_destroy");
    return KVIO_OK;
}

}  // extern "C"

namespace kvio {

// Validate the spans and layer range; translate host chunks to device
// addresses.  Nothing is enqueued here.
kvio_status validate_spans(const PoolGeom &g, const kvio_span *spans, int32_t n, int32_t l0, int32_t l1,
                           const char *fn, Resolved *out) {
    if (n < 0) return fail(KVIO_EINVAL, "%s: n_spans %d < 0", fn, n);
    if (n > 0 && spans == nullptr) return fail(KVIO_EINVAL, "%s: null span array", fn);
    if (l0 < 0 || l1 > g.num_layers || l0 >= l1)
        return fail(KVIO_EINVAL, "%s: layer range [%d, %d) outside [0, %d)", fn, l0, l1, g.num_layers);
    const int64_t R = g.row_bytes;
    for (int32_t i = 0; i < n; ++i) {
        const kvio_span &s = spans[i];
        if (s.num_tokens < 0 || s.host_tokens < 0 || s.num_tokens > s.host_tokens)
            return fail(KVIO_EINVAL, "%s: span %d: need 0 <= num_tokens (%lld) <= host_tokens (%lld)", fn, i,
                        (long long)s.num_tokens, (long long)s.host_tokens);
        if (s.num_tokens > INT32_MAX)
            return fail(KVIO_EINVAL, "%s: span %d: num_tokens %lld >= 2^31", fn, i, (long long)s.num_tokens);
        Resolved r{nullptr, s.page_idx, s.host_tokens, s.num_tokens};
        if (s.num_tokens > 0) {
            if (s.host == nullptr) return fail(KVIO_EINVAL, "%s: span %d: null host chunk", fn, i);
            if (s.page_idx == nullptr) return fail(KVIO_EINVAL, "%s: span %d: null page table", fn, i);
            if (!aligned16(s.host)) return fail(KVIO_EALIGN, "%s: span %d: host chunk not 16-byte aligned", fn, i);
            if ((reinterpret_cast<uintptr_t>(s.page_idx) & 3u) != 0)
                return fail(KVIO_EALIGN, "%s: span %d: page table not 4-byte aligned", fn, i);
            // One past the highest host byte the transfer can touch.
            uint64_t reach;
            const uint64_t P = uint64_t(g.page_size);
            if (g.host_layout == KVIO_HOST_PAGE_FIRST) {
                if (s.host_tokens % g.page_size != 0)
                    return fail(KVIO_EINVAL, "%s: span %d: page-first chunks need host_tokens (%lld) to be a "
                                "multiple of the page size %d", fn, i, (long long)s.host_tokens, g.page_size);
                // whole pages up to the one holding token num_tokens - 1
                reach = (uint64_t(s.num_tokens) + P - 1) / P * uint64_t(g.num_layers) * 2 * P * uint64_t(R);
            } else if (g.host_layout == KVIO_HOST_HEAD_MAJOR) {
                // segment (l1 - 1, V, H - 1, num_tokens - 1)
                reach = ((uint64_t(l1 - 1) * 2 + 1) * uint64_t(g.num_heads) + uint64_t(g.num_heads) - 1) *
                            uint64_t(s.host_tokens) * uint64_t(g.seg_bytes) +
                        uint64_t(s.num_tokens) * uint64_t(g.seg_bytes);
            } else {
                // row (l1 - 1, V, num_tokens - 1)
                reach = (uint64_t(l1 - 1) * 2 + 1) * uint64_t(s.host_tokens) * uint64_t(R) +
                        uint64_t(s.num_tokens) * uint64_t(R);
            }
            kvio_status st = device_view(s.host, reach, false, "host chunk", &r.host);
            if (st != KVIO_OK) return st;
            const int64_t pages = (s.num_tokens + g.page_size - 1) / g.page_size;
            const uint8_t *pt = nullptr;
            st = device_view(s.page_idx, uint64_t(pages) * 4u, false, "page table", &pt);
            if (st != KVIO_OK) {
                char why[512];
                snprintf(why, sizeof why, "%s", kvio_last_error());
                return fail(KVIO_EINVAL, "%s: span %d: %s", fn, i, why);
            }
            r.page_idx = reinterpret_cast<const int32_t *>(pt);
        }
        out[i] = r;
    }
    return KVIO_OK;
}

// Fields of a launch that do not depend on its spans.
void common_args(const PoolGeom &g, uint8_t *const *layers, unsigned long long *err, const Shape &shape,
                 int32_t l0, CopyArgs *a) {
    memset(a, 0, sizeof *a);
    const int64_t R = g.row_bytes;
    a->layers = layers;
    a->err = err;
    a->row_bytes = R;
    a->num_pages = g.num_slots / g.page_size;
    a->num_layers = g.num_layers;
    a->layer_begin = l0;
    a->page_size = g.page_size;
    a->page_shift = ilog2_exact(g.page_size);
    a->vec_per_row = static_cast<int32_t>(R / 16);
    a->vec_shift = ilog2_exact(R / 16);
    a->vec_step_rows = static_cast<int32_t>(64 / (R / 16));
    a->vec_step_cols = static_cast<int32_t>(64 % (R / 16));
    a->rows_per_tile = kvio::rows_per_tile(R, shape.tile_kib);
    a->host_layout = g.host_layout;
    a->num_heads = g.num_heads;
    a->seg_vecs = static_cast<int32_t>(g.seg_bytes / 16);
}

void common_args(kvio_pool_t p, const Shape &shape, int32_t l0, CopyArgs *a) {
    common_args(p->g, p->d_layers, p->d_err, shape, l0, a);
}

hipError_t launch_capped(const CopyArgs &a, Direction dir, Shape s, hipStream_t stream) {
    const int64_t waves_per_wg = s.threads / 64;
    const int64_t max_wgs = (a.total_tiles + waves_per_wg - 1) / waves_per_wg;
    if (s.workgroups > max_wgs) s.workgroups = static_cast<int>(max_wgs);
    return launch_copy(a, dir, s, stream);
}

Shape kernel_shape(const PoolGeom &g, const kvio_launch &l, const Shape &def) {
    Shape shape = resolve(l, def);
    // LDS staging of a head-major tile needs the whole tile (>= one row) in the
    // wave's U KiB slice.
    if (g.host_layout == KVIO_HOST_HEAD_MAJOR && g.row_bytes > int64_t(shape.tile_kib) * 1024)
        shape.head_major_lds = false;
    return shape;
}

kvio_status launch_spans(const PoolGeom &g, uint8_t *const *layers, unsigned long long *err, const Resolved *rs,
                         int32_t n, int32_t l0, int32_t l1, Direction dir, const Shape &shape, hipStream_t stream,
                         const char *fn) {
    for (int32_t first = 0; first < n; first += KVIO_MAX_SPANS_PER_LAUNCH) {
        const int32_t cnt = n - first < KVIO_MAX_SPANS_PER_LAUNCH ? n - first : KVIO_MAX_SPANS_PER_LAUNCH;
        CopyArgs a;
        common_args(g, layers, err, shape, l0, &a);
        a.n_spans = cnt;
        int64_t tiles = 0;
        for (int32_t i = 0; i < cnt; ++i) {
            const Resolved &r = rs[first + i];
            a.tile_prefix[i] = tiles;
            a.spans[i].host = r.host;
            a.spans[i].page_idx = r.page_idx;
            a.spans[i].host_tokens = r.host_tokens;
            a.spans[i].num_tokens = static_cast<int32_t>(r.num_tokens);
            a.spans[i].origin = first + i;
            tiles += (r.num_tokens + a.rows_per_tile - 1) / a.rows_per_tile;
        }
        a.tile_prefix[cnt] = tiles;
        a.plane_tiles = tiles;
        a.total_tiles = tiles * 2 * int64_t(l1 - l0);
        if (a.total_tiles == 0) continue;
        const hipError_t e = launch_capped(a, dir, shape, stream);
        if (e != hipSuccess) return fail_hip(e, fn);
    }
    return KVIO_OK;
}

}  // namespace kvio

namespace {

kvio_status run_copy(kvio_pool_t p, const kvio_span *spans, int32_t n, int32_t l0, int32_t l1,
                     hipStream_t stream, kvio::Direction dir, const char *fn) {
    kvio::clear_error();
    if (p == nullptr) return fail(KVIO_EINVAL, "%s: null pool", fn);
    std::vector<Resolved> rs(size_t(n > 0 ? n : 0));
    kvio_status st = kvio::validate_spans(p->g, spans, n, l0, l1, fn, rs.data());
    if (st != KVIO_OK) return st;
    kvio_launch lc = dir == kvio::kLoad ? p->load_launch : p->offload_launch;
    int64_t bytes = 0;                       // payload of the whole call
    for (const Resolved &r : rs) bytes += r.num_tokens;
    bytes *= 2 * int64_t(l1 - l0) * p->g.row_bytes;
    if (lc.flags & KVIO_LAUNCH_STAGED) {
        if (bytes >= std::min(kStagedMinBytes, p->slot_bytes))
            return run_staged(p, rs, spans, n, l0, l1, stream, dir,
                              kvio::kernel_shape(p->g, lc, kvio::kDefaultStaged), fn);
        lc = kvio_launch{0, 0, 0, lc.flags & ~KVIO_LAUNCH_STAGED};   // small: the kernel path, default shape
    }
    const kvio::Shape shape = kvio::kernel_shape(p->g, lc, kvio::default_shape(dir, bytes, p->g.host_layout, p->g.num_heads));
    return kvio::launch_spans(p->g, p->d_layers, p->d_err, rs.data(), n, l0, l1, dir, shape, stream, fn);
}

kvio_status run_naive(kvio_pool_t p, const kvio_span *spans, int32_t n, int32_t l0, int32_t l1,
                      hipStream_t stream, kvio::Direction dir, const char *fn) {
    kvio::clear_error();
    if (p == nullptr) return fail(KVIO_EINVAL, "%s: null pool", fn);
    std::vector<Resolved> rs(size_t(n > 0 ? n : 0));
    kvio_status st = kvio::validate_spans(p->g, spans, n, l0, l1, fn, rs.data());
    if (st != KVIO_OK) return st;
    if (p->g.host_layout == KVIO_HOST_HEAD_MAJOR)
        return fail(KVIO_EINVAL, "%s: the per-page copy baseline takes token-major or page-first chunks", fn);
    const int64_t R = p->g.row_bytes;
    const int64_t P = p->g.page_size;
    const int64_t num_pages = p->g.num_slots / P;
    std::vector<int32_t> table;
    for (int32_t i = 0; i < n; ++i) {
        const kvio_span &s = spans[i];
        if (s.num_tokens == 0) continue;
        const int64_t pages = (s.num_tokens + P - 1) / P;
        table.resize(size_t(pages));
        hipError_t e = hipMemcpy(table.data(), s.page_idx, size_t(pages) * 4, hipMemcpyDefault);
        if (e != hipSuccess) return fail_hip(e, fn);
        for (int64_t j = 0; j < pages; ++j)
            if (table[size_t(j)] < 0 || table[size_t(j)] >= num_pages)
                return fail(KVIO_ERANGE, "%s: span %d context page %lld holds page %d outside [0, %lld)", fn, i,
                            (long long)j, table[size_t(j)], (long long)num_pages);
        uint8_t *host = static_cast<uint8_t *>(s.host);
        for (int32_t l = l0; l < l1; ++l) {
            for (int kv = 0; kv < 2; ++kv) {
                uint8_t *pool = p->layers[size_t(kv) * p->g.num_layers + l];
                uint8_t *hrow0 = host + ((int64_t(l) * 2 + kv) * s.host_tokens) * R;
                for (int64_t j = 0; j < pages; ++j) {
                    const int64_t rows = (j + 1) * P <= s.num_tokens ? P : s.num_tokens - j * P;
                    uint8_t *prow = pool + int64_t(table[size_t(j)]) * P * R;
                    uint8_t *hrow = p->g.host_layout == KVIO_HOST_PAGE_FIRST
                        ? host + ((j * p->g.num_layers + l) * 2 + kv) * P * R
                        : hrow0 + j * P * R;
                    hipError_t e2 = dir == kvio::kLoad
                        ? hipMemcpyAsync(prow, hrow, size_t(rows * R), hipMemcpyHostToDevice, stream)
                        : hipMemcpyAsync(hrow, prow, size_t(rows * R), hipMemcpyDeviceToHost, stream);
                    if (e2 != hipSuccess) return fail_hip(e2, fn);
                }
            }
        }
    }
    return KVIO_OK;
}

}  // namespace

extern "C" {

kvio_status kvio_load(kvio_pool_t p, const kvio_span *spans, int32_t n, int32_t l0, int32_t l1,
                      hipStream_t stream) {
    return run_copy(p, spans, n, l0, l1, stream, kvio::kLoad, "kvio_load");
}

kvio_status kvio_offload(kvio_pool_t p, const kvio_span *spans, int32_t n, int32_t l0, int32_t l1,
                         hipStream_t stream) {
    return run_copy(p, spans, n, l0, l1, stream, kvio::kOffload, "kvio_offload");
}

kvio_status kvio_load_layer(kvio_pool_t p, const kvio_span *spans, int32_t n, int32_t layer,
                            hipStream_t stream, hipEvent_t done) {
    kvio_status st = run_copy(p, spans, n, layer, layer + 1, stream, kvio::kLoad, "kvio_load_layer");
    if (st != KVIO_OK) return st;
    if (done != nullptr) {
        hipError_t e = hipEventRecord(done, stream);
        if (e != hipSuccess) return fail_hip(e, "kvio_load_layer: hipEventRecord");
    }
    return KVIO_OK;
}

kvio_status kvio_check(kvio_pool_t p) {
    kvio::clear_error();
    if (p == nullptr) return fail(KVIO_EINVAL, "kvio_check: null pool");
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return fail_hip(e, "kvio_check: hipDeviceSynchronize");
    unsigned long long rec = 0;
    e = hipMemcpy(&rec, p->d_err, sizeof rec, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_hip(e, "kvio_check: read error record");
    if (rec == 0) return KVIO_OK;
    e = hipMemset(p->d_err, 0, sizeof rec);
    if (e != hipSuccess) return fail_hip(e, "kvio_check: clear error record");
    const unsigned long long span = (rec >> kvio::kErrSpanShift) - 1;
    const unsigned long long page = rec & ((1ull << kvio::kErrSpanShift) - 1);
    return fail(KVIO_ERANGE, "kvio_check: span %llu, context page %llu: pool page index outside [0, %lld); "
                "those rows were skipped", span, page, (long long)(p->g.num_slots / p->g.page_size));
}

kvio_status kvio_naive_load(kvio_pool_t p, const kvio_span *spans, int32_t n, int32_t l0, int32_t l1,
                            hipStream_t stream) {
    return run_naive(p, spans, n, l0, l1, stream, kvio::kLoad, "kvio_naive_load");
}

kvio_status kvio_naive_offload(kvio_pool_t p, const kvio_span *spans, int32_t n, int32_t l0, int32_t l1,
                               hipStream_t stream) {
    return run_naive(p, spans, n, l0, l1, stream, kvio::kOffload, "kvio_naive_offload");
}

kvio_status kvio_memcpy(void *dst, const void *src, size_t bytes, hipStream_t stream) {
    kvio::clear_error();
    if (bytes == 0) return KVIO_OK;
    if (dst == nullptr || src == nullptr) return fail(KVIO_EINVAL, "kvio_memcpy: null pointer");
    hipError_t e = hipMemcpyAsync(dst, src, bytes, hipMemcpyDefault, stream);
    if (e != hipSuccess) return fail_hip(e, "kvio_memcpy");
    return KVIO_OK;
}

kvio_status kvio_stream_create(const uint32_t *cu_mask, uint32_t mask_words, hipStream_t *out) {
    kvio::clear_error();
    if (out == nullptr) return fail(KVIO_EINVAL, "kvio_stream_create: null out");
    hipStream_t s = nullptr;
    hipError_t e;
    if (mask_words == 0) {
        e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
    } else {
        if (cu_mask == nullptr) return fail(KVIO_EINVAL, "kvio_stream_create: null CU mask");
        bool any = false;
        for (uint32_t i = 0; i < mask_words; ++i) any = any || cu_mask[i] != 0;
        if (!any) return fail(KVIO_EINVAL, "kvio_stream_create: empty CU mask");
        e = hipExtStreamCreateWithCUMask(&s, mask_words, cu_mask);
    }
    if (e != hipSuccess) return fail_hip(e, "kvio_stream_create");
    *out = s;
    return KVIO_OK;
}

kvio_status kvio_stream_destroy(hipStream_t stream) {
    kvio::clear_error();
    if (stream == nullptr) return fail(KVIO_EINVAL, "kvio_stream_destroy: null stream");
    hipError_t e = hipStreamDestroy(stream);
    if (e != hipSuccess) return fail_hip(e, "kvio_stream_destroy");
    return KVIO_OK;
}

kvio_status kvio_host_alloc(size_t bytes, uint32_t flags, void **out) {
    kvio::clear_error();
    if (out == nullptr || bytes == 0) return fail(KVIO_EINVAL, "kvio_host_alloc: null out or zero size");
    if ((flags & ~uint32_t(KVIO_HOST_NONCOHERENT)) != 0)
        return fail(KVIO_EINVAL, "kvio_host_alloc: unknown flags 0x%x", flags);
    unsigned hf = hipHostMallocMapped | hipHostMallocPortable |
                  ((flags & KVIO_HOST_NONCOHERENT) ? hipHostMallocNonCoherent : hipHostMallocCoherent);
    void *ptr = nullptr;
    hipError_t e = hipHostMalloc(&ptr, bytes, hf);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return e == hipErrorOutOfMemory
            ? fail(KVIO_ENOMEM, "kvio_host_alloc: %zu bytes: %s", bytes, hipGetErrorString(e))
            : fail_hip(e, "kvio_host_alloc");
    }
    *out = ptr;
    return KVIO_OK;
}

kvio_status kvio_host_free(void *ptr) {
    kvio::clear_error();
    if (ptr == nullptr) return KVIO_OK;
    hipError_t e = hipHostFree(ptr);
    if (e != hipSuccess) return fail_hip(e, "kvio_host_free");
    return KVIO_OK;
}

}  // extern "C"
