// kvio_pool.h -- what the C ABI layer's translation units share: the pool
// geometry and handle, resolved spans, argument checks, launch helpers, the
// error helpers and the staged-transfer entry.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "kvio.h"
#include "kvio_internal.h"

namespace kvio {

// The staging buffer is split into this many slots so the copy engine fills
// (drains) one while the kernel scatters (gathers) another.
constexpr int kStageSlots = 4;

// Record a thread-local error text (printf format) and return `st`.
kvio_status fail(kvio_status st, const char *fmt, ...);
kvio_status fail_hip(hipError_t e, const char *what);
// Empty the thread-local error text.
void clear_error();

// What a transfer needs to know of a pool besides its layer addresses.
struct PoolGeom {
    int32_t num_layers;
    int32_t num_heads;
    int32_t host_layout;
    int32_t page_size;
    int64_t num_slots;
    int64_t row_bytes;
    int64_t seg_bytes;               // head_dim * elem_bytes
};

// A validated span: the device-visible addresses of its chunk and page table.
struct Resolved {
    const uint8_t *host;       // device-visible chunk address
    const int32_t *page_idx;
    int64_t host_tokens;
    int64_t num_tokens;
};

// Check a pool description's sizes, layout and launch shapes (not its layer
// pointers) and fill in its geometry.
kvio_status check_desc(const kvio_pool_desc *d, const char *fn, PoolGeom *g);
// Check every layer pointer of a checked description (device memory of at
// least S * R bytes, 16-byte aligned) and write their device addresses to
// layers[kv * L + l] (2 * L entries).
kvio_status resolve_layers(const kvio_pool_desc *d, const PoolGeom &g, const char *fn, uint8_t **layers);
// Validate n spans and the layer range; write the resolved spans to
// out[0 .. n).  Nothing is enqueued.
kvio_status validate_spans(const PoolGeom &g, const kvio_span *spans, int32_t n, int32_t l0, int32_t l1,
                           const char *fn, Resolved *out);
// Validate a launch shape; fill in a shape from it and the defaults.
kvio_status check_launch(const kvio_launch &l, const char *which);
Shape resolve(const kvio_launch &l, const Shape &def);
// The kernel path's shape for a pool (head-major tiles too wide for LDS gather directly).
Shape kernel_shape(const PoolGeom &g, const kvio_launch &l, const Shape &def);
// Device-visible address of [p, p + bytes) (see kvio_api.cpp).
kvio_status device_view(const void *p, uint64_t bytes, bool want_device_memory, const char *what,
                        const uint8_t **out);
// Fields of a launch that do not depend on its spans.
void common_args(const PoolGeom &g, uint8_t *const *layers, unsigned long long *err, const Shape &shape,
                 int32_t l0, CopyArgs *a);
void common_args(kvio_pool_t p, const Shape &shape, int32_t l0, CopyArgs *a);
// Launch with the workgroup count capped at what the tiles can use.
hipError_t launch_capped(const CopyArgs &a, Direction dir, Shape s, hipStream_t stream);
// Enqueue the kernel launches of a transfer of validated spans, one launch
// per KVIO_MAX_SPANS_PER_LAUNCH spans; `layers` (device table of 2 * L layer
// addresses) and `err` (device error word) are what the kernels read and
// record into.  Launches with no rows are skipped.
kvio_status launch_spans(const PoolGeom &g, uint8_t *const *layers, unsigned long long *err, const Resolved *rs,
                         int32_t n, int32_t l0, int32_t l1, Direction dir, const Shape &shape, hipStream_t stream,
                         const char *fn);
// KVIO_LAUNCH_STAGED transfers (kvio_staged.cpp).
kvio_status run_staged(kvio_pool_t p, const std::vector<Resolved> &rs, const kvio_span *spans, int32_t n,
                       int32_t l0, int32_t l1, hipStream_t stream, Direction dir, const Shape &shape,
                       const char *fn);

}  // namespace kvio

struct kvio_pool {
    int device;
    kvio::PoolGeom g;
    std::vector<uint8_t *> layers;   // host copy: [kv * L + l]
    uint8_t **d_layers;              // device copy
    unsigned long long *d_err;       // device error record
    kvio_launch load_launch;
    kvio_launch offload_launch;
    // KVIO_LAUNCH_STAGED, per direction: HBM staging split into kStageSlots
    // slots, a side stream for the scatter / gather kernels, and the events
    // that hand slots between it and the caller's stream.
    uint8_t *stage[2];
    int64_t slot_bytes;
    hipStream_t side_stream[2];
    hipEvent_t ev_filled[2][kvio::kStageSlots];
    hipEvent_t ev_free[2][kvio::kStageSlots];
    hipEvent_t ev_start[2];
    hipEvent_t ev_done[2];
};
