// kvio_pool.h -- what the C ABI layer's translation units share: the pool
// handle, resolved spans, the error helpers and the staged-transfer entry.
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

// A validated span: the device-visible addresses of its chunk and page table.
struct Resolved {
    const uint8_t *host;       // device-visible chunk address
    const int32_t *page_idx;
    int64_t host_tokens;
    int64_t num_tokens;
};

// Fields of a launch that do not depend on its spans.
void common_args(kvio_pool_t p, const Shape &shape, int32_t l0, CopyArgs *a);
// Launch with the workgroup count capped at what the tiles can use.
hipError_t launch_capped(const CopyArgs &a, Direction dir, Shape s, hipStream_t stream);
// KVIO_LAUNCH_STAGED transfers (kvio_staged.cpp).
kvio_status run_staged(kvio_pool_t p, const std::vector<Resolved> &rs, const kvio_span *spans, int32_t n,
                       int32_t l0, int32_t l1, hipStream_t stream, Direction dir, const Shape &shape,
                       const char *fn);

}  // namespace kvio

struct kvio_pool {
    int device;
    int32_t num_layers;
    int32_t num_heads;
    int32_t host_layout;
    int64_t seg_bytes;               // head_dim * elem_bytes
    int32_t page_size;
    int64_t num_slots;
    int64_t row_bytes;
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
