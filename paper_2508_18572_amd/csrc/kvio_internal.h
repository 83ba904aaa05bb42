// kvio_internal.h -- what the C ABI layer hands to the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvio.h"

namespace kvio {

// One cached context as the kernel sees it: the device-visible address of its
// host chunk, its page table and its sizes.
struct SpanArg {
    const uint8_t *host;       // device-visible address of the chunk
    const int32_t *page_idx;   // device page table
    int64_t host_tokens;       // per-(layer, K|V) token stride of the chunk
    int32_t num_tokens;        // tokens to move, < 2^31
    int32_t origin;            // index of the caller's span (error records)
    int32_t page_base;         // context page of this span's first page (error records)
    int32_t pad_;
};

// Kernel arguments of one launch.  Passed by value (kernarg segment), so every
// launch carries its own span table and no device staging buffer is shared
// between calls on different streams.
//
// Work decomposition: a "plane" is one (layer, K|V) of the launch's layer
// range, planes ordered layer-major; a "tile" is up to rows_per_tile
// consecutive token rows of one span in one plane.  tile_prefix[s] is the
// first tile of span s inside a plane, so a plane holds plane_tiles =
// tile_prefix[n_spans] tiles and the launch total_tiles = planes * plane_tiles.
struct CopyArgs {
    uint8_t *const *layers;        // device table: layers[kv * num_layers + l]
    unsigned long long *err;       // device error record (0 = none)
    int64_t row_bytes;             // R
    int64_t plane_tiles;
    int64_t total_tiles;
    int64_t num_pages;             // S / P
    int32_t num_layers;            // L, stride of the layer table
    int32_t layer_begin;
    int32_t page_size;             // P
    int32_t page_shift;            // log2(P) when P is a power of two, else -1
    int32_t vec_per_row;           // V = R / 16
    int32_t vec_shift;             // log2(V) when V is a power of two, else -1
    int32_t vec_step_rows;         // 64 / V: rows a lane's vector index advances per 64 vectors
    int32_t vec_step_cols;         // 64 % V: and columns (carried into the row at V)
    int32_t rows_per_tile;         // 1 .. 64
    int32_t n_spans;               // spans in this launch, 1 .. KVIO_MAX_SPANS_PER_LAUNCH
    int32_t host_layout;           // KVIO_HOST_*
    int32_t num_heads;             // H (head-major chunks)
    int32_t seg_vecs;              // De / 16, 16-byte vectors per head segment (head-major)
    int64_t tile_prefix[KVIO_MAX_SPANS_PER_LAUNCH + 1];
    SpanArg spans[KVIO_MAX_SPANS_PER_LAUNCH];
};

enum Direction { kLoad = 0, kOffload = 1 };

// Resolved launch shape (every field valid).
struct Shape {
    int workgroups;
    int threads;
    int tile_kib;      // 4, 8 or 16: vectors of 16 B per lane per step
    bool nontemporal;
    bool head_major_lds;  // head-major chunks: stage the transpose through LDS
};

// Library defaults for the launch shape, chosen by measurement on MI355X
// (PCIe Gen5 x16 host link), on 16 of the 256 CUs for loads.
//   Load of 32 MiB or more: 16 workgroups x 3 waves, 4 KiB steps (192 KiB in
//   flight).  That saturates the link alone (57.6 GB/s at page size 1, the
//   contiguous memcpy peak) and, beside an offload running on a small quota,
//   leaves the offload's writes room on the link: 97.9 GB/s both ways
//   against 88.6 GB/s with 4 waves per workgroup, whose extra outstanding
//   reads slow both directions.
//   Smaller loads: 16 x 4 waves.  A 2 MiB context is 512 tiles of 4 KiB,
//   which 64 waves share evenly (8 each) and finish ~1 us sooner than 48.
//   Offload: 32 workgroups x 4 waves with 16 KiB steps (57.0 GB/s with the
//   device-scope host stores).
// Two host layouts differ on large transfers (2-4 GiB at page sizes 1 and 16,
// rows of 1-32 KV heads x 128 bf16 dims):
//   Head-major loads with 8 or more KV heads take 8 KiB steps.  A wave step
//   reads step / H bytes from each head's run, and at 4 KiB with 8 heads
//   those 512-byte runs cost up to 15% (57.3 against 48.7-56.9 GB/s at
//   8 KiB); with 16 and 32 heads the two steps are within 0.4%, with 1-4
//   heads 4 KiB is 0.1-0.2 GB/s ahead.  2 MiB contexts keep 4 KiB (51.1
//   against 48.6 GB/s with 4 heads).
//   Page-first offloads take 64 x 4 waves with 8 KiB steps: 56.6-57.1 GB/s
//   against 56.0-57.0 with 128 waves of 16 KiB (the same 2 MiB in flight),
//   ahead at every row width.
constexpr int kDefaultThreads = 256;
constexpr Shape kDefaultLoad = {16, 192, 4, true, true};
constexpr Shape kDefaultLoadHeadMajor = {16, 192, 8, true, true};
constexpr Shape kDefaultLoadSmall = {16, kDefaultThreads, 4, true, true};
constexpr int64_t kSmallLoadBytes = int64_t(32) << 20;
constexpr Shape kDefaultOffload = {32, kDefaultThreads, 16, true, true};
constexpr Shape kDefaultOffloadPageFirst = {64, kDefaultThreads, 8, true, true};

// The default shape of a call that moves `bytes` in direction `dir` between
// the pool (rows of `num_heads` KV heads) and host chunks of layout
// `host_layout` (KVIO_HOST_*).
inline Shape default_shape(int dir, int64_t bytes, int host_layout, int num_heads) {
    if (dir != 0) return host_layout == KVIO_HOST_PAGE_FIRST ? kDefaultOffloadPageFirst : kDefaultOffload;
    if (bytes < kSmallLoadBytes) return kDefaultLoadSmall;
    return host_layout == KVIO_HOST_HEAD_MAJOR && num_heads >= 8 ? kDefaultLoadHeadMajor : kDefaultLoad;
}
// Staged transfers: the scatter / gather between the HBM staging buffer and
// the pool is HBM-bound, so it takes the whole chip (4 GiB of 2 KiB rows at
// page size 1 in 1.75 ms, 2.4 TB/s of payload).
constexpr Shape kDefaultStaged = {1024, kDefaultThreads, 16, true, true};

// Rows per tile for a given step size: one step moves tile_kib KiB per wave.
int rows_per_tile(int64_t row_bytes, int tile_kib);

// Enqueue one copy kernel.  `a` must be fully populated.
hipError_t launch_copy(const CopyArgs &a, Direction dir, const Shape &shape, hipStream_t stream);

// Error record layout: bits 40..63 = span index + 1, bits 0..39 = context page.
constexpr int kErrSpanShift = 40;

}  // namespace kvio
