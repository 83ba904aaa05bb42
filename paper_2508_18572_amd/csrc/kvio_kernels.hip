// kvio_kernels.hip -- GPU-assisted paged-KV transfer kernels for gfx950 (CDNA4).
//
// Strata, Sec. 4.2: one kernel launch replaces many small DMA copies; each
// work item loads a small chunk of the source into registers and streams it
// to the destination, which may be pinned host memory read or written
// directly over the host link.  Sec. 4.2.1 / Fig. 6: the layout change between
// the contiguous host chunk and the layer-first paged pool is one extra
// offset computation per chunk.  Sec. 3.1 (Little's law, X = C * S / L): the
// host link is latency-bound for small transfers, so throughput comes from
// keeping many independent 16-byte requests in flight (C), not from larger
// pages (S).
//
// CDNA4 mapping
//   * A wavefront (64 lanes) owns one tile: up to 64 consecutive token rows of
//     one (layer, K|V) plane of one context.  Host rows of a tile are
//     contiguous, so each wave-wide 16-byte-per-lane access covers 1 KiB of
//     consecutive host bytes (fully coalesced).
//   * Page-offset expansion is wavefront-level: lane r resolves the pool slot
//     of the tile's row r with one coalesced page-table read, masks rows past
//     the end of the context (partial last page) and range-checks the page;
//     every vector then fetches its row's slot from the owning lane with a
//     cross-lane permute (ds_bpermute), so the page table is read once per row.
//   * A step issues all U loads of a wave before any store (U KiB in flight per
//     wave); many waves over few workgroups keep the host link busy while
//     using a small part of the chip (Sec. 4.2: confine the I/O kernel to a
//     few compute units).
//   * Non-temporal loads and stores (Sec. 4.2: bypass the cache to limit
//     pollution of co-running kernels).
//   * Grid-stride over tiles in host-address order, so the waves of a launch
//     sweep a sliding window of consecutive host memory.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvio_internal.h"

namespace kvio {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// Global address space: host-mapped and device memory are both reached with
// global_load / global_store (no flat-address aperture checks).
typedef __attribute__((address_space(1))) u32x4 gvec;

template <bool NT>
__device__ __forceinline__ u32x4 load16(const uint8_t *p) {
    const gvec *q = (const gvec *)(p);
    if constexpr (NT) {
        return __builtin_nontemporal_load(q);
    } else {
        return *q;
    }
}

template <bool NT>
__device__ __forceinline__ void store16(uint8_t *p, u32x4 v) {
    gvec *q = (gvec *)(p);
    if constexpr (NT) {
        __builtin_nontemporal_store(v, q);
    } else {
        *q = v;
    }
}

// Locate global tile g: its plane (layer, K|V), span and first token.  All
// operands are wave-uniform, so this runs on the scalar unit.
struct TileLoc {
    int span;
    int layer;
    int kv;
    int64_t t0;
    int nrows;
};

__device__ __forceinline__ TileLoc locate(const CopyArgs &a, int64_t g) {
    TileLoc L;
    const int64_t plane = g / a.plane_tiles;
    const int64_t w = g - plane * a.plane_tiles;
    int lo = 0, hi = a.n_spans - 1;          // largest s with tile_prefix[s] <= w
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.tile_prefix[mid] <= w) lo = mid; else hi = mid - 1;
    }
    L.span = lo;
    L.layer = a.layer_begin + static_cast<int>(plane >> 1);
    L.kv = static_cast<int>(plane & 1);
    L.t0 = (w - a.tile_prefix[lo]) * a.rows_per_tile;
    const int64_t left = a.spans[lo].num_tokens - L.t0;
    L.nrows = left < a.rows_per_tile ? static_cast<int>(left) : a.rows_per_tile;
    return L;
}

// Lane r < nrows: pool slot of token t0 + r, or -1 for rows past the tile or
// an out-of-range page (recorded once in the error word, never dereferenced).
// Lane r < nrows: pool slot of token t0 + r, or -1 for rows past the tile or
// an out-of-range page (recorded once in the error word, never dereferenced).
__device__ __forceinline__ int lane_slot(const CopyArgs &a, const SpanArg &sp, int span,
                                         int64_t t0, int nrows, int lane) {
    int slot = -1;
    if (lane < nrows) {
        const int64_t t = t0 + lane;
        int64_t cpage, off;
        if (a.page_shift >= 0) {             // wave-uniform branch
            cpage = t >> a.page_shift;
            off = t & (a.page_size - 1);
        } else {
            cpage = t / a.page_size;
            off = t - cpage * a.page_size;
        }
        const int32_t page = sp.page_idx[cpage];
        if (page >= 0 && page < a.num_pages) {
            slot = static_cast<int>(static_cast<int64_t>(page) * a.page_size + off);
        } else {
            const unsigned long long code =
                (static_cast<unsigned long long>(a.span_base + span + 1) << kErrSpanShift) |
                static_cast<unsigned long long>(cpage);
            atomicCAS(a.err, 0ull, code);
        }
    }
    return slot;
}

// Row of vector v of a tile (v / V).
__device__ __forceinline__ int row_of(const CopyArgs &a, int v) {
    return a.vec_shift >= 0 ? (v >> a.vec_shift) : (v / a.vec_per_row);
}

// Loads never carry a mask, so a wave's U loads issue back to back and the
// compiler can count them exactly (precise s_waitcnt before each store).  A
// chunk that must not move (past the end of a tile, or a row whose page was
// out of range) is read from the first bytes of the pool layer instead: in
// bounds, in device memory, and discarded.  Stores run unmasked when every
// chunk of the step is valid (the common case) and guarded otherwise.

// WIDE rows (R a multiple of 1 KiB): each wave-wide access of 64 x 16 B lies
// in one row, so the row, its slot (read from the owning lane with readlane)
// and both base addresses are wave-uniform scalars; each lane adds only its
// own 16-byte offset.
template <int DIR, int U, bool NT>
__device__ __forceinline__ void step_wide(const CopyArgs &a, uint8_t *host, uint8_t *pool, int slot,
                                          int base, int nvec, uint32_t lane_off) {
    const int64_t R = a.row_bytes;
    const int nk = (nvec - base) / 64;      // valid chunks in this step (uniform, >= 1)
    int64_t pool_off[U];                    // chunk k's byte offset in the pool layer, -1 = skip
    bool all_ok = true;
#pragma unroll
    for (int k = 0; k < U; ++k) {
        const int v0 = base + k * 64;
        const int r = row_of(a, v0);
        const int s = __builtin_amdgcn_readlane(slot, r & 63);
        pool_off[k] = (k < nk && s >= 0) ? static_cast<int64_t>(s) * R + (v0 - r * a.vec_per_row) * 16
                                         : -1;
        all_ok = all_ok && pool_off[k] >= 0;
    }
    u32x4 buf[U];
    if (DIR == kLoad) {
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const uint8_t *src = k < nk ? host + static_cast<int64_t>(base + k * 64) * 16 : pool;
            buf[k] = load16<NT>(src + lane_off);
        }
        if (all_ok) {
#pragma unroll
            for (int k = 0; k < U; ++k) store16<NT>(pool + pool_off[k] + lane_off, buf[k]);
        } else {
#pragma unroll
            for (int k = 0; k < U; ++k)
                if (pool_off[k] >= 0) store16<NT>(pool + pool_off[k] + lane_off, buf[k]);
        }
    } else {
#pragma unroll
        for (int k = 0; k < U; ++k)
            buf[k] = load16<NT>(pool + (pool_off[k] >= 0 ? pool_off[k] : 0) + lane_off);
        if (all_ok) {
#pragma unroll
            for (int k = 0; k < U; ++k)
                store16<NT>(host + static_cast<int64_t>(base + k * 64) * 16 + lane_off, buf[k]);
        } else {
#pragma unroll
            for (int k = 0; k < U; ++k)
                if (pool_off[k] >= 0)
                    store16<NT>(host + static_cast<int64_t>(base + k * 64) * 16 + lane_off, buf[k]);
        }
    }
}

// NARROW rows (any R multiple of 16 B): a wave-wide access may span several
// rows, so each lane fetches its row's slot from the owning lane with a
// cross-lane permute (ds_bpermute).
template <int DIR, int U, bool NT>
__device__ __forceinline__ void step_narrow(const CopyArgs &a, uint8_t *host, uint8_t *pool, int slot,
                                            int base, int nvec, int lane) {
    const int64_t R = a.row_bytes;
    const int V = a.vec_per_row;
    int64_t pool_off[U];                    // this lane's vector k offset in the pool layer, -1 = skip
    bool ok = true;
#pragma unroll
    for (int k = 0; k < U; ++k) {
        const int j = base + k * 64 + lane;
        const int r = row_of(a, j);
        const int s = __shfl(slot, r & 63);
        pool_off[k] = (j < nvec && s >= 0) ? static_cast<int64_t>(s) * R + (j - r * V) * 16 : -1;
        ok = ok && pool_off[k] >= 0;
    }
    const bool all_ok = __all(ok);          // wave-uniform
    u32x4 buf[U];
    if (DIR == kLoad) {
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int j = base + k * 64 + lane;
            buf[k] = load16<NT>(j < nvec ? host + static_cast<int64_t>(j) * 16 : pool);
        }
        if (all_ok) {
#pragma unroll
            for (int k = 0; k < U; ++k) store16<NT>(pool + pool_off[k], buf[k]);
        } else {
#pragma unroll
            for (int k = 0; k < U; ++k)
                if (pool_off[k] >= 0) store16<NT>(pool + pool_off[k], buf[k]);
        }
    } else {
#pragma unroll
        for (int k = 0; k < U; ++k) buf[k] = load16<NT>(pool + (pool_off[k] >= 0 ? pool_off[k] : 0));
        if (all_ok) {
#pragma unroll
            for (int k = 0; k < U; ++k)
                store16<NT>(host + static_cast<int64_t>(base + k * 64 + lane) * 16, buf[k]);
        } else {
#pragma unroll
            for (int k = 0; k < U; ++k)
                if (pool_off[k] >= 0) store16<NT>(host + static_cast<int64_t>(base + k * 64 + lane) * 16, buf[k]);
        }
    }
}

// DIR: kLoad (host chunk -> pool) or kOffload (pool -> host chunk).
// U: 16-byte vectors per lane per step (one step = U KiB per wave).
// WIDE: R is a multiple of 1 KiB (see step_wide).
template <int DIR, int U, bool NT, bool WIDE>
__global__ void __launch_bounds__(1024) kvio_copy_kernel(const CopyArgs a) {
    const int lane = threadIdx.x & 63;
    const int waves_per_wg = blockDim.x >> 6;
    const int wave_in_wg = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * waves_per_wg;
    const uint32_t lane_off = static_cast<uint32_t>(lane) * 16u;

#pragma unroll 1
    for (int64_t g = static_cast<int64_t>(blockIdx.x) * waves_per_wg + wave_in_wg;
         g < a.total_tiles; g += nwaves) {
        const TileLoc loc = locate(a, g);
        const SpanArg &sp = a.spans[loc.span];
        uint8_t *pool = a.layers[loc.kv * a.num_layers + loc.layer];
        // First byte of the tile's rows inside the host chunk (layer-major, K then V).
        uint8_t *host = const_cast<uint8_t *>(sp.host) +
                        ((static_cast<int64_t>(loc.layer) * 2 + loc.kv) * sp.host_tokens + loc.t0) *
                            a.row_bytes;
        const int slot = lane_slot(a, sp, loc.span, loc.t0, loc.nrows, lane);
        const int nvec = loc.nrows * a.vec_per_row;
#pragma unroll 1
        for (int base = 0; base < nvec; base += 64 * U) {
            if constexpr (WIDE) {
                step_wide<DIR, U, NT>(a, host, pool, slot, base, nvec, lane_off);
            } else {
                step_narrow<DIR, U, NT>(a, host, pool, slot, base, nvec, lane);
            }
        }
    }
}

int rows_per_tile(int64_t row_bytes, int tile_kib) {
    const int64_t r = (static_cast<int64_t>(tile_kib) * 1024) / row_bytes;
    return r < 1 ? 1 : (r > 64 ? 64 : static_cast<int>(r));
}

template <int DIR, int U, bool NT>
static hipError_t launch_u(const CopyArgs &a, const Shape &s, hipStream_t stream) {
    if (a.vec_per_row % 64 == 0) {
        hipLaunchKernelGGL((kvio_copy_kernel<DIR, U, NT, true>), dim3(s.workgroups), dim3(s.threads),
                           0, stream, a);
    } else {
        hipLaunchKernelGGL((kvio_copy_kernel<DIR, U, NT, false>), dim3(s.workgroups), dim3(s.threads),
                           0, stream, a);
    }
    return hipGetLastError();
}

template <int DIR, bool NT>
static hipError_t launch_nt(const CopyArgs &a, const Shape &s, hipStream_t stream) {
    switch (s.tile_kib) {
        case 4: return launch_u<DIR, 4, NT>(a, s, stream);
        case 8: return launch_u<DIR, 8, NT>(a, s, stream);
        default: return launch_u<DIR, 16, NT>(a, s, stream);
    }
}

hipError_t launch_copy(const CopyArgs &a, Direction dir, const Shape &s, hipStream_t stream) {
    if (dir == kLoad) {
        return s.nontemporal ? launch_nt<kLoad, true>(a, s, stream) : launch_nt<kLoad, false>(a, s, stream);
    }
    return s.nontemporal ? launch_nt<kOffload, true>(a, s, stream)
                         : launch_nt<kOffload, false>(a, s, stream);
}

}  // namespace kvio
