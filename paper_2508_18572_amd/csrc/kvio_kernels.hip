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
//     pollution of co-running kernels); stores into host memory also carry
//     the device-scope policy, which lets them fill the host link.
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

// Stores into pinned host memory (the offload's destination).  With the
// device-scope cache policy (SC1) a wave's 1 KiB stores reach the host link's
// full write rate, the copy engine's 57.0 GB/s, where the compiler's own
// stores (plain or non-temporal) top out 1-2.5% lower.  An SC1 store is
// acknowledged only once it has crossed the link, though, and a wave's next
// step waits for its earlier stores, so SC1 pays only when many bytes are in
// flight (the launcher decides, kSc1MinInflight).  No builtin selects SC1 for
// a global store, so that store is written out; "memory" keeps the compiler
// from moving other memory accesses across it, and the s_nop gives the two
// wait states CDNA3/4 require before a VALU may overwrite the data registers
// of a store wider than 64 bits (the compiler inserts them after its own
// stores but cannot see the store inside the asm).
template <bool NT, bool SC1>
__device__ __forceinline__ void store_host16(uint8_t *p, u32x4 v) {
    if constexpr (SC1) {
        gvec *q = (gvec *)(p);
        if constexpr (NT) {
            asm volatile("global_store_dwordx4 %0, %1, off sc1 nt\n\ts_nop 1" : : "v"(q), "v"(v) : "memory");
        } else {
            asm volatile("global_store_dwordx4 %0, %1, off sc1\n\ts_nop 1" : : "v"(q), "v"(v) : "memory");
        }
    } else {
        store16<NT>(p, v);
    }
}

// Where a tile lies: its span, plane (layer, K|V), first token and row count.
// All of it is wave-uniform, so it is computed on the scalar unit (locate,
// from the wave's TileCursor below).
struct TileLoc {
    int span;
    int layer;
    int kv;
    int64_t t0;
    int nrows;
};

// Largest span s with tile_prefix[s] <= w (binary search over the spans).
__device__ __forceinline__ int span_of(const CopyArgs &a, int64_t w, int lo) {
    int hi = a.n_spans - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.tile_prefix[mid] <= w) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// A wave's position in the tile order: plane, tile inside the plane and the
// span that holds it.  The wave's tiles lie `stride` (the number of waves)
// apart, so the next one is found from the last without a 64-bit division
// or a search in the common case (same plane, same span).
struct TileCursor {
    int64_t plane;
    int64_t w;
    int span;
};

__device__ __forceinline__ TileCursor cursor_at(const CopyArgs &a, int64_t g) {
    TileCursor c;
    c.plane = g / a.plane_tiles;
    c.w = g - c.plane * a.plane_tiles;
    c.span = span_of(a, c.w, 0);
    return c;
}

__device__ __forceinline__ void cursor_advance(const CopyArgs &a, TileCursor &c, int64_t stride) {
    c.w += stride;
    if (c.w >= a.plane_tiles) {                 // into a later plane: its spans start over
        if (c.w < 2 * a.plane_tiles) {
            c.w -= a.plane_tiles;
            ++c.plane;
        } else {
            c.plane += c.w / a.plane_tiles;
            c.w %= a.plane_tiles;
        }
        c.span = span_of(a, c.w, 0);
    } else if (c.span + 1 < a.n_spans && a.tile_prefix[c.span + 1] <= c.w) {
        c.span = span_of(a, c.w, c.span + 1);  // further on in the same plane
    }
}

__device__ __forceinline__ TileLoc locate(const CopyArgs &a, const TileCursor &c) {
    TileLoc L;
    L.span = c.span;
    L.layer = a.layer_begin + static_cast<int>(c.plane >> 1);
    L.kv = static_cast<int>(c.plane & 1);
    L.t0 = (c.w - a.tile_prefix[c.span]) * a.rows_per_tile;
    const int64_t left = a.spans[c.span].num_tokens - L.t0;
    L.nrows = left < a.rows_per_tile ? static_cast<int>(left) : a.rows_per_tile;
    return L;
}

// Lane r < nrows: the pool page that the span's page table gives token t0 + r
// (read only; checked by page_slot), or -1 for rows past the tile.
__device__ __forceinline__ int32_t lane_page(const CopyArgs &a, const SpanArg &sp, int64_t t0, int nrows,
                                             int lane) {
    if (lane >= nrows) return -1;
    const int64_t t = t0 + lane;
    const int64_t cpage = a.page_shift >= 0 ? (t >> a.page_shift) : t / a.page_size;   // wave-uniform branch
    return sp.page_idx[cpage];
}

// Lane r < nrows: pool slot of token t0 + r given its page from lane_page, or
// -1 for rows past the tile or an out-of-range page (recorded once in the
// error word, never dereferenced).
__device__ __forceinline__ int page_slot(const CopyArgs &a, const SpanArg &sp, int64_t t0, int nrows, int lane,
                                         int32_t page) {
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
        if (page >= 0 && page < a.num_pages) {
            slot = static_cast<int>(static_cast<int64_t>(page) * a.page_size + off);
        } else {
            const unsigned long long code =
                (static_cast<unsigned long long>(sp.origin + 1) << kErrSpanShift) |
                static_cast<unsigned long long>(sp.page_base + cpage);
            atomicCAS(a.err, 0ull, code);
        }
    }
    return slot;
}

// Lane r < nrows: pool slot of token t0 + r (lane_page, then page_slot).
__device__ __forceinline__ int lane_slot(const CopyArgs &a, const SpanArg &sp, int64_t t0, int nrows, int lane) {
    return page_slot(a, sp, t0, nrows, lane, lane_page(a, sp, t0, nrows, lane));
}

// Row of vector v of a tile (v / V).
__device__ __forceinline__ int row_of(const CopyArgs &a, int v) {
    return a.vec_shift >= 0 ? (v >> a.vec_shift) : (v / a.vec_per_row);
}

// Row and column of one lane's vectors of a step, which lie 64 apart: from
// vector j to j + 64 the row grows by 64 / V and the column by 64 % V (< V),
// with at most one carry, so only the first vector needs a division.
struct RowCol {
    int r, c;
};

__device__ __forceinline__ RowCol rowcol_of(const CopyArgs &a, int j) {
    const int r = row_of(a, j);
    return {r, j - r * a.vec_per_row};
}

__device__ __forceinline__ void advance64(const CopyArgs &a, RowCol &p) {
    p.r += a.vec_step_rows;
    p.c += a.vec_step_cols;
    if (p.c >= a.vec_per_row) {
        p.c -= a.vec_per_row;
        ++p.r;
    }
}

// Lane r < nrows, page-first host chunk (the layers of one context page stored
// together, Sec. 4.2.1 / Fig. 6): byte offset of row (layer, kv, t0 + r) from
// the chunk start.  Rows of one page are contiguous; pages are L * 2 * P rows
// apart.
__device__ __forceinline__ int64_t lane_host_row_page_first(const CopyArgs &a, int layer, int kv,
                                                            int64_t t0, int nrows, int lane) {
    if (lane >= nrows) return 0;
    const int64_t t = t0 + lane;
    int64_t cpage, off;
    if (a.page_shift >= 0) {
        cpage = t >> a.page_shift;
        off = t & (a.page_size - 1);
    } else {
        cpage = t / a.page_size;
        off = t - cpage * a.page_size;
    }
    return (((cpage * a.num_layers + layer) * 2 + kv) * a.page_size + off) * a.row_bytes;
}

__device__ __forceinline__ int64_t readlane64(int64_t v, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(v), lane);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(static_cast<uint64_t>(v) >> 32), lane);
    return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

// Host layouts handled by kvio_copy_kernel: the tile's rows are one contiguous
// run (token-major chunk), or each row sits at its own offset (page-first).
constexpr int kHostTokenMajor = KVIO_HOST_TOKEN_MAJOR;
constexpr int kHostPageFirst = KVIO_HOST_PAGE_FIRST;

// Loads never carry a mask, so a wave's U loads issue back to back and the
// compiler can count them exactly (precise s_waitcnt before each store).  A
// chunk that must not move (past the end of a tile, or a row whose page was
// out of range) is read from the first bytes of the pool layer instead: in
// bounds, in device memory, and discarded.  Stores run unmasked when every
// chunk of the step is valid (the common case) and guarded otherwise.
//
// `host` is the first byte of the tile's rows for a token-major chunk and the
// chunk start for a page-first chunk, where `hoff` is the lane's row offset.

// WIDE rows (R a multiple of 1 KiB): each wave-wide access of 64 x 16 B lies
// in one row, so the row, its slot (read from the owning lane with readlane)
// and both base addresses are wave-uniform scalars; each lane adds only its
// own 16-byte offset.
template <int DIR, int U, bool NT, bool SC1, int HL>
__device__ __forceinline__ void step_wide(const CopyArgs &a, uint8_t *host, uint8_t *pool, int slot,
                                          int64_t hoff, int base, int nvec, uint32_t lane_off) {
    const int64_t R = a.row_bytes;
    const int nk = (nvec - base) / 64;      // valid chunks in this step (uniform, >= 1)
    int64_t pool_off[U];                    // chunk k's byte offset in the pool layer, -1 = skip
    int64_t host_off[U];                    // chunk k's byte offset from `host`
    bool all_ok = true;
#pragma unroll
    for (int k = 0; k < U; ++k) {
        const int v0 = base + k * 64;
        const int r = row_of(a, v0);
        const int c0 = v0 - r * a.vec_per_row;
        const int s = __builtin_amdgcn_readlane(slot, r & 63);
        pool_off[k] = (k < nk && s >= 0) ? static_cast<int64_t>(s) * R + c0 * 16 : -1;
        if constexpr (HL == kHostPageFirst)
            host_off[k] = readlane64(hoff, r & 63) + c0 * 16;
        else
            host_off[k] = static_cast<int64_t>(v0) * 16;
        all_ok = all_ok && pool_off[k] >= 0;
    }
    u32x4 buf[U];
    if (DIR == kLoad) {
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const uint8_t *src = k < nk ? host + host_off[k] : pool;
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
            for (int k = 0; k < U; ++k) store_host16<NT, SC1>(host + host_off[k] + lane_off, buf[k]);
        } else {
#pragma unroll
            for (int k = 0; k < U; ++k)
                if (pool_off[k] >= 0) store_host16<NT, SC1>(host + host_off[k] + lane_off, buf[k]);
        }
    }
}

// NARROW rows (any R multiple of 16 B): a wave-wide access may span several
// rows, so each lane fetches its row's slot (and, page-first, its row's host
// offset) from the owning lane with a cross-lane permute (ds_bpermute).
// Which vectors move is kept as a bit mask, and token-major host addresses
// are formed where they are used, so at 16 KiB steps the kernel stays inside
// the 128 registers a 1024-thread workgroup leaves each lane: only the U
// loaded vectors and the U pool offsets of one direction are live at once.
template <int DIR, int U, bool NT, bool SC1, int HL>
__device__ __forceinline__ void step_narrow(const CopyArgs &a, uint8_t *host, uint8_t *pool, int slot,
                                            int64_t hoff, int base, int nvec, int lane) {
    static_assert(U <= 32, "the move mask holds one bit per vector");
    const int64_t R = a.row_bytes;
    const RowCol p0 = rowcol_of(a, base + lane);   // this lane's vector 0 of the step
    int sl[U];                              // vector k: the slot of its row
    int64_t host_off[HL == kHostPageFirst ? U : 1];   // page-first: its offset from `host`
    uint32_t moves = 0;                     // bit k: vector k moves
    auto resolve = [&]() {
        RowCol p = p0;
#pragma unroll
        for (int k = 0; k < U; ++k) {
            sl[k] = __shfl(slot, p.r & 63);
            if constexpr (HL == kHostPageFirst)
                host_off[k] = __shfl(static_cast<long long>(hoff), p.r & 63) + p.c * 16;
            moves |= (base + k * 64 + lane < nvec && sl[k] >= 0) ? (1u << k) : 0u;
            advance64(a, p);
        }
    };
    // Byte offset in the pool layer of vector k at row/column p (0 for a
    // vector that does not move: an in-bounds read, discarded).
    auto pool_at = [&](int k, const RowCol &p) -> int64_t {
        return ((moves >> k) & 1u) ? static_cast<int64_t>(sl[k]) * R + p.c * 16 : 0;
    };
    // This lane's vector k of a token-major chunk sits (base + k * 64 + lane) * 16
    // bytes from `host`.
    uint8_t *const host_lane = host + (static_cast<int64_t>(base) + lane) * 16;
    auto host_at = [&](int k) -> uint8_t * {
        if constexpr (HL == kHostPageFirst)
            return host + host_off[k];
        else
            return host_lane + k * 1024;
    };
    constexpr uint32_t kAll = U == 32 ? ~0u : (1u << U) - 1u;
    u32x4 buf[U];
    RowCol p = p0;
    if (DIR == kLoad) {
        // Token-major host reads need no slot, so they go out first and the
        // slots are resolved while they are in flight.
        if constexpr (HL == kHostPageFirst) resolve();
#pragma unroll
        for (int k = 0; k < U; ++k)
            buf[k] = load16<NT>(base + k * 64 + lane < nvec ? host_at(k) : pool);
        if constexpr (HL != kHostPageFirst) resolve();
        if (__all(moves == kAll)) {
#pragma unroll
            for (int k = 0; k < U; ++k) {
                store16<NT>(pool + pool_at(k, p), buf[k]);
                advance64(a, p);
            }
        } else {
#pragma unroll
            for (int k = 0; k < U; ++k) {
                if ((moves >> k) & 1u) store16<NT>(pool + pool_at(k, p), buf[k]);
                advance64(a, p);
            }
        }
    } else {
        resolve();
#pragma unroll
        for (int k = 0; k < U; ++k) {
            buf[k] = load16<NT>(pool + pool_at(k, p));
            advance64(a, p);
        }
        if (__all(moves == kAll)) {
#pragma unroll
            for (int k = 0; k < U; ++k) store_host16<NT, SC1>(host_at(k), buf[k]);
        } else {
#pragma unroll
            for (int k = 0; k < U; ++k)
                if ((moves >> k) & 1u) store_host16<NT, SC1>(host_at(k), buf[k]);
        }
    }
}

// The first tile of a load wave: its host reads are issued before anything
// else (their addresses come from the kernel arguments alone), and the pool
// layer and the slots are resolved while they are in flight, which shortens
// the start of every launch.  Chunks that do not move read the tile's first
// host row instead (in bounds, discarded).  Later tiles run through the step
// functions above.
template <int U, bool NT, bool WIDE, int HL>
__device__ __forceinline__ void first_load_step(const CopyArgs &a, const SpanArg &sp, const TileLoc &loc,
                                                uint8_t *host, uint8_t *&pool, int &slot, int64_t hoff,
                                                int nvec, int lane) {
    const int64_t R = a.row_bytes;
    const uint32_t lane_off = static_cast<uint32_t>(lane) * 16u;
    // Chunk k is (WIDE) vector k * 64 and the 63 after it, all in one row, or
    // this lane's vector k * 64 + lane.  Rows and columns are walked again for
    // the stores rather than kept, so only the U loaded vectors stay live
    // across the slot lookup.
    const RowCol p0 = rowcol_of(a, WIDE ? 0 : lane);
    u32x4 buf[U];
    {
        RowCol p = p0;
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int j = k * 64 + (WIDE ? 0 : lane);
            const bool valid = WIDE ? (k * 64 < nvec) : (j < nvec);
            int64_t host_off;
            if constexpr (HL == kHostPageFirst)
                host_off = (WIDE ? readlane64(hoff, p.r & 63)
                                 : static_cast<int64_t>(__shfl(static_cast<long long>(hoff), p.r & 63))) +
                           p.c * 16;
            else
                host_off = static_cast<int64_t>(j) * 16;
            buf[k] = load16<NT>(valid ? host + host_off + (WIDE ? lane_off : 0u) : host);
            advance64(a, p);
        }
    }
    pool = a.layers[loc.kv * a.num_layers + loc.layer];
    slot = lane_slot(a, sp, loc.t0, loc.nrows, lane);
    RowCol p = p0;
#pragma unroll
    for (int k = 0; k < U; ++k) {
        const int j = k * 64 + (WIDE ? 0 : lane);
        const bool valid = WIDE ? (k * 64 < nvec) : (j < nvec);
        const int s = WIDE ? __builtin_amdgcn_readlane(slot, p.r & 63) : __shfl(slot, p.r & 63);
        if (valid && s >= 0)
            store16<NT>(pool + static_cast<int64_t>(s) * R + p.c * 16 + (WIDE ? lane_off : 0u), buf[k]);
        advance64(a, p);
    }
}

// DIR: kLoad (host chunk -> pool) or kOffload (pool -> host chunk).
// U: 16-byte vectors per lane per step (one step = U KiB per wave).
// NT: non-temporal accesses.  SC1: offload host stores with the device-scope
// policy (store_host16).  WIDE: R is a multiple of 1 KiB (see step_wide).
// HL: host layout.
// Workgroup size bound of the kernels that need more than the 128 VGPRs per
// lane a 1024-thread workgroup leaves (page-first and head-major addressing,
// and loads of narrow token-major rows at 16 KiB steps); their launcher folds
// larger workgroups into more workgroups of this size.
constexpr int kNarrowBound = 256;

template <int DIR, int U, bool WIDE, int HL>
constexpr bool needs_narrow_bound() {
    return HL != KVIO_HOST_TOKEN_MAJOR || (DIR == kLoad && U == 16 && !WIDE);
}

template <int DIR, int U, bool NT, bool SC1, bool WIDE, int HL>
__global__ void __launch_bounds__((needs_narrow_bound<DIR, U, WIDE, HL>() ? kNarrowBound : 1024))
    kvio_copy_kernel(const CopyArgs a) {
    const int lane = threadIdx.x & 63;
    const int waves_per_wg = blockDim.x >> 6;
    const int wave_in_wg = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * waves_per_wg;
    const uint32_t lane_off = static_cast<uint32_t>(lane) * 16u;

    int64_t g = static_cast<int64_t>(blockIdx.x) * waves_per_wg + wave_in_wg;
    bool first = DIR == kLoad;
    TileCursor cur = cursor_at(a, g);
#pragma unroll 1
    for (; g < a.total_tiles; g += nwaves, cursor_advance(a, cur, nwaves)) {
        const TileLoc loc = locate(a, cur);
        const SpanArg &sp = a.spans[loc.span];
        uint8_t *host = const_cast<uint8_t *>(sp.host);
        int64_t hoff = 0;
        if constexpr (HL == kHostPageFirst) {
            hoff = lane_host_row_page_first(a, loc.layer, loc.kv, loc.t0, loc.nrows, lane);
        } else {
            // First byte of the tile's rows (layer-major chunk, K then V).
            host += ((static_cast<int64_t>(loc.layer) * 2 + loc.kv) * sp.host_tokens + loc.t0) * a.row_bytes;
        }
        const int nvec = loc.nrows * a.vec_per_row;
        uint8_t *pool;
        int slot;
        int base = 0;
        if (first) {
            first = false;
            first_load_step<U, NT, WIDE, HL>(a, sp, loc, host, pool, slot, hoff, nvec, lane);
            base = 64 * U;
        } else {
            pool = a.layers[loc.kv * a.num_layers + loc.layer];
            slot = lane_slot(a, sp, loc.t0, loc.nrows, lane);
        }
#pragma unroll 1
        for (; base < nvec; base += 64 * U) {
            if constexpr (WIDE) {
                step_wide<DIR, U, NT, SC1, HL>(a, host, pool, slot, hoff, base, nvec, lane_off);
            } else {
                step_narrow<DIR, U, NT, SC1, HL>(a, host, pool, slot, hoff, base, nvec, lane);
            }
        }
    }
}

// ----------------------------------------------------------------------------
// Head-major host chunk: one contiguous run per (layer, K|V, head), so a pool
// row (token-major [H][D]) gathers H segments of De = R / H bytes from H runs.
// This is the head/token transpose of the layout conversion.
//
// LDS = true: each wave owns one tile of n rows that fits its share of LDS.
// It reads the tile in host order (per head, n * De contiguous bytes), writes
// each 16-byte vector to its pool-order position in the wave's LDS slice,
// and then reads the slice back in pool order, so both sides are long
// contiguous runs: host reads of n * De bytes, pool writes of whole rows.
// Offload runs the same two phases the other way round.
// LDS = false: a direct gather in pool order (each wave-wide access reads
// 64 / (De / 16) head segments of De bytes from as many runs).
//
// Vector numbering inside a tile (Vd = De / 16 vectors per segment,
// V = H * Vd per row):
//   pool order  p = r * V + h * Vd + c     (pool row r, head h, vector c)
//   host order  q = (h * n + r) * Vd + c
// ----------------------------------------------------------------------------
template <int DIR, int U, bool NT, bool SC1, bool LDS>
__global__ void __launch_bounds__(kNarrowBound) kvio_head_major_kernel(const CopyArgs a) {
    extern __shared__ u32x4 lds[];           // U * 64 vectors per wave
    const int lane = threadIdx.x & 63;
    const int waves_per_wg = blockDim.x >> 6;
    const int wave_in_wg = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * waves_per_wg;
    u32x4 *slice = lds + wave_in_wg * (U * 64);
    const int64_t R = a.row_bytes;
    const int V = a.vec_per_row;
    const int Vd = a.seg_vecs;
    const int64_t De = static_cast<int64_t>(Vd) * 16;

    int64_t g0 = static_cast<int64_t>(blockIdx.x) * waves_per_wg + wave_in_wg;
    TileCursor cur = cursor_at(a, g0);
#pragma unroll 1
    for (int64_t g = g0; g < a.total_tiles; g += nwaves, cursor_advance(a, cur, nwaves)) {
        const TileLoc loc = locate(a, cur);
        const SpanArg &sp = a.spans[loc.span];
        uint8_t *pool = a.layers[loc.kv * a.num_layers + loc.layer];
        const int n = loc.nrows;
        // Start of head 0's run at token t0; head h's run is h * host_tokens * De further.
        uint8_t *host = const_cast<uint8_t *>(sp.host) +
                        ((static_cast<int64_t>(loc.layer) * 2 + loc.kv) * a.num_heads * sp.host_tokens + loc.t0) * De;
        const int64_t head_stride = sp.host_tokens * De;
        // The page-table read goes out first.  A load through LDS with steps of
        // 8 KiB or more then issues its host reads and checks the page once
        // they are in flight: the table read is older than them, so waiting
        // for it leaves them outstanding (workload-size head-major loads:
        // 57.2-57.3 against 56.8-56.9 GB/s).  With 4 KiB steps, the small-call
        // default, checking first is faster (2 MiB contexts: 51.0 against
        // 48.8-49.2 GB/s), and the other paths need the slot before their
        // first access.
        constexpr bool kLateSlot = LDS && DIR == kLoad && U >= 8;
        const int32_t page = lane_page(a, sp, loc.t0, n, lane);
        int slot = kLateSlot ? -1 : page_slot(a, sp, loc.t0, n, lane, page);
        const int nvec = n * V;
#pragma unroll 1
        for (int base = 0; base < nvec; base += 64 * U) {
            if constexpr (LDS) {
                // The whole tile is one step (rows_per_tile keeps n * R <= U KiB).
                if (DIR == kLoad) {
                    u32x4 buf[U];
                    int pos[U];                             // pool-order position of vector q, -1 = none
#pragma unroll
                    for (int k = 0; k < U; ++k) {          // host order, contiguous per head
                        const int q = k * 64 + lane;
                        const int hr = q / Vd;              // h * n + r
                        const int h = hr / n;
                        const int r = hr - h * n;
                        const int c = q - hr * Vd;
                        pos[k] = q < nvec ? r * V + h * Vd + c : -1;
                        buf[k] = load16<NT>(q < nvec ? host + h * head_stride + (static_cast<int64_t>(r) * Vd + c) * 16
                                                     : pool);
                    }
                    slot = page_slot(a, sp, loc.t0, n, lane, page);
                    // All U loads are in flight before the first LDS write waits for one.
#pragma unroll
                    for (int k = 0; k < U; ++k)
                        if (pos[k] >= 0) slice[pos[k]] = buf[k];
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                    __builtin_amdgcn_wave_barrier();
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
                    for (int k = 0; k < U; ++k) {          // pool order, whole rows
                        const int p = k * 64 + lane;
                        const int r = p / V;
                        const int s = __shfl(slot, r & 63);
                        if (p < nvec && s >= 0)
                            store16<NT>(pool + static_cast<int64_t>(s) * R + (p - r * V) * 16, slice[p]);
                    }
                } else {
                    u32x4 buf[U];
#pragma unroll
                    for (int k = 0; k < U; ++k) {          // pool order, whole rows
                        const int p = k * 64 + lane;
                        const int r = p / V;
                        const int s = __shfl(slot, r & 63);
                        buf[k] = load16<NT>(pool + (p < nvec && s >= 0
                                                        ? static_cast<int64_t>(s) * R + (p - r * V) * 16
                                                        : 0));
                    }
#pragma unroll
                    for (int k = 0; k < U; ++k)
                        if (k * 64 + lane < nvec) slice[k * 64 + lane] = buf[k];
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                    __builtin_amdgcn_wave_barrier();
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
                    for (int k = 0; k < U; ++k) {          // host order, contiguous per head
                        const int q = k * 64 + lane;
                        const int hr = q / Vd;
                        const int h = hr / n;
                        const int r = hr - h * n;
                        const int c = q - hr * Vd;
                        const int s = __shfl(slot, r & 63);
                        if (q < nvec && s >= 0)
                            store_host16<NT, SC1>(host + h * head_stride + (static_cast<int64_t>(r) * Vd + c) * 16,
                                        slice[r * V + h * Vd + c]);
                    }
                }
                // The slice is reused by the wave's next tile.
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            } else {
                u32x4 buf[U];
                int64_t pool_off[U];
                int64_t host_off[U];
#pragma unroll
                for (int k = 0; k < U; ++k) {              // pool order
                    const int p = base + k * 64 + lane;
                    const int r = p / V;
                    const int hv = p - r * V;
                    const int h = hv / Vd;
                    const int c = hv - h * Vd;
                    const int s = __shfl(slot, r & 63);
                    pool_off[k] = (p < nvec && s >= 0) ? static_cast<int64_t>(s) * R + hv * 16 : -1;
                    host_off[k] = h * head_stride + (static_cast<int64_t>(r) * Vd + c) * 16;
                }
                if (DIR == kLoad) {
#pragma unroll
                    for (int k = 0; k < U; ++k)
                        buf[k] = load16<NT>(base + k * 64 + lane < nvec ? host + host_off[k] : pool);
#pragma unroll
                    for (int k = 0; k < U; ++k)
                        if (pool_off[k] >= 0) store16<NT>(pool + pool_off[k], buf[k]);
                } else {
#pragma unroll
                    for (int k = 0; k < U; ++k) buf[k] = load16<NT>(pool + (pool_off[k] >= 0 ? pool_off[k] : 0));
#pragma unroll
                    for (int k = 0; k < U; ++k)
                        if (pool_off[k] >= 0) store_host16<NT, SC1>(host + host_off[k], buf[k]);
                }
            }
        }
    }
}

int rows_per_tile(int64_t row_bytes, int tile_kib) {
    const int64_t r = (static_cast<int64_t>(tile_kib) * 1024) / row_bytes;
    return r < 1 ? 1 : (r > 64 ? 64 : static_cast<int>(r));
}

// Offloads whose launch keeps at least this many bytes in flight (waves x
// step) store into host memory with the SC1 policy: enough to cover the
// longer acknowledgement of those stores, so the link runs at its full write
// rate (57.0 against 55.7 GB/s at the default 128 waves x 16 KiB).  Smaller
// quotas (16 waves x 4 KiB: 27 against 44 GB/s) keep the plain policy.  A
// build may move the threshold (-DKVIO_SC1_MIN_INFLIGHT=0 stores every
// offload with SC1; a huge value never does), which is how both policies
// were measured over launch shapes.
#ifndef KVIO_SC1_MIN_INFLIGHT
#define KVIO_SC1_MIN_INFLIGHT (int64_t(512) << 10)
#endif
constexpr int64_t kSc1MinInflight = KVIO_SC1_MIN_INFLIGHT;

template <int DIR, int U, bool NT, bool SC1>
static hipError_t launch_policy(const CopyArgs &a, dim3 grid, dim3 block, const Shape &s, hipStream_t stream) {
    const bool wide = a.vec_per_row % 64 == 0;
    switch (a.host_layout) {
        case kHostPageFirst:
            if (wide)
                hipLaunchKernelGGL((kvio_copy_kernel<DIR, U, NT, SC1, true, kHostPageFirst>), grid, block, 0, stream,
                                   a);
            else
                hipLaunchKernelGGL((kvio_copy_kernel<DIR, U, NT, SC1, false, kHostPageFirst>), grid, block, 0, stream,
                                   a);
            break;
        case KVIO_HOST_HEAD_MAJOR:
            if (s.head_major_lds)
                hipLaunchKernelGGL((kvio_head_major_kernel<DIR, U, NT, SC1, true>), grid, block,
                                   static_cast<size_t>(block.x / 64) * U * 1024, stream, a);
            else
                hipLaunchKernelGGL((kvio_head_major_kernel<DIR, U, NT, SC1, false>), grid, block, 0, stream, a);
            break;
        default:
            if (wide)
                hipLaunchKernelGGL((kvio_copy_kernel<DIR, U, NT, SC1, true, kHostTokenMajor>), grid, block, 0, stream,
                                   a);
            else
                hipLaunchKernelGGL((kvio_copy_kernel<DIR, U, NT, SC1, false, kHostTokenMajor>), grid, block, 0,
                                   stream, a);
    }
    return hipGetLastError();
}

template <int DIR, int U, bool NT>
static hipError_t launch_u(const CopyArgs &a, const Shape &s, hipStream_t stream) {
    dim3 grid(s.workgroups), block(s.threads);
    const bool wide = a.vec_per_row % 64 == 0;
    const bool narrow_bound = a.host_layout != KVIO_HOST_TOKEN_MAJOR ||
                              (wide ? needs_narrow_bound<DIR, U, true, kHostTokenMajor>()
                                    : needs_narrow_bound<DIR, U, false, kHostTokenMajor>());
    if (narrow_bound && s.threads > kNarrowBound) {
        grid = dim3(static_cast<unsigned>(int64_t(s.workgroups) * s.threads / kNarrowBound));
        block = dim3(kNarrowBound);
    }
    if constexpr (DIR == kOffload && NT) {
        const int64_t inflight = int64_t(grid.x) * (block.x / 64) * U * 1024;
        if (inflight >= kSc1MinInflight) return launch_policy<DIR, U, NT, true>(a, grid, block, s, stream);
    }
    return launch_policy<DIR, U, NT, false>(a, grid, block, s, stream);
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
