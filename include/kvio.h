/*
 * kvio.h -- C ABI of libkvio.so: paged-KV transfers between pinned host memory
 * and a GPU's paged KV pool, on AMD Instinct MI355X (gfx950).
 *
 * The operation is Strata's GPU-assisted I/O (Sec. 4.2, "Efficient KV Cache
 * I/O"): instead of one DMA copy per small page, one kernel launch whose
 * wavefronts each read a small chunk of the source into registers and stream
 * it to the destination.  The source may be pinned host memory that the GPU
 * reads directly over the host link.  Because every work item computes its
 * own addresses, the kernel converts layouts on the fly (Sec. 4.2.1, Fig. 6):
 * the host keeps one contiguous, transfer-friendly chunk per cached context,
 * while the GPU keeps the compute-friendly, layer-first paged pool of Sec. 2.2.
 *
 * Layouts (R = num_kv_heads * head_dim * elem_bytes = bytes of one token row,
 * P = page_size tokens, S = num_slots token slots per per-layer pool):
 *   pool  : per layer l, one K array and one V array of S rows of R bytes,
 *           token-major ([S][H][D]); slot s belongs to pool page s / P.
 *   host  : one chunk per cached context, layer-major then K before V, then
 *           token-major: row (l, kv, t) starts at byte
 *           ((l * 2 + kv) * host_tokens + t) * R of the chunk (kv 0 = K, 1 = V).
 *   pages : page_idx[j] is the pool page that holds context page j, so token
 *           t lives in slot page_idx[t / P] * P + t % P.  At P = 1 the page
 *           table is the slot list.
 *
 * Semantics of a transfer of context tokens [0, num_tokens) over the layer
 * range [layer_begin, layer_end):
 *   load    : pool row slot(t) of layer l, K or V  := host row (l, kv, t)
 *   offload : host row (l, kv, t) := pool row slot(t)
 * No other pool byte (load) or host byte (offload) is written.  The tail of a
 * partial last page is left untouched.
 *
 * Conventions
 *   - Every call returns kvio_status (0 = OK, negative = error); no exception
 *     crosses the ABI.  On error kvio_last_error() holds a thread-local text.
 *   - Transfers are asynchronous on the given stream (NULL = the default
 *     stream); completion follows stream order.  Validation errors are
 *     reported synchronously and enqueue nothing.  A HIP call that fails
 *     inside the library is reported by the status and kvio_last_error();
 *     the runtime's per-thread last error is cleared, so the caller's next
 *     HIP call does not report it again.  The transfer calls enqueue
 *     no memset and allocate nothing, so they can be captured into a HIP
 *     graph (a staged call forks its side stream from the captured stream and
 *     joins it back through events).
 *   - The caller owns every buffer: pools, host chunks, page tables.  The
 *     library owns only the pool handle (a device copy of the layer-pointer
 *     table, a device error record and, for directions launched with
 *     KVIO_LAUNCH_STAGED, HBM staging slots with a side stream and events).
 *   - A pool handle is immutable after creation and may be used from several
 *     threads and streams at once.  Transfers that run concurrently must write
 *     disjoint bytes (and staged transfers of one direction must not overlap);
 *     a load whose page tables name one pool slot twice leaves each 16-byte
 *     piece of that slot holding the same piece of one of the rows named
 *     for it (unspecified which; the pieces may come from different rows).
 *   - Page indices are range-checked on the device at no measurable cost: a
 *     row whose page lies outside [0, S / P) is skipped, never dereferenced,
 *     and the first such (span, context page) is recorded for kvio_check().
 */
#ifndef KVIO_H
#define KVIO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same opaque handle types as the HIP runtime API (redeclaring an identical
 * typedef is legal in C11 and C++). */
typedef struct ihipStream_t *hipStream_t;
typedef struct ihipEvent_t *hipEvent_t;

typedef enum kvio_status {
    KVIO_OK = 0,
    KVIO_EINVAL = -1,      /* null pointer, bad size, bad layer range, num_tokens > host_tokens,
                              buffer smaller than the transfer reaches                        */
    KVIO_ERANGE = -2,      /* kvio_check: a page index was outside [0, S / P)                */
    KVIO_EALIGN = -3,      /* R, a pool layer or a host chunk not 16-byte aligned            */
    KVIO_ENOTMAPPED = -4,  /* host chunk not accessible from the device (e.g. plain malloc)  */
    KVIO_EHIP = -5,        /* a HIP runtime call failed; its message is in kvio_last_error  */
    KVIO_ENOMEM = -6,      /* allocation failed                                              */
    KVIO_EIO = -7          /* a disk read or write failed or came up short (errno in the text) */
} kvio_status;

/* Host chunk layouts (kvio_pool_desc.host_layout).  All hold the same rows;
 * they differ in where row (l, kv, t) -- head-major: its head h segment of
 * De = head_dim * elem_bytes bytes -- starts inside one context's chunk:
 *   KVIO_HOST_TOKEN_MAJOR  layer-major, K before V, token-major (above):
 *                          ((l*2 + kv)*host_tokens + t) * R
 *   KVIO_HOST_PAGE_FIRST   the paper's transfer-friendly layout (Sec. 4.2.1,
 *                          Fig. 6): all layers of one context page together,
 *                          [page][L][2][P][H][D]; host_tokens must be a
 *                          multiple of P:  (((t/P)*L + l)*2 + kv)*P*R + (t%P)*R
 *   KVIO_HOST_HEAD_MAJOR   one run per (layer, K|V, head), [L][2][H][T][D]:
 *                          (((l*2 + kv)*H + h)*host_tokens + t) * De;
 *                          De must be a multiple of 16.  Converting it to
 *                          the token-major pool is a head/token transpose,
 *                          staged through LDS unless KVIO_LAUNCH_NO_LDS. */
#define KVIO_HOST_TOKEN_MAJOR 0
#define KVIO_HOST_PAGE_FIRST 1
#define KVIO_HOST_HEAD_MAJOR 2

/* Launch shaping (Sec. 4.2: a small number of large workgroups keeps the I/O
 * kernel on few compute units; cache bypass limits pollution).  Zero fields
 * take the library defaults.  Results never depend on these. */
#define KVIO_LAUNCH_CACHED 0x1     /* plain loads/stores instead of non-temporal ones */
#define KVIO_LAUNCH_NO_LDS 0x2     /* head-major chunks: gather directly, no LDS staging */
/* KVIO_LAUNCH_STAGED (token-major and head-major chunks): instead of
 * wavefronts reading (writing) the pinned chunk across the host link, the
 * copy engine moves the chunk's contiguous runs to (from) an HBM staging buffer
 * of the pool handle with hipMemcpyAsync, and a kernel scatters (gathers) the
 * rows between the staging buffer and the paged pool -- the layout conversion
 * then runs at HBM speed on the whole chip for short bursts, and the long
 * host-link phase occupies no compute unit.  The staging buffer is split into
 * 4 slots: the copies run on the call's stream while the kernels run on a
 * side stream the pool handle owns for that direction, each slot handed
 * between them by events, so the copy engine never waits for a kernel that
 * is queued behind other work.  The call keeps stream order: it starts after
 * the work already on the call's stream, and the call's stream has passed
 * all of its work (a load: its last scatter) when the call completes in
 * stream order.  The launch fields shape the scatter / gather kernel (defaults
 * 1024 x 256, 16 KiB steps).  A call that moves less than 64 MiB in total
 * (or less than one slot, if slots are smaller) runs on the kernel path
 * (default shape) instead: staging cannot amortise its per-copy and hand-over
 * costs on small transfers.  Calls in one direction on one handle share that
 * direction's staging, so they must not overlap (same stream, or ordered by
 * events).  An out-of-range page is still skipped and reported by kvio_check,
 * but a staged offload then leaves unspecified bytes in the host rows of its
 * tokens. */
#define KVIO_LAUNCH_STAGED 0x4
typedef struct kvio_launch {
    int32_t workgroups;   /* workgroups per launch, >= 1; 0 = default                       */
    int32_t threads;      /* threads per workgroup: multiple of 64 in [64, 1024]; 0 = default */
    int32_t tile_kib;     /* bytes each wavefront moves per step, in KiB: 4, 8 or 16; 0 = default */
    int32_t flags;        /* KVIO_LAUNCH_* bits                                              */
} kvio_launch;

/* Describes caller-owned device memory; copied by kvio_pool_create.  The
 * memory is the GPU's paged KV cache (Sec. 2.2: KV states kept in fixed-size
 * pages of token slots, one pool per layer), addressed through a page table
 * that the caller's cache index maintains (Sec. 4.1: the HiRadixTree maps
 * cached tokens to pool indices; Sec. 4.2.1: the pool is layer-first). */
typedef struct kvio_pool_desc {
    int32_t num_layers;       /* L >= 1                                                  */
    int32_t num_kv_heads;     /* H >= 1                                                  */
    int32_t head_dim;         /* D >= 1                                                  */
    int32_t elem_bytes;       /* bytes per element (2 for fp16/bf16); R % 16 must be 0  */
    int32_t page_size;        /* P >= 1 tokens                                           */
    int32_t host_layout;      /* KVIO_HOST_TOKEN_MAJOR | _PAGE_FIRST | _HEAD_MAJOR       */
    int64_t num_slots;        /* S token slots per per-layer pool, S % P == 0, S < 2^31 */
    void *const *k_layers;    /* host array of L device pointers, each S * R bytes       */
    void *const *v_layers;    /* host array of L device pointers, each S * R bytes       */
    kvio_launch load_launch;  /* launch shape of load kernels                            */
    kvio_launch offload_launch; /* launch shape of offload kernels                       */
    int64_t staging_bytes;    /* HBM staging per direction with KVIO_LAUNCH_STAGED: 4 slots
                                 of staging_bytes / 4 (rounded down to 16 B), each >= 2 * P
                                 * R; 0 = 4 GiB.  Allocated by kvio_pool_create, with a
                                 side stream and events, only for staged directions.      */
} kvio_pool_desc;

typedef struct kvio_pool *kvio_pool_t;

/* One cached context (one "span" of a batched transfer): its contiguous host
 * chunk (Sec. 4.2.1: the host keeps each context in one transfer-friendly
 * chunk) and the page table that places its tokens in the pool (Sec. 2.2 paged
 * KV; Sec. 4.1: the cache index resolves a context to pool pages).  A batched
 * call moves several contexts at once, as the scheduler issues one load per
 * batch (Sec. 4.3.2). */
typedef struct kvio_span {
    void *host;               /* pinned, device-mapped host chunk (or device memory),
                                 16-byte aligned, L * 2 * host_tokens * R bytes        */
    int64_t host_tokens;      /* token capacity of the chunk: its per-(layer, K|V) stride */
    int64_t num_tokens;       /* move context tokens [0, num_tokens); <= host_tokens     */
    const int32_t *page_idx;  /* DEVICE int32[ceil(num_tokens / P)]                      */
} kvio_span;

/* Most spans one kernel launch carries; a larger batch is split into
 * consecutive launches on the same stream. */
#define KVIO_MAX_SPANS_PER_LAUNCH 64

/* Create a pool handle on the current device (Sec. 2.2 / Sec. 4.1: the paged
 * pool and its page addressing that every transfer names).  Checks that every layer
 * pointer is device memory of at least S * R bytes and 16-byte aligned
 * (KVIO_EINVAL / KVIO_EALIGN), then allocates the handle (KVIO_ENOMEM /
 * KVIO_EHIP).  *out is set only on success. */
kvio_status kvio_pool_create(const kvio_pool_desc *desc, kvio_pool_t *out);

/* Free the handle (waiting for its own side streams first).  The caller must
 * have synchronised every stream that still runs a transfer on it.  NULL is
 * accepted. */
kvio_status kvio_pool_destroy(kvio_pool_t pool);

/* Load (Sec. 4.2): move tokens [0, num_tokens) of each of the n_spans contexts,
 * layers [layer_begin, layer_end), from the host chunks into the pool, in one
 * launch per KVIO_MAX_SPANS_PER_LAUNCH spans.  Host reads are sequential per
 * (layer, K|V); pool writes are scattered by page.  n_spans == 0 or all
 * num_tokens == 0 enqueues nothing and returns KVIO_OK. */
kvio_status kvio_load(kvio_pool_t pool, const kvio_span *spans, int32_t n_spans,
                      int32_t layer_begin, int32_t layer_end, hipStream_t stream);

/* Offload (Sec. 4.1 backup to lower tiers; Sec. 4.2 I/O kernel): the inverse
 * gather, pool rows into the contiguous host chunks.  Host bytes of rows
 * t >= num_tokens are not written.  Duplicate page indices are allowed. */
kvio_status kvio_offload(kvio_pool_t pool, const kvio_span *spans, int32_t n_spans,
                         int32_t layer_begin, int32_t layer_end, hipStream_t stream);

/* Layer-wise load (Sec. 4.1: the executor waits until a layer's KV cache is
 * present before computing that layer; Sec. 3.2 / Sec. 4.2.1 layer-wise
 * overlap): kvio_load of the single layer `layer` on `stream`, then, if `done`
 * is not NULL, hipEventRecord(done, stream), also when there was nothing to
 * move.  A compute stream that waits on `done` may use layer `layer`. */
kvio_status kvio_load_layer(kvio_pool_t pool, const kvio_span *spans, int32_t n_spans,
                            int32_t layer, hipStream_t stream, hipEvent_t done);

/* For callers that cannot allocate -- code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc: kvio_load without a pool
 * handle, allocating nothing (no hipMalloc, hipFree or other allocating
 * call; no host-to-device copy).  `desc` describes the pool as for
 * kvio_pool_create and is checked the same way on every call (staged loads,
 * which need staging memory, are refused); spans, layer range, stream and
 * result are those of kvio_load.  The device memory a pool handle would own
 * -- the table of layer addresses and the error word -- lives in a static
 * 4 KiB device array of the library (one per GPU, held until the process
 * ends), so the call takes at most KVIO_NOALLOC_MAX_LAYERS layers and at most
 * KVIO_MAX_SPANS_PER_LAUNCH spans (KVIO_EINVAL beyond either).  Each call
 * first enqueues a one-workgroup kernel that writes the layer table and
 * clears the error word, then the load kernel.  Every call on a GPU shares
 * that array: calls that overlap on one GPU (on different streams, or from
 * different threads) race and must be ordered by the caller.  A page index
 * outside [0, S / P) is skipped, never dereferenced, and not reported (use a
 * pool handle and kvio_check to diagnose one).  n_spans == 0 or all
 * num_tokens == 0 enqueues nothing. */
#define KVIO_NOALLOC_MAX_LAYERS 128
kvio_status kvio_load_noalloc(const kvio_pool_desc *desc, const kvio_span *spans, int32_t n_spans,
                              int32_t layer_begin, int32_t layer_end, hipStream_t stream);

/* The library's own error reporting; no passage of the paper defines it.
 * Synchronise the device, then report and clear the device error record:
 * KVIO_ERANGE (with the span and context page in kvio_last_error) if an
 * earlier transfer met an out-of-range page index, else KVIO_OK. */
kvio_status kvio_check(kvio_pool_t pool);

/* Naive baseline (Sec. 3.1, the DMA path of the baselines): one
 * hipMemcpyAsync per contiguous (page, layer, K|V) segment of up to P rows,
 * all on `stream`.  Same arguments and result as kvio_load / kvio_offload.
 * Page indices are validated on the host first (KVIO_ERANGE), so the
 * page tables must be readable from the host here: host memory or pinned
 * memory, or device memory (copied to the host first, synchronously). */
kvio_status kvio_naive_load(kvio_pool_t pool, const kvio_span *spans, int32_t n_spans,
                            int32_t layer_begin, int32_t layer_end, hipStream_t stream);
kvio_status kvio_naive_offload(kvio_pool_t pool, const kvio_span *spans, int32_t n_spans,
                               int32_t layer_begin, int32_t layer_end, hipStream_t stream);

/* One contiguous hipMemcpyAsync(dst, src, bytes, hipMemcpyDefault, stream):
 * the host-link peak that the transfers are measured against. */
kvio_status kvio_memcpy(void *dst, const void *src, size_t bytes, hipStream_t stream);

/* One contiguous copy of `bytes` from src to dst by a plain kernel (16-byte
 * vectors; 16 workgroups of 192 threads into device memory, 32 of 256 into
 * host memory; enqueued on `stream`), in either
 * direction between pinned host memory (kvio_host_alloc) and device memory,
 * or within either.  It is the rate compute units reach on the host link with
 * no paging at all: the ceiling of the kernel path, beside kvio_memcpy's
 * copy-engine rate.  Defined by no passage of the paper; a measurement aid.
 * bytes must be a multiple of 16 and both pointers 16-byte aligned
 * (KVIO_EINVAL otherwise), and each range must lie whole inside one
 * allocation the device can reach (KVIO_ENOTMAPPED for memory the runtime
 * does not know, KVIO_EINVAL for a range past its allocation's end); all
 * checked before anything is enqueued.  Zero bytes is a no-op.  The caller owns both buffers and keeps them alive until the copy
 * has completed on `stream`. */
kvio_status kvio_kernel_memcpy(void *dst, const void *src, size_t bytes, hipStream_t stream);

/* Pinned, device-mapped host memory for host chunks (hipHostMalloc).
 * flags: KVIO_HOST_COHERENT (fine-grained, the default) or
 * KVIO_HOST_NONCOHERENT (coarse-grained).  The returned pointer is also the
 * device address.  Free with kvio_host_free. */
#define KVIO_HOST_COHERENT 0x0
#define KVIO_HOST_NONCOHERENT 0x1
kvio_status kvio_host_alloc(size_t bytes, uint32_t flags, void **out);
kvio_status kvio_host_free(void *ptr);

/* Stream for transfers or for the kernels they run beside (Sec. 4.2: the
 * I/O kernel is confined to a small part of the GPU so that co-running
 * compute is not disturbed).  With mask_words > 0 the stream's kernels run
 * only on the compute units whose bits are set in cu_mask (bit b of word w =
 * CU 32 * w + b, hipExtStreamCreateWithCUMask); a transfer stream and a
 * compute stream with complementary masks never wait for each other's
 * workgroups.  With mask_words == 0 it is an ordinary non-blocking stream.
 * Streams keep the default priority.  Destroy with kvio_stream_destroy after
 * synchronising it. */
kvio_status kvio_stream_create(const uint32_t *cu_mask, uint32_t mask_words, hipStream_t *out);
kvio_status kvio_stream_destroy(hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Storage tier (Sec. 4.2.1): cached contexts kept on disk are prefetched
 * into pinned host chunks, from where kvio_load moves them to the pool; the
 * reverse (kvio_disk_store_pages) backs a host chunk up to disk.  The paper
 * stores host and disk copies page-first, so every page is one large
 * contiguous transfer instead of L * 2 small ones (Fig. 12).
 *
 * A disk store is one file of KV pages of one model, P tokens per page,
 * R = H * D * elem_bytes bytes per row, in one of two layouts:
 *   KVIO_DISK_PAGE_FIRST   [disk page][L][2][P][H][D]: row (l, kv, o) of disk
 *                          page p at byte ((p*L + l)*2 + kv)*P*R + o*R
 *   KVIO_DISK_LAYER_FIRST  the pool's own order, [L][2][disk page][P][H][D]:
 *                          at ((l*2 + kv)*num_disk_pages + p)*P*R + o*R
 * Context page j (tokens [j*P, j*P + P)) lives in disk page disk_pages[j].
 * Transfers copy whole pages: the host chunk (token-major or page-first host
 * layout, see KVIO_HOST_*) must hold host_tokens >= n_pages * P tokens.
 * Contiguous pieces are merged; `threads` positioned reads / writes run in
 * parallel.  With an O_DIRECT descriptor every file offset and length must
 * be a multiple of the device's logical block size (P * R a multiple of
 * 4 KiB is always enough).  Host memory that the OS cannot pin for direct I/O
 * -- the HIP runtime's pinned allocations among it -- makes a direct transfer
 * fail with EFAULT; the call then stages the rest through 4 KiB-aligned
 * 16 MiB bounce buffers, one per thread.  `host` must be a valid mapping of
 * the whole chunk.  Pure host code; the calls block until done and may run
 * concurrently on distinct chunks.
 * ------------------------------------------------------------------------- */
#define KVIO_DISK_PAGE_FIRST 0
#define KVIO_DISK_LAYER_FIRST 1
typedef struct kvio_disk_store {
    int32_t fd;               /* open file descriptor                              */
    int32_t disk_layout;      /* KVIO_DISK_PAGE_FIRST | KVIO_DISK_LAYER_FIRST      */
    int64_t num_disk_pages;   /* pages the file holds                              */
    int32_t num_layers;       /* L                                                 */
    int32_t page_size;        /* P tokens                                          */
    int64_t row_bytes;        /* R                                                 */
} kvio_disk_store;

/* Read the n_pages disk pages of one context into `host` (host_layout
 * KVIO_HOST_TOKEN_MAJOR or KVIO_HOST_PAGE_FIRST).  KVIO_EINVAL on bad
 * arguments or a disk page outside [0, num_disk_pages); KVIO_EIO on a failed
 * or short read. */
kvio_status kvio_disk_prefetch(const kvio_disk_store *store, const int64_t *disk_pages, int32_t n_pages,
                               void *host, int64_t host_tokens, int32_t host_layout, int32_t threads);

/* Write the n_pages context pages of `host` to the disk pages (backup). */
kvio_status kvio_disk_store_pages(const kvio_disk_store *store, const int64_t *disk_pages, int32_t n_pages,
                                  const void *host, int64_t host_tokens, int32_t host_layout,
                                  int32_t threads);

/* Background prefetch (Sec. 4.2.1): a storage hit starts the prefetch while
 * the request waits in the queue; at dispatch the controller stops whatever is
 * still in flight and uses the pages that already reached host memory.
 *
 * kvio_disk_prefetch_start validates like kvio_disk_prefetch, then returns at
 * once with `threads` worker threads reading in the background; *out is the
 * job handle (NULL on error).  The store's descriptor and the host chunk must
 * stay valid until kvio_disk_prefetch_finish returns.
 * kvio_disk_prefetch_progress: pages complete so far (never blocks).
 * kvio_disk_prefetch_finish: with cancel != 0 the workers stop at their next
 * transfer boundary (at most one piece or one bounce buffer each); then it
 * waits for them, writes page_done[j] = 1 for every context page j whose bytes
 * have all arrived and 0 otherwise (page_done may be NULL; it holds n_pages
 * bytes), stores the count in *pages_done (may be NULL), and frees the job.
 * Bytes of incomplete pages are unspecified.  Returns KVIO_EIO if a read
 * failed (page_done still names the complete pages), else KVIO_OK -- also
 * after a cancellation.  Every job must be finished exactly once. */
typedef struct kvio_prefetch *kvio_prefetch_t;
kvio_status kvio_disk_prefetch_start(const kvio_disk_store *store, const int64_t *disk_pages, int32_t n_pages,
                                     void *host, int64_t host_tokens, int32_t host_layout, int32_t threads,
                                     kvio_prefetch_t *out);
kvio_status kvio_disk_prefetch_progress(kvio_prefetch_t job, int32_t *pages_done);
kvio_status kvio_disk_prefetch_finish(kvio_prefetch_t job, int32_t cancel, uint8_t *page_done, int32_t *pages_done);

/* ---------------------------------------------------------------------------
 * Cache-aware batch formation (Sec. 4.3): the host-side step that decides
 * which queued prefill requests the next batch loads and computes.
 *
 * One scheduling round:
 *   1. Deferral on delay hit (Sec. 4.3.1): a request whose tokens match
 *      transient (in-queue / in-flight) cache entries by more than
 *      delay_hit_threshold tokens waits for the next round, at the front of
 *      the queue.
 *   2. Balanced batch formation (Sec. 4.3.2, Algorithm 1) over the others: the
 *      queue head always joins, followed by every queued request that
 *      bundle-hits the batch (reuses a context already in it; that context
 *      is loaded once).  Then, while the batch is not full, requests are taken
 *      in queue order: one that would make the batch loading-bound --
 *      aggregated load tokens > loading_bound_ratio * aggregated compute
 *      tokens, decided exactly on the integer token sums and the ratio's
 *      binary value (no rounding) -- is deprioritized, otherwise it
 *      joins and pulls in its own bundle hits.  Deprioritized requests then
 *      fill any room left, in their original order.
 * "Full" means the batch's compute tokens reached max_tokens or its size
 * reached max_requests; as in Algorithm 1, a joining request is not checked
 * against the remaining room.  The call is pure host code (no device work).
 * ------------------------------------------------------------------------- */
typedef struct kvio_request {
    int64_t load_tokens;        /* cached tokens to load from host memory, >= 0           */
    int64_t compute_tokens;     /* new tokens to prefill, >= 0                            */
    int64_t context;            /* id of the cached context it reuses; < 0 = none         */
    int64_t transient_matches;  /* tokens matched on in-queue / in-flight entries, >= 0   */
} kvio_request;

typedef struct kvio_batch_policy {
    int64_t max_tokens;           /* token budget of a batch, >= 1                          */
    int32_t max_requests;         /* request cap of a batch, >= 1                           */
    int32_t reserved;             /* 0                                                      */
    double loading_bound_ratio;   /* > 0; 0 = the paper's default 100; INFINITY = FIFO      */
    int64_t delay_hit_threshold;  /* deferral threshold in matched tokens; < 0 = default 100 */
} kvio_batch_policy;

/* Form the next batch from `queue` (n requests, index 0 = head).  Writes the
 * batch as queue indices in the order they joined to batch[0 .. *n_batch) and
 * the next round's queue (deferred requests first, then the rest in queue
 * order) to next_queue[0 .. *n_next); both arrays must hold n entries.
 * n == 0 gives an empty batch.  KVIO_EINVAL on bad arguments. */
kvio_status kvio_schedule_round(const kvio_request *queue, int32_t n, const kvio_batch_policy *policy,
                                int32_t *batch, int32_t *n_batch, int32_t *next_queue, int32_t *n_next);

/* Static text for a status code. */
const char *kvio_strerror(kvio_status status);

/* Thread-local detail of the last failure on this thread ("" if none). */
const char *kvio_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KVIO_H */
