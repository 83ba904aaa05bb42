/*
 * kvoracle.c -- CPU oracle for the paged-KV host<->pool transfer.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library may link, call or
 * include this file; only the tests, the smoke check and the benchmark's CPU
 * baseline use it.  It shares no header, table or helper with the GPU path.
 *
 * What it computes (Strata, Sec. 4.2 "Efficient KV Cache I/O" and Sec. 4.2.1
 * "Data Management Beyond Host Memory", Fig. 6): a GPU-assisted I/O job moves
 * each small chunk of a cached context from its source into its destination,
 * and the layout change between the transfer-friendly host copy and the
 * compute-friendly, layer-first paged pool is one extra offset computation per
 * chunk.  The copy is exact: no arithmetic touches the payload, so the result
 * has a plain definition, written out here as plain loops with one memcpy per
 * token row.
 *
 * Notation (all byte counts):
 *   L layers, K and V per layer (kv = 0 is K, kv = 1 is V),
 *   R = row bytes = KV heads * head_dim * element bytes (one token of one
 *       layer's K or V),
 *   P = page size in tokens, S = token slots per per-layer pool (S % P == 0),
 *   page_idx[j] = pool page that holds context page j (Sec. 2.2, paged KV;
 *       the HiRadixTree of Sec. 4.1 acts as the page table),
 *   host chunk of one context, layer-major and token-major:
 *       host[((l*2 + kv)*host_tokens + t)*R + b], b < R,
 *   pool: per-layer K and V arrays, pool_kv[l][slot*R + b].
 *
 * Definition, for every l in [l0, l1), kv in {K, V}, t in [0, num_tokens):
 *   slot(t) = page_idx[t / P] * P + t % P
 *   load:    pool_kv[l][slot(t)] row := host row (l, kv, t)
 *   offload: host row (l, kv, t)     := pool_kv[l][slot(t)] row
 * Every other pool byte (load) and host byte (offload) is left unchanged.
 * A load that would write one slot twice (a duplicate page, or two contexts
 * sharing a page) is rejected; an offload may read a slot twice.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/*
 * Host chunk layouts.  All three hold the same rows; they differ only in where
 * row (l, kv, t) -- or, head-major, its head h segment -- sits in the chunk:
 *   TOKEN_MAJOR (layer-major chunk per context):
 *       ((l*2 + kv)*host_tokens + t) * R
 *   PAGE_FIRST (Sec. 4.2.1, Fig. 6: the layers of one page stored together, the
 *   transfer-friendly layout for host and disk; host_tokens is a multiple of P):
 *       (((t/P)*L + l)*2 + kv) * P*R + (t%P) * R
 *   HEAD_MAJOR (one contiguous run per (layer, K|V, head); the segment of head h
 *   of row t, De = head_dim * element bytes bytes long):
 *       (((l*2 + kv)*H + h)*host_tokens + t) * De
 */
#define KVO_TOKEN_MAJOR 0
#define KVO_PAGE_FIRST 1
#define KVO_HEAD_MAJOR 2

#define KVO_OK 0
#define KVO_EINVAL (-1)   /* bad sizes, null pointers, num_tokens > host_tokens */
#define KVO_ERANGE (-2)   /* a page index outside [0, S/P)                       */
#define KVO_EDUP (-3)     /* a load would write one pool slot twice              */
#define KVO_ENOMEM (-4)

/* Byte offset of host row (layer, kv, token) inside one context's chunk. */
int64_t kvo_host_row_offset(int32_t layer, int32_t kv, int64_t host_tokens,
                            int64_t token, int64_t row_bytes)
{
    return (((int64_t)layer * 2 + kv) * host_tokens + token) * row_bytes;
}

/* Page-first layout: byte offset of host row (layer, kv, token). */
int64_t kvo_host_row_offset_page_first(int32_t layer, int32_t kv, int32_t num_layers,
                                       int32_t page_size, int64_t token, int64_t row_bytes)
{
    int64_t page = token / page_size;
    int64_t in_page = token % page_size;
    return (((page * num_layers + layer) * 2 + kv) * page_size + in_page) * row_bytes;
}

/* Head-major layout: byte offset of the head `head` segment of row (layer, kv, token). */
int64_t kvo_host_seg_offset_head_major(int32_t layer, int32_t kv, int32_t head, int32_t num_heads,
                                       int64_t host_tokens, int64_t token, int64_t seg_bytes)
{
    return ((((int64_t)layer * 2 + kv) * num_heads + head) * host_tokens + token) * seg_bytes;
}

/*
 * Page-offset expansion: the pool slot of every context token t < num_tokens.
 * Context page j = t / P lives in pool page page_idx[j]; the token sits at
 * offset t % P inside it.  Tokens at or beyond num_tokens (the unused tail of
 * a partial last page) get no slot.
 */
int kvo_expand_slots(const int32_t *page_idx, int32_t page_size,
                     int64_t num_tokens, int64_t num_slots, int64_t *slots_out)
{
    int64_t t;
    int64_t num_pages;
    if (page_size < 1 || num_tokens < 0 || num_slots < 0 || num_slots % page_size != 0)
        return KVO_EINVAL;
    if (num_tokens > 0 && (page_idx == NULL || slots_out == NULL))
        return KVO_EINVAL;
    num_pages = num_slots / page_size;
    for (t = 0; t < num_tokens; ++t) {
        int64_t ctx_page = t / page_size;
        int64_t in_page = t % page_size;
        int64_t pool_page = page_idx[ctx_page];
        if (pool_page < 0 || pool_page >= num_pages)
            return KVO_ERANGE;
        slots_out[t] = pool_page * page_size + in_page;
    }
    return KVO_OK;
}

/* One (layer, kv) slab: host_slab holds rows t = 0.. of that slab. */
int kvo_load_slab(uint8_t *pool_slab, int64_t num_slots, int32_t page_size,
                  int64_t row_bytes, const uint8_t *host_slab,
                  int64_t num_tokens, const int32_t *page_idx)
{
    int64_t t;
    int64_t num_pages;
    if (pool_slab == NULL || host_slab == NULL || row_bytes <= 0 || page_size < 1 ||
        num_tokens < 0 || num_slots < 0 || num_slots % page_size != 0)
        return KVO_EINVAL;
    if (num_tokens > 0 && page_idx == NULL)
        return KVO_EINVAL;
    num_pages = num_slots / page_size;
    for (t = 0; t < num_tokens; ++t) {
        int64_t pool_page = page_idx[t / page_size];
        int64_t slot;
        if (pool_page < 0 || pool_page >= num_pages)
            return KVO_ERANGE;
        slot = pool_page * page_size + t % page_size;
        memcpy(pool_slab + slot * row_bytes, host_slab + t * row_bytes, (size_t)row_bytes);
    }
    return KVO_OK;
}

int kvo_offload_slab(const uint8_t *pool_slab, int64_t num_slots, int32_t page_size,
                     int64_t row_bytes, uint8_t *host_slab,
                     int64_t num_tokens, const int32_t *page_idx)
{
    int64_t t;
    int64_t num_pages;
    if (pool_slab == NULL || host_slab == NULL || row_bytes <= 0 || page_size < 1 ||
        num_tokens < 0 || num_slots < 0 || num_slots % page_size != 0)
        return KVO_EINVAL;
    if (num_tokens > 0 && page_idx == NULL)
        return KVO_EINVAL;
    num_pages = num_slots / page_size;
    for (t = 0; t < num_tokens; ++t) {
        int64_t pool_page = page_idx[t / page_size];
        int64_t slot;
        if (pool_page < 0 || pool_page >= num_pages)
            return KVO_ERANGE;
        slot = pool_page * page_size + t % page_size;
        memcpy(host_slab + t * row_bytes, pool_slab + slot * row_bytes, (size_t)row_bytes);
    }
    return KVO_OK;
}

/*
 * Validate a batch of contexts against one pool before anything is moved:
 * sizes, page range, and (for a load) that no pool slot is written twice.
 * Spans are given as parallel arrays, one entry per cached context.
 */
static int kvo_check_batch(int32_t n_spans, const int64_t *host_tokens,
                           const int64_t *num_tokens, const int32_t *const *page_idx,
                           int64_t num_slots, int32_t page_size, int reject_duplicates)
{
    int32_t s;
    int64_t t;
    int64_t num_pages;
    uint8_t *written = NULL;
    if (n_spans < 0 || page_size < 1 || num_slots < 0 || num_slots % page_size != 0)
        return KVO_EINVAL;
    num_pages = num_slots / page_size;
    if (reject_duplicates) {
        written = (uint8_t *)calloc((size_t)(num_slots / 8 + 1), 1);
        if (written == NULL)
            return KVO_ENOMEM;
    }
    for (s = 0; s < n_spans; ++s) {
        if (num_tokens[s] < 0 || num_tokens[s] > host_tokens[s] ||
            (num_tokens[s] > 0 && page_idx[s] == NULL)) {
            free(written);
            return KVO_EINVAL;
        }
        for (t = 0; t < num_tokens[s]; ++t) {
            int64_t pool_page = page_idx[s][t / page_size];
            int64_t slot;
            if (pool_page < 0 || pool_page >= num_pages) {
                free(written);
                return KVO_ERANGE;
            }
            slot = pool_page * page_size + t % page_size;
            if (reject_duplicates) {
                if (written[slot / 8] & (uint8_t)(1u << (slot % 8))) {
                    free(written);
                    return KVO_EDUP;
                }
                written[slot / 8] |= (uint8_t)(1u << (slot % 8));
            }
        }
    }
    free(written);
    return KVO_OK;
}

/*
 * Load a batch of cached contexts (host chunks) into the paged pool, over the
 * layer range [layer_begin, layer_end).  k_pool[l] / v_pool[l] are the
 * per-layer pool images (S rows of R bytes each).
 */
int kvo_load_batch(uint8_t *const *k_pool, uint8_t *const *v_pool, int32_t num_layers,
                   int64_t num_slots, int32_t page_size, int64_t row_bytes,
                   int32_t n_spans, const uint8_t *const *host,
                   const int64_t *host_tokens, const int64_t *num_tokens,
                   const int32_t *const *page_idx, int32_t layer_begin, int32_t layer_end)
{
    int32_t s, l, kv;
    int rc;
    if (k_pool == NULL || v_pool == NULL || row_bytes <= 0 || layer_begin < 0 ||
        layer_end > num_layers || layer_begin >= layer_end)
        return KVO_EINVAL;
    if (n_spans > 0 && (host == NULL || host_tokens == NULL || num_tokens == NULL || page_idx == NULL))
        return KVO_EINVAL;
    rc = kvo_check_batch(n_spans, host_tokens, num_tokens, page_idx, num_slots, page_size, 1);
    if (rc != KVO_OK)
        return rc;
    for (s = 0; s < n_spans; ++s) {
        if (num_tokens[s] > 0 && host[s] == NULL)
            return KVO_EINVAL;
        for (l = layer_begin; l < layer_end; ++l) {
            for (kv = 0; kv < 2; ++kv) {
                uint8_t *slab = kv == 0 ? k_pool[l] : v_pool[l];
                const uint8_t *src = host[s] + kvo_host_row_offset(l, kv, host_tokens[s], 0, row_bytes);
                if (num_tokens[s] == 0)
                    continue;
                rc = kvo_load_slab(slab, num_slots, page_size, row_bytes, src,
                                   num_tokens[s], page_idx[s]);
                if (rc != KVO_OK)
                    return rc;
            }
        }
    }
    return KVO_OK;
}

/* Offload: the inverse gather, pool rows -> contiguous host rows. */
int kvo_offload_batch(const uint8_t *const *k_pool, const uint8_t *const *v_pool,
                      int32_t num_layers, int64_t num_slots, int32_t page_size,
                      int64_t row_bytes, int32_t n_spans, uint8_t *const *host,
                      const int64_t *host_tokens, const int64_t *num_tokens,
                      const int32_t *const *page_idx, int32_t layer_begin, int32_t layer_end)
{
    int32_t s, l, kv;
    int rc;
    if (k_pool == NULL || v_pool == NULL || row_bytes <= 0 || layer_begin < 0 ||
        layer_end > num_layers || layer_begin >= layer_end)
        return KVO_EINVAL;
    if (n_spans > 0 && (host == NULL || host_tokens == NULL || num_tokens == NULL || page_idx == NULL))
        return KVO_EINVAL;
    rc = kvo_check_batch(n_spans, host_tokens, num_tokens, page_idx, num_slots, page_size, 0);
    if (rc != KVO_OK)
        return rc;
    for (s = 0; s < n_spans; ++s) {
        if (num_tokens[s] > 0 && host[s] == NULL)
            return KVO_EINVAL;
        for (l = layer_begin; l < layer_end; ++l) {
            for (kv = 0; kv < 2; ++kv) {
                const uint8_t *slab = kv == 0 ? k_pool[l] : v_pool[l];
                uint8_t *dst = host[s] + kvo_host_row_offset(l, kv, host_tokens[s], 0, row_bytes);
                if (num_tokens[s] == 0)
                    continue;
                rc = kvo_offload_slab(slab, num_slots, page_size, row_bytes, dst,
                                      num_tokens[s], page_idx[s]);
                if (rc != KVO_OK)
                    return rc;
            }
        }
    }
    return KVO_OK;
}

/*
 * Load / offload for any host layout.  `num_heads` is H (R = H * seg bytes);
 * for PAGE_FIRST, host_tokens must be a multiple of the page size.  Same
 * validation and semantics as kvo_load_batch / kvo_offload_batch.
 */
static int kvo_move_layout(uint8_t *const *k_pool, uint8_t *const *v_pool, int32_t num_layers,
                           int64_t num_slots, int32_t page_size, int64_t row_bytes, int32_t num_heads,
                           int32_t host_layout, int32_t n_spans, uint8_t *const *host,
                           const int64_t *host_tokens, const int64_t *num_tokens,
                           const int32_t *const *page_idx, int32_t layer_begin, int32_t layer_end,
                           int to_pool)
{
    int32_t s, l, kv, h;
    int64_t t;
    int rc;
    int64_t seg;
    if (k_pool == NULL || v_pool == NULL || row_bytes <= 0 || num_heads < 1 ||
        row_bytes % num_heads != 0 || layer_begin < 0 || layer_end > num_layers ||
        layer_begin >= layer_end)
        return KVO_EINVAL;
    if (host_layout != KVO_TOKEN_MAJOR && host_layout != KVO_PAGE_FIRST && host_layout != KVO_HEAD_MAJOR)
        return KVO_EINVAL;
    if (n_spans > 0 && (host == NULL || host_tokens == NULL || num_tokens == NULL || page_idx == NULL))
        return KVO_EINVAL;
    rc = kvo_check_batch(n_spans, host_tokens, num_tokens, page_idx, num_slots, page_size, to_pool);
    if (rc != KVO_OK)
        return rc;
    seg = row_bytes / num_heads;
    for (s = 0; s < n_spans; ++s) {
        if (num_tokens[s] == 0)
            continue;
        if (host[s] == NULL)
            return KVO_EINVAL;
        if (host_layout == KVO_PAGE_FIRST && host_tokens[s] % page_size != 0)
            return KVO_EINVAL;
        for (l = layer_begin; l < layer_end; ++l) {
            for (kv = 0; kv < 2; ++kv) {
                uint8_t *slab = kv == 0 ? k_pool[l] : v_pool[l];
                for (t = 0; t < num_tokens[s]; ++t) {
                    int64_t slot = (int64_t)page_idx[s][t / page_size] * page_size + t % page_size;
                    uint8_t *prow = slab + slot * row_bytes;
                    if (host_layout == KVO_HEAD_MAJOR) {
                        for (h = 0; h < num_heads; ++h) {
                            uint8_t *hseg = host[s] + kvo_host_seg_offset_head_major(
                                                          l, kv, h, num_heads, host_tokens[s], t, seg);
                            if (to_pool)
                                memcpy(prow + h * seg, hseg, (size_t)seg);
                            else
                                memcpy(hseg, prow + h * seg, (size_t)seg);
                        }
                    } else {
                        int64_t off = host_layout == KVO_TOKEN_MAJOR
                            ? kvo_host_row_offset(l, kv, host_tokens[s], t, row_bytes)
                            : kvo_host_row_offset_page_first(l, kv, num_layers, page_size, t, row_bytes);
                        if (to_pool)
                            memcpy(prow, host[s] + off, (size_t)row_bytes);
                        else
                            memcpy(host[s] + off, prow, (size_t)row_bytes);
                    }
                }
            }
        }
    }
    return KVO_OK;
}

int kvo_load_layout(uint8_t *const *k_pool, uint8_t *const *v_pool, int32_t num_layers,
                    int64_t num_slots, int32_t page_size, int64_t row_bytes, int32_t num_heads,
                    int32_t host_layout, int32_t n_spans, const uint8_t *const *host,
                    const int64_t *host_tokens, const int64_t *num_tokens,
                    const int32_t *const *page_idx, int32_t layer_begin, int32_t layer_end)
{
    return kvo_move_layout(k_pool, v_pool, num_layers, num_slots, page_size, row_bytes, num_heads,
                           host_layout, n_spans, (uint8_t *const *)host, host_tokens, num_tokens,
                           page_idx, layer_begin, layer_end, 1);
}

int kvo_offload_layout(uint8_t *const *k_pool, uint8_t *const *v_pool, int32_t num_layers,
                       int64_t num_slots, int32_t page_size, int64_t row_bytes, int32_t num_heads,
                       int32_t host_layout, int32_t n_spans, uint8_t *const *host,
                       const int64_t *host_tokens, const int64_t *num_tokens,
                       const int32_t *const *page_idx, int32_t layer_begin, int32_t layer_end)
{
    return kvo_move_layout(k_pool, v_pool, num_layers, num_slots, page_size, row_bytes, num_heads,
                           host_layout, n_spans, host, host_tokens, num_tokens, page_idx,
                           layer_begin, layer_end, 0);
}
