/*
 * kvio_abi_demo.c -- drives libkvio.so from plain C (no Python, no torch):
 * validation errors (no device needed), then, with "gpu" as argument, a
 * small paged load and offload whose results are checked against a direct
 * C computation of the definition (slot = page_idx[t / P] * P + t % P).
 * Exit status 0 = every check passed.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "kvio.h"

#define CHECK(cond, ...)                                           \
    do {                                                           \
        if (!(cond)) {                                             \
            fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__);   \
            fprintf(stderr, __VA_ARGS__);                          \
            fprintf(stderr, "\n");                                 \
            return 1;                                              \
        }                                                          \
    } while (0)

static int host_only(void)
{
    kvio_pool_desc d;
    kvio_pool_t pool = NULL;
    memset(&d, 0, sizeof d);
    d.num_layers = 2;
    d.num_kv_heads = 4;
    d.head_dim = 64;
    d.elem_bytes = 2;
    d.page_size = 16;
    d.num_slots = 4096;
    CHECK(kvio_pool_create(&d, &pool) == KVIO_EINVAL, "null layer table must be EINVAL");
    CHECK(strstr(kvio_last_error(), "null layer table") != NULL, "error text: %s", kvio_last_error());
    d.head_dim = 5;
    d.num_kv_heads = 3;
    {
        void *layers[2] = {(void *)16, (void *)16};
        d.k_layers = layers;
        d.v_layers = layers;
        CHECK(kvio_pool_create(&d, &pool) == KVIO_EALIGN, "30-byte rows must be EALIGN");
    }
    CHECK(kvio_load(NULL, NULL, 0, 0, 1, NULL) == KVIO_EINVAL, "null pool must be EINVAL");
    CHECK(kvio_pool_destroy(NULL) == KVIO_OK, "destroy(NULL) is OK");
    CHECK(strcmp(kvio_strerror(KVIO_ERANGE), "KVIO_ERANGE: page index out of range") == 0, "strerror");
    {
        kvio_request q[4] = {{80000, 1000, 3, 0}, {60000, 200, 7, 0}, {60000, 200, 7, 0}, {0, 2000, -1, 0}};
        kvio_batch_policy pol = {8000, 2, 0, 0.0, -1};
        int32_t b[4], nq[4], nb = 0, nn = 0;
        CHECK(kvio_schedule_round(q, 4, &pol, b, &nb, nq, &nn) == KVIO_OK, "schedule_round");
        CHECK(nb == 2 && b[0] == 0 && b[1] == 3 && nn == 2 && nq[0] == 1 && nq[1] == 2, "figure-7 batch");
    }
    printf("host-only checks passed\n");
    return 0;
}

static int gpu(void)
{
    enum { L = 2, H = 4, D = 64, P = 16, S = 1024, T = 200 };
    const int64_t R = H * D * 2;
    const int npages = (T + P - 1) / P;
    uint8_t *pool_dev = NULL, *chunk = NULL, *out = NULL;
    int32_t *pidx_dev = NULL;
    int32_t pidx[(T + P - 1) / P];
    void *kl[L], *vl[L];
    kvio_pool_desc d;
    kvio_pool_t pool = NULL;
    kvio_span span;
    uint8_t *img;
    int i, l, kv, mode;
    int64_t t;

    CHECK(hipMalloc((void **)&pool_dev, (size_t)(2 * L * S * R)) == hipSuccess, "hipMalloc pool");
    CHECK(hipMalloc((void **)&pidx_dev, sizeof pidx) == hipSuccess, "hipMalloc page table");
    for (i = 0; i < npages; ++i) pidx[i] = (i * 7 + 3) % (S / P);   /* distinct pages */
    CHECK(hipMemcpy(pidx_dev, pidx, sizeof pidx, hipMemcpyHostToDevice) == hipSuccess, "page table copy");
    CHECK(kvio_host_alloc((size_t)(L * 2 * T * R), KVIO_HOST_COHERENT, (void **)&chunk) == KVIO_OK, "host alloc");
    CHECK(kvio_host_alloc((size_t)(L * 2 * T * R), KVIO_HOST_COHERENT, (void **)&out) == KVIO_OK, "host alloc");
    for (i = 0; i < L * 2 * T * R; ++i) chunk[i] = (uint8_t)(i * 131 + (i >> 9));
    for (l = 0; l < L; ++l) {
        kl[l] = pool_dev + (int64_t)l * S * R;
        vl[l] = pool_dev + (int64_t)(L + l) * S * R;
    }
    /* mode 0: the transfer kernels read / write the pinned chunk; mode 1:
     * staged through HBM slots (three pages of K and V rows each) */
    for (mode = 0; mode < 2; ++mode) {
        CHECK(hipMemset(pool_dev, 0x5A, (size_t)(2 * L * S * R)) == hipSuccess, "hipMemset");
        memset(out, 0xA5, (size_t)(L * 2 * T * R));
        memset(&d, 0, sizeof d);
        if (mode == 1) {
            d.load_launch.flags = KVIO_LAUNCH_STAGED;
            d.offload_launch.flags = KVIO_LAUNCH_STAGED;
            d.staging_bytes = 4 * 3 * 2 * P * R;
        }
        d.num_layers = L;
        d.num_kv_heads = H;
        d.head_dim = D;
        d.elem_bytes = 2;
        d.page_size = P;
        d.num_slots = S;
        d.k_layers = kl;
        d.v_layers = vl;
        CHECK(kvio_pool_create(&d, &pool) == KVIO_OK, "pool create: %s", kvio_last_error());
        span.host = chunk;
        span.host_tokens = T;
        span.num_tokens = T;
        span.page_idx = pidx_dev;
        CHECK(kvio_load(pool, &span, 1, 0, L, NULL) == KVIO_OK, "load (mode %d): %s", mode, kvio_last_error());
        span.host = out;
        CHECK(kvio_offload(pool, &span, 1, 0, L, NULL) == KVIO_OK, "offload: %s", kvio_last_error());
        CHECK(kvio_check(pool) == KVIO_OK, "check: %s", kvio_last_error());
        img = (uint8_t *)malloc((size_t)(2 * L * S * R));
        CHECK(img != NULL, "malloc");
        CHECK(hipMemcpy(img, pool_dev, (size_t)(2 * L * S * R), hipMemcpyDeviceToHost) == hipSuccess, "readback");
        /* every moved row, by the definition; every other row still 0x5A */
        for (l = 0; l < L; ++l)
            for (kv = 0; kv < 2; ++kv) {
                const uint8_t *plane = img + (int64_t)(kv * L + l) * S * R;
                char *used = (char *)calloc(S, 1);
                for (t = 0; t < T; ++t) {
                    const int64_t slot = (int64_t)pidx[t / P] * P + t % P;
                    const uint8_t *src = chunk + ((int64_t)(l * 2 + kv) * T + t) * R;
                    used[slot] = 1;
                    CHECK(memcmp(plane + slot * R, src, (size_t)R) == 0, "row l=%d kv=%d t=%lld", l, kv, (long long)t);
                }
                for (t = 0; t < S; ++t)
                    if (!used[t])
                        for (i = 0; i < R; ++i) CHECK(plane[t * R + i] == 0x5A, "untouched slot %lld", (long long)t);
                free(used);
            }
        CHECK(memcmp(out, chunk, (size_t)(L * 2 * T * R)) == 0, "offload round trip (mode %d)", mode);
        free(img);
        CHECK(kvio_pool_destroy(pool) == KVIO_OK, "destroy");
    }
    kvio_host_free(chunk);
    kvio_host_free(out);
    (void)hipFree(pool_dev);
    (void)hipFree(pidx_dev);
    printf("gpu checks passed\n");
    return 0;
}

int main(int argc, char **argv)
{
    int rc = host_only();
    if (rc == 0 && argc > 1 && strcmp(argv[1], "gpu") == 0) rc = gpu();
    return rc;
}
