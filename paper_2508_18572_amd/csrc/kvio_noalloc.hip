// kvio_noalloc.hip -- kvio_load_noalloc: the load for callers that cannot
// allocate (code under HIP graph capture, tight serving loops, harnesses that
// forbid hipMalloc).  It takes the pool description instead of a pool handle
// and keeps the two pieces of device memory a handle would own -- the table of
// layer addresses the kernels read and the error word they record into -- in
// one static device array of this file.  Every call on a GPU uses that GPU's
// copy of the array, so calls that overlap on one GPU race.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <mutex>

#include "kvio.h"
#include "kvio_internal.h"
#include "kvio_pool.h"

namespace {

// Layout of the static array: the error word at byte 0, the layer table
// (layers[kv * L + l], 2 * L addresses) from byte kTableOffset.
constexpr int kMaxLayers = KVIO_NOALLOC_MAX_LAYERS;
constexpr size_t kTableOffset = 256;
constexpr size_t kScratchBytes = 4096;
static_assert(kTableOffset + 2 * kMaxLayers * sizeof(uint8_t *) <= kScratchBytes, "layer table does not fit");

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

// Device address of `scratch` on each device, looked up on the first call on
// that device (in host code the array's name is not a device address).
constexpr int kMaxDevices = 64;
std::mutex g_lookup;
uint8_t *g_scratch[kMaxDevices];

// What the set-up kernel writes: every layer address into the table, zero
// into the error word.  Passed by value (kernel arguments), so the call needs
// no host-to-device copy.
struct ScratchInit {
    unsigned long long *err;
    uint8_t **table;
    int32_t n;
    uint8_t *layers[2 * kMaxLayers];
};

__global__ void __launch_bounds__(256) kvio_noalloc_setup(const ScratchInit a) {
    const int i = static_cast<int>(threadIdx.x);
    if (i < a.n) a.table[i] = a.layers[i];
    if (i == 0) *a.err = 0;
}

kvio_status scratch_address(const char *fn, uint8_t **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return kvio::fail_hip(e, fn);
    if (dev < 0 || dev >= kMaxDevices)
        return kvio::fail(KVIO_EINVAL, "%s: device %d beyond the %d devices the library tracks", fn, dev,
                          kMaxDevices);
    std::lock_guard<std::mutex> lock(g_lookup);
    if (g_scratch[dev] == nullptr) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return kvio::fail_hip(e, "kvio_load_noalloc: hipGetSymbolAddress");
        if (ptr == nullptr) return kvio::fail(KVIO_EHIP, "%s: no device address for the static scratch array", fn);
        g_scratch[dev] = static_cast<uint8_t *>(ptr);
    }
    *out = g_scratch[dev];
    return KVIO_OK;
}

}  // namespace

extern "C" kvio_status kvio_load_noalloc(const kvio_pool_desc *desc, const kvio_span *spans, int32_t n_spans,
                                         int32_t layer_begin, int32_t layer_end, hipStream_t stream) {
    const char *fn = "kvio_load_noalloc";
    kvio::clear_error();
    if (desc == nullptr) return kvio::fail(KVIO_EINVAL, "%s: null pool description", fn);
    kvio::PoolGeom g;
    kvio_status st = kvio::check_desc(desc, fn, &g);
    if (st != KVIO_OK) return st;
    if (g.num_layers > kMaxLayers)
        return kvio::fail(KVIO_EINVAL, "%s: %d layers exceed the %d its static layer table holds", fn,
                          g.num_layers, kMaxLayers);
    if (desc->load_launch.flags & KVIO_LAUNCH_STAGED)
        return kvio::fail(KVIO_EINVAL, "%s: staged loads need staging memory; use a pool handle", fn);
    if (n_spans > KVIO_MAX_SPANS_PER_LAUNCH)
        return kvio::fail(KVIO_EINVAL, "%s: %d spans exceed the %d of one call", fn, n_spans,
                          KVIO_MAX_SPANS_PER_LAUNCH);
    ScratchInit init;
    init.n = 2 * g.num_layers;
    st = kvio::resolve_layers(desc, g, fn, init.layers);
    if (st != KVIO_OK) return st;
    kvio::Resolved rs[KVIO_MAX_SPANS_PER_LAUNCH];
    st = kvio::validate_spans(g, spans, n_spans, layer_begin, layer_end, fn, rs);
    if (st != KVIO_OK) return st;
    int64_t tokens = 0;
    for (int32_t i = 0; i < n_spans; ++i) tokens += rs[i].num_tokens;
    if (tokens == 0) return KVIO_OK;              // nothing to move: nothing enqueued
    uint8_t *base = nullptr;
    st = scratch_address(fn, &base);
    if (st != KVIO_OK) return st;
    init.err = reinterpret_cast<unsigned long long *>(base);
    init.table = reinterpret_cast<uint8_t **>(base + kTableOffset);
    hipLaunchKernelGGL(kvio_noalloc_setup, dim3(1), dim3(256), 0, stream, init);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return kvio::fail_hip(e, fn);
    const kvio::Shape shape = kvio::kernel_shape(
        g, desc->load_launch,
        kvio::default_shape(kvio::kLoad, tokens * 2 * (layer_end - layer_begin) * g.row_bytes, g.host_layout, g.num_heads));
    return kvio::launch_spans(g, init.table, init.err, rs, n_spans, layer_begin, layer_end, kvio::kLoad, shape,
                              stream, fn);
}
