// kvio_linkpeak.hip -- kvio_kernel_memcpy: one contiguous copy by a plain
// kernel.  It is the rate compute units reach on the host link when nothing
// is paged (no page table, no slot lookup, no layout change), the ceiling of
// the kernel path in each direction, beside kvio_memcpy's copy-engine rate.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "kvio.h"
#include "kvio_pool.h"

namespace {

typedef uint32_t vec16 __attribute__((ext_vector_type(4)));   // one 16-byte vector

// 16 workgroups of 3 waves, two per XCD; each wave moves 4 KiB per step (4
// vectors per lane), so 192 KiB is in flight across the grid: what the link
// needs (Little's law on its read latency), without the longer queues that
// more reads in flight build up.
constexpr int kWorkgroups = 16;
constexpr int kThreads = 192;
constexpr int kVecPerLane = 4;

__global__ void __launch_bounds__(kThreads) kvio_plain_copy_kernel(const vec16 *__restrict__ src,
                                                                    vec16 *__restrict__ dst, int64_t nvec) {
    const int lane = static_cast<int>(threadIdx.x & 63);
    const int64_t waves = static_cast<int64_t>(gridDim.x) * (kThreads / 64);
    const int64_t wave = static_cast<int64_t>(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6);
    constexpr int64_t kStep = 64 * kVecPerLane;      // vectors per wave step
#pragma unroll 1
    for (int64_t base = wave * kStep; base < nvec; base += waves * kStep) {
        vec16 buf[kVecPerLane];
        if (base + kStep <= nvec) {                  // a whole step (wave-uniform): no per-vector checks
#pragma unroll
            for (int k = 0; k < kVecPerLane; ++k) buf[k] = __builtin_nontemporal_load(src + base + k * 64 + lane);
#pragma unroll
            for (int k = 0; k < kVecPerLane; ++k) __builtin_nontemporal_store(buf[k], dst + base + k * 64 + lane);
        } else {                                     // the last, partial step
#pragma unroll
            for (int k = 0; k < kVecPerLane; ++k) {
                const int64_t j = base + k * 64 + lane;
                if (j < nvec) __builtin_nontemporal_store(__builtin_nontemporal_load(src + j), dst + j);
            }
        }
    }
}

}  // namespace

extern "C" kvio_status kvio_kernel_memcpy(void *dst, const void *src, size_t bytes, hipStream_t stream) {
    const char *fn = "kvio_kernel_memcpy";
    kvio::clear_error();
    if (bytes == 0) return KVIO_OK;
    if (dst == nullptr || src == nullptr) return kvio::fail(KVIO_EINVAL, "%s: null pointer", fn);
    if (bytes % 16 != 0)
        return kvio::fail(KVIO_EINVAL, "%s: %zu bytes is not a multiple of 16", fn, bytes);
    if (reinterpret_cast<uintptr_t>(dst) % 16 != 0 || reinterpret_cast<uintptr_t>(src) % 16 != 0)
        return kvio::fail(KVIO_EINVAL, "%s: pointers must be 16-byte aligned", fn);
    if (bytes > static_cast<size_t>(INT64_MAX))
        return kvio::fail(KVIO_EINVAL, "%s: %zu bytes is too large", fn, bytes);
    // Both ranges must lie in allocations the device can reach, whole: the
    // kernel never touches memory past either.
    const uint8_t *s = nullptr, *d = nullptr;
    kvio_status st = kvio::device_view(src, bytes, false, "kvio_kernel_memcpy: source", &s);
    if (st != KVIO_OK) return st;
    st = kvio::device_view(dst, bytes, false, "kvio_kernel_memcpy: destination", &d);
    if (st != KVIO_OK) return st;
    hipLaunchKernelGGL(kvio_plain_copy_kernel, dim3(kWorkgroups), dim3(kThreads), 0, stream,
                       reinterpret_cast<const vec16 *>(s), reinterpret_cast<vec16 *>(const_cast<uint8_t *>(d)),
                       static_cast<int64_t>(bytes / 16));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return kvio::fail_hip(e, fn);
    return KVIO_OK;
}
