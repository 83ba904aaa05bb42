// kvio_linkpeak.hip -- kvio_kernel_memcpy: one contiguous copy by a plain
// kernel.  It is the rate compute units reach on the host link when nothing
// is paged (no page table, no slot lookup, no layout change), the ceiling of
// the kernel path in each direction, beside kvio_memcpy's copy-engine rate.
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <string.h>

#include "kvio.h"
#include "kvio_pool.h"

namespace {

typedef uint32_t vec16 __attribute__((ext_vector_type(4)));   // one 16-byte vector

// Launch shapes, both multiples of 8 workgroups (even over the XCDs).
//  * Into device memory (host reads): 16 workgroups of 3 waves, 4 KiB per
//    wave step: 192 KiB in flight, what the link needs by Little's law on its
//    read latency, without the longer queues that more reads in flight build.
//  * Into host memory (host writes): 32 workgroups of 4 waves, 16 KiB steps:
//    2 MiB in flight, enough to cover the acknowledgement of device-scope
//    stores (below).
struct Shape {
    int workgroups, threads;
};
constexpr Shape kIntoDevice = {16, 192};
constexpr Shape kIntoHost = {32, 256};

// One 16-byte store.  SC1: non-temporal with the device-scope (SC1) cache
// policy, the fastest way for a wave to write pinned host memory over the
// link (the compiler's plain or non-temporal stores reach 1-2.5% less).  No
// builtin selects SC1 for a global store; the s_nop gives the two wait
// states required before a VALU may overwrite the data registers of a store
// wider than 64 bits (the compiler cannot see the store inside the asm).
template <bool SC1>
__device__ __forceinline__ void store16(vec16 *p, vec16 v) {
    if constexpr (SC1) {
        asm volatile("global_store_dwordx4 %0, %1, off sc1 nt\n\ts_nop 1" : : "v"(p), "v"(v) : "memory");
    } else {
        __builtin_nontemporal_store(v, p);
    }
}

// Grid-stride over wave steps of 64 x VPL vectors; whole steps run without
// per-vector checks, the last partial step with them.
template <int VPL, bool SC1>
__global__ void __launch_bounds__(256) kvio_plain_copy_kernel(const vec16 *__restrict__ src, vec16 *__restrict__ dst,
                                                              int64_t nvec) {
    const int lane = static_cast<int>(threadIdx.x & 63);
    const int64_t wpg = blockDim.x >> 6;
    const int64_t waves = static_cast<int64_t>(gridDim.x) * wpg;
    const int64_t wave = static_cast<int64_t>(blockIdx.x) * wpg + (threadIdx.x >> 6);
    constexpr int64_t kStep = 64 * VPL;              // vectors per wave step
#pragma unroll 1
    for (int64_t base = wave * kStep; base < nvec; base += waves * kStep) {
        vec16 buf[VPL];
        if (base + kStep <= nvec) {                  // a whole step (wave-uniform)
#pragma unroll
            for (int k = 0; k < VPL; ++k) buf[k] = __builtin_nontemporal_load(src + base + k * 64 + lane);
#pragma unroll
            for (int k = 0; k < VPL; ++k) store16<SC1>(dst + base + k * 64 + lane, buf[k]);
        } else {                                     // the last, partial step
#pragma unroll
            for (int k = 0; k < VPL; ++k) {
                const int64_t j = base + k * 64 + lane;
                if (j < nvec) store16<SC1>(dst + j, __builtin_nontemporal_load(src + j));
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
    hipPointerAttribute_t attr;
    memset(&attr, 0, sizeof attr);
    const hipError_t ea = hipPointerGetAttributes(&attr, dst);   // succeeded inside device_view already
    if (ea != hipSuccess) return kvio::fail_hip(ea, fn);
    const vec16 *sv = reinterpret_cast<const vec16 *>(s);
    vec16 *dv = reinterpret_cast<vec16 *>(const_cast<uint8_t *>(d));
    const int64_t nvec = static_cast<int64_t>(bytes / 16);
    if (attr.type == hipMemoryTypeHost)
        hipLaunchKernelGGL((kvio_plain_copy_kernel<16, true>), dim3(kIntoHost.workgroups), dim3(kIntoHost.threads), 0,
                           stream, sv, dv, nvec);
    else
        hipLaunchKernelGGL((kvio_plain_copy_kernel<4, false>), dim3(kIntoDevice.workgroups),
                           dim3(kIntoDevice.threads), 0, stream, sv, dv, nvec);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return kvio::fail_hip(e, fn);
    return KVIO_OK;
}
