// The stream side of the copy proxy's start/finish flag handshake (Stream
// Manager section), as one gfx950 dispatch of one lane.
//
// Publish START once everything before it is visible to the copy engines (a
// system-scope release), wait until the proxy acknowledges by clearing
// START, wait until it writes FINISH after the copies completed, then
// acquire at system scope (later work sees the copied bytes) and clear
// FINISH.  Every flag access is a system-scope vector atomic on host memory
// mapped for the device.  The lane sleeps between polls, and both waits give
// up once limit_ticks of the constant-rate device wall clock have passed,
// recording that in *status, so the dispatch always ends.
#include <hip/hip_runtime.h>

#include "hoccl_internal.h"

namespace hoccl {
namespace {

__device__ inline uint32_t poll_flag(uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__device__ inline bool wait_flag(uint32_t *p, uint32_t want, uint64_t t0, uint64_t limit) {
    while (poll_flag(p) != want) {
        if ((uint64_t)wall_clock64() - t0 > limit) return false;
        __builtin_amdgcn_s_sleep(4);
    }
    return true;
}

__global__ void __launch_bounds__(64) handshake_kernel(HandshakeArgs a) {
    if (threadIdx.x != 0) return;
    __hip_atomic_store(a.start, a.start_value, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    const uint64_t t0 = (uint64_t)wall_clock64();
    if (!wait_flag(a.start, 0u, t0, a.limit_ticks) ||
        !wait_flag(a.finish, a.finish_value, t0, a.limit_ticks)) {
        __hip_atomic_store(a.status, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
        return;
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
    __hip_atomic_store(a.finish, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

}  // namespace

hipError_t launch_handshake(const HandshakeArgs &a, hipStream_t s) {
    void *args[] = {const_cast<HandshakeArgs *>(&a)};
    return hipLaunchKernel((const void *)handshake_kernel, dim3(1), dim3(64), args, 0, s);
}

}  // namespace hoccl
