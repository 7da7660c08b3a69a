// Test helper: a kernel that holds CU wave slots for a fixed wall-clock time
// and then exits, so a test can ask whether other work needs a CU.  The
// time bound uses the GPU's constant 100 MHz real-time counter, so every
// block ends after `ticks` whatever else runs.
#include <hip/hip_runtime.h>

#include <cstdint>

__global__ void __launch_bounds__(1024) occupy_kernel(uint64_t ticks) {
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    while (__builtin_amdgcn_s_memrealtime() - t0 < ticks) __builtin_amdgcn_s_sleep(8);
}

// Launches `blocks` blocks of 1024 threads on `stream`, each spinning for
// `ticks` counts of the 100 MHz counter.  Returns the hipError_t of the launch.
extern "C" int occupy_launch(int blocks, uint64_t ticks, hipStream_t stream) {
    hipLaunchKernelGGL(occupy_kernel, dim3((unsigned)blocks), dim3(1024), 0, stream, ticks);
    return (int)hipGetLastError();
}
