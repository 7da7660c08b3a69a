// Streaming-ceiling kernels (ceilings.hip): reference rates of the memory
// system for reading the collectives' kernels against.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstddef>

namespace hoccl {

// mode 0 read a, 1 write c, 2 copy a -> c, 3 c = a + b (fp32), 4 c += 1 in
// place (fp32), 5 and 6 modes 2 and 3 with non-temporal stores; `bytes` per
// operand, a multiple of 16, operands 16-byte aligned.  Mode 0 may write 4
// bytes at c (it never does in practice).
hipError_t launch_stream_ceiling(int mode, const void *a, const void *b, void *c, size_t bytes, int wg,
                                 int threads, hipStream_t s);

}  // namespace hoccl
