// Static device scratch for the entry point that allocates nothing
// (hoccl_reduce_scatter_noalloc).
//
// A file-scope device array, loaded with this file's code object on every
// device the library runs on and held there until the process ends.  Host
// code never passes the array's name to a kernel (on the host it is only a
// stand-in for the symbol): the library takes each device's own address of
// it once, at initialisation with that device current, and passes that
// pointer wherever the ring's fp32 partials would otherwise live in the
// allocated workspace.  Nothing in it has to start at zero: every ring step
// writes its partials before the next step reads them.
#include <hip/hip_runtime.h>

#include "hoccl_internal.h"

namespace hoccl {
namespace {

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

}  // namespace

hipError_t scratch_address(void **out) {
    *out = nullptr;
    void *p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e == hipSuccess) *out = p;
    return e;
}

}  // namespace hoccl
