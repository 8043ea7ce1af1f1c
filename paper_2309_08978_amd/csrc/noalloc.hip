// Device buffers that the library never allocates at run time: the fixed
// split-K scratch of the allocation-free entry point and the zero block
// that out-of-range GEMM loads read.  Both are file-scope device arrays, so
// each GPU that loads the library holds its own copy for the life of the
// process.  Host code must not pass these names to a kernel (on the host
// they stand for a host-side shadow, not device memory): it takes each
// array's device address once per device, with hipGetSymbolAddress, and
// passes that address instead.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace nnjit {

static __device__ __align__(256) float scratch[kNoAllocScratchBytes / sizeof(float)];
static __device__ __align__(256) unsigned zero_block[64];

hipError_t static_buffer_addresses(void **scratch_ptr, void **zero_ptr)
{
    hipError_t e = hipGetSymbolAddress(scratch_ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    return hipGetSymbolAddress(zero_ptr, HIP_SYMBOL(zero_block));
}

}  // namespace nnjit
