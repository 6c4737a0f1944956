// lamp_noalloc.hip -- the fixed device scratch of lamp_attn_fwd_noalloc, the
// entry point for callers that cannot allocate device memory (code under graph
// capture, serving loops, harnesses that forbid hipMalloc).
//
// The scratch is a file-scope device array of NOALLOC_SCRATCH_BYTES: each GPU
// the library runs on holds its own copy from module load until the process
// ends.  Host code never uses the array's name as an address (in host code it
// is only a stand-in for the symbol): the device address of each GPU's copy
// comes from hipGetSymbolAddress, called once per device at initialisation
// with that device current (noalloc_scratch_address), and is kept per device.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lamp_kernels.h"

namespace lamp {

static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

hipError_t noalloc_scratch_address(void **ptr)
{
    *ptr = nullptr;
    return hipGetSymbolAddress(ptr, HIP_SYMBOL(scratch));
}

} // namespace lamp
