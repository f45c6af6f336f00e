// Internal interface between the C-ABI entry points and the MX-FP8 quantisation kernel.
#ifndef DSATTN_QUANT_LAUNCH_H
#define DSATTN_QUANT_LAUNCH_H

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace dsattn {

// n_blocks blocks of 32 bf16 values (src, 64 bytes each, 16-byte aligned) become 32 E4M3
// codes each (codes, 16-byte aligned) and one E8M0 scale code each (scales).
hipError_t launch_quantize_mxfp8(const void* src, void* codes, void* scales,
                                 long long n_blocks, hipStream_t stream);

}  // namespace dsattn

#endif
