// Internal interface between the C-ABI entry points and the MX-FP8 quantisation kernel.
#ifndef DSATTN_QUANT_LAUNCH_H
#define DSATTN_QUANT_LAUNCH_H

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace dsattn {

// n_blocks blocks of 32 bf16 values (src, 64 bytes each, 16-byte aligned) become 32 E4M3
// codes each (codes, 16-byte aligned) and one E8M0 scale code each (scales).  With a
// shift (float32, 16-byte aligned), row i (blocks_per_row blocks) first has vector
// i / group_rows subtracted.
hipError_t launch_quantize_mxfp8(const void* src, void* codes, void* scales,
                                 long long n_blocks, const float* shift, int blocks_per_row,
                                 long long group_rows, hipStream_t stream);

// mean[h][c] = (1/N) sum_n k[h][n][c] for bh heads of N rows of d bf16 values (d a power
// of two in [8, 1024], k 16-byte aligned); deterministic.
hipError_t launch_key_mean(const void* k, float* mean, int bh, int N, int d,
                           hipStream_t stream);

}  // namespace dsattn

#endif
