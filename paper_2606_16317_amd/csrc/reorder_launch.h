// Internal interface between the C-ABI entry points and the row gather/scatter kernels.
#ifndef DSATTN_REORDER_LAUNCH_H
#define DSATTN_REORDER_LAUNCH_H

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace dsattn {

// dst[b][i] = src[b][index[i]] for b < bh, i < N, rows of row_bytes (a multiple of 4);
// indexes outside [0, N) give zero rows.  `wide` moves 16-byte chunks (row_bytes a
// multiple of 16, src and dst 16-byte aligned), otherwise 4-byte words.  Requires
// N * row_bytes / 4 < 2^32.
hipError_t launch_gather_rows(const void* src, void* dst, const int32_t* index, int bh, int N,
                              int row_bytes, bool wide, hipStream_t stream);

// dst[b][index[i]] = src[b][i]; rows whose index lies outside [0, N) are dropped.
hipError_t launch_scatter_rows(const void* src, void* dst, const int32_t* index, int bh, int N,
                               int row_bytes, bool wide, hipStream_t stream);

}  // namespace dsattn

#endif
