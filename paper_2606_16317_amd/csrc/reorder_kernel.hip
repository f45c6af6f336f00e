// Row gather / scatter over the sequence axis, for the spatio-temporal token reordering
// that precedes the attention loop (Section 3.1, end of the hyperparameter paragraph:
// tokens are regrouped by their position in the latent video so that a tile holds
// neighbours in time and space).
//
// A tensor [BH][N][row_bytes] is moved row by row:
//   gather:  dst[bh][i] = src[bh][index[i]]
//   scatter: dst[bh][index[i]] = src[bh][i]
// Each thread moves one 16-byte chunk (one 4-byte word when row_bytes is not a multiple
// of 16 or a pointer is not 16-byte aligned), so consecutive lanes read and write
// consecutive bytes of a row: a 256-byte bf16 row of d = 128 is one fully used 16-lane
// segment.  The work is pure HBM streaming; blockIdx.y is the head, blockIdx.x walks the
// chunks of that head.
//
// An index outside [0, N) never causes an access: gather writes a zero row for it and
// scatter drops the row.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "reorder_launch.h"

namespace dsattn {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

template <typename T, bool kScatter>
__global__ __launch_bounds__(kThreads) void move_rows_kernel(const T* __restrict__ src,
                                                            T* __restrict__ dst,
                                                            const int32_t* __restrict__ index,
                                                            int N, int per_row) {
  const uint32_t c = blockIdx.x * kThreads + threadIdx.x;   // chunk inside this head
  const uint32_t head_chunks = (uint32_t)N * (uint32_t)per_row;
  if (c >= head_chunks) return;
  const uint32_t i = c / (uint32_t)per_row;
  const uint32_t w = c - i * (uint32_t)per_row;
  const size_t head = (size_t)blockIdx.y * head_chunks;
  const uint32_t s = (uint32_t)index[i];
  const bool ok = s < (uint32_t)N;
  const size_t moved = head + (size_t)s * per_row + w;   // row named by the index
  if constexpr (kScatter) {
    if (ok) dst[moved] = src[head + c];
  } else {
    dst[head + c] = ok ? src[moved] : T{};
  }
}

template <bool kScatter>
hipError_t launch(const void* src, void* dst, const int32_t* index, int bh, int N,
                  int row_bytes, bool wide, hipStream_t stream) {
  const int per_row = wide ? row_bytes / 16 : row_bytes / 4;
  const uint32_t chunks = (uint32_t)N * (uint32_t)per_row;
  const dim3 grid((chunks + kThreads - 1) / kThreads, (unsigned)bh);
  if (wide)
    hipLaunchKernelGGL((move_rows_kernel<u32x4, kScatter>), grid, dim3(kThreads), 0, stream,
                       static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), index, N,
                       per_row);
  else
    hipLaunchKernelGGL((move_rows_kernel<uint32_t, kScatter>), grid, dim3(kThreads), 0,
                       stream, static_cast<const uint32_t*>(src), static_cast<uint32_t*>(dst),
                       index, N, per_row);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gather_rows(const void* src, void* dst, const int32_t* index, int bh, int N,
                              int row_bytes, bool wide, hipStream_t stream) {
  return launch<false>(src, dst, index, bh, N, row_bytes, wide, stream);
}

hipError_t launch_scatter_rows(const void* src, void* dst, const int32_t* index, int bh, int N,
                               int row_bytes, bool wide, hipStream_t stream) {
  return launch<true>(src, dst, index, bh, N, row_bytes, wide, stream);
}

}  // namespace dsattn
