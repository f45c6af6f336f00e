// MX-FP8 quantisation of bf16 rows (the storage of a quantised Q K^T; the Conclusion,
// Section 5, lists quantisation among the methods the rule combines with), optionally of rows minus
// a float32 shift vector (key smoothing), and the per-head mean key that serves as that
// shift.
//
// Every run of 32 consecutive values of a row is one block: it shares the power-of-two
// scale 2^E with E = floor(log2(max |x|)) - 8, stored as the E8M0 code E + 127 (0 for an
// all-zero block), and each value becomes the FP8 E4M3 number nearest to x / 2^E -- ties
// to the even code, magnitudes above 448 saturating to 448.  One thread handles one
// block: four 16-byte loads, two 16-byte stores and one scale byte, so consecutive lanes
// touch consecutive memory; the kernel is pure HBM streaming.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "quant_launch.h"

namespace dsattn {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

// E4M3 code of a finite float, rounded to nearest with ties to the even code, saturating
// at 448 (0x7e); -0 and values that round to zero give +0.
__device__ __forceinline__ uint32_t e4m3_code(float y) {
  const uint32_t bits = __float_as_uint(y);
  const uint32_t sign = bits >> 31;
  const uint32_t a = bits & 0x7fffffffu;
  uint32_t code;
  if (a >= 0x43e00000u) {                 // |y| >= 448
    code = 0x7eu;
  } else if (a < 0x3c800000u) {           // |y| < 2^-6: subnormal step 2^-9
    code = (uint32_t)__builtin_rintf(__uint_as_float(a) * 512.0f);   // 0..8; 8 = 2^-6
  } else {
    const uint32_t e = (a >> 23) - 127u + 7u;        // biased E4M3 exponent, 1..15
    const uint32_t m = a & 0x7fffffu;
    uint32_t keep = m >> 20;
    const uint32_t rem = m & 0xfffffu;
    keep += (rem > 0x80000u || (rem == 0x80000u && (keep & 1u))) ? 1u : 0u;
    code = (e << 3) + keep;                          // a mantissa carry bumps the exponent
    if (code > 0x7eu) code = 0x7eu;
  }
  return code == 0 ? 0u : (code | (sign << 7));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// SHIFT: every value first has its column's entry of a float32 shift vector subtracted
// (rounded to nearest float32); row i uses vector i / group_rows.
template <bool SHIFT>
__global__ __launch_bounds__(kThreads) void quantize_mxfp8_kernel(
    const u32x4* __restrict__ src, u32x4* __restrict__ codes, uint8_t* __restrict__ scales,
    long long n_blocks, const float* __restrict__ shift, int blocks_per_row,
    long long group_rows) {
  const long long blk = (long long)blockIdx.x * kThreads + threadIdx.x;
  if (blk >= n_blocks) return;
  u32x4 w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = src[blk * 4 + i];      // 32 bf16 values
  float x[32];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[8 * i + 2 * j] = bf16_lo(w[i][j]);
      x[8 * i + 2 * j + 1] = bf16_hi(w[i][j]);
    }
  if constexpr (SHIFT) {
    const long long row = blk / blocks_per_row;
    const int cb = (int)(blk - row * blocks_per_row);
    const float4* sh = reinterpret_cast<const float4*>(
        shift + (row / group_rows) * (long long)blocks_per_row * 32 + cb * 32);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float4 s4 = sh[i];
      x[4 * i] -= s4.x;
      x[4 * i + 1] -= s4.y;
      x[4 * i + 2] -= s4.z;
      x[4 * i + 3] -= s4.w;
    }
  }
  float amax = 0.f;
#pragma unroll
  for (int i = 0; i < 32; ++i) amax = fmaxf(amax, fabsf(x[i]));
  uint32_t scode = 0;
  float inv = 1.f;
  if (amax > 0.f) {
    int e2;
    (void)frexpf(amax, &e2);                 // amax = f * 2^e2, f in [0.5, 1)
    const int e = e2 - 1 - 8;                // floor(log2 amax) - 8
    scode = (uint32_t)min(254, max(0, e + 127));
    inv = __uint_as_float((254u - scode) << 23);           // 2^(127 - scode), exact
  }
  u32x4 out[2];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t packed = e4m3_code(x[4 * i] * inv) | (e4m3_code(x[4 * i + 1] * inv) << 8) |
                            (e4m3_code(x[4 * i + 2] * inv) << 16) |
                            (e4m3_code(x[4 * i + 3] * inv) << 24);
    out[i >> 2][i & 3] = packed;
  }
  codes[blk * 2] = out[0];
  codes[blk * 2 + 1] = out[1];
  scales[blk] = (uint8_t)scode;
}

// Mean over the N keys of every head.  Workgroup (g, h) takes column group g of head h:
// kMeanCols columns (64 bytes of every row; all of a row when d is smaller).  Thread t
// sums 16-byte chunk t % C of rows t / C, t / C + P, ... (C chunks per group, P =
// kMeanThreads / C rows in flight per step, eight steps unrolled); then the P partial sums
// of every column are added in row order from LDS.  The order is fixed, so repeated
// calls agree bit for bit.
constexpr int kMeanThreads = 256;
constexpr int kMeanCols = 32;

__global__ __launch_bounds__(kMeanThreads) void key_mean_kernel(const u32x4* __restrict__ k,
                                                                float* __restrict__ mean,
                                                                int N, int d) {
  __shared__ float part[kMeanThreads * 8];
  const int cols = d < kMeanCols ? d : kMeanCols;
  const int cpg = cols >> 3;                 // 16-byte chunks per group and row
  const int cpr = d >> 3;                    // chunks per row
  const int par = kMeanThreads / cpg;        // rows per step
  const int t = threadIdx.x;
  const int c = t % cpg;
  const int head = blockIdx.y;
  const u32x4* base = k + (size_t)head * (size_t)N * cpr + (size_t)blockIdx.x * cpg + c;
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  int r = t / cpg;
  for (; r + 7 * par < N; r += 8 * par) {
    u32x4 x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = base[(size_t)(r + u * par) * cpr];
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc[2 * j] += bf16_lo(x[u][j]);
        acc[2 * j + 1] += bf16_hi(x[u][j]);
      }
  }
  for (; r < N; r += par) {
    const u32x4 x = base[(size_t)r * cpr];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      acc[2 * j] += bf16_lo(x[j]);
      acc[2 * j + 1] += bf16_hi(x[j]);
    }
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) part[t * 8 + i] = acc[i];
  __syncthreads();
  const float inv_n = 1.0f / (float)N;
  for (int e = t; e < cols; e += kMeanThreads) {
    const int ch = e >> 3, i = e & 7;
    float sum = 0.f;
    for (int rl = 0; rl < par; ++rl) sum += part[(rl * cpg + ch) * 8 + i];
    mean[(size_t)head * d + (size_t)blockIdx.x * cols + e] = sum * inv_n;
  }
}

}  // namespace

hipError_t launch_quantize_mxfp8(const void* src, void* codes, void* scales,
                                 long long n_blocks, const float* shift, int blocks_per_row,
                                 long long group_rows, hipStream_t stream) {
  const long long grid = (n_blocks + kThreads - 1) / kThreads;
  if (shift == nullptr)
    hipLaunchKernelGGL(quantize_mxfp8_kernel<false>, dim3((unsigned)grid), dim3(kThreads), 0,
                       stream, static_cast<const u32x4*>(src), static_cast<u32x4*>(codes),
                       static_cast<uint8_t*>(scales), n_blocks, shift, blocks_per_row,
                       group_rows);
  else
    hipLaunchKernelGGL(quantize_mxfp8_kernel<true>, dim3((unsigned)grid), dim3(kThreads), 0,
                       stream, static_cast<const u32x4*>(src), static_cast<u32x4*>(codes),
                       static_cast<uint8_t*>(scales), n_blocks, shift, blocks_per_row,
                       group_rows);
  return hipGetLastError();
}

hipError_t launch_key_mean(const void* k, float* mean, int bh, int N, int d,
                           hipStream_t stream) {
  const int groups = d < kMeanCols ? 1 : d / kMeanCols;
  hipLaunchKernelGGL(key_mean_kernel, dim3((unsigned)groups, (unsigned)bh), dim3(kMeanThreads),
                     0, stream, static_cast<const u32x4*>(k), mean, N, d);
  return hipGetLastError();
}

}  // namespace dsattn
