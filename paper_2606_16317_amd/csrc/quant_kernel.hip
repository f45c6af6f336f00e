// MX-FP8 quantisation of bf16 rows (the storage of a quantised Q K^T; Section 1 lists
// quantised attention among the methods the rule combines with).
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

__global__ __launch_bounds__(kThreads) void quantize_mxfp8_kernel(
    const u32x4* __restrict__ src, u32x4* __restrict__ codes, uint8_t* __restrict__ scales,
    long long n_blocks) {
  const long long blk = (long long)blockIdx.x * kThreads + threadIdx.x;
  if (blk >= n_blocks) return;
  u32x4 w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = src[blk * 4 + i];      // 32 bf16 values
  float amax = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      amax = fmaxf(amax, fmaxf(fabsf(bf16_lo(w[i][j])), fabsf(bf16_hi(w[i][j]))));
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
  for (int i = 0; i < 4; ++i) {
    uint32_t packed[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t lo = e4m3_code(bf16_lo(w[i][2 * h]) * inv);
      const uint32_t hi = e4m3_code(bf16_hi(w[i][2 * h]) * inv);
      const uint32_t lo2 = e4m3_code(bf16_lo(w[i][2 * h + 1]) * inv);
      const uint32_t hi2 = e4m3_code(bf16_hi(w[i][2 * h + 1]) * inv);
      packed[h] = lo | (hi << 8) | (lo2 << 16) | (hi2 << 24);
    }
    out[i >> 1][2 * (i & 1)] = packed[0];
    out[i >> 1][2 * (i & 1) + 1] = packed[1];
  }
  codes[blk * 2] = out[0];
  codes[blk * 2 + 1] = out[1];
  scales[blk] = (uint8_t)scode;
}

}  // namespace

hipError_t launch_quantize_mxfp8(const void* src, void* codes, void* scales,
                                 long long n_blocks, hipStream_t stream) {
  const long long grid = (n_blocks + kThreads - 1) / kThreads;
  hipLaunchKernelGGL(quantize_mxfp8_kernel, dim3((unsigned)grid), dim3(kThreads), 0, stream,
                     static_cast<const u32x4*>(src), static_cast<u32x4*>(codes),
                     static_cast<uint8_t*>(scales), n_blocks);
  return hipGetLastError();
}

}  // namespace dsattn
