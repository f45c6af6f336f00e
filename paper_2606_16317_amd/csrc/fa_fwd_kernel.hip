// Tile-filtered FlashAttention forward kernels for gfx950 (CDNA4).
//
// One workgroup computes one (b, h, query tile of 128 rows); its four waves own 32 query
// rows each.  The loop visits key tiles of 64 keys in ascending order (Section 1,
// tile-based attention), and for every tile:
//
//   1. S^T = K_j Q_i^T on MFMA (bf16 inputs, fp32 accumulation) -- always computed;
//   2. per-row tile maximum m_hat (always);
//   3. the rule's decision (Section 3.1, Eq. 5 for DynSparse; the running-max test for
//      BLASST), reduced over all valid rows of the 128-row tile;
//   4. only for kept tiles: online-softmax update of the running max m and row sum l,
//      P = exp(S - m), O = alpha O + P V_j on MFMA.
//
// Register layout (lane l of a wave, r = l % 32, g = l / 32):
//   * the MFMA 32x32x16 output places column (l % 32) in lane l, so computing S^T = K Q^T
//     puts one query row per lane pair (l, l ^ 32): row statistics need a single
//     cross-half exchange instead of a 32-lane reduction;
//   * the same lane owns P^T[., row], which is exactly what the B operand of
//     O^T = V^T P^T needs, so P never leaves registers;
//   * O^T accumulates in the output layout with one query row per lane, so the rescale
//     by alpha is a per-lane scalar multiply.
// The PV contraction runs over key "slots": slot i of lane half g in PV step s is the
// key whose S^T value sits in register 8*(s%2) + i of block s/2.  V is transposed into
// LDS in that slot order, so each V^T operand is one 16-byte LDS read.
//
// LDS (double buffered, 64 KiB per workgroup): K tile [64 keys][128 d] with 16-byte
// chunks XOR-swizzled by (key % 16); V^T tile [128 d][64 slots] with 16-byte chunks
// XOR-swizzled by ((d / 2) % 8).  Both swizzles make the 16-lane phases of the
// ds_read_b128 operand fetches hit 16 distinct bank quads.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fa_fwd_launch.h"

namespace dsattn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kD = 128;        // head dimension
constexpr int kTQ = 128;       // query rows per workgroup (decision granularity)
constexpr int kTK = 64;        // keys per tile
constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;

struct Smem {
  alignas(16) uint16_t k[2][kTK * kD];
  alignas(16) uint16_t vt[2][kD * kTK];
  int vote[kWaves];
};

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float log2_fast(float x) { return __builtin_amdgcn_logf(x); }

// Position of tile-local key `key` (0..63) in the V^T slot order.
__device__ __forceinline__ int slot_of_key(int key) {
  const int b = key >> 5;           // 32-key S^T block
  const int m = (key >> 3) & 3;     // register group (v / 4) inside the block
  const int gg = (key >> 2) & 1;    // lane half holding the key
  const int i4 = key & 3;
  const int s = 2 * b + (m >> 1);   // PV step
  const int i = ((m & 1) << 2) | i4;
  return 16 * s + 8 * gg + i;
}

__device__ __forceinline__ int k_lds_index(int key, int chunk) {
  return key * kD + ((chunk ^ (key & 15)) << 3);
}

__device__ __forceinline__ int vt_lds_index(int d, int slot) {
  return d * kTK + ((((slot >> 3) ^ ((d >> 1) & 7))) << 3) + (slot & 7);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 x) {
  return __builtin_bit_cast(bf16x8, x);
}

// Global -> register prefetch of one K/V tile (zero-filled past the sequence end).
struct TileRegs {
  u32x4 k[4];
  u32x4 v[4];
};

__device__ __forceinline__ void load_tile(TileRegs& t, const uint16_t* __restrict__ kb,
                                          const uint16_t* __restrict__ vb, int key0, int N,
                                          int tid) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int ci = tid + kThreads * u;
    // K: 16 lanes cover one key row (256 contiguous bytes).
    const int kkey = ci >> 4, kc = ci & 15;
    const int kg = key0 + kkey;
    t.k[u] = (kg < N) ? *reinterpret_cast<const u32x4*>(kb + (size_t)kg * kD + kc * 8)
                      : u32x4{0, 0, 0, 0};
    // V: a wave covers 64 keys of one 8-wide d chunk (the LDS writes then stay in one
    // V^T row per instruction).
    const int vkey = ci & 63, vc = ci >> 6;
    const int vg = key0 + vkey;
    t.v[u] = (vg < N) ? *reinterpret_cast<const u32x4*>(vb + (size_t)vg * kD + vc * 8)
                      : u32x4{0, 0, 0, 0};
  }
}

__device__ __forceinline__ void store_tile(const TileRegs& t, uint16_t* __restrict__ ks,
                                           uint16_t* __restrict__ vts, int tid) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int ci = tid + kThreads * u;
    const int kkey = ci >> 4, kc = ci & 15;
    *reinterpret_cast<u32x4*>(ks + k_lds_index(kkey, kc)) = t.k[u];
    const int vkey = ci & 63, vc = ci >> 6;
    const int slot = slot_of_key(vkey);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t w = t.v[u][e >> 1];
      vts[vt_lds_index(vc * 8 + e, slot)] = (uint16_t)((e & 1) ? (w >> 16) : (w & 0xFFFF));
    }
  }
}

template <int RULE>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads),
                          amdgpu_waves_per_eu(2, 2))) void
fa_fwd_kernel(FwdParams p) {
  __shared__ __attribute__((aligned(16))) Smem sm;

  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int lane = tid & 63;
  const int r = lane & 31;
  const int g = lane >> 5;
  const int qt = blockIdx.x;
  const int bh = blockIdx.y;
  const int N = p.N;
  const int n_kt = p.n_kt;

  const size_t head_off = (size_t)bh * (size_t)N * kD;
  const uint16_t* __restrict__ qb = p.q + head_off;
  const uint16_t* __restrict__ kb = p.k + head_off;
  const uint16_t* __restrict__ vb = p.v + head_off;

  const int q0 = qt * kTQ;
  const int qrow = q0 + w * 32 + r;
  const bool valid = qrow < N;
  const int rows_valid = min(kTQ, N - q0);

  // Q^T B-operand fragments: d = 16 s + 8 g + (0..7) of this lane's query row.
  bf16x8 qf[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    u32x4 x = valid ? *reinterpret_cast<const u32x4*>(qb + (size_t)qrow * kD + 16 * s + 8 * g)
                    : u32x4{0, 0, 0, 0};
    qf[s] = as_bf16x8(x);
  }

  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) o[db] = f32x16{};
  float m_run = -__builtin_inff();   // running max of kept tiles, log2 units
  float l_half = 0.f;                // this lane's share of the kept row sum

  uint64_t tiles_skipped = 0, elems_skipped = 0;

  TileRegs tr;
  load_tile(tr, kb, vb, 0, N, tid);
  store_tile(tr, sm.k[0], sm.vt[0], tid);
  __syncthreads();

  const float c = p.c;
  for (int j = 0; j < n_kt; ++j) {
    const int buf = j & 1;
    const int key0 = j * kTK;
    const bool has_next = (j + 1) < n_kt;
    if (has_next) load_tile(tr, kb, vb, key0 + kTK, N, tid);

    // ---- S^T = K_j Q^T: two 32-key blocks, eight 16-wide d steps each --------------
    f32x16 st[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      st[b] = f32x16{};
      const int key = 32 * b + r;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const bf16x8 a = as_bf16x8(
            *reinterpret_cast<const u32x4*>(sm.k[buf] + k_lds_index(key, 2 * s + g)));
        st[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[s], st[b], 0, 0, 0);
      }
    }
    // Keys past the end of the sequence take no part in max or sum.
    if (key0 + kTK > N) {
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = key0 + 32 * b + (v >> 2) * 8 + g * 4 + (v & 3);
          if (key >= N) st[b][v] = -__builtin_inff();
        }
    }

    // ---- tile row max (raw logits; c > 0 so scaling commutes with max) ------------
    float mx = st[0][0];
#pragma unroll
    for (int v = 1; v < 16; ++v) mx = fmaxf(mx, st[0][v]);
#pragma unroll
    for (int v = 0; v < 16; ++v) mx = fmaxf(mx, st[1][v]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_hat = mx * c;

    // ---- decision --------------------------------------------------------------
    bool keep = true;
    if constexpr (RULE != kRuleDense) {
      float t;
      if constexpr (RULE == kRuleDynSparse) {
        const float l_row = l_half + __shfl_xor(l_half, 32);
        t = m_hat - (m_run + log2_fast(l_row));   // Eq. 5 in log2 units
      } else {
        t = m_hat - m_run;
      }
      const bool row_keeps = valid && !(t < p.thr);
      const bool wave_keeps = __ballot(row_keeps) != 0;
      if (lane == 0) sm.vote[w] = wave_keeps ? 1 : 0;
      __syncthreads();
      keep = (sm.vote[0] | sm.vote[1] | sm.vote[2] | sm.vote[3]) != 0;
      if (!keep) {
        tiles_skipped += 1;
        elems_skipped += (uint64_t)rows_valid * (uint64_t)min(kTK, N - key0);
      }
      if (p.mask != nullptr && tid == 0)
        p.mask[((size_t)bh * p.n_qt + qt) * n_kt + j] = keep ? 0 : 1;
    } else {
      if (p.mask != nullptr && tid == 0) p.mask[((size_t)bh * p.n_qt + qt) * n_kt + j] = 0;
    }

    if (keep) {
      // ---- online softmax (Eq. 6 state) --------------------------------------
      const float m_new = fmaxf(m_run, m_hat);
      const float alpha = exp2_fast(m_run - m_new);
      const float neg_m = -m_new;
      float psum = 0.f;
      bf16x8 pf[4];
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float e = exp2_fast(fmaf(st[b][v], c, neg_m));
          psum += e;
          pf[2 * b + (v >> 3)][v & 7] = (__bf16)e;
        }
      l_half = fmaf(alpha, l_half, psum);
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
      m_run = m_new;

      // ---- O^T += V^T P^T ------------------------------------------------------
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const int d = 32 * db + r;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const bf16x8 a = as_bf16x8(*reinterpret_cast<const u32x4*>(
              sm.vt[buf] + vt_lds_index(d, 16 * s + 8 * g)));
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[s], o[db], 0, 0, 0);
        }
      }
    }

    if (has_next) store_tile(tr, sm.k[buf ^ 1], sm.vt[buf ^ 1], tid);
    __syncthreads();
  }

  // ---- epilogue: renormalise over kept keys, store O (bf16) and the row LSE --------
  const float l_row = l_half + __shfl_xor(l_half, 32);
  const float inv = 1.0f / l_row;
  if (valid) {
    uint16_t* __restrict__ orow = p.o + head_off + (size_t)qrow * kD;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        __bf16 h0 = (__bf16)(o[db][4 * grp + 0] * inv);
        __bf16 h1 = (__bf16)(o[db][4 * grp + 1] * inv);
        __bf16 h2 = (__bf16)(o[db][4 * grp + 2] * inv);
        __bf16 h3 = (__bf16)(o[db][4 * grp + 3] * inv);
        const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, h0) |
                            ((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16);
        const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, h2) |
                            ((uint32_t)__builtin_bit_cast(uint16_t, h3) << 16);
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        *reinterpret_cast<u32x2*>(orow + 32 * db + 8 * grp + 4 * g) = u32x2{lo, hi};
      }
    if (p.lse != nullptr && g == 0)
      p.lse[(size_t)bh * N + qrow] = (m_run + log2_fast(l_row)) * 0.69314718055994530942f;
  }
  if (p.stats != nullptr && tid == 0) {
    unsigned long long* st = reinterpret_cast<unsigned long long*>(p.stats) + (size_t)bh * 4;
    atomicAdd(st + 0, (unsigned long long)n_kt);
    atomicAdd(st + 1, (unsigned long long)tiles_skipped);
    atomicAdd(st + 2, (unsigned long long)rows_valid * (unsigned long long)N);
    atomicAdd(st + 3, (unsigned long long)elems_skipped);
  }
}

__global__ void zero_u64_kernel(uint64_t* __restrict__ p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

}  // namespace

hipError_t launch_fa_fwd(int rule, const FwdParams& p, int bh, hipStream_t stream) {
  const dim3 grid((unsigned)p.n_qt, (unsigned)bh);
  const dim3 block(kThreads);
  switch (rule) {
    case kRuleDense:
      hipLaunchKernelGGL(fa_fwd_kernel<kRuleDense>, grid, block, 0, stream, p);
      break;
    case kRuleBlasst:
      hipLaunchKernelGGL(fa_fwd_kernel<kRuleBlasst>, grid, block, 0, stream, p);
      break;
    case kRuleDynSparse:
      hipLaunchKernelGGL(fa_fwd_kernel<kRuleDynSparse>, grid, block, 0, stream, p);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_zero_u64(uint64_t* ptr, int n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int threads = 256;
  hipLaunchKernelGGL(zero_u64_kernel, dim3((n + threads - 1) / threads), dim3(threads), 0,
                     stream, ptr, n);
  return hipGetLastError();
}

}  // namespace dsattn
