// Tile-filtered FlashAttention forward kernels for gfx950 (CDNA4).
//
// One workgroup computes one (b, h, query tile of 128 rows); its four waves own 32 query
// rows each.  Key tiles of 64 keys are visited in ascending order by default (Section 1,
// tile-based attention).  For every tile the kernel
//
//   1. computes S^T = K_j Q_i^T on MFMA (bf16 inputs, fp32 accumulation) -- always;
//   2. takes the per-row tile maximum m_hat -- always;
//   3. decides, for all valid rows of the 128-row tile together, whether the tile is
//      kept: DynSparse (Section 3.1, Eq. 5) compares m_hat - LSE^(j-1) with lambda,
//      BLASST compares m_hat - m^(j-1) with ln(tau), dense keeps everything;
//   4. only for kept tiles: updates the online-softmax state (reference max, row sum),
//      forms P = exp(S - m) and accumulates O += P V_j on MFMA.
//
// Register layout (lane l of a wave, r = l % 32, g = l / 32):
//   * the 32x32x16 MFMA puts output column (l % 32) in lane l, so S^T = K Q^T leaves one
//     query row per lane pair (l, l ^ 32): row statistics need one cross-half exchange;
//   * that lane pair also owns P^T[., row], which is exactly the B operand of
//     O^T = V^T P^T, so P never leaves registers;
//   * O^T accumulates with one query row per lane, so rescaling is a per-lane multiply.
// The PV contraction runs over key "slots": slot i of lane half g in PV step s is the
// key whose S^T value sits in register 8*(s%2) + i of block s/2, i.e. key
// 32*(s/2) + 8*(2*(s%2) + i/4) + 4*g + i%4.  Slots 4c..4c+3 are four consecutive keys,
// which is what one ds_read_b64_tr_b16 delivers from a row-major V tile.
//
// Pipeline (one barrier per key tile): S_{j+1} is computed during iteration j, so the
// decision for tile j+1 is voted before the barrier that closes iteration j.  A wave
// writes its vote byte only when its vote changes, and only waves that vote skip read
// the others' after the barrier (the read's latency overlaps the issue of the next K-tile
// DMA), so with nothing skipped the votes touch no LDS.  K is
// prefetched two tiles ahead and V one tile ahead, straight from global memory into LDS
// (buffer loads with the LDS bit; rows past the sequence end come back as zeros from the
// buffer range check); V is fetched only for tiles that follow a kept tile or are
// themselves kept, so runs of skipped tiles stream K alone.  Inside an iteration the
// instruction order is fixed by scheduling fences: the 16 S_{j+1} MFMAs carry 24 elements
// of the tile-j softmax, the first eight P V MFMAs the other 8 (the ones the last four
// P V MFMAs read) and the last eight the row max of S_{j+1}; the row sum is added after the
// P V MFMAs; MFMA operands are read from LDS two MFMAs ahead.
//
// Variants, all compile-time parameters of fa_fwd_kernel:
//   * UNIT: the query rows that share a decision, the workgroup's 128 or each wave's 32;
//   * ORDER: key tiles in ascending or diagonal-first order;
//   * Q8: Q and K in MX-FP8 on the scaled fp8 MFMA (the rest of the tile is unchanged);
//   * BC: keys per decision, 64 (one tile), 128 (two tiles deciding together) or 32 (the
//     halves of each tile deciding in turn).
// fa_fwd_mask_kernel applies a given skip mask instead of a rule (mask reuse).
//
// Online softmax uses a lazily updated reference max m_ref: O and l are rescaled only
// when a kept tile's max exceeds m_ref by more than 8 (log2 units), so P <= 2^8.  The
// row LSE = m_ref + log2(l) is exact either way, which is all the DynSparse rule reads.
//
// LDS (64 KiB per workgroup): K[2][64][128] and V[2][64][128] bf16, row-major, with
// 16-byte chunks XOR-swizzled per row (K by key % 16, V by 4 * (key % 4)) so that the
// MFMA operand reads of every 16- and 32-lane group touch distinct banks.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fa_fwd_launch.h"

namespace dsattn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

constexpr int kD = 128;        // head dimension
constexpr int kTQ = 128;       // query rows per workgroup (decision granularity)
constexpr int kTK = 64;        // keys per tile
constexpr int kXcds = 8;       // accelerator dies; workgroups are dealt to them round-robin
constexpr int kWaves = 4;
constexpr uint32_t kAllSkip = 0x01010101u;  // skip word in which every wave votes skip
constexpr int kThreads = kWaves * 64;
constexpr int kTileElems = kTK * kD;         // 8192 bf16 = 16 KiB
constexpr float kRescaleSlack = 8.0f;        // log2 units

struct Smem {
  alignas(16) uint16_t k[2][kTileElems];     // bf16 K tiles, or MX-FP8 K tiles (first half)
  alignas(16) uint16_t v[2][kTileElems];
  // Per wave, double-buffered by step.  64- and 128-key decisions: 1 while the wave's last
  // vote here was skip.  32-key decisions: the wave's vote bits on the next tile.
  alignas(4) uint8_t vote[2][kWaves];
  alignas(16) uint8_t ks[2][kTK * 4];        // MX-FP8 K: E8M0 exponents, 4 blocks per key
  alignas(4) uint8_t vote_mid[kWaves];       // B_c = 32: second-half votes taken mid-step
};

// Mask-reuse workgroups also hold the list of key tiles they visit (at most
// kMaxMaskTiles, so N <= 262144 in that mode).
constexpr int kMaxMaskTiles = 4096;
struct MaskSmem {
  Smem t;
  alignas(4) uint16_t list[kMaxMaskTiles];   // (key tile << 4) | keep bit of each wave
  alignas(4) uint16_t count[kThreads];       // kept tiles per thread, then their prefix
  uint32_t total;                            // number of visited tiles
};

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float log2_fast(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// Combine a per-lane value with the one held by lane ^ 32 (the other half of the same
// query row) using v_permlane32_swap: no LDS round trip.
__device__ __forceinline__ float half_sum(float x) {
  const uint32_t b = __builtin_bit_cast(uint32_t, x);
  const auto sw = __builtin_amdgcn_permlane32_swap(b, b, false, false);
  return __builtin_bit_cast(float, (uint32_t)sw[0]) + __builtin_bit_cast(float, (uint32_t)sw[1]);
}

__device__ __forceinline__ int k_swz(int key) { return key & 15; }
__device__ __forceinline__ int v_swz(int key) { return (key & 3) << 2; }

// Element offset of (key, 16-byte chunk) inside a swizzled tile.
__device__ __forceinline__ int k_off(int key, int chunk) {
  return key * kD + ((chunk ^ k_swz(key)) << 3);
}
__device__ __forceinline__ int v_off(int key, int chunk) {
  return key * kD + ((chunk ^ v_swz(key)) << 3);
}

// Copy the 64 x 128 tile starting at key `key0` of one head into a swizzled LDS tile.
// Wave w writes four 1 KiB blocks u*4 + w (4 key rows each); lane l of a block lands in
// chunk slot l % 16 of row l / 16 and fetches the global chunk that the swizzle maps
// there.  `rs` covers the whole head (N rows of 256 bytes), so keys >= N fail the buffer
// range check and arrive as zeros.  `voff` is the lane's byte offset inside a block,
// which is the same for all four blocks of every tile (the swizzles depend on the key
// modulo 16 only).
//
// The loads are issued from inline assembly on purpose: the compiler cannot tell which
// LDS tile a buffer-to-LDS load writes, so it would otherwise wait for every such load
// before the next LDS read of any tile.  The loop's own barrier waits for them instead.
// M0 (the LDS base of the transfer) is saved and restored inside the statement, with
// the wait state an M0 write needs before an LDS-DMA instruction.
__device__ __forceinline__ void load_tile_lds(uint16_t* tile, __amdgpu_buffer_rsrc_t rs,
                                              uint32_t voff, int key0, int w) {
  const uint32_t o0 = voff + (uint32_t)key0 * (kD * 2);
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(tile + w * 512));
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %[sv], m0\n\t"
      "s_mov_b32 m0, %[l0]\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %[o0], %[rs], 0 offen lds\n\t"
      "s_add_u32 m0, %[l0], 0x1000\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %[o1], %[rs], 0 offen lds\n\t"
      "s_add_u32 m0, %[l0], 0x2000\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %[o2], %[rs], 0 offen lds\n\t"
      "s_add_u32 m0, %[l0], 0x3000\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %[o3], %[rs], 0 offen lds\n\t"
      "s_mov_b32 m0, %[sv]"
      : [sv] "=&s"(saved)
      : [l0] "s"(lds0), [o0] "v"(o0), [o1] "v"(o0 + 4096u), [o2] "v"(o0 + 8192u),
        [o3] "v"(o0 + 12288u), [rs] "s"(rs)
      : "memory", "scc");
}

// Lane offset inside a 1 KiB block (4 key rows) for a K (swizzle key % 16) or V
// (swizzle 4 * (key % 4)) tile.
template <bool kIsV>
__device__ __forceinline__ uint32_t tile_lane_offset(int w, int lane) {
  const int row = lane >> 4;
  const int key = 4 * w + row;              // key index modulo 16 of this lane's row
  const int chunk = (lane & 15) ^ (kIsV ? v_swz(key) : k_swz(key));
  return (uint32_t)(key * (kD * 2) + chunk * 16);
}


__device__ __forceinline__ bf16x8 lds_b128(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ bf16x4 lds_tr_b64(const uint16_t* p) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  const i16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
  return __builtin_bit_cast(bf16x4, x);
}

// ---- MX-FP8 Q K^T ------------------------------------------------------------------
// Quantised Q and K (E4M3 values, one E8M0 exponent per 32 values of a row) feed
// v_mfma_scale_f32_32x32x64_f8f6f4, which multiplies a 32 x 64 block of K by a 64 x 32
// block of Q^T and applies the exponents itself.  In its operands lane l holds row l % 32
// and 32 bytes.  Bytes 0-15 of both lane halves form the first 32-value exponent block of
// the 64-wide step and bytes 16-31 the second; the exponent of the first block comes from
// the lane of the low half, that of the second from the lane of the high half (measured
// with an in-bounds probe).  So for d-step s, lane half g reads d in [64 s + 16 g, +16)
// and [64 s + 32 + 16 g, +16) and supplies the exponent of block 2 s + g of its row.
//
// The fp8 K tile (64 keys x 128 bytes = 8 KiB) lives in 32 lines of 256 bytes: line L
// holds key L in its first 128 bytes and key L + 32 in its last 128, in 16-byte chunks
// XOR-swizzled by L % 16 like the bf16 tiles, so every 16-lane group of an operand read
// touches each bank once.

__device__ __forceinline__ int k8_slot(int line, int half, int chunk) {
  return (8 * half + chunk) ^ (line & 15);
}

// Lane offset (bytes, relative to the tile's first key) of wave w's first 1 KiB block of
// the fp8 K tile (lines 4 w .. 4 w + 3); its second block, 16 lines on, holds keys 16
// further on: 2 KiB further in global memory.
__device__ __forceinline__ uint32_t k8_lane_offset(int w, int lane) {
  const int line = 4 * w + (lane >> 4);       // line of this lane's slot
  const int s = (lane & 15) ^ (line & 15);    // logical chunk stored in that slot
  const int key = line + 32 * (s >> 3);
  return (uint32_t)(key * kD + (s & 7) * 16);
}

// Copy the fp8 K tile starting at key key0 into LDS (two 1 KiB blocks per wave) and, from
// wave 0, the tile's exponents (one dword per key).  Keys >= N come back as zeros.
__device__ __forceinline__ void load_k8_tile(uint8_t* tile, uint8_t* scales,
                                             __amdgpu_buffer_rsrc_t rs,
                                             __amdgpu_buffer_rsrc_t srs, uint32_t off,
                                             int key0, int w, int lane) {
  const uint32_t o0 = off + (uint32_t)key0 * kD;
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(tile + w * 1024));
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %[sv], m0\n\t"
      "s_mov_b32 m0, %[l0]\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %[o0], %[rs], 0 offen lds\n\t"
      "s_add_u32 m0, %[l0], 0x1000\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %[o1], %[rs], 0 offen lds\n\t"
      "s_mov_b32 m0, %[sv]"
      : [sv] "=&s"(saved)
      : [l0] "s"(lds0), [o0] "v"(o0), [o1] "v"(o0 + 2048u), [rs] "s"(rs)
      : "memory", "scc");
  if (w == 0) {
    const uint32_t s0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)scales);
    const uint32_t so = ((uint32_t)key0 + (uint32_t)lane) * 4u;
    asm volatile(
        "s_mov_b32 %[sv], m0\n\t"
        "s_mov_b32 m0, %[l0]\n\t"
        "s_nop 0\n\t"
        "buffer_load_dword %[o0], %[rs], 0 offen lds\n\t"
        "s_mov_b32 m0, %[sv]"
        : [sv] "=&s"(saved)
        : [l0] "s"(s0), [o0] "v"(so), [rs] "s"(srs)
        : "memory", "scc");
  }
}

// K operand of key block kb (keys 32 kb + r) and d-step s for lane half g.
__device__ __forceinline__ i32x8 k8_operand(const uint8_t* kt, int kb, int s, int r, int g) {
  const uint8_t* line = kt + r * 256;
  const u32x4 lo = *reinterpret_cast<const u32x4*>(line + k8_slot(r, kb, 4 * s + g) * 16);
  const u32x4 hi = *reinterpret_cast<const u32x4*>(line + k8_slot(r, kb, 4 * s + 2 + g) * 16);
  return i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
               (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
}

// Exponent word of key 32 kb + r for lane half g: byte 0 = block g (d-step 0), byte 2 =
// block 2 + g (d-step 1), picked by the MFMA's op_sel.
__device__ __forceinline__ uint32_t k8_scales(const uint8_t* ks, int kb, int r, int g) {
  const uint32_t w = *reinterpret_cast<const uint32_t*>(ks + (32 * kb + r) * 4);
  return (w >> (8 * g)) & 0x00ff00ffu;
}

// One MX-FP8 MFMA of d-step S (exponent byte 2 S of both scale words).  The empty
// statement after it reads the result together with a and b, so all three are live at
// once and the result registers never share storage with the operands (with a zero
// accumulator the compiler would otherwise reuse their registers, which gives wrong
// results for this instruction).
template <int S>
__device__ __forceinline__ f32x16 mfma_q8(const i32x8& a, const i32x8& b, const f32x16& acc,
                                          uint32_t sa, uint32_t sb) {
  f32x16 r = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
      a, b, acc, 0, 0, (S == 0 ? 0 : 2), (int)sa, (S == 0 ? 0 : 2), (int)sb);
  asm volatile("" : "+v"(r) : "v"(a), "v"(b));
  return r;
}

// Q^T operand registers of one lane in the MX-FP8 path: both d-steps and the exponent word.
struct QFrag8 {
  i32x8 q[2];
  uint32_t sc;
};

// K^T operand registers of one lane for the current tile: the first d-step of both key
// blocks (refilled with the second d-step as the MFMAs consume them) and the exponents.
struct KFrag8 {
  i32x8 a[2];
  uint32_t sc[2];
};

__device__ __forceinline__ void k8_begin(KFrag8& kf, const uint8_t* kt, const uint8_t* ks,
                                         int r, int g) {
  kf.sc[0] = k8_scales(ks, 0, r, g);
  kf.sc[1] = k8_scales(ks, 1, r, g);
  kf.a[0] = k8_operand(kt, 0, 0, r, g);
  kf.a[1] = k8_operand(kt, 1, 0, r, g);
}

// MFMA i (0..3) of S^T = K Q^T on the MX-FP8 path: key block i % 2, d-step i / 2.  The two
// first-step MFMAs also refill their block's operand with the second d-step.
__device__ __forceinline__ void qk_q8_step(int i, f32x16 (&s_next)[2], KFrag8& kf,
                                           const uint8_t* kt, const QFrag8& qf, int r, int g) {
  const int kb = i & 1;
  const i32x8 a = kf.a[kb];
  if (i < 2) {
    kf.a[kb] = k8_operand(kt, kb, 1, r, g);
    s_next[kb] = mfma_q8<0>(a, qf.q[0], f32x16{}, kf.sc[kb], qf.sc);
  } else {
    s_next[kb] = mfma_q8<1>(a, qf.q[1], s_next[kb], kf.sc[kb], qf.sc);
  }
}

// K operand of S^T MFMA number i (chains alternate: block b = i % 2, d step s = i / 2).
__device__ __forceinline__ bf16x8 k_operand(const uint16_t* kt, int i, int r, int g) {
  return lds_b128(kt + k_off(32 * (i & 1) + r, 2 * (i >> 1) + g));
}

// V^T operand of PV MFMA number i (output block db = i % 4, key step s = i / 4): two
// transposed 8-byte reads of four consecutive keys each.
__device__ __forceinline__ bf16x8 v_operand(const uint16_t* vt, int i, int lane) {
  const int db = i & 3, s = i >> 2;
  const int grp = lane >> 4;                 // 16-lane group
  const int lg = lane & 15;
  const int g = grp >> 1;
  const int d = 32 * db + 16 * (grp & 1) + 4 * (lg & 3);
  const int chunk = d >> 3, half = (d >> 2) & 1;
  bf16x8 out;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int key = 32 * (s >> 1) + 8 * (2 * (s & 1) + c) + 4 * g + (lg >> 2);
    const bf16x4 x = lds_tr_b64(vt + v_off(key, chunk) + 4 * half);
#pragma unroll
    for (int t = 0; t < 4; ++t) out[4 * c + t] = x[t];
  }
  return out;
}

// Keys past the sequence end take no part in max or sum.  Register v of block b holds
// key key0 + 4g + (32b + 8(v/4) + v%4): compare that compile-time offset with one
// per-lane limit so no per-element index stays live.
__device__ __forceinline__ void mask_tail(f32x16 (&st)[2], int key0, int N, int g) {
  const int lim = N - key0 - 4 * g;
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int v = 0; v < 16; ++v)
      if (32 * b + (v >> 2) * 8 + (v & 3) >= lim) st[b][v] = -__builtin_inff();
}

// Maxima (of score rows, and the running ones) use IEEE maximum (v_maximum / v_maximum3):
// with no NaN in the scores it equals fmaxf, and unlike fmaxf it needs no canonicalising
// copy of its operands.
__device__ __forceinline__ float fmax_row(float a, float b) { return __builtin_elementwise_maximum(a, b); }

__device__ __forceinline__ float row_max(const f32x16 (&st)[2]) {
  float mx = st[0][0];
#pragma unroll
  for (int v = 1; v < 16; ++v) mx = fmax_row(mx, st[0][v]);
#pragma unroll
  for (int v = 0; v < 16; ++v) mx = fmax_row(mx, st[1][v]);
  const uint32_t b = __builtin_bit_cast(uint32_t, mx);
  const auto sw = __builtin_amdgcn_permlane32_swap(b, b, false, false);
  return fmax_row(__builtin_bit_cast(float, (uint32_t)sw[0]), __builtin_bit_cast(float, (uint32_t)sw[1]));
}

// Four elements of a running lane-local row max over a score tile, elements
// 1 + 4k .. 4 + 4k (k = 0..7; element 0 starts the chain), for the MFMA slots that carry
// no other VALU work.
__device__ __forceinline__ void row_max_part(const f32x16 (&st)[2], int k, float& mx) {
#pragma unroll
  for (int e = 1 + 4 * k; e <= 4 + 4 * k && e < 32; ++e) mx = fmax_row(mx, st[e >> 4][e & 15]);
}

// Combine a lane-local row max with the other lane half of the row.
__device__ __forceinline__ float row_max_join(float mx) {
  const uint32_t b = __builtin_bit_cast(uint32_t, mx);
  const auto sw = __builtin_amdgcn_permlane32_swap(b, b, false, false);
  return fmax_row(__builtin_bit_cast(float, (uint32_t)sw[0]), __builtin_bit_cast(float, (uint32_t)sw[1]));
}

struct RowState {
  float m_ref;   // reference max (log2 units) of P = exp2(S*c - m_ref)
  float m_true;  // running max of the kept tiles (BLASST metric)
  float l_half;  // this lane's share of the kept row sum, relative to m_ref
  float lse;     // MX-FP8 64-key steps: m_ref + log2(row sum) after the last kept tile
};

// Lazy rescale at the start of a kept tile with row max m_hat (log2 units).
__device__ __forceinline__ void rescale_if_needed(RowState& rs, f32x16 (&o)[4], float m_hat) {
  rs.m_true = fmax_row(rs.m_true, m_hat);
  const bool need = m_hat > rs.m_ref + kRescaleSlack;
  if (__ballot(need) != 0) {
    const float m_new = need ? m_hat : rs.m_ref;
    const float alpha = exp2_fast(rs.m_ref - m_new);
    rs.l_half *= alpha;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
    rs.m_ref = m_new;
  }
}

// An empty asm statement that reads x: the value must exist at this point of the
// instruction stream.  With 32-key decisions the consumers of a softmax sit under branches;
// this keeps its exponentials under the S_{j+1} MFMAs that hide them instead of letting the
// compiler sink them into the branches, after the MFMAs.
__device__ __forceinline__ void pin_here(float x) { asm volatile("" ::"v"(x)); }
__device__ __forceinline__ void pin_here(const bf16x8& x) { asm volatile("" ::"v"(x)); }

// Softmax numerator of S^T element e (0..31, block e / 16, register e % 16).
__device__ __forceinline__ void softmax_elem(const f32x16 (&st)[2], int e, float c, float neg_m,
                                             float& psum, bf16x8 (&pf)[4]) {
  const int b = e >> 4, v = e & 15;
  const float x = exp2_fast(fmaf(st[b][v], c, neg_m));
  psum += x;
  pf[2 * b + (v >> 3)][v & 7] = (__bf16)x;
}

// Softmax numerator of element e without the row sum: the value is kept in xs[e] and
// added up after the P V MFMAs are issued, in element order.
__device__ __forceinline__ void softmax_elem_keep(const f32x16 (&st)[2], int e, float c,
                                                  float neg_m, float (&xs)[32],
                                                  bf16x8 (&pf)[4]) {
  const int b = e >> 4, v = e & 15;
  const float x = exp2_fast(fmaf(st[b][v], c, neg_m));
  xs[e] = x;
  pf[2 * b + (v >> 3)][v & 7] = (__bf16)x;
}

// Kept tile j: softmax of S_j interleaved with the 16 MFMAs of S_{j+1} = K_{j+1} Q^T,
// then O += P V_j.  MFMA operands are read from LDS two MFMAs ahead.
__device__ __forceinline__ void kept_tile(RowState& rs, f32x16 (&o)[4], const f32x16 (&s_cur)[2],
                                          float m_hat, float c, f32x16 (&s_next)[2],
                                          const uint16_t* kt, const uint16_t* vt,
                                          const bf16x8 (&qf)[8], int r, int g, int lane,
                                          float& rmax_next, bool contribute = true) {
  // contribute == false (uniform): the tile runs the same instructions but adds nothing --
  // exp2(S c - inf) = 0 for every element (S is finite or -inf), and the running max and
  // sum stay as they are.
  if (contribute) rescale_if_needed(rs, o, m_hat);
  const float neg_m = contribute ? -rs.m_ref : -__builtin_inff();
  float xs[32];
  bf16x8 pf[4];
  constexpr int RK = 3;   // operand ring: reads issued two MFMAs ahead
  bf16x8 ka[RK], va[RK];
#pragma unroll
  for (int i = 0; i < RK - 1; ++i) ka[i] = k_operand(kt, i, r, g);
  sched_fence();
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    if (i + RK - 1 < 16)
      ka[(i + RK - 1) % RK] = k_operand(kt, i + RK - 1, r, g);
    else
      va[i + RK - 1 - 16] = v_operand(vt, i + RK - 1 - 16, lane);
    f32x16& acc = s_next[i & 1];
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[i % RK], qf[i >> 1],
                                                  i < 2 ? f32x16{} : acc, 0, 0, 0);
    // elements 0-23 here: two under each of the first eight MFMAs, one under the rest
    if (i < 8) {
      softmax_elem_keep(s_cur, 2 * i, c, neg_m, xs, pf);
      softmax_elem_keep(s_cur, 2 * i + 1, c, neg_m, xs, pf);
    } else {
      softmax_elem_keep(s_cur, 16 + (i - 8), c, neg_m, xs, pf);
    }
    sched_fence();
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    if (i + RK - 1 < 16) va[(i + RK - 1) % RK] = v_operand(vt, i + RK - 1, lane);
    o[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[i % RK], pf[i >> 2], o[i & 3], 0, 0, 0);
    // elements 24-31 (P block 3, first read by MFMA 12) under the first eight; the row
    // max of S_{j+1} (complete by now) under the other eight
    if (i < 8) {
      softmax_elem_keep(s_cur, 24 + i, c, neg_m, xs, pf);
    } else {
      if (i == 8) rmax_next = s_next[0][0];
      row_max_part(s_next, i - 8, rmax_next);
    }
    sched_fence();
  }
  __builtin_amdgcn_s_setprio(0);
  rmax_next = row_max_join(rmax_next);
  // The row sum goes after the P V MFMAs, where the VALU is otherwise idle, rather than
  // into the softmax phase, which is VALU-bound.
  float psum = 0.f;
#pragma unroll
  for (int e = 0; e < 32; ++e) psum += xs[e];
  rs.l_half += psum;
}

// Kept tile j on the MX-FP8 path: as kept_tile, with S_{j+1} from four scaled fp8 MFMAs
// that carry eight softmax elements each.  (The P V loop is written out in both tile
// bodies: moving it into a shared inline function changes the bf16 kernel's schedule.)
__device__ __forceinline__ void kept_tile_q8(RowState& rs, f32x16 (&o)[4],
                                             const f32x16 (&s_cur)[2], float m_hat, float c,
                                             f32x16 (&s_next)[2], const uint8_t* kt,
                                             const uint8_t* ks, const uint16_t* vt,
                                             const QFrag8& qf, int r, int g, int lane,
                                             float& rmax_next) {
  rescale_if_needed(rs, o, m_hat);
  const float neg_m = -rs.m_ref;
  float xs[32];
  bf16x8 pf[4];
  bf16x8 va[3];
  KFrag8 kf;
  k8_begin(kf, kt, ks, r, g);
  sched_fence();
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    qk_q8_step(i, s_next, kf, kt, qf, r, g);
    if (i >= 2) va[i - 2] = v_operand(vt, i - 2, lane);
#pragma unroll
    for (int e = 0; e < 6; ++e) softmax_elem_keep(s_cur, 6 * i + e, c, neg_m, xs, pf);
    sched_fence();
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    if (i + 2 < 16) va[(i + 2) % 3] = v_operand(vt, i + 2, lane);
    o[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[i % 3], pf[i >> 2], o[i & 3], 0, 0, 0);
    if (i < 8) {
      softmax_elem_keep(s_cur, 24 + i, c, neg_m, xs, pf);   // P block 3, as in kept_tile
    } else {
      if (i == 8) rmax_next = s_next[0][0];                  // the row max, as in kept_tile
      row_max_part(s_next, i - 8, rmax_next);
    }
    sched_fence();
  }
  __builtin_amdgcn_s_setprio(0);
  rmax_next = row_max_join(rmax_next);
  float psum = 0.f;                          // after the P V MFMAs, as in kept_tile
#pragma unroll
  for (int e = 0; e < 32; ++e) psum += xs[e];
  rs.l_half += psum;
}

// Skipped tile j: only S_{j+1} = K_{j+1} Q^T.
__device__ __forceinline__ void skipped_tile(f32x16 (&s_next)[2], const uint16_t* kt,
                                             const bf16x8 (&qf)[8], int r, int g) {
  constexpr int RK = 3;   // operand ring: reads issued two MFMAs ahead
  bf16x8 ka[RK];
#pragma unroll
  for (int i = 0; i < RK - 1; ++i) ka[i] = k_operand(kt, i, r, g);
  sched_fence();
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    if (i + RK - 1 < 16) ka[(i + RK - 1) % RK] = k_operand(kt, i + RK - 1, r, g);
    f32x16& acc = s_next[i & 1];
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[i % RK], qf[i >> 1],
                                                  i < 2 ? f32x16{} : acc, 0, 0, 0);
    sched_fence();
  }
}

// Skipped tile j with the row max of S_{j+1} (before any tail mask), taken after its
// MFMAs.
__device__ __forceinline__ float skipped_tile_rmax(f32x16 (&s_next)[2], const uint16_t* kt,
                                                   const bf16x8 (&qf)[8], int r, int g) {
  skipped_tile(s_next, kt, qf, r, g);
  return row_max(s_next);
}

// Skipped tile j on the MX-FP8 path: only S_{j+1}.
__device__ __forceinline__ void skipped_tile_q8(f32x16 (&s_next)[2], const uint8_t* kt,
                                                const uint8_t* ks, const QFrag8& qf, int r,
                                                int g) {
  KFrag8 kf;
  k8_begin(kf, kt, ks, r, g);
  sched_fence();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    qk_q8_step(i, s_next, kf, kt, qf, r, g);
    sched_fence();
  }
}

// The same with the row max of S_{j+1}, as skipped_tile_rmax.
__device__ __forceinline__ float skipped_tile_q8_rmax(f32x16 (&s_next)[2], const uint8_t* kt,
                                                      const uint8_t* ks, const QFrag8& qf,
                                                      int r, int g) {
  skipped_tile_q8(s_next, kt, ks, qf, r, g);
  return row_max(s_next);
}

// Q operand registers of the bf16 path (eight d-steps) and of the MX-FP8 path.
template <bool Q8>
struct QFragOf {
  typedef bf16x8 type[8];
};
template <>
struct QFragOf<true> {
  typedef QFrag8 type;
};

template <int RULE>
__device__ __forceinline__ bool row_keeps(const RowState& rs, float m_hat, float thr) {
  if constexpr (RULE == kRuleDynSparse) {
    const float l_row = half_sum(rs.l_half);
    return !(m_hat - (rs.m_ref + log2_fast(l_row)) < thr);   // Eq. 5, log2 units
  } else {
    return !(m_hat - rs.m_true < thr);
  }
}

// The same against the LSE cached in rs.lse.  The LSE changes only when a tile is kept,
// so a run of skipped tiles reuses it instead of recomputing it before every vote.
template <int RULE>
__device__ __forceinline__ bool row_keeps_cached(const RowState& rs, float m_hat, float thr) {
  if constexpr (RULE == kRuleDynSparse)
    return !(m_hat - rs.lse < thr);
  else
    return !(m_hat - rs.m_true < thr);
}

// Per-thread constants of the key-tile loop.
struct LoopCtx {
  __amdgpu_buffer_rsrc_t krs;   // K / V of this head as buffer resources
  __amdgpu_buffer_rsrc_t vrs;
  __amdgpu_buffer_rsrc_t ksrs;  // MX-FP8 path: the exponents of K (4 bytes per key)
  uint32_t koff, voff;          // lane offsets inside a 1 KiB tile block
  uint8_t* mask_row;            // this decision unit's row of the skip mask, or null
  float c;
  float thr;
  // The rule's threshold on this lane's query row, +inf past the last row: a vote taken
  // against it is "skip" for rows past N (their margin is finite once a tile is kept, and
  // every vote follows the first kept tile), so the votes need no row mask.
  float thr_row;
  int N, n_kt, w, lane, r, g;
  int rows_valid;               // valid query rows of this decision unit
  bool valid, ragged;
  // Diagonal-first visit order around key tile diag_c (the tile holding the workgroup's
  // first query row): diag_c, diag_c + 1, diag_c - 1, ..., then on along the longer side
  // once the shorter one (diag_m tiles) is used up.
  bool diag_right;
  int diag_c, diag_m;
};

// Key tile visited at loop step s (0 <= s < n_kt) in order ORDER.
template <int ORDER>
__device__ __forceinline__ int key_tile_at(int s, const LoopCtx& cx) {
  if constexpr (ORDER == kOrderAscending) {
    return s;
  } else {
    if (s <= 2 * cx.diag_m) return (s & 1) ? cx.diag_c + ((s + 1) >> 1) : cx.diag_c - (s >> 1);
    const int t = s - 2 * cx.diag_m;
    return cx.diag_right ? cx.diag_c + cx.diag_m + t : cx.diag_c - cx.diag_m - t;
  }
}

// Key tile of step s, or the first tile past the sequence for steps beyond the loop (its
// loads come back as zeros and are never read).
template <int ORDER>
__device__ __forceinline__ int key_tile_or_past(int s, const LoopCtx& cx) {
  if constexpr (ORDER == kOrderAscending) return s;   // already past the end when s >= n_kt
  return s < cx.n_kt ? key_tile_at<ORDER>(s, cx) : cx.n_kt;
}

// Epilogue of one lane: renormalise O over the kept keys, store it as bf16, and the
// natural-log LSE of the row over its kept keys.  A row whose unit kept no key tile
// (possible only with a reused mask) gets zeros and -inf.
__device__ __forceinline__ void store_rows(const FwdParams& p, const f32x16 (&o)[4],
                                           const RowState& rs, const LoopCtx& cx,
                                           size_t head_off, int bh, int qrow) {
  const float l_row = half_sum(rs.l_half);
  const bool any = l_row > 0.f;
  const float inv = any ? 1.0f / l_row : 0.f;
  if (cx.valid) {
    uint16_t* orow = p.o + head_off + (size_t)qrow * kD;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        bf16x4 h;
#pragma unroll
        for (int i = 0; i < 4; ++i) h[i] = (__bf16)(o[db][4 * grp + i] * inv);
        *reinterpret_cast<u32x2*>(orow + 32 * db + 8 * grp + 4 * cx.g) =
            __builtin_bit_cast(u32x2, h);
      }
    if (p.lse != nullptr && cx.g == 0)
      p.lse[(size_t)bh * cx.N + qrow] =
          any ? (rs.m_ref + log2_fast(l_row)) * 0.69314718055994530942f : -__builtin_inff();
  }
}

// Skipped key tiles (or 32-key halves) of one decision unit, and the keys they hold; the
// skipped elements are rows_valid times the keys, formed once after the loop.
struct SkipCount {
  uint32_t tiles = 0;
  uint32_t keys = 0;
};

// Stage the K tile starting at key key0 into K buffer buf (bf16, or MX-FP8 codes and
// exponents).
template <bool Q8>
__device__ __forceinline__ void load_k_tile(Smem& sm, int buf, const LoopCtx& cx, int key0) {
  if constexpr (Q8)
    load_k8_tile(reinterpret_cast<uint8_t*>(sm.k[buf]), sm.ks[buf], cx.krs, cx.ksrs, cx.koff,
                 key0, cx.w, cx.lane);
  else
    load_tile_lds(sm.k[buf], cx.krs, cx.koff, key0, cx.w);
}

// One loop step j, visiting key tile key_tile_at(j) (written "tile j" below; LDS buffers
// rotate with the step).  On entry s_cur holds S_j, mhat its row max (log2 units), vote the
// workgroup's skip word for tile j as this wave needs it (below), keep_own the decision for
// tile j of this wave's decision unit when that unit is the wave's own 32 rows (UNIT = 32;
// with the workgroup's 128 rows it comes from the vote), and v_ready whether V_j is already
// in LDS (buffer j % 2).  keep_any (some unit of the workgroup keeps tile j) is set from
// the vote.  On exit s_next holds S_{j+1}, the other state refers to tile j+1, and every
// wave has passed the barrier that publishes K_{j+2}, the V_{j+1} buffer if it was
// requested, and the tile-(j+1) votes.
//
// Votes.  Byte w of vote buffer b is 1 while wave w's last vote in that buffer was "skip".
// A wave writes its byte only when its vote changes (marks records which of its two bytes
// are set), and only a wave that votes skip reads the word back: one that keeps the tile
// knows that the workgroup keeps it.  The workgroup skips a tile when all four bytes are 1.
// With nothing skipped the votes therefore cost no LDS traffic at all.
//
// V tiles are fetched for tiles some unit keeps.  V_{j+1} is requested one iteration
// ahead when tile j is kept (runs of kept tiles are the common case); after a skipped
// tile, a kept tile's V is requested at the start of its own iteration, so a run of
// skipped tiles streams K alone.
template <int RULE, int UNIT, int ORDER, bool Q8>
__device__ __forceinline__ void key_tile_step(int j, const f32x16 (&s_cur)[2], f32x16 (&s_next)[2],
                                              float& mhat, bool& keep_own, bool& keep_any,
                                              uint32_t& vote, uint32_t& marks, bool& v_ready,
                                              RowState& rs, f32x16 (&o)[4],
                                              const typename QFragOf<Q8>::type& qf, Smem& sm,
                                              const LoopCtx& cx, SkipCount& sk) {
  const int nb = (j + 1) & 1;
  const bool has_next = (j + 1) < cx.n_kt;
  const int tj = key_tile_at<ORDER>(j, cx);          // key tiles of steps j, j+1, j+2
  const int tn = key_tile_or_past<ORDER>(j + 1, cx);
  const int tn2 = key_tile_or_past<ORDER>(j + 2, cx);
  // The K tile two steps ahead does not depend on the decision: its DMA goes out while a
  // vote word read after the last barrier is still in flight.
  load_k_tile<Q8>(sm, j & 1, cx, tn2 * kTK);
  if constexpr (RULE != kRuleDense) {
    keep_any = __builtin_amdgcn_readfirstlane(vote) != kAllSkip;
    if constexpr (UNIT == kTQ) keep_own = keep_any;
  }
  if (cx.mask_row != nullptr && (UNIT == kTQ ? cx.w == 0 : true) && cx.lane == 0)
    cx.mask_row[tj] = keep_own ? 0 : 1;

  // Tile loads.  Past the last tile the range check returns zeros into buffers nobody
  // reads.  A kept tile after a skipped one fetches its own V first and waits for it (all
  // waves' shares) before anything else: real masks change between kept and skipped
  // rarely (about one tile in twenty at 30 % sparsity on video inputs), and this keeps
  // the kept-tile code identical to the dense kernel's.
  const bool late_v = keep_any && !v_ready;
  if (late_v) {
    load_tile_lds(sm.v[j & 1], cx.vrs, cx.voff, tj * kTK, cx.w);
    asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
  }
  if (keep_any) load_tile_lds(sm.v[nb], cx.vrs, cx.voff, tn * kTK, cx.w);

  // S_{j+1} is computed on both paths (on the last tile it reads a stale buffer and is
  // dropped), with its row max before any tail mask: under the P V MFMAs of a kept tile,
  // after the MFMAs of a skipped one.
  float rmax = 0.f;
  if (keep_own) {
    if constexpr (Q8)
      kept_tile_q8(rs, o, s_cur, mhat, cx.c, s_next, reinterpret_cast<const uint8_t*>(sm.k[nb]),
                   sm.ks[nb], sm.v[j & 1], qf, cx.r, cx.g, cx.lane, rmax);
    else
      kept_tile(rs, o, s_cur, mhat, cx.c, s_next, sm.k[nb], sm.v[j & 1], qf, cx.r, cx.g,
                cx.lane, rmax);
    // The MX-FP8 path caches the LSE for its votes (its kept tiles are shorter, and taking
    // the log out of the vote chain pays there); the bf16 path keeps it in the chain.
    if constexpr (Q8 && RULE == kRuleDynSparse)
      rs.lse = rs.m_ref + log2_fast(half_sum(rs.l_half));
  } else {
    sk.tiles += 1;
    sk.keys += (uint32_t)min(kTK, cx.N - tj * kTK);
    if constexpr (Q8)
      rmax = skipped_tile_q8_rmax(s_next, reinterpret_cast<const uint8_t*>(sm.k[nb]), sm.ks[nb],
                                  qf, cx.r, cx.g);
    else
      rmax = skipped_tile_rmax(s_next, sm.k[nb], qf, cx.r, cx.g);
  }
  v_ready = keep_any;

  float mhat_next = 0.f;
  bool wave_keeps = true;
  if (has_next) {
    if (cx.ragged && tn == cx.n_kt - 1) {
      mask_tail(s_next, tn * kTK, cx.N, cx.g);
      rmax = row_max(s_next);
    }
    mhat_next = rmax * cx.c;
    if constexpr (RULE != kRuleDense) {
      wave_keeps = __ballot(Q8 ? row_keeps_cached<RULE>(rs, mhat_next, cx.thr_row)
                               : row_keeps<RULE>(rs, mhat_next, cx.thr_row)) != 0;
      const uint32_t mark = wave_keeps ? 0u : 1u;
      if (mark != ((marks >> nb) & 1u)) {
        if (cx.lane == 0) sm.vote[nb][cx.w] = (uint8_t)mark;
        marks ^= 1u << nb;
      }
    }
  }
  // Publish this wave's LDS traffic and its tile loads (read in the next iteration), then
  // meet the other waves.  (__syncthreads() would add a fence that makes the compiler
  // drain every load again on its own.)
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  if (has_next) {
    if constexpr (RULE != kRuleDense) {
      // Consumed by the next step.  The atomic load keeps the read under the branch.
      if (wave_keeps)
        vote = 0u;
      else
        vote = __atomic_load_n(reinterpret_cast<const uint32_t*>(sm.vote[nb]),
                               __ATOMIC_RELAXED);
      if constexpr (UNIT != kTQ) keep_own = wave_keeps;
    }
    mhat = mhat_next;
  }
}

// ---- 128-key decisions -------------------------------------------------------------
// With B_c = 128 one decision covers two consecutive 64-key tiles 2m, 2m+1 (a "pair"),
// visited in ascending order.  The pipeline keeps its 64-key steps and two score tiles in
// registers:
//   * first step of pair m (tile j = 2m, S_j already in registers): compute S_{j+1}, take
//     the pair's row max over both, vote (Eq. 5 against the LSE after pair m-1) and meet
//     the other waves at a barrier in the middle of the step; if the pair is kept, form
//     P_j and accumulate P_j V_j, the softmax running under the P.V MFMAs;
//   * second step (tile j+1): the ordinary kept or skipped tile body, which also computes
//     S of the next pair's first tile; no vote.
// V tiles follow the same policy as with 64-key decisions: the next tile's V is
// requested when the current pair is kept, and a kept pair after a skipped one fetches its
// first V tile late.

// 64-key tile of loop step j with 128-key decisions: tile j in ascending order; in
// diagonal-first order pair key_tile_at(j / 2) (the order runs over 128-key tiles, centred
// on the workgroup's own) and its tile j % 2.  A partial last pair still takes two steps:
// its second tile lies past the sequence end, so every key of it is masked.  Steps past
// the loop name a tile past the end.
template <int ORDER>
__device__ __forceinline__ int pair_tile(int j, const LoopCtx& cx) {
  if constexpr (ORDER == kOrderAscending) {
    return j;
  } else {
    const int n_pairs = (cx.n_kt + 1) >> 1;
    if ((j >> 1) >= n_pairs) return 2 * n_pairs;
    return 2 * key_tile_at<ORDER>(j >> 1, cx) + (j & 1);
  }
}

// Softmax of S_j (lazy reference max already updated) and O += P_j V_j: the first eight
// elements up front, then two under each of the first twelve P.V MFMAs, so that P block s
// is complete before MFMA 4 s reads it.
__device__ __forceinline__ void softmax_pv_tile(RowState& rs, f32x16 (&o)[4],
                                                const f32x16 (&s_cur)[2], float c,
                                                const uint16_t* vt, int lane) {
  const float neg_m = -rs.m_ref;
  float psum = 0.f;
  bf16x8 pf[4];
  bf16x8 va[3];
#pragma unroll
  for (int e = 0; e < 8; ++e) softmax_elem(s_cur, e, c, neg_m, psum, pf);
  va[0] = v_operand(vt, 0, lane);
  va[1] = v_operand(vt, 1, lane);
  sched_fence();
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    if (i + 2 < 16) va[(i + 2) % 3] = v_operand(vt, i + 2, lane);
    o[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[i % 3], pf[i >> 2], o[i & 3], 0, 0, 0);
    if (i < 12) {
      softmax_elem(s_cur, 8 + 2 * i, c, neg_m, psum, pf);
      softmax_elem(s_cur, 9 + 2 * i, c, neg_m, psum, pf);
    }
    sched_fence();
  }
  __builtin_amdgcn_s_setprio(0);
  rs.l_half += psum;
}

// First step of pair m = j / 2.  On entry s_cur holds S_j and mhat its row max; v_ready
// tells whether V_j was requested in the previous step.  On exit s_next holds S_{j+1},
// mhat the pair's row max, keep_own / keep_any the pair's decisions.
template <int RULE, int UNIT, bool Q8, int ORDER>
__device__ __forceinline__ void pair_first_step(int j, const f32x16 (&s_cur)[2],
                                                f32x16 (&s_next)[2], float& mhat,
                                                bool& keep_own, bool& keep_any, bool& v_ready,
                                                RowState& rs, f32x16 (&o)[4],
                                                const typename QFragOf<Q8>::type& qf,
                                                Smem& sm, const LoopCtx& cx, SkipCount& sk) {
  const int nb = (j + 1) & 1;
  const int tj = pair_tile<ORDER>(j, cx);             // the pair's two tiles: tj, tj + 1
  load_k_tile<Q8>(sm, j & 1, cx, pair_tile<ORDER>(j + 2, cx) * kTK);
  if constexpr (Q8)
    skipped_tile_q8(s_next, reinterpret_cast<const uint8_t*>(sm.k[nb]), sm.ks[nb], qf, cx.r,
                    cx.g);
  else
    skipped_tile(s_next, sm.k[nb], qf, cx.r, cx.g);
  // Keys past the end (a partial last tile, or no second tile at all) do not count.
  if ((tj + 2) * kTK > cx.N) mask_tail(s_next, (tj + 1) * kTK, cx.N, cx.g);
  const float mhat_pair = fmax_row(mhat, row_max(s_next) * cx.c);
  if constexpr (RULE != kRuleDense) {
    const bool wave_keeps = __ballot(row_keeps<RULE>(rs, mhat_pair, cx.thr_row)) != 0;
    if (cx.lane == 0) sm.vote[0][cx.w] = wave_keeps ? 1 : 0;
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    keep_any = __builtin_amdgcn_readfirstlane(*reinterpret_cast<const uint32_t*>(sm.vote[0])) != 0;
    keep_own = UNIT == kTQ ? keep_any : wave_keeps;
  }
  if (cx.mask_row != nullptr && (UNIT == kTQ ? cx.w == 0 : true) && cx.lane == 0)
    cx.mask_row[tj >> 1] = keep_own ? 0 : 1;
  if (keep_any && !v_ready) {
    load_tile_lds(sm.v[j & 1], cx.vrs, cx.voff, tj * kTK, cx.w);
    asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
  }
  if (keep_any) load_tile_lds(sm.v[nb], cx.vrs, cx.voff, (tj + 1) * kTK, cx.w);
  if (keep_own) {
    rescale_if_needed(rs, o, mhat_pair);
    softmax_pv_tile(rs, o, s_cur, cx.c, sm.v[j & 1], cx.lane);
  } else {
    sk.tiles += 1;
    sk.keys += (uint32_t)min(2 * kTK, cx.N - tj * kTK);
  }
  v_ready = keep_any;
  mhat = mhat_pair;
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Second step of the pair (tile j = 2m + 1, decisions from the first step): the tile
// body, which also computes S_{j+1} of the next pair's first tile.
template <int RULE, int UNIT, bool Q8, int ORDER>
__device__ __forceinline__ void pair_second_step(int j, const f32x16 (&s_cur)[2],
                                                 f32x16 (&s_next)[2], float& mhat,
                                                 bool keep_own, bool keep_any, bool& v_ready,
                                                 RowState& rs, f32x16 (&o)[4],
                                                 const typename QFragOf<Q8>::type& qf,
                                                 Smem& sm, const LoopCtx& cx) {
  const int nb = (j + 1) & 1;
  const int tn = pair_tile<ORDER>(j + 1, cx);        // the next pair's first tile
  load_k_tile<Q8>(sm, j & 1, cx, pair_tile<ORDER>(j + 2, cx) * kTK);
  if (keep_any) load_tile_lds(sm.v[nb], cx.vrs, cx.voff, tn * kTK, cx.w);
  float rmax;                                        // row max of S_{j+1}, as in key_tile_step
  if (keep_own) {
    if constexpr (Q8)
      kept_tile_q8(rs, o, s_cur, mhat, cx.c, s_next, reinterpret_cast<const uint8_t*>(sm.k[nb]),
                   sm.ks[nb], sm.v[j & 1], qf, cx.r, cx.g, cx.lane, rmax);
    else
      kept_tile(rs, o, s_cur, mhat, cx.c, s_next, sm.k[nb], sm.v[j & 1], qf, cx.r, cx.g,
                cx.lane, rmax);
  } else {
    if constexpr (Q8)
      rmax = skipped_tile_q8_rmax(s_next, reinterpret_cast<const uint8_t*>(sm.k[nb]), sm.ks[nb],
                                  qf, cx.r, cx.g);
    else
      rmax = skipped_tile_rmax(s_next, sm.k[nb], qf, cx.r, cx.g);
  }
  v_ready = keep_any;
  if (tn < cx.n_kt) {
    if ((tn + 1) * kTK > cx.N) {
      mask_tail(s_next, tn * kTK, cx.N, cx.g);
      rmax = row_max(s_next);
    }
    mhat = rmax * cx.c;
  }
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// ---- 32-key decisions ---------------------------------------------------------------
// With B_c = 32 every 64-key tile holds two decision tiles, its key halves h0 (S block 0)
// and h1 (block 1), visited in ascending order.  h0 of tile j is voted at the end of step
// j-1 against the LSE after tile j-1, as with 64-key decisions but on its own row max.
// h1 is voted against the LSE after h0:
//   * if h0 is skipped that LSE is the same, so h1 is voted together with h0;
//   * if h0 is kept, the step computes the softmax of both halves under the MFMAs of
//     S_{j+1} (h1 speculatively, its row sum kept apart), adds h0's sum, takes h1's
//     decision (from the certain-keep bit voted with h0 when some row holds it, see
//     half_votes; otherwise voted here, with an LDS exchange and a barrier for 128-row
//     units, the wave alone for 32-row units) and then adds h1's sum and issues h1's
//     eight P.V MFMAs only if h1 is kept.  h0's eight P.V MFMAs carry the lane-local
//     block maxima of S_{j+1}; the other paths take them after their MFMAs.
// The lazy reference max is raised to the larger half max of the tile whenever the tile
// is entered with a kept half; a half skipped after that only lowers P of the other half
// by a bounded factor (its max is below the LSE), never the LSE itself.

// Raise the lazy reference max (as rescale_if_needed, without the BLASST running max).
__device__ __forceinline__ void raise_reference(RowState& rs, f32x16 (&o)[4], float m_hat) {
  const bool need = m_hat > rs.m_ref + kRescaleSlack;
  if (__ballot(need) != 0) {
    const float m_new = need ? m_hat : rs.m_ref;
    const float alpha = exp2_fast(rs.m_ref - m_new);
    rs.l_half *= alpha;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
    rs.m_ref = m_new;
  }
}

// Row max of one 32-key block of S^T.
__device__ __forceinline__ float block_max(const f32x16& st) {
  float mx = st[0];
#pragma unroll
  for (int v = 1; v < 16; ++v) mx = fmax_row(mx, st[v]);
  return row_max_join(mx);
}

// S_{j+1} = K_{j+1} Q^T with the softmax of both halves of S_j under its 16 MFMAs (block
// b relative to reference -neg_m_b; -inf makes a block contribute nothing), the row sums
// of the halves kept apart.  Also reads the first two V operands.
__device__ __forceinline__ void qk_softmax_halves(const f32x16 (&s_cur)[2], float c,
                                                  float neg_m0, float neg_m1, float& psum0,
                                                  float& psum1, bf16x8 (&pf)[4],
                                                  bf16x8 (&va)[3], f32x16 (&s_next)[2],
                                                  const uint16_t* kt, const uint16_t* vt,
                                                  const bf16x8 (&qf)[8], int r, int g,
                                                  int lane) {
  bf16x8 ka[3];
  ka[0] = k_operand(kt, 0, r, g);
  ka[1] = k_operand(kt, 1, r, g);
  sched_fence();
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    if (i + 2 < 16)
      ka[(i + 2) % 3] = k_operand(kt, i + 2, r, g);
    else
      va[i - 14] = v_operand(vt, i - 14, lane);
    f32x16& acc = s_next[i & 1];
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[i % 3], qf[i >> 1],
                                                  i < 2 ? f32x16{} : acc, 0, 0, 0);
    if (i < 8) {
      softmax_elem(s_cur, 2 * i, c, neg_m0, psum0, pf);
      softmax_elem(s_cur, 2 * i + 1, c, neg_m0, psum0, pf);
      pin_here(psum0);
    } else {
      softmax_elem(s_cur, 2 * i, c, neg_m1, psum1, pf);
      softmax_elem(s_cur, 2 * i + 1, c, neg_m1, psum1, pf);
      pin_here(psum1);
    }
    if ((i & 3) == 3) pin_here(pf[i >> 2]);
    sched_fence();
  }
  __builtin_amdgcn_s_setprio(0);
}

// The same on the MX-FP8 path: the four scaled MFMAs of S_{j+1} carry eight elements
// each, the first two h0's and the last two h1's.
__device__ __forceinline__ void qk_softmax_halves_q8(const f32x16 (&s_cur)[2], float c,
                                                     float neg_m0, float neg_m1, float& psum0,
                                                     float& psum1, bf16x8 (&pf)[4],
                                                     bf16x8 (&va)[3], f32x16 (&s_next)[2],
                                                     const uint8_t* kt, const uint8_t* ks,
                                                     const uint16_t* vt, const QFrag8& qf,
                                                     int r, int g, int lane) {
  KFrag8 kf;
  k8_begin(kf, kt, ks, r, g);
  sched_fence();
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    qk_q8_step(i, s_next, kf, kt, qf, r, g);
    if (i >= 2) va[i - 2] = v_operand(vt, i - 2, lane);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (i < 2)
        softmax_elem(s_cur, 8 * i + e, c, neg_m0, psum0, pf);
      else
        softmax_elem(s_cur, 8 * i + e, c, neg_m1, psum1, pf);
    }
    pin_here(i < 2 ? psum0 : psum1);
    pin_here(pf[i]);
    sched_fence();
  }
  __builtin_amdgcn_s_setprio(0);
}

// Lane-local maxima of the two 32-key blocks of a score tile: elements 1 + 2k and 2 + 2k
// of each block (k = 0..7; element 0 starts each chain), for P.V MFMA slots that carry no
// other VALU work.  block_max_join completes them.
__device__ __forceinline__ void block_max_part(const f32x16 (&st)[2], int k, float (&bm)[2]) {
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    if (k == 0) bm[b] = st[b][0];
#pragma unroll
    for (int v = 1 + 2 * k; v <= 2 + 2 * k && v < 16; ++v) bm[b] = fmax_row(bm[b], st[b][v]);
  }
}

// O += P V_j for the first key half (MFMAs 0-7, keys 0-31; va holds the operands of MFMAs
// 0 and 1 on entry, those of 8 and 9 on exit) and for the second (MFMAs 8-15).  The first
// half's eight MFMAs also carry the lane-local block maxima of st (S_{j+1}); the pins keep
// the compiler from merging them with the other paths' copies behind the MFMAs.
__device__ __forceinline__ void pv_first_half(f32x16 (&o)[4], const bf16x8 (&pf)[4],
                                              bf16x8 (&va)[3], const uint16_t* vt, int lane,
                                              const f32x16 (&st)[2], float (&bm)[2]) {
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    va[(i + 2) % 3] = v_operand(vt, i + 2, lane);
    o[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[i % 3], pf[i >> 2], o[i & 3], 0, 0, 0);
    block_max_part(st, i, bm);
    pin_here(bm[0]);
    pin_here(bm[1]);
    sched_fence();
  }
  __builtin_amdgcn_s_setprio(0);
}
__device__ __forceinline__ void pv_second_half(f32x16 (&o)[4], const bf16x8 (&pf)[4],
                                               bf16x8 (&va)[3], const uint16_t* vt, int lane) {
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int i = 8; i < 16; ++i) {
    if (i + 2 < 16) va[(i + 2) % 3] = v_operand(vt, i + 2, lane);
    o[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[i % 3], pf[i >> 2], o[i & 3], 0, 0, 0);
    sched_fence();
  }
  __builtin_amdgcn_s_setprio(0);
}

// Votes of this wave's rows on the two 32-key halves h0, h1 of the next tile, one bit each
// (a bit is set when some valid row keeps):
//   1  h0 is kept (Eq. 5 against the state after this tile),
//   2  h1 is kept against the same state (its decision when h0 is skipped),
//   4  h1 is kept once h0 is.  BLASST: exact, the running max then being max(m, m_h0).
//      DynSparse: a sufficient condition.  h0 adds at most 32 terms of at most 2^m_h0, so
//      the LSE afterwards is at most max(LSE, m_h0 + 5) + 1 (log2 units); 1/16 more covers
//      the rounding of the kernel's own sum and logarithm.  A decision unit without this
//      bit decides h1 mid-step against the LSE that includes h0.
// Contraction is off so that every comparison sees the rounded m_hat, as the mid-step
// decision does.
template <int RULE>
__device__ __forceinline__ uint32_t half_votes(const RowState& rs, const float (&mh)[2],
                                               const LoopCtx& cx) {
#pragma clang fp contract(off)
  float ref, ref1;
  if constexpr (RULE == kRuleDynSparse) {
    ref = rs.m_ref + log2_fast(half_sum(rs.l_half));
    ref1 = fmax_row(ref, mh[0] + 5.0f) + 1.0625f;
  } else {
    ref = rs.m_true;
    ref1 = fmax_row(rs.m_true, mh[0]);
  }
  const bool k0 = !(mh[0] - ref < cx.thr_row);
  const bool k1 = !(mh[1] - ref < cx.thr_row);
  const bool s1 = !(mh[1] - ref1 < cx.thr_row);
  return (__ballot(k0) != 0 ? 1u : 0u) | (__ballot(k1) != 0 ? 2u : 0u) |
         (__ballot(s1) != 0 ? 4u : 0u);
}

// One 64-key step j with 32-key decisions.  On entry s_cur holds S_j and mh its half row
// maxima (log2 units); vote[b] is nonzero when some wave of the workgroup set bit b of
// half_votes for tile j (the decisions of 128-row units), own[b] this wave's bit (those
// of 32-row units); lds_bytes mirrors this wave's bytes in the two vote buffers, which
// are stored only when they change.  On exit the same for tile j+1.
template <int RULE, int UNIT, bool Q8>
__device__ __forceinline__ void half_tile_step(int j, const f32x16 (&s_cur)[2],
                                               f32x16 (&s_next)[2], float (&mh)[2],
                                               uint32_t (&vote)[3], bool (&own)[3],
                                               uint32_t& lds_bytes,
                                               bool& v_ready, RowState& rs, f32x16 (&o)[4],
                                               const typename QFragOf<Q8>::type& qf,
                                               Smem& sm, const LoopCtx& cx, SkipCount& sk) {
  const int nb = (j + 1) & 1;
  const bool has_next = (j + 1) < cx.n_kt;
  load_k_tile<Q8>(sm, j & 1, cx, (j + 2) * kTK);
  bool keep0 = true, keep1_pre = true, sure1 = true, need_v = true;
  if constexpr (RULE != kRuleDense) {
    const bool any0 = __builtin_amdgcn_readfirstlane(vote[0]) != 0;
    const bool any1 = __builtin_amdgcn_readfirstlane(vote[1]) != 0;
    const bool anys = __builtin_amdgcn_readfirstlane(vote[2]) != 0;
    sure1 = UNIT == kTQ ? anys : __builtin_amdgcn_readfirstlane((int)own[2]) != 0;
    need_v = any0 || any1;
    // (readfirstlane keeps the 32-row units' own votes visibly wave-uniform, so the
    // compiler branches on them instead of predicating both paths)
    keep0 = UNIT == kTQ ? any0 : __builtin_amdgcn_readfirstlane((int)own[0]) != 0;
    keep1_pre = UNIT == kTQ ? any1 : __builtin_amdgcn_readfirstlane((int)own[1]) != 0;
  }
  if (need_v && !v_ready) {
    load_tile_lds(sm.v[j & 1], cx.vrs, cx.voff, j * kTK, cx.w);
    asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
  }
  if (need_v) load_tile_lds(sm.v[nb], cx.vrs, cx.voff, (j + 1) * kTK, cx.w);

  const bool h1_exists = j * kTK + 32 < cx.N;
  bool keep1 = false;
  bf16x8 pf[4], va[3];
  float psum0 = 0.f, psum1 = 0.f;
  float bm[2];   // lane-local block maxima of S_{j+1}
  if (keep0 || keep1_pre) {
    // h0 kept (h1 decided below), or h0 skipped and h1 kept: one body, h0's elements
    // relative to -inf in the second case.
    raise_reference(rs, o, keep0 ? fmax_row(mh[0], mh[1]) : mh[1]);
    if (keep0) rs.m_true = fmax_row(rs.m_true, mh[0]);
    if constexpr (Q8)
      qk_softmax_halves_q8(s_cur, cx.c, keep0 ? -rs.m_ref : -__builtin_inff(), -rs.m_ref,
                           psum0, psum1, pf, va, s_next,
                           reinterpret_cast<const uint8_t*>(sm.k[nb]), sm.ks[nb], sm.v[j & 1],
                           qf, cx.r, cx.g, cx.lane);
    else
      qk_softmax_halves(s_cur, cx.c, keep0 ? -rs.m_ref : -__builtin_inff(), -rs.m_ref, psum0,
                        psum1, pf, va, s_next, sm.k[nb], sm.v[j & 1], qf, cx.r, cx.g, cx.lane);
    sched_fence();
    keep1 = true;
    if (keep0) {
      rs.l_half += psum0;
      // h1 after h0: from the sure bit, or decided here against the state that includes h0
      // (DynSparse without a sure vote; the first tile, which has no votes).  The sure bit
      // is uniform over the decision unit, so every wave of the workgroup meets the barrier.
      const bool exact = RULE != kRuleDense && !sure1 && (RULE == kRuleDynSparse || j == 0);
      bool own1 = true;
      if (exact) {
        own1 = __ballot(row_keeps<RULE>(rs, mh[1], cx.thr_row)) != 0;
        if (UNIT == kTQ && cx.lane == 0) sm.vote_mid[cx.w] = own1 ? 1 : 0;
      }
      sched_fence();
      pv_first_half(o, pf, va, sm.v[j & 1], cx.lane, s_next, bm);  // under the vote exchange
      if constexpr (RULE != kRuleDense) {
        keep1 = sure1;
        if (exact) {
          if constexpr (UNIT == kTQ) {
            asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
            keep1 = __builtin_amdgcn_readfirstlane(
                        *reinterpret_cast<const uint32_t*>(sm.vote_mid)) != 0;
          } else {
            keep1 = __builtin_amdgcn_readfirstlane((int)own1) != 0;
          }
        }
      }
    } else {
      va[8 % 3] = v_operand(sm.v[j & 1], 8, cx.lane);
      va[9 % 3] = v_operand(sm.v[j & 1], 9, cx.lane);
#pragma unroll
      for (int k = 0; k < 8; ++k) block_max_part(s_next, k, bm);
    }
    if (keep1) {
      rs.l_half += psum1;
      rs.m_true = fmax_row(rs.m_true, mh[1]);
      sched_fence();
      pv_second_half(o, pf, va, sm.v[j & 1], cx.lane);
    }
  } else {
    if constexpr (Q8)
      skipped_tile_q8(s_next, reinterpret_cast<const uint8_t*>(sm.k[nb]), sm.ks[nb], qf, cx.r,
                      cx.g);
    else
      skipped_tile(s_next, sm.k[nb], qf, cx.r, cx.g);
#pragma unroll
    for (int k = 0; k < 8; ++k) block_max_part(s_next, k, bm);
  }
  keep1 = keep1 && h1_exists;
  if (cx.mask_row != nullptr && (UNIT == kTQ ? cx.w == 0 : true) && cx.lane == 0) {
    cx.mask_row[2 * j] = keep0 ? 0 : 1;
    if (h1_exists) cx.mask_row[2 * j + 1] = keep1 ? 0 : 1;
  }
  if (!keep0) {
    sk.tiles += 1;
    sk.keys += (uint32_t)min(32, cx.N - j * kTK);
  }
  if (h1_exists && !keep1) {
    sk.tiles += 1;
    sk.keys += (uint32_t)min(32, cx.N - j * kTK - 32);
  }
  v_ready = need_v;

  bool next_own0 = true, next_own1 = true, next_s1 = true;
  if (has_next) {
    if (cx.ragged && j + 1 == cx.n_kt - 1) {
      mask_tail(s_next, (j + 1) * kTK, cx.N, cx.g);
#pragma unroll
      for (int k = 0; k < 8; ++k) block_max_part(s_next, k, bm);
    }
    mh[0] = row_max_join(bm[0]) * cx.c;
    mh[1] = row_max_join(bm[1]) * cx.c;
    if constexpr (RULE != kRuleDense) {
      const uint32_t b = half_votes<RULE>(rs, mh, cx);
      next_own0 = (b & 1u) != 0;
      next_own1 = (b & 2u) != 0;
      next_s1 = (b & 4u) != 0;
      const uint32_t sh = 8u * (uint32_t)nb;
      if (((lds_bytes >> sh) & 0xffu) != b) {
        if (cx.lane == 0) sm.vote[nb][cx.w] = (uint8_t)b;
        lds_bytes ^= (((lds_bytes >> sh) & 0xffu) ^ b) << sh;
      }
    }
  }
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  if (has_next) {
    if constexpr (RULE != kRuleDense) {
      const uint32_t word = *reinterpret_cast<const uint32_t*>(sm.vote[nb]);
      vote[0] = word & 0x01010101u;
      vote[1] = word & 0x02020202u;
      vote[2] = word & 0x04040404u;
      own[0] = next_own0;
      own[1] = next_own1;
      own[2] = next_s1;
    }
  }
}

// UNIT: query rows per skip decision, 128 (the workgroup's tile) or 32 (one wave).
// ORDER: key-tile visit order (ascending or diagonal-first).
// Q8: Q and K in MX-FP8 (codes p.q8 / p.k8, exponents p.q_scales / p.k_scales), S = Q K^T
// on the scaled fp8 MFMA; everything after S is the same as with bf16 Q and K.
// BC: keys per skip decision: 64 (one tile), 128 (two tiles) or 32 (half a tile); 32
// walks keys in ascending order only.
template <int RULE, int UNIT, int ORDER, bool Q8, int BC = kTK>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads),
                          amdgpu_waves_per_eu(2, 2))) void
fa_fwd_kernel(FwdParams p) {
  static_assert(UNIT == kTQ || UNIT == 32, "decision unit is the tile or one wave");
  static_assert(BC == kTK || BC == 2 * kTK || BC == kTK / 2, "B_c is 32, 64 or 128");
  constexpr bool PAIR = BC == 2 * kTK;
  constexpr bool HALF = BC == kTK / 2;
  __shared__ __attribute__((aligned(16))) Smem sm;

  const int tid = threadIdx.x;
  // Query tile of this workgroup.  In ascending order every workgroup of a head streams
  // K/V from tile 0 on, so neighbours in dispatch order share tiles in L2 whatever query
  // tile they hold.  In diagonal-first order each query tile starts at its own position;
  // there the grid is padded to kXcds chunks of consecutive query tiles and x % kXcds (the
  // XCD the workgroup lands on) picks the chunk, so the workgroups sharing one XCD's L2
  // start close together and their outward walks overlap.  Padding workgroups exit here.
  int qt = blockIdx.x;
  if constexpr (ORDER == kOrderDiagonal) {
    const int chunk = (p.n_qt + kXcds - 1) / kXcds;
    qt = (int)(blockIdx.x % kXcds) * chunk + (int)(blockIdx.x / kXcds);
    if (qt >= p.n_qt) return;
  }
  const int bh = blockIdx.y;
  const int N = p.N;
  const size_t head_off = (size_t)bh * (size_t)N * kD;

  LoopCtx cx;
  const int head_bytes = N * (kD * 2);
  if constexpr (Q8) {
    cx.krs = __builtin_amdgcn_make_buffer_rsrc((void*)(p.k8 + head_off), (short)0, N * kD,
                                               0x00020000);
    cx.ksrs = __builtin_amdgcn_make_buffer_rsrc((void*)(p.k_scales + (size_t)bh * N * 4),
                                                (short)0, N * 4, 0x00020000);
  } else {
    cx.krs = __builtin_amdgcn_make_buffer_rsrc((void*)(p.k + head_off), (short)0, head_bytes,
                                               0x00020000);
  }
  cx.vrs = __builtin_amdgcn_make_buffer_rsrc((void*)(p.v + head_off), (short)0, head_bytes,
                                             0x00020000);
  cx.c = p.c;
  cx.thr = p.thr;
  cx.N = N;
  cx.n_kt = p.n_kt;
  cx.w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index, kept in an SGPR
  cx.lane = tid & 63;
  cx.koff = Q8 ? k8_lane_offset(cx.w, cx.lane) : tile_lane_offset<false>(cx.w, cx.lane);
  cx.voff = tile_lane_offset<true>(cx.w, cx.lane);
  cx.r = cx.lane & 31;
  cx.g = cx.lane >> 5;
  const int q0 = qt * kTQ;
  const int qrow = q0 + cx.w * 32 + cx.r;
  cx.valid = qrow < N;
  cx.thr_row = cx.valid ? p.thr : __builtin_inff();
  cx.ragged = (N % kTK) != 0;
  // This wave's decision unit: the workgroup's tile, or the wave's own 32 rows.
  const int unit = UNIT == kTQ ? qt : qt * (kTQ / UNIT) + cx.w;
  const int unit_row0 = unit * UNIT;
  cx.rows_valid = max(0, min(UNIT, N - unit_row0));
  cx.mask_row = (p.mask != nullptr && cx.rows_valid > 0)
                    ? p.mask + ((size_t)bh * p.n_qu + unit) * (BC == kTK ? p.n_kt : p.n_kd)
                    : nullptr;
  // Diagonal-first order starts at the key tile holding the first query row: over 64-key
  // tiles, or over 128-key tiles with 128-key decisions.
  const int n_order = PAIR ? (cx.n_kt + 1) / 2 : cx.n_kt;
  cx.diag_c = PAIR ? q0 / (2 * kTK) : q0 / kTK;       // < n_order since q0 < N
  cx.diag_m = min(cx.diag_c, n_order - 1 - cx.diag_c);
  cx.diag_right = (n_order - 1 - cx.diag_c) > cx.diag_c;

  // Stage K and V of the first visited tile, then K of the second.
  const int t0 = PAIR ? pair_tile<ORDER>(0, cx) : key_tile_at<ORDER>(0, cx);
  load_k_tile<Q8>(sm, 0, cx, t0 * kTK);
  load_tile_lds(sm.v[0], cx.vrs, cx.voff, t0 * kTK, cx.w);

  typename QFragOf<Q8>::type qf;
  if constexpr (Q8) {
    // d in [64 s + 16 g, +16) and [64 s + 32 + 16 g, +16) of the row for d-step s; the
    // exponent word carries blocks g (byte 0) and 2 + g (byte 2).
    const uint8_t* qrow8 = p.q8 + head_off + (size_t)qrow * kD;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const u32x4 lo = cx.valid ? *reinterpret_cast<const u32x4*>(qrow8 + 64 * s + 16 * cx.g)
                                : u32x4{0, 0, 0, 0};
      const u32x4 hi = cx.valid
                           ? *reinterpret_cast<const u32x4*>(qrow8 + 64 * s + 32 + 16 * cx.g)
                           : u32x4{0, 0, 0, 0};
      qf.q[s] = i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
                      (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
    }
    const uint32_t qs =
        cx.valid ? *reinterpret_cast<const uint32_t*>(p.q_scales + ((size_t)bh * N + qrow) * 4)
                 : 0u;
    qf.sc = (qs >> (8 * cx.g)) & 0x00ff00ffu;
  } else {
    // Q^T B-operand fragments: d = 16 s + 8 g + (0..7) of this lane's query row.
    const uint16_t* qb = p.q + head_off;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      u32x4 x = cx.valid
                    ? *reinterpret_cast<const u32x4*>(qb + (size_t)qrow * kD + 16 * s + 8 * cx.g)
                    : u32x4{0, 0, 0, 0};
      qf[s] = __builtin_bit_cast(bf16x8, x);
    }
  }
  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) o[db] = f32x16{};
  RowState rs{-__builtin_inff(), -__builtin_inff(), 0.f, -__builtin_inff()};

  load_k_tile<Q8>(sm, 1, cx, (PAIR ? pair_tile<ORDER>(1, cx) : key_tile_or_past<ORDER>(1, cx)) * kTK);
  if (cx.lane == 0) {                        // vote bytes start at 0 (not skipping)
    sm.vote[0][cx.w] = 0;
    sm.vote[1][cx.w] = 0;
  }
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");

  f32x16 sa[2], sb[2];
  if constexpr (Q8)                            // S of the first visited tile
    skipped_tile_q8(sa, reinterpret_cast<const uint8_t*>(sm.k[0]), sm.ks[0], qf, cx.r, cx.g);
  else
    skipped_tile(sa, sm.k[0], qf, cx.r, cx.g);
  if (cx.ragged && t0 == cx.n_kt - 1) mask_tail(sa, t0 * kTK, N, cx.g);
  float mhat = row_max(sa) * cx.c;
  bool keep_own = true;                      // the first tile is always kept
  bool keep_any = true;
  uint32_t vote = 0;                         // the first tile's skip word: kept
  uint32_t marks = 0;                        // this wave's vote bytes that hold 1
  bool v_ready = true;                       // V_0 was staged above
  SkipCount sk;
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");  // K_0 consumed

  if constexpr (HALF) {
    static_assert(ORDER == kOrderAscending, "32-key decisions walk keys in ascending order");
    float mh[2] = {block_max(sa[0]) * cx.c, block_max(sa[1]) * cx.c};
    // h0 of the first tile is always kept and its h1 decided mid-step; the vote buffers
    // were cleared above.
    uint32_t votes[3] = {1u, 1u, 0u};
    bool own[3] = {true, true, false};
    uint32_t lds_bytes = 0u;
    for (int j = 0; j < cx.n_kt; j += 2) {
      half_tile_step<RULE, UNIT, Q8>(j, sa, sb, mh, votes, own, lds_bytes, v_ready, rs, o, qf,
                                     sm, cx, sk);
      if (j + 1 < cx.n_kt)
        half_tile_step<RULE, UNIT, Q8>(j + 1, sb, sa, mh, votes, own, lds_bytes, v_ready, rs, o,
                                       qf, sm, cx, sk);
    }
  } else if constexpr (PAIR) {
    // Ascending: the last pair is the partial one and may end after one step.  Diagonal:
    // every pair takes two steps (a partial pair's second tile is all masked).
    const int n_steps = ORDER == kOrderAscending ? cx.n_kt : 2 * ((cx.n_kt + 1) / 2);
    for (int j = 0; j < n_steps; j += 2) {
      pair_first_step<RULE, UNIT, Q8, ORDER>(j, sa, sb, mhat, keep_own, keep_any, v_ready, rs,
                                             o, qf, sm, cx, sk);
      if (j + 1 < n_steps)
        pair_second_step<RULE, UNIT, Q8, ORDER>(j + 1, sb, sa, mhat, keep_own, keep_any,
                                                v_ready, rs, o, qf, sm, cx);
    }
  } else {
    // Unrolled by two so that S_j / S_{j+1} alternate between sa and sb without copies.
    for (int j = 0; j < cx.n_kt; j += 2) {
      key_tile_step<RULE, UNIT, ORDER, Q8>(j, sa, sb, mhat, keep_own, keep_any, vote, marks,
                                           v_ready, rs, o, qf, sm, cx, sk);
      if (j + 1 < cx.n_kt)
        key_tile_step<RULE, UNIT, ORDER, Q8>(j + 1, sb, sa, mhat, keep_own, keep_any, vote,
                                             marks, v_ready, rs, o, qf, sm, cx, sk);
    }
  }

  store_rows(p, o, rs, cx, head_off, bh, qrow);
  // One set of counters per decision unit (the workgroup's tile, or each wave's rows).
  if (p.stats != nullptr && (UNIT == kTQ ? cx.w == 0 : true) && cx.lane == 0 &&
      cx.rows_valid > 0) {
    unsigned long long* st = reinterpret_cast<unsigned long long*>(p.stats) + (size_t)bh * 4;
    atomicAdd(st + 0, (unsigned long long)(BC == kTK ? cx.n_kt : p.n_kd));
    atomicAdd(st + 1, (unsigned long long)sk.tiles);
    atomicAdd(st + 2, (unsigned long long)cx.rows_valid * (unsigned long long)N);
    atomicAdd(st + 3, (unsigned long long)cx.rows_valid * (unsigned long long)sk.keys);
  }
}

// ---- mask reuse -----------------------------------------------------------------------
// A skip mask from an earlier call (for instance an earlier denoising step of the same
// layer) is applied as given: the workgroup visits only the key tiles some of its units
// keep, in ascending order; a unit that skips a visited tile (UNIT = 32) adds nothing for
// it.  Tiles nobody keeps cost nothing at all, not even QK^T.  A mask of 128-key
// decisions keeps or skips both 64-key tiles of each decision.

// Visited tiles of one workgroup, ascending: (key tile << 4) | keep bit of each wave.
__device__ __forceinline__ int list_tile(const MaskSmem& sm, int s) {
  return (int)__builtin_amdgcn_readfirstlane((uint32_t)sm.list[s] >> 4);
}

// One visited tile per step, with the pipeline of the dense kernel: S of the next visited
// tile is computed while this one's softmax runs, V is requested one tile and K two tiles
// ahead.  The list entries of steps j, j+1 and j+2 travel in registers (e0, e1, e2; past
// the end they name the tile after the last one); the entry of step j+3 is read from LDS
// here and used a step later, so no list read waits in front of the tile loads.
template <int UNIT>
__device__ __forceinline__ void mask_tile_step(int j, int n_keep, const f32x16 (&s_cur)[2],
                                               f32x16 (&s_next)[2], float& mhat, RowState& rs,
                                               f32x16 (&o)[4], const bf16x8 (&qf)[8],
                                               MaskSmem& sm, const LoopCtx& cx, uint32_t& e0,
                                               uint32_t& e1, uint32_t& e2) {
  const int nb = (j + 1) & 1;
  const bool has_next = j + 1 < n_keep;
  const int tn = (int)(e1 >> 4);
  const int tn2 = (int)(e2 >> 4);
  const uint32_t e3_raw = j + 3 < n_keep ? (uint32_t)sm.list[j + 3]
                                         : (uint32_t)cx.n_kt << 4;
  bool keep_own = true;
  if constexpr (UNIT != kTQ) keep_own = ((e0 >> cx.w) & 1u) != 0;
  load_tile_lds(sm.t.v[nb], cx.vrs, cx.voff, tn * kTK, cx.w);
  load_tile_lds(sm.t.k[j & 1], cx.krs, cx.koff, tn2 * kTK, cx.w);
  // Some unit of the workgroup keeps every visited tile and the step's barrier waits for
  // it, so a wave whose own unit skips the tile runs the kept path without contributing
  // rather than a second code path.
  float rmax_kept;
  kept_tile(rs, o, s_cur, mhat, cx.c, s_next, sm.t.k[nb], sm.t.v[j & 1], qf, cx.r, cx.g,
            cx.lane, rmax_kept, keep_own);
  float mhat_next = 0.f;
  if (has_next) {
    if (cx.ragged && tn == cx.n_kt - 1) {
      mask_tail(s_next, tn * kTK, cx.N, cx.g);
      rmax_kept = row_max(s_next);
    }
    mhat_next = rmax_kept * cx.c;
  }
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  mhat = mhat_next;
  e0 = e1;
  e1 = e2;
  e2 = __builtin_amdgcn_readfirstlane(e3_raw);
}

template <int UNIT>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads),
                          amdgpu_waves_per_eu(2, 2))) void
fa_fwd_mask_kernel(FwdParams p) {
  static_assert(UNIT == kTQ || UNIT == 32, "decision unit is the tile or one wave");
  __shared__ __attribute__((aligned(16))) MaskSmem sm;

  const int tid = threadIdx.x;
  const int qt = blockIdx.x;
  const int bh = blockIdx.y;
  const int N = p.N;
  const size_t head_off = (size_t)bh * (size_t)N * kD;

  LoopCtx cx;
  const int head_bytes = N * (kD * 2);
  cx.krs = __builtin_amdgcn_make_buffer_rsrc((void*)(p.k + head_off), (short)0, head_bytes,
                                             0x00020000);
  cx.vrs = __builtin_amdgcn_make_buffer_rsrc((void*)(p.v + head_off), (short)0, head_bytes,
                                             0x00020000);
  cx.c = p.c;
  cx.thr = p.thr;
  cx.N = N;
  cx.n_kt = p.n_kt;
  cx.w = __builtin_amdgcn_readfirstlane(tid >> 6);
  cx.lane = tid & 63;
  cx.koff = tile_lane_offset<false>(cx.w, cx.lane);
  cx.voff = tile_lane_offset<true>(cx.w, cx.lane);
  cx.r = cx.lane & 31;
  cx.g = cx.lane >> 5;
  const int q0 = qt * kTQ;
  const int qrow = q0 + cx.w * 32 + cx.r;
  cx.valid = qrow < N;
  cx.thr_row = cx.valid ? p.thr : __builtin_inff();
  cx.ragged = (N % kTK) != 0;
  const int unit = UNIT == kTQ ? qt : qt * (kTQ / UNIT) + cx.w;
  cx.rows_valid = max(0, min(UNIT, N - unit * UNIT));

  // ---- compact the visited tiles into sm.list ----------------------------------------
  const int n_units = UNIT == kTQ ? 1 : kTQ / UNIT;
  const uint8_t* rows[kTQ / 32];
#pragma unroll
  for (int u = 0; u < kTQ / 32; ++u) {
    const int uu = UNIT == kTQ ? qt : qt * (kTQ / UNIT) + u;
    rows[u] = (u < n_units && uu * UNIT < N) ? p.mask_in + ((size_t)bh * p.n_qu + uu) * p.n_kd
                                             : nullptr;
  }
  // Mask columns are decisions of key_tile keys: 64-key tile t reads column t (64) or
  // t / 2 (128, two tiles per decision).
  const int col_shift = p.key_tile == 2 * kTK ? 1 : 0;
  auto keep_bits = [&](int t) -> uint32_t {
    const int col = t >> col_shift;
    if constexpr (UNIT == kTQ) {
      return rows[0][col] == 0 ? 0xFu : 0u;
    } else {
      uint32_t b = 0;
#pragma unroll
      for (int u = 0; u < kTQ / 32; ++u)
        if (rows[u] != nullptr && rows[u][col] == 0) b |= 1u << u;
      return b;
    }
  };
  const int per = (cx.n_kt + kThreads - 1) / kThreads;
  const int t_lo = min(cx.n_kt, tid * per), t_hi = min(cx.n_kt, t_lo + per);
  uint32_t mine = 0;
  for (int t = t_lo; t < t_hi; ++t) mine += keep_bits(t) != 0 ? 1u : 0u;
  sm.count[tid] = (uint16_t)mine;
  __syncthreads();
  if (tid == 0) {
    uint32_t run = 0;
    for (int i = 0; i < kThreads; ++i) {
      const uint32_t c = sm.count[i];
      sm.count[i] = (uint16_t)run;
      run += c;
    }
    sm.total = run;
  }
  __syncthreads();
  {
    uint32_t at = sm.count[tid];
    for (int t = t_lo; t < t_hi; ++t) {
      const uint32_t b = keep_bits(t);
      if (b != 0) sm.list[at++] = (uint16_t)((t << 4) | b);
    }
  }
  const int n_keep = (int)__builtin_amdgcn_readfirstlane(sm.total);

  // The caller's mask is also the output mask; counters from this unit's own mask row.
  if (p.mask != nullptr) {
    for (int u = 0; u < n_units; ++u) {
      if (rows[u] == nullptr) continue;
      const int uu = UNIT == kTQ ? qt : qt * (kTQ / UNIT) + u;
      uint8_t* out = p.mask + ((size_t)bh * p.n_qu + uu) * p.n_kd;
      for (int t = tid; t < p.n_kd; t += kThreads) out[t] = rows[u][t] != 0 ? 1 : 0;
    }
  }
  if (p.stats != nullptr && (UNIT == kTQ ? cx.w == 0 : true) && cx.rows_valid > 0) {
    const uint8_t* own = rows[UNIT == kTQ ? 0 : cx.w];
    uint32_t skipped = 0, width = 0;
    for (int t = cx.lane; t < p.n_kd; t += 64)
      if (own[t] != 0) {
        skipped += 1;
        width += (uint32_t)min(p.key_tile, N - t * p.key_tile);
      }
#pragma unroll
    for (int sh = 32; sh >= 1; sh >>= 1) {
      skipped += __shfl_xor(skipped, sh);
      width += __shfl_xor(width, sh);
    }
    if (cx.lane == 0) {
      unsigned long long* st = reinterpret_cast<unsigned long long*>(p.stats) + (size_t)bh * 4;
      atomicAdd(st + 0, (unsigned long long)p.n_kd);
      atomicAdd(st + 1, (unsigned long long)skipped);
      atomicAdd(st + 2, (unsigned long long)cx.rows_valid * (unsigned long long)N);
      atomicAdd(st + 3, (unsigned long long)cx.rows_valid * (unsigned long long)width);
    }
  }
  __syncthreads();   // the list is complete

  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) o[db] = f32x16{};
  RowState rs{-__builtin_inff(), -__builtin_inff(), 0.f, -__builtin_inff()};

  if (n_keep > 0) {
    const int t0 = list_tile(sm, 0);
    load_tile_lds(sm.t.k[0], cx.krs, cx.koff, t0 * kTK, cx.w);
    load_tile_lds(sm.t.v[0], cx.vrs, cx.voff, t0 * kTK, cx.w);
    const uint16_t* qb = p.q + head_off;
    bf16x8 qf[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      u32x4 x = cx.valid
                    ? *reinterpret_cast<const u32x4*>(qb + (size_t)qrow * kD + 16 * s + 8 * cx.g)
                    : u32x4{0, 0, 0, 0};
      qf[s] = __builtin_bit_cast(bf16x8, x);
    }
    load_tile_lds(sm.t.k[1], cx.krs, cx.koff, (n_keep > 1 ? list_tile(sm, 1) : cx.n_kt) * kTK,
                  cx.w);
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");

    f32x16 sa[2], sb[2];
    skipped_tile(sa, sm.t.k[0], qf, cx.r, cx.g);
    if (cx.ragged && t0 == cx.n_kt - 1) mask_tail(sa, t0 * kTK, N, cx.g);
    float mhat = row_max(sa) * cx.c;
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");

    const uint32_t past = (uint32_t)cx.n_kt << 4;
    uint32_t e0 = __builtin_amdgcn_readfirstlane((uint32_t)sm.list[0]);
    uint32_t e1 = n_keep > 1 ? __builtin_amdgcn_readfirstlane((uint32_t)sm.list[1]) : past;
    uint32_t e2 = n_keep > 2 ? __builtin_amdgcn_readfirstlane((uint32_t)sm.list[2]) : past;
    for (int j = 0; j < n_keep; j += 2) {
      mask_tile_step<UNIT>(j, n_keep, sa, sb, mhat, rs, o, qf, sm, cx, e0, e1, e2);
      if (j + 1 < n_keep)
        mask_tile_step<UNIT>(j + 1, n_keep, sb, sa, mhat, rs, o, qf, sm, cx, e0, e1, e2);
    }
  }
  store_rows(p, o, rs, cx, head_off, bh, qrow);
}

__global__ void zero_u64_kernel(uint64_t* __restrict__ p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

}  // namespace

namespace {

template <int UNIT, int ORDER, bool Q8 = false>
hipError_t launch_unit(int rule, const FwdParams& p, dim3 grid, hipStream_t stream) {
  const dim3 block(kThreads);
  switch (rule) {
    case kRuleDense:
      // Every tile is kept, so the visit order changes nothing but the rounding of the
      // sums: the dense kernel always walks ascending.
      hipLaunchKernelGGL((fa_fwd_kernel<kRuleDense, UNIT, kOrderAscending, Q8>), grid, block, 0,
                         stream, p);
      break;
    case kRuleBlasst:
      hipLaunchKernelGGL((fa_fwd_kernel<kRuleBlasst, UNIT, ORDER, Q8>), grid, block, 0, stream,
                         p);
      break;
    case kRuleDynSparse:
      hipLaunchKernelGGL((fa_fwd_kernel<kRuleDynSparse, UNIT, ORDER, Q8>), grid, block, 0,
                         stream, p);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int UNIT, bool Q8, int ORDER>
hipError_t launch_pair(int rule, const FwdParams& p, dim3 grid, hipStream_t stream) {
  const dim3 block(kThreads);
  switch (rule) {
    case kRuleDense:
      hipLaunchKernelGGL((fa_fwd_kernel<kRuleDense, UNIT, kOrderAscending, Q8, 2 * kTK>), grid,
                         block, 0, stream, p);
      break;
    case kRuleBlasst:
      hipLaunchKernelGGL((fa_fwd_kernel<kRuleBlasst, UNIT, ORDER, Q8, 2 * kTK>), grid, block, 0,
                         stream, p);
      break;
    case kRuleDynSparse:
      hipLaunchKernelGGL((fa_fwd_kernel<kRuleDynSparse, UNIT, ORDER, Q8, 2 * kTK>), grid, block,
                         0, stream, p);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int UNIT, bool Q8>
hipError_t launch_half(int rule, const FwdParams& p, dim3 grid, hipStream_t stream) {
  const dim3 block(kThreads);
  switch (rule) {
    case kRuleDense:
      hipLaunchKernelGGL((fa_fwd_kernel<kRuleDense, UNIT, kOrderAscending, Q8, kTK / 2>), grid,
                         block, 0, stream, p);
      break;
    case kRuleBlasst:
      hipLaunchKernelGGL((fa_fwd_kernel<kRuleBlasst, UNIT, kOrderAscending, Q8, kTK / 2>), grid,
                         block, 0, stream, p);
      break;
    case kRuleDynSparse:
      hipLaunchKernelGGL((fa_fwd_kernel<kRuleDynSparse, UNIT, kOrderAscending, Q8, kTK / 2>),
                         grid, block, 0, stream, p);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int UNIT, bool Q8>
hipError_t launch_order(int rule, const FwdParams& p, dim3 grid, hipStream_t stream) {
  if (p.key_tile == 2 * kTK) {
    if (p.key_order == kOrderDiagonal && rule != kRuleDense) {
      const int chunk = (p.n_qt + kXcds - 1) / kXcds;
      return launch_pair<UNIT, Q8, kOrderDiagonal>(rule, p,
                                                   dim3((unsigned)(chunk * kXcds), grid.y),
                                                   stream);
    }
    return launch_pair<UNIT, Q8, kOrderAscending>(rule, p, grid, stream);
  }
  if (p.key_tile == kTK / 2) {
    if (p.key_order != kOrderAscending) return hipErrorInvalidValue;
    return launch_half<UNIT, Q8>(rule, p, grid, stream);
  }
  if (p.key_order == kOrderDiagonal && rule != kRuleDense) {
    const int chunk = (p.n_qt + kXcds - 1) / kXcds;
    return launch_unit<UNIT, kOrderDiagonal, Q8>(rule, p,
                                                 dim3((unsigned)(chunk * kXcds), grid.y), stream);
  }
  return launch_unit<UNIT, kOrderAscending, Q8>(rule, p, grid, stream);
}

}  // namespace

hipError_t launch_fa_fwd(int rule, int unit_rows, const FwdParams& p, int bh,
                         hipStream_t stream) {
  const dim3 grid((unsigned)p.n_qt, (unsigned)bh);
  if (rule == kRuleMask) {
    if (p.n_kt > kMaxMaskTiles || p.mask_in == nullptr) return hipErrorInvalidValue;
    if (unit_rows == kTQ)
      hipLaunchKernelGGL((fa_fwd_mask_kernel<kTQ>), grid, dim3(kThreads), 0, stream, p);
    else if (unit_rows == 32)
      hipLaunchKernelGGL((fa_fwd_mask_kernel<32>), grid, dim3(kThreads), 0, stream, p);
    else
      return hipErrorInvalidValue;
    return hipGetLastError();
  }
  if (p.qk_format == kQkMxfp8) {
    if (p.q8 == nullptr || p.k8 == nullptr || p.q_scales == nullptr || p.k_scales == nullptr)
      return hipErrorInvalidValue;
    if (unit_rows == kTQ) return launch_order<kTQ, true>(rule, p, grid, stream);
    if (unit_rows == 32) return launch_order<32, true>(rule, p, grid, stream);
    return hipErrorInvalidValue;
  }
  if (unit_rows == kTQ) return launch_order<kTQ, false>(rule, p, grid, stream);
  if (unit_rows == 32) return launch_order<32, false>(rule, p, grid, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_zero_u64(uint64_t* ptr, int n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int threads = 256;
  hipLaunchKernelGGL(zero_u64_kernel, dim3((n + threads - 1) / threads), dim3(threads), 0,
                     stream, ptr, n);
  return hipGetLastError();
}

}  // namespace dsattn
