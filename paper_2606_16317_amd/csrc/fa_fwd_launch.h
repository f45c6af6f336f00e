// Internal interface between the C-ABI entry points and the gfx950 kernels.
#ifndef DSATTN_FA_FWD_LAUNCH_H
#define DSATTN_FA_FWD_LAUNCH_H

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace dsattn {

enum { kRuleDense = 0, kRuleBlasst = 1, kRuleDynSparse = 2, kRuleMask = 3 };
enum { kOrderAscending = 0, kOrderDiagonal = 1 };
enum { kQkBf16 = 0, kQkMxfp8 = 1 };

struct FwdParams {
  const uint16_t* q;   // bf16 [BH][N][128]
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  int N;
  int n_qt;            // ceil(N / 128): query tiles (workgroups per head)
  int n_qu;            // ceil(N / unit rows): skip-decision units per head (mask rows)
  int n_kt;            // ceil(N / 64)
  float c;             // scale * log2(e): logits are handled in log2 units
  float thr;           // skip threshold in log2 units (lambda*log2(e) or log2(tau))
  uint64_t* stats;     // [BH][4] or null (zeroed beforehand)
  uint8_t* mask;       // [BH][n_qu][n_kt] or null
  float* lse;          // [BH][N] or null
  int key_order;       // kOrderAscending or kOrderDiagonal
  const uint8_t* mask_in;  // kRuleMask: [BH][n_qu][n_kt], 1 = skip (else unused)
  int qk_format;           // kQkBf16 (q, k) or kQkMxfp8 (q8, k8 and their exponents)
  const uint8_t* q8;       // kQkMxfp8: E4M3 codes [BH][N][128]
  const uint8_t* k8;
  const uint8_t* q_scales; // kQkMxfp8: E8M0 exponents [BH][N][4]
  const uint8_t* k_scales;
  int key_tile;            // keys per skip decision: 64, or 128 (two 64-key tiles)
  int n_kd;                // ceil(N / key_tile): decisions per row of the mask
};

// Enqueue one forward pass over `bh` heads on `stream`; unit_rows (128 or 32) is the
// number of query rows that share one skip decision.
hipError_t launch_fa_fwd(int rule, int unit_rows, const FwdParams& p, int bh,
                         hipStream_t stream);

// Enqueue a fill of n uint64 zeros (a kernel rather than a memset node, so the call can be
// captured into a graph and replayed).
hipError_t launch_zero_u64(uint64_t* ptr, int n, hipStream_t stream);

}  // namespace dsattn

#endif
