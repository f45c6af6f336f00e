/*
 * dsattn.h -- C ABI of libdsattn.so: FlashAttention-style forward pass with online
 * tile filtering (DynSparse, BLASST) and a dense reference rule, for AMD MI355X (gfx950).
 *
 * Problem (Section 2.1.1): produce the attention output O' = softmax(S) V with
 * S = scale * Q K^T at the least compute while staying close to the dense output.  The
 * kernels walk key tiles j = 0, 1, ... in ascending order for every query tile i
 * (Section 1: tile-based attention over (Q_i, K_j) pairs), always compute S_ij and its
 * per-row maximum m_hat, and then decide whether the tile's exponentials, row sums and
 * P.V product are computed at all:
 *
 *   DynSparse (Section 3.1, Eq. 5 and Eq. 6): t = m_hat - LSE^(j-1), where LSE^(j-1) is
 *     the log-sum-exp of the logits of the key tiles kept so far; skip when t < lambda.
 *   BLASST (Section 1, Section 2.1.1 item 4): t = m_hat - m^(j-1), the tile maximum
 *     minus the running maximum of the kept tiles; skip when t < ln(tau).
 *   dense: never skip.
 *
 * A tile is skipped only when every valid row of the query tile satisfies the skip
 * condition (this keeps the per-row recall bound of Section 3.1); t == threshold keeps
 * the tile; the first key tile is always kept.  Skipped tiles change neither the running
 * maximum nor the LSE.  The output is renormalised over the kept keys (Eq. 1).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Layout: q, k, v, o are contiguous bf16 arrays [B][H][N][d], row-major (d fastest).
 * Shapes: d must be 128; (tile_q, tile_k) must be (128, 64).  B, H, N >= 0 and
 *   B*H <= 65535; B == 0, H == 0 or N == 0 is an empty problem: nothing is read or
 *   written except stats_out, which is zeroed.
 * Memory: every pointer is a device pointer allocated by the caller on the current HIP
 *   device; the library never allocates, frees or retains memory.  q, k, v are read-only;
 *   o must not alias q, k or v.
 * Execution: asynchronous on `stream` (0 = the null stream).  Argument errors are found
 *   on the host before anything is enqueued.  Calls that share output buffers on one
 *   stream are ordered by the stream; on different streams they race.
 * Optional outputs (NULL = not produced):
 *   stats_out uint64 [B*H][4] = {tiles_total, tiles_skipped, elems_total, elems_skipped}
 *     per (b, h), where tiles are (query tile, key tile) pairs and elems are the valid
 *     (query row, key) pairs they cover.  Zeroed by the library on `stream` first.
 *   mask_out  uint8 [B*H][ceil(N/tile_q)][ceil(N/tile_k)], 1 = the pair was skipped.
 *   lse_out   float [B*H][N], natural-log log-sum-exp of each row over its kept keys.
 * Return value: DSATTN_OK, or a negative dsattn_status; dsattn_last_error() then holds a
 *   message (thread-local, valid until the next call on the same thread).  Faults inside
 *   the kernels surface as HIP errors on `stream`, not through the return value.
 */
#ifndef DSATTN_H
#define DSATTN_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum dsattn_status {
  DSATTN_OK = 0,
  DSATTN_EINVAL = -1,      /* null pointer, negative size, bad scale/threshold, host pointer */
  DSATTN_EUNSUPPORTED = -2, /* head dim or tile shape not built into the library */
  DSATTN_ELAUNCH = -3      /* the HIP runtime refused a launch */
} dsattn_status;

typedef enum dsattn_rule {
  DSATTN_RULE_DENSE = 0,
  DSATTN_RULE_BLASST = 1,            /* param = tau in [0, 1] */
  DSATTN_RULE_DYNSPARSE_RECALL = 2,  /* param = recall target in (0, 1] */
  DSATTN_RULE_DYNSPARSE_LAMBDA = 3   /* param = lambda (finite, or -inf for dense) */
} dsattn_rule;

/*
 * Threshold that guarantees a per-row recall of at least recall_target
 * (Section 3.1, recall bound): each skipped key carries at most e^lambda of the dense
 * softmax mass, so lambda = ln((1 - recall_target) / N) keeps at least recall_target of
 * it.  Returns -inf for recall_target == 1 and NaN when recall_target is outside (0, 1]
 * or N <= 0.
 */
float dsattn_lambda_from_recall(float recall_target, int N);

/*
 * DynSparse forward pass (Section 3.1, Eq. 5-6) with lambda derived from recall_target
 * by dsattn_lambda_from_recall(recall_target, N).  recall_target must lie in (0, 1];
 * 1 reproduces the dense rule exactly.  scale must be finite and > 0.
 */
int dynsparse_attn_fwd(const void* q, const void* k, const void* v, void* o,
                       int B, int H, int N, int d, float scale, float recall_target,
                       int tile_q, int tile_k, hipStream_t stream, uint64_t* stats_out);

/*
 * DynSparse forward pass with an explicit threshold lambda in natural-log units
 * (Section 3.1, hyperparameter selection, Eq. 7 suggests ln(P_real) + ln(B_c / L)).  lambda must be finite or -inf
 * (-inf = dense).
 */
int dynsparse_attn_fwd_lambda(const void* q, const void* k, const void* v, void* o,
                              int B, int H, int N, int d, float scale, float lambda,
                              int tile_q, int tile_k, hipStream_t stream, uint64_t* stats_out);

/*
 * BLASST-style forward pass: skip a key tile when every valid row has
 * m_hat - m^(j-1) < ln(threshold).  threshold (tau) must lie in [0, 1]; 0 = dense.
 */
int blasst_attn_fwd(const void* q, const void* k, const void* v, void* o,
                    int B, int H, int N, int d, float scale, float threshold,
                    int tile_q, int tile_k, hipStream_t stream, uint64_t* stats_out);

/* Dense FlashAttention forward pass of the same kernel family (no skip decisions). */
int dense_attn_fwd(const void* q, const void* k, const void* v, void* o,
                   int B, int H, int N, int d, float scale,
                   int tile_q, int tile_k, hipStream_t stream, uint64_t* stats_out);

/* All rules, plus the optional mask_out and lse_out outputs. */
typedef struct dsattn_args {
  int rule;              /* dsattn_rule */
  float param;           /* tau, recall target or lambda, as the rule says; unused for dense */
  const void* q;
  const void* k;
  const void* v;
  void* o;
  int B, H, N, d;
  float scale;
  int tile_q, tile_k;
  hipStream_t stream;
  uint64_t* stats_out;   /* may be NULL */
  uint8_t* mask_out;     /* may be NULL */
  float* lse_out;        /* may be NULL */
} dsattn_args;

int dsattn_attn_fwd_ex(const dsattn_args* args);

/* Message describing the last error on this thread ("" after a successful call). */
const char* dsattn_last_error(void);

/* Library version string. */
const char* dsattn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DSATTN_H */
