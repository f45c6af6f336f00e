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
 * Shapes: d must be 128; tile_q is 128 or 32 and tile_k 32, 64 or 128.  tile_k is the
 *   key tile B_c, the number of keys one skip decision covers (Section 4.2.1 uses 128 for
 *   the 14B model and 32 for the 5B model).  The kernels work on 64-key tiles: 128 is two
 *   of them deciding together, 32 their two halves deciding in turn (ascending order
 *   only); tile_q is the number of query rows that share one skip
 *   decision ("query tile" below): 128 decides per workgroup tile, 32 lets every 32-row
 *   slice decide on its own (a finer granularity of the same rule, which the paper
 *   leaves open).  B, H, N >= 0, N <= 8388607 and B*H <= 65535; B == 0, H == 0 or
 *   N == 0 is an empty problem: nothing is read or written except stats_out, which is
 *   zeroed.
 * Memory: every pointer is a device pointer allocated by the caller on the current HIP
 *   device; the library never allocates, frees or retains memory.  q, k, v are read-only;
 *   the outputs (o, lse_out, mask_out, stats_out) must not overlap any input or each
 *   other (checked on byte ranges); q, k, v, o must be 16-byte aligned and lse_out 4-byte
 *   aligned.
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

#include <stddef.h>
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

typedef enum dsattn_key_order {
  DSATTN_ORDER_ASCENDING = 0,  /* key tiles 0, 1, 2, ... for every query tile */
  DSATTN_ORDER_DIAGONAL = 1    /* from the query tile's own position outward, see below */
} dsattn_key_order;

typedef enum dsattn_qk_format {
  DSATTN_QK_BF16 = 0,   /* q and k are bf16 [B][H][N][d] */
  DSATTN_QK_MXFP8 = 1   /* q and k are MX-FP8 codes with E8M0 exponents, see below */
} dsattn_qk_format;

typedef enum dsattn_rule {
  DSATTN_RULE_DENSE = 0,
  DSATTN_RULE_BLASST = 1,            /* param = tau in [0, 1] */
  DSATTN_RULE_DYNSPARSE_RECALL = 2,  /* param = recall target in (0, 1] */
  DSATTN_RULE_DYNSPARSE_LAMBDA = 3,  /* param = lambda (finite, or -inf for dense) */
  DSATTN_RULE_MASK = 4               /* reuse a skip mask: args->mask_in; param unused */
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
  int key_order;         /* dsattn_key_order; the named entry points use ascending */
  const uint8_t* mask_in; /* DSATTN_RULE_MASK only, else ignored (see below) */
  int qk_format;         /* dsattn_qk_format; the named entry points use bf16 */
  const uint8_t* q_scales; /* DSATTN_QK_MXFP8 only, else ignored (see below) */
  const uint8_t* k_scales;
} dsattn_args;

/*
 * Key-tile visit order.  The rule is order dependent (Eq. 5 compares with the LSE of the
 * tiles kept before), and the paper walks key tiles in ascending order.  With
 * DSATTN_ORDER_DIAGONAL every 128-row query block starts at the key tile c that holds its
 * first row (c = 128 i / tile_k for block i), then visits c+1, c-1, c+2, c-2, ... and,
 * once one side is used up, the rest of the other side in order; query tiles of 32 rows
 * use the order of their 128-row block.  With tile_k = 128 the order runs over 128-key
 * tiles (c = i); tile_k = 32 takes ascending order only.  For self-attention this visits
 * the keys nearest each query first.  mask_out is indexed by key tile whatever the order.
 */
int dsattn_attn_fwd_ex(const dsattn_args* args);

/*
 * Mask reuse (DSATTN_RULE_MASK).  The skip decisions of an earlier call -- typically the
 * same layer at an earlier denoising step, whose attention changes slowly (the reuse the
 * paper cites from LiteAttention in Section 1) -- are applied as given: mask_in is a
 * device uint8 array laid out like mask_out ([B*H][ceil(N/tile_q)][ceil(N/tile_k)],
 * nonzero = skip), and the output is attention over the kept key tiles, renormalised as
 * for the rules.  Skipped tiles cost nothing, not even Q K^T: each workgroup visits only
 * the tiles one of its rows keeps, in ascending order.  A unit that keeps no tile gets
 * zeros and an LSE of -inf.  Reusing the mask a rule call wrote with tile_k = 64 (same
 * inputs, tile_q and ascending order) reproduces that call's output bit for bit.  tile_k
 * may be 64 or 128 (a 128-key decision keeps or skips two 64-key tiles).  Requirements:
 * mask_in non-NULL, key_order ascending, N <= 262144, else DSATTN_EINVAL /
 * DSATTN_EUNSUPPORTED.  mask_out, if given, receives mask_in (as 0/1).
 */

/*
 * Quantised Q K^T (DSATTN_QK_MXFP8; the Conclusion, Section 5, lists quantisation among
 * the methods the rule combines with).  q and k then point at E4M3 codes (uint8 [B][H][N][d], 16-byte
 * aligned) and q_scales / k_scales at their E8M0 block exponents (uint8 [B][H][N][d/32],
 * 4-byte aligned), as written by dsattn_quantize_mxfp8: element x of block b of a row
 * stands for e4m3(x) * 2^(scale[b] - 127).  S = Q K^T is computed from these values with
 * fp32 accumulation; v stays bf16, and the rule, the softmax and P V are as in the bf16
 * path.  Supported for the dense, BLASST and DynSparse rules at both decision units
 * (tile_q = 128 or 32) and both key orders; not for mask reuse or by the reordered entry
 * point (DSATTN_EUNSUPPORTED).
 */

/*
 * Spatio-temporal token reordering (Section 3.1, closing remark on hyperparameter
 * selection; Section 1 describes the same grouping of tokens that are near in time and
 * space).  A video transformer flattens its T x Y x X latent grid row-major (x fastest),
 * so a 128-token query tile spans whole rows of x and a key tile's neighbours in y and t
 * lie far away in the sequence.  Regrouping the tokens into bt x by x bx blocks before the
 * attention puts neighbours into the same tile.
 */

/*
 * Host function.  Writes the gather map of the blocked order into perm_out (host memory,
 * int32 [T*Y*X]): blocks are visited in row-major block order (the last block along an
 * axis may be clipped by the grid), the tokens of a block in row-major order; position i
 * of the reordered sequence holds original token perm_out[i] = (t*Y + y)*X + x.
 * All extents must be positive and T*Y*X < 2^31.  Returns DSATTN_EINVAL otherwise, or
 * when perm_out is NULL or device-only memory.
 */
int dsattn_block_order(int T, int Y, int X, int bt, int by, int bx, int32_t* perm_out);

/*
 * Row moves along the sequence axis of a device tensor [BH][N][row_bytes]:
 *   dsattn_gather_rows:  dst[b][i] = src[b][index[i]]
 *   dsattn_scatter_rows: dst[b][index[i]] = src[b][i]
 * index is a device int32 [N] array shared by all BH heads.  An entry outside [0, N)
 * never causes a memory access: gather writes a zero row for it, scatter drops the row.
 * With a non-injective index, scatter writes the duplicates in an unspecified order.
 * row_bytes must be a positive multiple of 4 and N * row_bytes <= 2^33; src, dst and
 * index must be 4-byte aligned device pointers and src and dst must not overlap
 * (16-byte alignment and row_bytes % 16 == 0 select the 16-byte-per-lane path).
 * 0 <= BH <= 65535.  Asynchronous on `stream`.
 */
int dsattn_gather_rows(const void* src, void* dst, const int32_t* index, int BH, int N,
                       int row_bytes, hipStream_t stream);
int dsattn_scatter_rows(const void* src, void* dst, const int32_t* index, int BH, int N,
                        int row_bytes, hipStream_t stream);

/*
 * Workspace, in bytes, that dsattn_attn_fwd_reordered needs for a [B][H][N][d] problem
 * (with_lse != 0 when lse_out will be requested): reordered copies of q, k, v and o
 * (and of the LSE).  0 for an empty problem.
 */
size_t dsattn_reordered_workspace_bytes(int B, int H, int N, int d, int with_lse);

/*
 * dsattn_attn_fwd_ex over a reordered sequence: queries are taken in the order q_index
 * (a gather map, e.g. from dsattn_block_order), keys and values in the order kv_index,
 * the key-tile loop and its skip decisions run over the reordered tiles, and o and
 * lse_out are returned in the ORIGINAL query order.  mask_out and stats_out describe the
 * reordered (query tile, key tile) pairs.  q_index and kv_index are device int32 [N]
 * arrays that must be permutations of 0..N-1 (not checked; see dsattn_gather_rows for
 * entries outside [0, N)).  workspace is a caller-owned device buffer of at least
 * dsattn_reordered_workspace_bytes(B, H, N, d, lse_out != NULL) bytes, 256-byte aligned,
 * overlapping no other buffer of the call (q, k, v, o, lse_out, mask_out, stats_out,
 * mask_in, q_index, kv_index); its contents are overwritten.  q_index and kv_index must
 * not overlap any output either.  Everything else as dsattn_attn_fwd_ex.
 */
int dsattn_attn_fwd_reordered(const dsattn_args* args, const int32_t* q_index,
                              const int32_t* kv_index, void* workspace,
                              size_t workspace_bytes);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): dsattn_attn_fwd_reordered with its
 * workspace taken from a scratch array inside the library, so the call allocates
 * nothing.  Each GPU the library runs on holds one such array of
 * DSATTN_STATIC_SCRATCH_BYTES until the process ends; a problem whose workspace
 * (dsattn_reordered_workspace_bytes) exceeds it is rejected with DSATTN_EINVAL.  Every
 * call on one GPU uses that GPU's array: calls that overlap in time on one GPU (other
 * streams, other threads) race and give undefined results; calls ordered on one stream
 * are safe.  The array keeps the last call's contents (nothing in it needs clearing: every
 * byte a call reads there it has written first).  Everything else as
 * dsattn_attn_fwd_reordered.
 */
#define DSATTN_STATIC_SCRATCH_BYTES ((size_t)96 << 20)
int dsattn_attn_fwd_reordered_noalloc(const dsattn_args* args, const int32_t* q_index,
                                      const int32_t* kv_index);

/*
 * MX-FP8 quantisation of bf16 rows, the storage of the quantised Q K^T variant (the
 * Conclusion, Section 5, lists quantisation among the methods the rule combines with).  src holds `rows`
 * rows of `row_len` bf16 values (row_len a multiple of 32); every 32 consecutive values
 * of a row form a block that shares the scale 2^E, E = floor(log2(max |x|)) - 8, written
 * to `scales` as the E8M0 code E + 127 (uint8 [rows][row_len / 32]; 0 for an all-zero
 * block), and each value becomes the FP8 E4M3 code nearest to x / 2^E in `codes` (uint8
 * [rows][row_len]): ties to the even code, magnitudes above 448 saturate to 448, values
 * that round to zero give +0.  Inputs must be finite.  src and codes must be 16-byte
 * aligned device pointers; scales a device pointer.  Asynchronous on `stream`.
 */
int dsattn_quantize_mxfp8(const void* src, void* codes, void* scales, long long rows,
                          int row_len, hipStream_t stream);

/*
 * Key smoothing for the quantised path.  Subtracting one vector m from every key of a head
 * shifts all scores of a query row by the same -q.m, which the softmax removes: the
 * attention output and the rule's decisions (they compare score differences) are
 * unchanged in exact arithmetic, while keys that share a large common component quantise
 * with a much smaller error once it is removed.  The LSE of the smoothed scores is the
 * original one minus scale * q.m.
 *
 * dsattn_key_mean: mean_out[h][c] = (1/N) sum_n k[h][n][c] in float32 for BH heads of N
 * bf16 keys of d values (d a power of two in [8, 1024]; k 16-byte aligned, mean_out 4-byte
 * aligned, both device pointers).  The summation order is fixed, so repeated calls give
 * the same bits.  N must be > 0 when BH > 0.
 *
 * dsattn_quantize_mxfp8_shift: as dsattn_quantize_mxfp8 on the float32 values
 * x - shift[i / group_rows][c] (each difference rounded to nearest float32) for element c
 * of row i; shift is a 16-byte aligned device array of float32 [ceil(rows/group_rows)]
 * [row_len].  For keys [B][H][N][d] and the mean of dsattn_key_mean, group_rows = N.
 * x - shift must stay finite.
 */
int dsattn_key_mean(const void* k, float* mean_out, int BH, int N, int d, hipStream_t stream);
int dsattn_quantize_mxfp8_shift(const void* src, const float* shift, void* codes, void* scales,
                                long long rows, int row_len, long long group_rows,
                                hipStream_t stream);

/* Message describing the last error on this thread ("" after a successful call). */
const char* dsattn_last_error(void);

/* Library version string. */
const char* dsattn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DSATTN_H */
